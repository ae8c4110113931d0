"""ctypes wrapper of the CPU fp64 oracle (oracle/mla_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg; never by the product path.  The C file states
the definition it computes (mixed decode + chunked-prefill step, section 2.3
and section 4.3.1 Eq. 4 of the paper; absorbed latent attention of the model
of section 6).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")
HEADS, DQK, DV = 16, 576, 512

_lib = None

_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_u16p = ctypes.POINTER(ctypes.c_uint16)
_f64p = ctypes.POINTER(ctypes.c_double)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b  # noqa: F401  (compiles on first use in a source tree)
            _b.build()
        L = ctypes.CDLL(LIB_PATH)
        L.oracle_append.argtypes = [ctypes.c_int32] * 4 + [_i32p, _i32p, _i32p, _u16p, _u16p]
        L.oracle_append.restype = ctypes.c_int
        L.oracle_attend_row.argtypes = [ctypes.c_int32] * 3 + [_i32p, ctypes.c_long, _u16p, _u16p,
                                                               ctypes.c_double, _f64p, _f64p, _f64p]
        L.oracle_attend_row.restype = ctypes.c_int
        L.oracle_attend_rows.argtypes = [ctypes.c_int32] * 4 + [_i32p, _i32p, _i32p, _u16p, _u16p,
                                                                ctypes.c_double, ctypes.c_long, _i64p,
                                                                _f64p, _f64p, ctypes.c_int32]
        L.oracle_attend_rows.restype = ctypes.c_int
        L.oracle_max_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray, t):
    return a.ctypes.data_as(t)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def append(batch, new_latents: np.ndarray, pool: np.ndarray) -> np.ndarray:
    """Return a copy of `pool` with the step's new latents scattered in."""
    out = np.array(pool, dtype=np.uint16, copy=True, order="C")
    ql = _c(batch.q_lens, np.int32)
    pl = _c(batch.prefix_lens, np.int32)
    bt = _c(batch.block_table, np.int32)
    nl = _c(new_latents, np.uint16)
    rc = lib().oracle_append(batch.num_reqs, batch.page_size, batch.num_pages, batch.max_pages_per_req,
                             _ptr(ql, _i32p), _ptr(pl, _i32p), _ptr(bt, _i32p), _ptr(nl, _u16p),
                             _ptr(out, _u16p))
    if rc != 0:
        raise ValueError("oracle_append: slot outside the block table or pool")
    return out


def attend(batch, q: np.ndarray, pool_after_append: np.ndarray, scale: float,
           rows: Optional[Sequence[int]] = None, threads: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Attention output [n][16][512] and lse [n][16] (fp64) for `rows` (default: all)."""
    ql = _c(batch.q_lens, np.int32)
    pl = _c(batch.prefix_lens, np.int32)
    bt = _c(batch.block_table, np.int32)
    qq = _c(q, np.uint16)
    pool = _c(pool_after_append, np.uint16)
    if rows is None:
        n = batch.num_rows
        rp = None
    else:
        rr = _c(rows, np.int64)
        n = int(rr.shape[0])
        rp = _ptr(rr, _i64p)
    out = np.zeros((n, HEADS, DV), dtype=np.float64)
    lse = np.zeros((n, HEADS), dtype=np.float64)
    if n == 0:
        return out, lse
    rc = lib().oracle_attend_rows(batch.num_reqs, batch.page_size, batch.num_pages, batch.max_pages_per_req,
                                  _ptr(ql, _i32p), _ptr(pl, _i32p), _ptr(bt, _i32p), _ptr(qq, _u16p),
                                  _ptr(pool, _u16p), float(np.float64(np.float32(scale))), n, rp,
                                  _ptr(out, _f64p), _ptr(lse, _f64p), int(threads))
    if rc != 0:
        raise ValueError("oracle_attend_rows: bad row or slot")
    return out, lse


def attend_row_weights(batch, req: int, n_keys: int, q_row: np.ndarray, pool_after_append: np.ndarray,
                       scale: float) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One row with n_keys visible keys: (out [16][512], lse [16], weights [16][n_keys])."""
    bt = _c(batch.block_table[req], np.int32)
    qq = _c(q_row, np.uint16)
    pool = _c(pool_after_append, np.uint16)
    out = np.zeros((HEADS, DV), dtype=np.float64)
    lse = np.zeros(HEADS, dtype=np.float64)
    w = np.zeros((HEADS, n_keys), dtype=np.float64)
    rc = lib().oracle_attend_row(batch.page_size, batch.num_pages, batch.max_pages_per_req, _ptr(bt, _i32p),
                                 int(n_keys), _ptr(qq, _u16p), _ptr(pool, _u16p),
                                 float(np.float64(np.float32(scale))), _ptr(out, _f64p), _ptr(lse, _f64p),
                                 _ptr(w, _f64p))
    if rc != 0:
        raise ValueError("oracle_attend_row: bad slot")
    return out, lse, w


def step(batch, layer_inputs, scale: float, rows=None, threads: int = 0):
    """Append then attend: (pool_after, out, lse)."""
    pool_after = append(batch, layer_inputs.new_latents, layer_inputs.pool)
    out, lse = attend(batch, layer_inputs.q, pool_after, scale, rows=rows, threads=threads)
    return pool_after, out, lse


def max_threads() -> int:
    return int(lib().oracle_max_threads())
