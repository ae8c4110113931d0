"""Python binding of libmlastep (include/mla_step.h): argument marshalling only.

Every step of the computation runs in the library's HIP kernels; this module
turns torch tensors into raw pointers and the caller's HIP stream.  There is
no CPU fallback: if the library is not built, loading it raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmlastep.so")

MLA_OK = 0
MLA_ERR_INVALID_ARG = -1
MLA_ERR_UNSUPPORTED = -2
MLA_ERR_WORKSPACE = -3
MLA_ERR_HIP = -4
MLA_OUT_F32 = 0
MLA_OUT_BF16 = 1
NUM_HEADS, D_QK, D_V = 16, 576, 512

EXPORTED = ("mla_abi_version", "mla_last_error", "mla_device_flags", "mla_debug_set", "mixed_step_workspace_bytes",
            "append_latent_kv", "mixed_step_attn", "mixed_step", "mixed_step_noalloc")
NOALLOC_SCRATCH_BYTES = 128 << 20
MLA_FLAG_BAD_PAGE = 1
MLA_FLAG_WAIT_EXPIRED = 2
MLA_DEBUG_CHECK = 0
MLA_DEBUG_SPIN_LIMIT = 1
MLA_DEBUG_CHUNK_KEYS = 2
MLA_DEBUG_WARM_PLAN = 3
MLA_DEBUG_DEC_UNIT = 4
MLA_DEBUG_DEC_FIRST = 5
# include/mla_layer.h
EXPORTED_LAYER = ("mla_proj_workspace_bytes", "mla_pre_attn", "mla_post_attn", "mla_layer_workspace_bytes",
                  "mla_attention_layer", "mla_layer_tune")
# mla_layer_tune knobs (include/mla_layer.h)
TUNE_GEMM_BM, TUNE_GEMM_BN, TUNE_GEMM_DEPTH, TUNE_MHA_MIN_ROWS, TUNE_MHA_PAIRS = range(5)
HIDDEN = 2048


class MlaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libmlastep error {code}: {msg}")
        self.code = code


class mla_batch(ctypes.Structure):
    _fields_ = [
        ("num_reqs", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("num_pages", ctypes.c_int32),
        ("max_pages_per_req", ctypes.c_int32),
        ("q_lens", ctypes.POINTER(ctypes.c_int32)),
        ("prefix_lens", ctypes.POINTER(ctypes.c_int32)),
        ("cu_q_dev", ctypes.c_void_p),
        ("prefix_lens_dev", ctypes.c_void_p),
        ("block_table_dev", ctypes.c_void_p),
    ]


class mla_proj_weights(ctypes.Structure):
    _fields_ = [
        ("w_q", ctypes.c_void_p),
        ("w_dkv", ctypes.c_void_p),
        ("kv_gain", ctypes.c_void_p),
        ("w_uk_t", ctypes.c_void_p),
        ("w_uv", ctypes.c_void_p),
        ("w_uk", ctypes.c_void_p),
        ("w_o", ctypes.c_void_p),
        ("rms_eps", ctypes.c_float),
        ("rope_base", ctypes.c_float),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libmlastep.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2607_02043_amd/build.py "
                              "(or __graft_entry__.build())")
        # torch first: the library's HIP runtime dependency then resolves to
        # the runtime torch has loaded, so the process holds one HIP runtime
        # (loading ours first would leave torch a second one, and the first
        # runtime to open the device keeps it)
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        L.mla_abi_version.restype = ctypes.c_int
        L.mla_last_error.restype = ctypes.c_char_p
        L.mixed_step_workspace_bytes.argtypes = [ctypes.POINTER(mla_batch)]
        L.mixed_step_workspace_bytes.restype = ctypes.c_size_t
        L.append_latent_kv.argtypes = [ctypes.POINTER(mla_batch), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.append_latent_kv.restype = ctypes.c_int
        L.mixed_step_attn.argtypes = [ctypes.POINTER(mla_batch), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float,
                                      ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_size_t, ctypes.c_void_p]
        L.mixed_step_attn.restype = ctypes.c_int
        L.mixed_step.argtypes = [ctypes.POINTER(mla_batch), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_float, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_size_t, ctypes.c_void_p]
        L.mixed_step.restype = ctypes.c_int
        L.mixed_step_noalloc.argtypes = [ctypes.POINTER(mla_batch), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_float, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.c_void_p]
        L.mixed_step_noalloc.restype = ctypes.c_int
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.mla_device_flags.argtypes = [i32, ctypes.POINTER(ctypes.c_int32), vp]
        L.mla_device_flags.restype = ctypes.c_int
        L.mla_debug_set.argtypes = [i32, i32]
        L.mla_debug_set.restype = ctypes.c_int
        wp = ctypes.POINTER(mla_proj_weights)
        L.mla_proj_workspace_bytes.argtypes = [i32]
        L.mla_proj_workspace_bytes.restype = sz
        L.mla_pre_attn.argtypes = [ctypes.POINTER(mla_batch), vp, wp, vp, vp, vp, sz, vp]
        L.mla_pre_attn.restype = ctypes.c_int
        L.mla_post_attn.argtypes = [i32, vp, i32, wp, vp, i32, vp, sz, vp]
        L.mla_post_attn.restype = ctypes.c_int
        L.mla_layer_workspace_bytes.argtypes = [ctypes.POINTER(mla_batch)]
        L.mla_layer_workspace_bytes.restype = sz
        L.mla_attention_layer.argtypes = [ctypes.POINTER(mla_batch), vp, wp, vp, ctypes.c_float, vp, i32, vp, sz,
                                          vp]
        L.mla_attention_layer.restype = ctypes.c_int
        L.mla_layer_tune.argtypes = [i32, i32]
        L.mla_layer_tune.restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc: int) -> None:
    if rc != MLA_OK:
        raise MlaError(rc, lib().mla_last_error().decode())


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


class DeviceBatch:
    """Host and device copies of one step's lengths and block table.

    q_lens / prefix_lens stay on the host (numpy int32, kept alive here);
    cu_q, prefix_lens and the block table are torch int32 tensors on `device`.
    """

    def __init__(self, q_lens, prefix_lens, block_table, page_size: int, num_pages: int, device="cuda"):
        import torch
        self.q_lens = np.ascontiguousarray(q_lens, dtype=np.int32)
        self.prefix_lens = np.ascontiguousarray(prefix_lens, dtype=np.int32)
        bt = np.ascontiguousarray(block_table, dtype=np.int32)
        if bt.ndim != 2 or bt.shape[0] != self.q_lens.shape[0]:
            raise ValueError("block_table must be [num_reqs][max_pages_per_req]")
        cu = np.zeros(self.q_lens.shape[0] + 1, dtype=np.int32)
        np.cumsum(self.q_lens, out=cu[1:])
        self.num_rows = int(cu[-1])
        self.cu_q_dev = torch.from_numpy(cu).to(device)
        self.prefix_dev = torch.from_numpy(self.prefix_lens.copy()).to(device)
        self.bt_dev = torch.from_numpy(bt.copy()).to(device)
        self.page_size = int(page_size)
        self.num_pages = int(num_pages)
        self.max_pages = int(bt.shape[1])
        self.c = mla_batch(
            num_reqs=int(self.q_lens.shape[0]), page_size=self.page_size, num_pages=self.num_pages,
            max_pages_per_req=self.max_pages,
            q_lens=self.q_lens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            prefix_lens=self.prefix_lens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            cu_q_dev=_ptr(self.cu_q_dev), prefix_lens_dev=_ptr(self.prefix_dev), block_table_dev=_ptr(self.bt_dev))

    @classmethod
    def from_batch(cls, batch, device="cuda") -> "DeviceBatch":
        """From a paper_2607_02043_amd.workloads.Batch."""
        return cls(batch.q_lens, batch.prefix_lens, batch.block_table, batch.page_size, batch.num_pages, device)


def abi_version() -> int:
    return int(lib().mla_abi_version())


def device_flags(clear: bool = True, stream=None) -> int:
    """The current device's sticky kernel error flags (MLA_FLAG_*), after
    synchronising `stream`; cleared unless clear is False."""
    f = ctypes.c_int32(0)
    _check(lib().mla_device_flags(1 if clear else 0, ctypes.byref(f), _stream(stream)))
    return int(f.value)


def debug_set(knob: int, value: int) -> None:
    """Process-wide debug setting (MLA_DEBUG_CHECK: 0/1; MLA_DEBUG_SPIN_LIMIT: >= 0, -1 = default)."""
    _check(lib().mla_debug_set(int(knob), int(value)))


def mixed_step_workspace_bytes(batch: DeviceBatch) -> int:
    n = int(lib().mixed_step_workspace_bytes(ctypes.byref(batch.c)))
    err = lib().mla_last_error().decode()
    if n == 0 and err:
        raise MlaError(MLA_ERR_INVALID_ARG, err)
    return n


def append_latent_kv(batch: DeviceBatch, new_latents, kv_cache, stream=None) -> None:
    """new_latents: uint16/bf16 [T][576] (device); kv_cache: [num_pages][P][576] updated in place."""
    _check(lib().append_latent_kv(ctypes.byref(batch.c), _ptr(new_latents), _ptr(kv_cache), _stream(stream)))


def _out_mode(out) -> int:
    import torch
    if out.dtype == torch.float32:
        return MLA_OUT_F32
    if out.dtype in (torch.bfloat16, torch.uint16, torch.int16):
        return MLA_OUT_BF16
    raise TypeError("out must be float32 or bfloat16")


def mixed_step_attn(batch: DeviceBatch, q, kv_cache, softmax_scale: float, out, lse=None, workspace=None,
                    stream=None) -> None:
    """q: [T][16][576] bf16 bits; out: [T][16][512] float32 or bf16 (dtype picks the mode)."""
    mode = _out_mode(out)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().mixed_step_attn(ctypes.byref(batch.c), _ptr(q), _ptr(kv_cache), float(softmax_scale), _ptr(out),
                                 mode, _ptr(lse), _ptr(workspace), ws_bytes, _stream(stream)))


def mixed_step(batch: DeviceBatch, q, new_latents, kv_cache, softmax_scale: float, out, lse=None, workspace=None,
               stream=None) -> None:
    """append_latent_kv + mixed_step_attn in one launch (bit-identical results)."""
    mode = _out_mode(out)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().mixed_step(ctypes.byref(batch.c), _ptr(q), _ptr(new_latents), _ptr(kv_cache), float(softmax_scale),
                            _ptr(out), mode, _ptr(lse), _ptr(workspace), ws_bytes, _stream(stream)))


def mixed_step_noalloc(batch: DeviceBatch, q, new_latents, kv_cache, softmax_scale: float, out, lse=None,
                       stream=None) -> None:
    """mixed_step on the library's own per-device scratch (no workspace argument)."""
    mode = _out_mode(out)
    _check(lib().mixed_step_noalloc(ctypes.byref(batch.c), _ptr(q), _ptr(new_latents), _ptr(kv_cache),
                                    float(softmax_scale), _ptr(out), mode, _ptr(lse), _stream(stream)))


def workspace_for(batch: DeviceBatch, device="cuda"):
    """A zeroed workspace tensor of the size mixed_step_attn / mixed_step need
    for `batch` (None if 0).  It may be reused for any batch that needs no more
    bytes: every completed call leaves its counters zero."""
    import torch
    n = mixed_step_workspace_bytes(batch)
    return torch.zeros(n, dtype=torch.uint8, device=device) if n > 0 else None


# --------------------------------------------------------------------------
# Projections around the attention and the whole layer (include/mla_layer.h)
# --------------------------------------------------------------------------
class DeviceProjWeights:
    """Device copies (int16 tensors holding bf16 bits) of one layer's
    projection weights, from a workloads.ProjWeights or any object with the
    same fields (numpy uint16 arrays in the C ABI's layouts)."""

    FIELDS = ("w_q", "w_dkv", "kv_gain", "w_uk_t", "w_uv", "w_uk", "w_o")

    def __init__(self, weights, device="cuda"):
        import torch
        self.tensors = {}
        for f in self.FIELDS:
            arr = np.ascontiguousarray(getattr(weights, f)).view(np.int16)
            self.tensors[f] = torch.from_numpy(arr.copy()).to(device)
        self.c = mla_proj_weights(**{f: _ptr(self.tensors[f]) for f in self.FIELDS},
                                  rms_eps=float(weights.rms_eps), rope_base=float(weights.rope_base))


def mla_proj_workspace_bytes(num_rows: int) -> int:
    return int(lib().mla_proj_workspace_bytes(int(num_rows)))


def mla_layer_workspace_bytes(batch: DeviceBatch) -> int:
    n = int(lib().mla_layer_workspace_bytes(ctypes.byref(batch.c)))
    err = lib().mla_last_error().decode()
    if n == 0 and err:
        raise MlaError(MLA_ERR_INVALID_ARG, err)
    return n


def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def mla_pre_attn(batch: DeviceBatch, hidden, weights: DeviceProjWeights, q_abs, new_latents, workspace,
                 stream=None) -> None:
    """hidden bf16 [T][2048] -> q_abs bf16 [T][16][576], new_latents bf16 [T][576]."""
    _check(lib().mla_pre_attn(ctypes.byref(batch.c), _ptr(hidden), ctypes.byref(weights.c), _ptr(q_abs),
                              _ptr(new_latents), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def mla_post_attn(attn_out, weights: DeviceProjWeights, out, workspace, stream=None) -> None:
    """attn_out [T][16][512] (fp32 or bf16) -> out [T][2048] (fp32 or bf16: dtypes pick the modes)."""
    T = int(attn_out.shape[0])
    _check(lib().mla_post_attn(T, _ptr(attn_out), _out_mode(attn_out), ctypes.byref(weights.c), _ptr(out),
                               _out_mode(out), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def mla_attention_layer(batch: DeviceBatch, hidden, weights: DeviceProjWeights, kv_cache, softmax_scale: float, out,
                        workspace, stream=None) -> None:
    """One attention layer: projections, append + attention, projections."""
    _check(lib().mla_attention_layer(ctypes.byref(batch.c), _ptr(hidden), ctypes.byref(weights.c), _ptr(kv_cache),
                                     float(softmax_scale), _ptr(out), _out_mode(out), _ptr(workspace),
                                     _nbytes(workspace), _stream(stream)))


def layer_workspace_for(batch: DeviceBatch, device="cuda"):
    """A workspace for mla_attention_layer with its counters zeroed (None if 0 bytes)."""
    import torch
    n = mla_layer_workspace_bytes(batch)
    return torch.zeros(n, dtype=torch.uint8, device=device) if n > 0 else None


def layer_tune(knob: int, value: int) -> None:
    """Process-wide tuning override of the layer (mla_layer_tune); -1 restores the default."""
    _check(lib().mla_layer_tune(int(knob), int(value)))


class tuned:
    """Context manager: set layer tuning knobs ({knob: value}) and restore
    the library defaults (-1) on exit."""

    def __init__(self, settings):
        self.settings = dict(settings)

    def __enter__(self):
        for k, v in self.settings.items():
            layer_tune(k, v)
        return self

    def __exit__(self, *exc):
        for k in self.settings:
            layer_tune(k, -1)
        return False
