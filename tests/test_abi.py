"""The C ABI library without a GPU: it loads, exports every entry point the
header declares, and rejects bad arguments on the host before any launch."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2607_02043_amd as mla

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mla_step.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([A-Za-z_][A-Za-z0-9_]*)\s*\(", text, re.M)
    return sorted(set(n for n in names if n not in ("if", "while", "return")))


def test_library_loads_and_exports_every_declared_symbol():
    L = mla.lib()
    declared = _declared_functions()
    assert set(declared) == set(mla.EXPORTED), declared
    for name in declared:
        assert hasattr(L, name), f"libmlastep.so does not export {name}"
    version = int(re.search(r"#define\s+MLA_ABI_VERSION\s+(\d+)", open(HEADER).read()).group(1))
    assert L.mla_abi_version() == version


class _HostBatch:
    """An mla_batch with host arrays and fake (never dereferenced) device pointers."""

    def __init__(self, q_lens, prefix_lens, page=64, num_pages=100, max_pages=64):
        self.ql = np.ascontiguousarray(q_lens, dtype=np.int32)
        self.pl = np.ascontiguousarray(prefix_lens, dtype=np.int32)
        self.c = mla.mla_batch(
            num_reqs=len(self.ql), page_size=page, num_pages=num_pages, max_pages_per_req=max_pages,
            q_lens=self.ql.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            prefix_lens=self.pl.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            cu_q_dev=0x1000, prefix_lens_dev=0x2000, block_table_dev=0x3000)


FAKE = 0x10000  # 16-byte aligned, never touched: every call below fails validation first


def _append(b, new=FAKE, kv=FAKE):
    return mla.lib().append_latent_kv(ctypes.byref(b.c) if b is not None else None, new, kv, None)


def _attn(b, scale=0.07, dtype=0, q=FAKE, kv=FAKE, out=FAKE, lse=None):
    return mla.lib().mixed_step_attn(ctypes.byref(b.c), q, kv, scale, out, dtype, lse, None, 0, None)


def _step(b, scale=0.07, dtype=0, q=FAKE, new=FAKE, kv=FAKE, out=FAKE, lse=None):
    return mla.lib().mixed_step(ctypes.byref(b.c), q, new, kv, scale, out, dtype, lse, None, 0, None)


def _err():
    return mla.lib().mla_last_error().decode()


def test_null_batch_is_rejected():
    assert mla.lib().append_latent_kv(None, FAKE, FAKE, None) == mla.MLA_ERR_INVALID_ARG
    assert "NULL" in _err()


def test_empty_batch_is_a_no_op():
    b = _HostBatch([], [])
    assert _append(b) == mla.MLA_OK
    assert _attn(b) == mla.MLA_OK


@pytest.mark.parametrize("page,code", [(0, mla.MLA_ERR_UNSUPPORTED), (48, mla.MLA_ERR_UNSUPPORTED),
                                       (2048, mla.MLA_ERR_UNSUPPORTED)])
def test_page_size_must_be_a_power_of_two(page, code):
    b = _HostBatch([1], [3], page=page)
    assert _append(b) == code
    assert "page_size" in _err()


@pytest.mark.parametrize("ql,pl,frag", [([0], [3], "q_lens"), ([1], [-1], "prefix_lens"),
                                        ([1, 5], [4095, 4092], "exceeds the block table")])
def test_bad_lengths_are_rejected(ql, pl, frag):
    b = _HostBatch(ql, pl, page=64, max_pages=64)
    assert _append(b) == mla.MLA_ERR_INVALID_ARG
    assert frag in _err()
    assert _attn(b) == mla.MLA_ERR_INVALID_ARG


def test_null_device_pointers_are_rejected():
    b = _HostBatch([1], [3])
    assert _append(b, new=None) == mla.MLA_ERR_INVALID_ARG
    assert _attn(b, q=None) == mla.MLA_ERR_INVALID_ARG
    assert _attn(b, out=None) == mla.MLA_ERR_INVALID_ARG
    b.c.block_table_dev = None
    assert _append(b) == mla.MLA_ERR_INVALID_ARG


def test_misaligned_pointers_are_rejected():
    b = _HostBatch([1], [3])
    assert _append(b, new=FAKE + 2) == mla.MLA_ERR_INVALID_ARG
    assert "aligned" in _err()
    assert _attn(b, q=FAKE + 8) == mla.MLA_ERR_INVALID_ARG
    assert _step(b, new=FAKE + 4) == mla.MLA_ERR_INVALID_ARG
    assert "aligned" in _err()


def test_fused_step_checks_its_arguments():
    b = _HostBatch([1], [3])
    assert _step(b, new=None) == mla.MLA_ERR_INVALID_ARG
    assert "new_latents" in _err()
    assert _step(b, scale=0.0) == mla.MLA_ERR_INVALID_ARG
    assert _step(b, dtype=3) == mla.MLA_ERR_INVALID_ARG
    assert _step(_HostBatch([0], [3])) == mla.MLA_ERR_INVALID_ARG
    assert _step(_HostBatch([], []), new=None) == mla.MLA_OK


@pytest.mark.parametrize("scale", [0.0, -1.0, float("inf"), float("nan")])
def test_bad_scale_is_rejected(scale):
    b = _HostBatch([1], [3])
    assert _attn(b, scale=scale) == mla.MLA_ERR_INVALID_ARG
    assert "softmax_scale" in _err()


def test_bad_out_dtype_is_rejected():
    b = _HostBatch([1], [3])
    assert _attn(b, dtype=7) == mla.MLA_ERR_INVALID_ARG


def test_error_message_is_cleared_by_a_good_call():
    b = _HostBatch([1], [3])
    assert _attn(b, dtype=7) != mla.MLA_OK
    assert _err() != ""
    assert _attn(_HostBatch([], [])) == mla.MLA_OK
    assert _err() == ""


def test_debug_settings_are_checked_on_the_host():
    L = mla.lib()
    assert L.mla_debug_set(7, 1) == mla.MLA_ERR_INVALID_ARG
    assert "knob" in _err()
    assert L.mla_debug_set(mla.MLA_DEBUG_CHECK, 2) == mla.MLA_ERR_INVALID_ARG
    assert L.mla_debug_set(mla.MLA_DEBUG_SPIN_LIMIT, -5) == mla.MLA_ERR_INVALID_ARG
    assert L.mla_debug_set(mla.MLA_DEBUG_SPIN_LIMIT, -1) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_CHECK, 0) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_CHUNK_KEYS, 100) == mla.MLA_ERR_INVALID_ARG
    assert L.mla_debug_set(mla.MLA_DEBUG_CHUNK_KEYS, -64) == mla.MLA_ERR_INVALID_ARG
    assert L.mla_debug_set(mla.MLA_DEBUG_CHUNK_KEYS, 128) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_CHUNK_KEYS, -1) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_WARM_PLAN, 2) == mla.MLA_ERR_INVALID_ARG
    assert L.mla_debug_set(mla.MLA_DEBUG_WARM_PLAN, 0) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_WARM_PLAN, -1) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_DEC_UNIT, -2) == mla.MLA_ERR_INVALID_ARG
    assert L.mla_debug_set(mla.MLA_DEBUG_DEC_UNIT, 5) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_DEC_UNIT, -1) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_DEC_FIRST, -2) == mla.MLA_ERR_INVALID_ARG
    assert L.mla_debug_set(mla.MLA_DEBUG_DEC_FIRST, 96) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_DEC_FIRST, 0) == mla.MLA_OK
    assert L.mla_debug_set(mla.MLA_DEBUG_DEC_FIRST, -1) == mla.MLA_OK
    assert L.mla_device_flags(1, None, None) == mla.MLA_ERR_INVALID_ARG


def test_library_shares_torch_hip_runtime():
    """Loading the library first (a fresh process) still leaves one HIP
    runtime in the process: the one torch loads."""
    import subprocess
    import sys
    code = ("import paper_2607_02043_amd as m; m.lib(); "
            "print('\\n'.join(sorted({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l})))")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, check=True,
                         cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__)))).stdout.split()
    assert len(out) == 1, out


def test_binding_constants_match_the_headers():
    """Every error code, flag, output mode, debug and tuning knob and size the
    headers define has the same value in the Python binding."""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    text = "".join(open(os.path.join(root, "include", h)).read() for h in ("mla_step.h", "mla_layer.h"))
    values = {name: int(v) for name, v in re.findall(r"\b(MLA_[A-Z0-9_]+)\s*=\s*(-?\d+)", text)}
    for name, base, shift in re.findall(r"#define\s+(MLA_[A-Z0-9_]+)\s+\(?(\d+)u?(?:\s*<<\s*(\d+))?", text):
        values[name] = int(base) << int(shift or 0)

    def py_name(name):
        if name == "MLA_NOALLOC_SCRATCH_BYTES":
            return "NOALLOC_SCRATCH_BYTES"
        return name[len("MLA_"):] if name.startswith("MLA_TUNE_") else name

    for must in ("MLA_OK", "MLA_ERR_INVALID_ARG", "MLA_ERR_UNSUPPORTED", "MLA_ERR_WORKSPACE", "MLA_ERR_HIP",
                 "MLA_OUT_F32", "MLA_OUT_BF16", "MLA_FLAG_BAD_PAGE", "MLA_FLAG_WAIT_EXPIRED", "MLA_DEBUG_CHECK",
                 "MLA_DEBUG_SPIN_LIMIT", "MLA_DEBUG_CHUNK_KEYS", "MLA_DEBUG_WARM_PLAN", "MLA_DEBUG_DEC_UNIT",
                 "MLA_DEBUG_DEC_FIRST", "MLA_TUNE_GEMM_BM",
                 "MLA_TUNE_GEMM_BN", "MLA_TUNE_GEMM_DEPTH", "MLA_TUNE_MHA_MIN_ROWS", "MLA_TUNE_MHA_PAIRS",
                 "MLA_NOALLOC_SCRATCH_BYTES"):
        assert must in values, must
        assert getattr(mla, py_name(must)) == values[must], (must, getattr(mla, py_name(must)), values[must])
    for name, v in values.items():  # anything else the binding also names
        if hasattr(mla, py_name(name)):
            assert getattr(mla, py_name(name)) == v, name
