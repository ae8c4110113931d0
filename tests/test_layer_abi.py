"""The layer entry points of the C ABI (include/mla_layer.h) without a GPU:
every declared symbol is exported, and bad arguments are rejected on the host
before anything is launched."""
import ctypes
import os
import re

import pytest

import paper_2607_02043_amd as mla
from test_abi import FAKE, _HostBatch, _declared_functions

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mla_layer.h")


def _err():
    return mla.lib().mla_last_error().decode()


def test_layer_header_symbols_are_exported():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    names = set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([A-Za-z_][A-Za-z0-9_]*)\s*\(", text, re.M))
    assert names == set(mla.EXPORTED_LAYER), names
    for n in names:
        assert hasattr(mla.lib(), n)
    assert not names & set(_declared_functions())


def _weights(**kw):
    w = mla.mla_proj_weights(w_q=FAKE, w_dkv=FAKE, kv_gain=FAKE, w_uk_t=FAKE, w_uv=FAKE, w_uk=FAKE, w_o=FAKE,
                             rms_eps=1e-6, rope_base=10000.0)
    for k, v in kw.items():
        setattr(w, k, v)
    return w


def _pre(b, w=None, hidden=FAKE, q=FAKE, lat=FAKE, ws=FAKE, ws_bytes=1 << 40):
    w = _weights() if w is None else w
    return mla.lib().mla_pre_attn(ctypes.byref(b.c), hidden, ctypes.byref(w), q, lat, ws, ws_bytes, None)


def _post(T=4, w=None, a=FAKE, adt=0, out=FAKE, odt=0, ws=FAKE, ws_bytes=1 << 40):
    w = _weights() if w is None else w
    return mla.lib().mla_post_attn(T, a, adt, ctypes.byref(w), out, odt, ws, ws_bytes, None)


def test_workspace_sizes():
    L = mla.lib()
    assert L.mla_proj_workspace_bytes(0) == 0 and L.mla_proj_workspace_bytes(-3) == 0
    # qn bf16 [16][128] + qpe fp32 [16][64] + latent fp32 [576] per row, 256-byte aligned parts
    n = L.mla_proj_workspace_bytes(100)
    assert n >= 100 * (4096 + 4096 + 2304) and n % 256 == 0
    assert L.mla_proj_workspace_bytes(100) >= 100 * 2048 * 2
    b = _HostBatch([1, 1, 7], [10, 300, 0])
    need = L.mla_layer_workspace_bytes(ctypes.byref(b.c))
    attn = L.mixed_step_workspace_bytes(ctypes.byref(b.c))
    if attn == 0:  # planning needs the device's CU count: no device here, and both sizes report it
        assert need == 0 and "hip" in _err().lower()
    else:
        T = 9
        assert need >= attn + T * (18432 + 1152 + 16384) + L.mla_proj_workspace_bytes(T)
    assert L.mla_layer_workspace_bytes(ctypes.byref(_HostBatch([], []).c)) == 0
    assert L.mla_layer_workspace_bytes(ctypes.byref(_HostBatch([0], [3]).c)) == 0
    assert "q_lens" in _err()


def test_pre_attn_checks():
    b = _HostBatch([1, 3], [5, 0])
    assert _pre(_HostBatch([], []), hidden=None) == mla.MLA_OK  # empty batch: nothing to do
    assert _pre(b, hidden=None) == mla.MLA_ERR_INVALID_ARG
    assert _pre(b, q=FAKE + 2) == mla.MLA_ERR_INVALID_ARG and "aligned" in _err()
    assert _pre(b, w=_weights(w_uk_t=None)) == mla.MLA_ERR_INVALID_ARG
    assert _pre(b, w=_weights(kv_gain=FAKE + 8)) == mla.MLA_ERR_INVALID_ARG
    for eps in (0.0, -1e-6, float("nan"), float("inf")):
        assert _pre(b, w=_weights(rms_eps=eps)) == mla.MLA_ERR_INVALID_ARG and "rms_eps" in _err()
    for base in (1.0, 0.5, float("inf")):
        assert _pre(b, w=_weights(rope_base=base)) == mla.MLA_ERR_INVALID_ARG and "rope_base" in _err()
    need = mla.lib().mla_proj_workspace_bytes(4)
    assert _pre(b, ws_bytes=need - 1) == mla.MLA_ERR_WORKSPACE
    assert _pre(b, ws=None) == mla.MLA_ERR_WORKSPACE
    assert _pre(_HostBatch([0], [1])) == mla.MLA_ERR_INVALID_ARG and "q_lens" in _err()
    assert mla.lib().mla_pre_attn(ctypes.byref(b.c), FAKE, None, FAKE, FAKE, FAKE, 1 << 40, None) == \
        mla.MLA_ERR_INVALID_ARG


def test_post_attn_checks():
    assert _post(T=0, a=None) == mla.MLA_OK
    assert _post(T=-1) == mla.MLA_ERR_INVALID_ARG
    assert _post(adt=2) == mla.MLA_ERR_INVALID_ARG and "attn_dtype" in _err()
    assert _post(odt=-1) == mla.MLA_ERR_INVALID_ARG and "out_dtype" in _err()
    assert _post(out=None) == mla.MLA_ERR_INVALID_ARG
    assert _post(a=FAKE + 4) == mla.MLA_ERR_INVALID_ARG
    assert _post(w=_weights(w_o=None)) == mla.MLA_ERR_INVALID_ARG
    assert _post(ws_bytes=mla.lib().mla_proj_workspace_bytes(4) - 256) == mla.MLA_ERR_WORKSPACE
    # a rejected call leaves a message; a no-op call clears it
    assert _post(T=-1) != mla.MLA_OK and _err() != ""
    assert _post(T=0) == mla.MLA_OK and _err() == ""


def test_layer_checks():
    b = _HostBatch([1, 3], [5, 0])
    w = _weights()
    L = mla.lib()
    need = L.mla_layer_workspace_bytes(ctypes.byref(b.c))

    def layer(ws_bytes=need, scale=0.07, odt=0, batch=b):
        return L.mla_attention_layer(ctypes.byref(batch.c), FAKE, ctypes.byref(w), FAKE, scale, FAKE, odt, FAKE,
                                     ws_bytes, None)

    if need > 0:
        assert layer(ws_bytes=need - 1) == mla.MLA_ERR_WORKSPACE
    else:  # no device: the planning step reports the HIP error
        assert layer(ws_bytes=1 << 40) == mla.MLA_ERR_HIP
    assert layer(batch=_HostBatch([], [])) == mla.MLA_OK
    assert layer(batch=_HostBatch([1], [-2])) == mla.MLA_ERR_INVALID_ARG
