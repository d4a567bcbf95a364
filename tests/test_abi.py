"""The C ABI from the host: the library loads, exports every function that
include/sas.h declares, sizes workspaces and rejects bad arguments before
touching the GPU (every call here fails validation, so nothing is launched)."""
import ctypes as C
import os
import re

import pytest

from paper_2609_13141_amd import configs, sas

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "sas.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\s*\*?\s*(sas_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(sas.LIB_PATH):
        pytest.skip("libsas.so not built")
    return sas.lib()


def test_header_declares_the_entry_points():
    fns = header_functions()
    for f in ("sas_attention_prefill", "sas_mlp_forward", "sas_layer_forward", "sas_decode_step",
              "sas_workspace_size", "sas_last_error"):
        assert f in fns


def test_library_exports_every_declared_symbol(L):
    for f in header_functions():
        assert hasattr(L, f), f"{f} not exported"
    assert b"gfx950" in L.sas_version()


def test_workspace_sizes(L):
    for w in configs.WORKLOADS:
        cfg = sas.make_config(w)
        n_att = sas.workspace_size(cfg, sas.OP_ATTENTION, w.batch, w.seq_len)
        n_lay = sas.workspace_size(cfg, sas.OP_LAYER, w.batch, w.seq_len)
        assert 0 < n_att < n_lay
        assert sas.workspace_size(cfg, sas.OP_MLP, w.tokens, 0) > 0
    bad = sas.make_config(configs.L7B_1K)
    bad.head_dim = 96
    assert sas.workspace_size(bad, sas.OP_LAYER, 1, 16) == 0


def _call_attention(L, cfg, q=0x1000, k=0x1000, v=0x1000, o=0x1000, batch=1, n=16, ws=None, ws_bytes=0):
    ain = sas.AttnIn(q, k, v, None, None)
    aout = sas.AttnOut(o, None, None, None, None, None)
    return L.sas_attention_prefill(C.byref(cfg), batch, n, C.byref(ain), C.byref(aout), ws, ws_bytes, None)


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, sas.SAS_ERR_UNSUPPORTED),
    ("n_kv_heads", 3, sas.SAS_ERR_INVALID_ARGUMENT),
    ("block_size", 48, sas.SAS_ERR_UNSUPPORTED),
    ("top_k", -1, sas.SAS_ERR_INVALID_ARGUMENT),
    ("top_k", 33, sas.SAS_ERR_UNSUPPORTED),
    ("dtype", 7, sas.SAS_ERR_INVALID_ARGUMENT),
    ("mode", 5, sas.SAS_ERR_INVALID_ARGUMENT),
])
def test_bad_config_is_rejected(L, field, value, status):
    cfg = sas.make_config(configs.L7B_1K)
    setattr(cfg, field, value)
    assert _call_attention(L, cfg) == status
    assert len(L.sas_last_error()) > 0


def test_null_and_misaligned_pointers_and_small_workspace(L):
    cfg = sas.make_config(configs.L7B_1K)
    assert _call_attention(L, cfg, q=None) == sas.SAS_ERR_INVALID_ARGUMENT
    assert b"in.q" in L.sas_last_error()
    assert _call_attention(L, cfg, o=None) == sas.SAS_ERR_INVALID_ARGUMENT
    assert _call_attention(L, cfg, k=0x1002) == sas.SAS_ERR_INVALID_ARGUMENT
    assert b"aligned" in L.sas_last_error()
    assert _call_attention(L, cfg, n=0) == sas.SAS_ERR_INVALID_ARGUMENT
    assert _call_attention(L, cfg, ws=None, ws_bytes=0) == sas.SAS_ERR_WORKSPACE
    assert _call_attention(L, cfg, ws=0x1000, ws_bytes=16) == sas.SAS_ERR_WORKSPACE
    assert L.sas_attention_prefill(None, 1, 16, None, None, None, 0, None) == sas.SAS_ERR_INVALID_ARGUMENT


def test_layer_and_mlp_reject_missing_weights(L):
    cfg = sas.make_config(configs.L7B_1K)
    W = sas.LayerWeights()
    st = L.sas_mlp_forward(C.byref(cfg), 4, 0x1000, C.byref(W), 0x1000, None, 0, None)
    assert st == sas.SAS_ERR_INVALID_ARGUMENT and b"w.rms2" in L.sas_last_error()
    st = L.sas_layer_forward(C.byref(cfg), 1, 4, 0x1000, C.byref(W), 0x1000, None, None, None, None, 0, None)
    assert st == sas.SAS_ERR_INVALID_ARGUMENT and b"w.rms1" in L.sas_last_error()
    bad = sas.make_config(configs.L7B_1K)
    bad.d_ff = 1001
    assert L.sas_mlp_forward(C.byref(bad), 4, 0x1000, C.byref(W), 0x1000, None, 0, None) == sas.SAS_ERR_UNSUPPORTED


def test_noalloc_decode_rejects_oversized_calls_before_touching_the_gpu(L):
    # batch 16 over 8192 blocks needs 16 * 32 * 8192 doubles of selector scores alone (32 MiB):
    # more than the static scratch holds; the call fails on the host with a clear message
    import ctypes as C
    w = configs.STACK_DECODE
    cfg = sas.make_config(w, "sparse")
    fake = C.c_void_p(256)
    cache = sas.PagedKV(fake, fake, fake, fake, 1, 16, 1, 8192)
    st = L.sas_decode_step_noalloc(C.byref(cfg), 16, fake, fake, C.byref(sas.weights_struct({})), C.byref(cache),
                                   fake, None, None)
    assert st == -3   # SAS_ERR_WORKSPACE
    assert b"static" in L.sas_last_error() and b"scratch" in L.sas_last_error()


def test_packed_decode_layout_size_and_validation(L):
    # the packed copy holds every linear weight exactly once when the column
    # groups divide the products (16 columns, 8 rotary or gate/up pairs)
    for w in (configs.STACK_DECODE, configs.BY_NAME["gqa28x4_layer_16k"]):
        cfg = sas.make_config(w, "sparse")
        d, H, Hkv, dh, F = w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.d_ff
        weights = 2 * (d * (H + 2 * Hkv) * dh + d * H * dh + 2 * d * F + F * d)
        assert L.sas_decode_packed_bytes(C.byref(cfg)) == weights
    f32 = sas.make_config(configs.BY_NAME["tiny_1layer_f32"], "sparse")
    assert L.sas_decode_packed_bytes(C.byref(f32)) == 0
    # validation fails before any launch: missing weights, misalignment, short buffer
    cfg = sas.make_config(configs.STACK_DECODE, "sparse")
    n = L.sas_decode_packed_bytes(C.byref(cfg))
    ws = sas.LayerWeights(*([0x1000] * 9 + [None, None, None]))
    assert L.sas_pack_decode_weights(C.byref(cfg), None, 0x1000, n, None) == sas.SAS_ERR_INVALID_ARGUMENT
    assert L.sas_pack_decode_weights(C.byref(cfg), C.byref(ws), 0x1010, n, None) == sas.SAS_ERR_INVALID_ARGUMENT
    assert L.sas_pack_decode_weights(C.byref(cfg), C.byref(ws), 0x1000, n - 1, None) == sas.SAS_ERR_WORKSPACE
    assert L.sas_pack_decode_weights(C.byref(f32), C.byref(ws), 0x1000, n, None) == sas.SAS_ERR_UNSUPPORTED
