"""GPU parity of the prefill entry points against the fp64 oracle, on the same
seeded inputs: selected block indices and block summaries bit-exact; O, LSE,
log gate and tau within the activation tolerance (2e-2 bf16, 1e-5 fp32,
max|gpu - ref| / max|ref|).  Shapes span several tiles with ragged tails,
GQA, every block size and the degenerate budgets (K = 0, K >= C)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_13141_amd import configs, inputs, sas

from oracle.selector import select
from helpers import (TOL, assert_close, assert_close_with_infs, assert_selection_near_ties, f64, score_bounds,
                     spec_of)

pytestmark = pytest.mark.gpu


def W_(**kw):
    base = dict(name="t", dtype="bf16", batch=2, seq_len=300, d_model=256, n_heads=4, n_kv_heads=2,
                head_dim=128, d_ff=688, block_size=64, top_k=2, mode="gated", segments=(), index=50)
    base.update(kw)
    n = base["seq_len"]
    base["segments"] = (("img", n // 2), ("txt", n - n // 2))
    return configs.Workload(**base)


ATTN_CASES = [
    W_(),                                                                     # 3 q-tiles, ragged
    W_(head_dim=64, block_size=16, top_k=3, seq_len=200, index=51),
    W_(n_heads=14, n_kv_heads=2, block_size=32, top_k=4, seq_len=257, batch=1, index=52),   # GQA G=7
    W_(block_size=128, top_k=1, seq_len=520, batch=1, index=53),
    W_(top_k=0, seq_len=190, index=54),                                        # K = 0: block-local
    W_(top_k=32, seq_len=400, batch=1, index=55),                              # K >= C: all kept
    W_(seq_len=1, batch=3, index=56),                                         # single token
    W_(dtype="f32", seq_len=64, n_heads=4, n_kv_heads=4, head_dim=64, block_size=16, top_k=2, batch=1,
       index=0),                                                              # the tiny fp32 layer shape
    W_(dtype="f32", seq_len=150, head_dim=128, block_size=32, top_k=3, index=57),
]


def _ids(cases):
    return [f"{w.dtype}-n{w.seq_len}-H{w.n_heads}/{w.n_kv_heads}-dh{w.head_dim}-B{w.block_size}-K{w.top_k}"
            for w in cases]


@pytest.mark.parametrize("mode", ["gated", "sparse", "dense"])
@pytest.mark.parametrize("w", ATTN_CASES, ids=_ids(ATTN_CASES))
def test_attention_prefill_matches_oracle(w, mode):
    print(f"\n[case] attention {w.dtype} b={w.batch} n={w.seq_len} H={w.n_heads}/{w.n_kv_heads} "
          f"dh={w.head_dim} B={w.block_size} K={w.top_k} mode={mode}", flush=True)
    q, k, v = inputs.qkv(w)
    cfg = sas.make_config(w, mode)
    dq, dk, dv = (sas.to_device(a, w.dtype) for a in (q, k, v))
    out = sas.attention_prefill(cfg, dq, dk, dv, log_gate=True, tau=True)
    torch.cuda.synchronize()
    ref = oracle.attention_prefill(f64(q), f64(k), f64(v), spec_of(w, mode))
    np.testing.assert_array_equal(out["sel_idx"].cpu().numpy(), ref["sel"])
    np.testing.assert_array_equal(out["k_summary"].float().cpu().numpy()[:, :, :ref["k_summary"].shape[2]],
                                  ref["k_summary"])
    assert_close(out["o"].float().cpu().numpy(), ref["O_exact"], w.dtype, "O")
    assert_close(out["lse"].cpu().numpy(), ref["LSE"], w.dtype, "LSE", tol=1e-5 if w.dtype == "f32" else 1e-3)
    assert_close_with_infs(out["log_gate"].cpu().numpy(), ref["log_gate"], w.dtype, "log_gate", tol=1e-5)
    assert_close_with_infs(out["tau"].cpu().numpy(), ref["tau"], w.dtype, "tau", tol=1e-5)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_attention_with_selector_projections(dtype):
    w = W_(dtype=dtype, seq_len=260, index=58)
    q, k, v = inputs.qkv(w)
    Wl = inputs.layer_weights(w, selector_proj=True)
    cfg = sas.make_config(w)
    out = sas.attention_prefill(cfg, *(sas.to_device(a, dtype) for a in (q, k, v)),
                                w_gq=sas.to_device(Wl["w_gq"], dtype), w_gk=sas.to_device(Wl["w_gk"], dtype))
    torch.cuda.synchronize()
    ref = oracle.attention_prefill(f64(q), f64(k), f64(v), spec_of(w), w_gq=f64(Wl["w_gq"]),
                                   w_gk=f64(Wl["w_gk"]))
    np.testing.assert_array_equal(out["sel_idx"].cpu().numpy(), ref["sel"])
    assert_close(out["o"].float().cpu().numpy(), ref["O_exact"], dtype, "O")


def test_zero_query_closed_form_on_gpu():
    # q = 0 makes every score tie: the lowest blocks are kept, g = 1/C_t
    w = W_(seq_len=330, batch=1, top_k=3, index=59)
    q, k, v = inputs.qkv(w)
    q[:] = 0.0
    cfg = sas.make_config(w, "gated")
    out = sas.attention_prefill(cfg, *(sas.to_device(a, "bf16") for a in (q, k, v)))
    torch.cuda.synchronize()
    sel = out["sel_idx"].cpu().numpy()
    for t in range(w.seq_len):
        c = t // w.block_size
        kk = min(w.top_k, c)
        assert list(sel[0, 0, t, :kk]) == list(range(kk))
    ref = oracle.attention_prefill(f64(q), f64(k), f64(v), spec_of(w, "gated"))
    assert_close(out["o"].float().cpu().numpy(), ref["O_exact"], "bf16", "O")


@pytest.mark.parametrize("dtype,M", [("bf16", 100), ("bf16", 300), ("f32", 64)])
def test_mlp_matches_oracle(dtype, M):
    w = W_(dtype=dtype, index=60)
    print(f"\n[case] mlp {dtype} M={M}", flush=True)
    Wl = inputs.layer_weights(w)
    x = inputs.normal(w, "h", (M, w.d_model), 1.0)
    cfg = sas.make_config(w)
    y = sas.mlp_forward(cfg, sas.to_device(x, dtype), sas.weights_to_device(Wl, dtype))
    torch.cuda.synchronize()
    ref = oracle.mlp_forward(f64(x), {k: (None if a is None else f64(a)) for k, a in Wl.items()}, spec_of(w))
    assert_close(y.float().cpu().numpy(), ref, dtype, "y")


LAYER_CASES = [
    configs.TINY,
    W_(n_heads=4, n_kv_heads=2, head_dim=64, block_size=32, top_k=2, seq_len=200, index=61),
    W_(d_model=512, n_heads=4, n_kv_heads=4, head_dim=128, d_ff=1024, seq_len=333, batch=1, top_k=3,
       index=62),
]


@pytest.mark.parametrize("w", LAYER_CASES, ids=[w.name + str(w.index) for w in LAYER_CASES])
def test_layer_forward_matches_oracle(w):
    print(f"\n[case] layer {w.name} {w.dtype} b={w.batch} n={w.seq_len} d={w.d_model}", flush=True)
    x = inputs.embeddings(w)
    Wl = inputs.layer_weights(w)
    cfg = sas.make_config(w)
    out = sas.layer_forward(cfg, sas.to_device(x, w.dtype), sas.weights_to_device(Wl, w.dtype), taps=True)
    torch.cuda.synchronize()
    ref = oracle.layer_forward(f64(x), {k: (None if a is None else f64(a)) for k, a in Wl.items()}, spec_of(w))
    assert_close(out["q"].float().cpu().numpy(), ref["Q"], w.dtype, "Q")
    assert_close(out["k"].float().cpu().numpy(), ref["K"], w.dtype, "K")
    assert_close(out["v"].float().cpu().numpy(), ref["V"], w.dtype, "V")
    assert_close(out["o"].float().cpu().numpy(), ref["O"], w.dtype, "O")
    assert_close(out["h1"].float().cpu().numpy(), ref["h1"], w.dtype, "h1")
    assert_close(out["y"].float().cpu().numpy(), ref["y"], w.dtype, "y")
    sel = out["sel_idx"].cpu().numpy()
    qg, kg = out["q"].float().cpu().numpy(), out["k"].float().cpu().numpy()
    sp = spec_of(w)
    for bi in range(w.batch):
        # the oracle's selector on the GPU's own materialised Q/K: bit-exact
        st = select(f64(qg[bi]), f64(kg[bi]), w.block_size, w.top_k, w.dtype)
        np.testing.assert_array_equal(sel[bi], st["sel"])
        # against the oracle's own Q/K: rows may differ only at near-ties within one ulp of Q/K
        r, bd = score_bounds(ref["Q"][bi], ref["K"][bi], w.block_size, sp.group, w.dtype)
        np.testing.assert_array_equal(r, ref["r"][bi])
        nd = assert_selection_near_ties(sel[bi], ref["sel"][bi], r, bd, "layer")
        print(f"  sequence {bi}: {nd} of {sel[bi].shape[0] * sel[bi].shape[1]} rows differ from the "
              f"oracle's own selection, each at a near-tie", flush=True)
