"""Pins of the oracle's layer, MLP, decode step and model ends: a dense
single-block layer against a torch composition of library routines (RMSNorm,
nn.Linear, scaled_dot_product_attention, SiLU), decode against SPARSE prefill
(Alg. 2 applied token by token must equal Alg. 2 applied to every row at
once), and the greedy tie rule."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle.layer import Spec, qkv_projection

from paper_2609_13141_amd import configs, inputs


def small_workload(**kw):
    base = dict(name="t", dtype="f32", batch=2, seq_len=40, d_model=64, n_heads=4, n_kv_heads=2,
                head_dim=16, d_ff=96, block_size=8, top_k=2, mode="gated",
                segments=(("img", 24), ("txt", 16)), index=90)
    base.update(kw)
    return configs.Workload(**base)


def spec_of(w, mode=None):
    return Spec(w.n_heads, w.n_kv_heads, w.head_dim, w.block_size, w.top_k, mode or w.mode,
                w.dtype, w.rope_base, w.rms_eps)


def f64(a):
    return np.asarray(a, dtype=np.float64)


def test_dense_single_block_layer_matches_torch_composition():
    w = small_workload(block_size=64)
    x = f64(inputs.embeddings(w))
    W = {k: (None if v is None else f64(v)) for k, v in inputs.layer_weights(w).items()}
    out = oracle.layer_forward(x, W, spec_of(w))
    rho = lambda a: torch.from_numpy(oracle.round_f32(a.numpy()))
    t = lambda a: torch.from_numpy(a)
    b, n, d = x.shape
    H, Hkv, dh = w.n_heads, w.n_kv_heads, w.head_dim
    u1 = rho(F.rms_norm(t(x), (d,), weight=t(W["rms1"]), eps=w.rms_eps))
    pos = np.arange(n)
    q = rho(t(oracle.rope(F.linear(u1, t(W["wq"])).reshape(b, n, H, dh).numpy(), pos, w.rope_base)))
    k = rho(t(oracle.rope(F.linear(u1, t(W["wk"])).reshape(b, n, Hkv, dh).numpy(), pos, w.rope_base)))
    v = rho(F.linear(u1, t(W["wv"])).reshape(b, n, Hkv, dh))
    G = H // Hkv
    o = F.scaled_dot_product_attention(q.transpose(1, 2), k.transpose(1, 2).repeat_interleave(G, 1),
                                       v.transpose(1, 2).repeat_interleave(G, 1), is_causal=True)
    o = rho(o.transpose(1, 2).reshape(b, n, H * dh))
    h1 = rho(t(x) + F.linear(o, t(W["wo"])))
    u2 = rho(F.rms_norm(h1, (d,), weight=t(W["rms2"]), eps=w.rms_eps))
    a = rho(F.silu(F.linear(u2, t(W["w_gate"]))) * F.linear(u2, t(W["w_up"])))
    y = rho(h1 + F.linear(a, t(W["w_down"])))
    np.testing.assert_allclose(out["y"], y.numpy(), rtol=0, atol=2e-6 * float(y.abs().max()))
    np.testing.assert_allclose(out["h1"], h1.numpy(), rtol=0, atol=2e-6 * float(h1.abs().max()))


def test_mlp_with_zero_down_projection_is_identity():
    w = small_workload()
    W = {k: (None if v is None else f64(v)) for k, v in inputs.layer_weights(w).items()}
    W["w_down"] = np.zeros_like(W["w_down"])
    h = oracle.round_f32(np.random.default_rng(1).standard_normal((5, w.d_model)))
    np.testing.assert_array_equal(oracle.mlp_forward(h, W, spec_of(w)), h)


def test_layer_rows_subset_matches_full():
    w = small_workload(dtype="bf16")
    x = f64(inputs.embeddings(w))
    W = {k: (None if v is None else f64(v)) for k, v in inputs.layer_weights(w).items()}
    full = oracle.layer_forward(x, W, spec_of(w))
    rows = np.array([3, 17, 39])
    part = oracle.layer_forward(x, W, spec_of(w), rows=rows)
    np.testing.assert_array_equal(part["y"], full["y"][:, rows])
    np.testing.assert_array_equal(part["sel"], full["sel"][:, :, rows])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_decode_equals_sparse_prefill_row_by_row(dtype):
    # Dense prefill of the first n0 tokens fills the cache; decoding tokens
    # n0..n-1 one at a time (teacher forced on the same inputs) must equal the
    # SPARSE-mode layer applied to the whole sequence at those rows.
    w = small_workload(dtype=dtype, seq_len=56, segments=(("img", 40), ("txt", 16)))
    x = f64(inputs.embeddings(w))
    W = {k: (None if v is None else f64(v)) for k, v in inputs.layer_weights(w, selector_proj=True).items()}
    n, n0 = w.seq_len, 21
    sp = spec_of(w, "sparse")
    ref = oracle.layer_forward(x, W, sp)
    cache = oracle.DecodeCache(w.batch, n, sp)
    pre = oracle.layer_forward(x[:, :n0], W, spec_of(w, "dense"))
    for bi in range(w.batch):
        cache.fill_prefill(bi, pre["K"][bi], pre["V"][bi], pre["k_summary"][bi])
    np.testing.assert_array_equal(pre["y"], oracle.layer_forward(x[:, :n0], W, spec_of(w, "dense"))["y"])
    for t in range(n0, n):
        y, sel = oracle.decode_step(x[:, t], np.full(w.batch, t), W, cache, sp)
        np.testing.assert_allclose(y, ref["y"][:, t], rtol=0, atol=1e-12)
        np.testing.assert_array_equal(sel, ref["sel"][:, :, t])
    np.testing.assert_array_equal(cache.K[:, :n], ref["K"])


def test_lm_head_greedy_lowest_id_on_ties():
    d, V = 8, 6
    h = np.ones((2, d))
    w_lm = np.zeros((V, d))
    w_lm[2] = 1.0
    w_lm[4] = 1.0          # tie between ids 2 and 4
    w_lm[5, 0] = -1.0
    tok, logits = oracle.lm_head_argmax(h, np.ones(d), w_lm, 1e-6, "bf16")
    assert list(tok) == [2, 2]
    u = oracle.round_bf16(np.array([1 / math.sqrt(1 + 1e-6)]))[0]    # RMSNorm of a constant row
    assert logits[0, 2] == d * u and logits[0, 5] == -u


def test_embed_tokens_places_image_rows_in_order():
    table = np.arange(12.0).reshape(4, 3)
    ids = np.array([[-1, 2, -1, 0]])
    img = np.array([[[100.0, 101, 102], [200, 201, 202]]])
    x = oracle.embed_tokens(ids, table, img)
    np.testing.assert_array_equal(x[0], [[100, 101, 102], [6, 7, 8], [200, 201, 202], [0, 1, 2]])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dense_prefill_layer_equals_layer_forward_dense(dtype):
    # the serving prefill's layer (masked-matrix attention) equals the per-row
    # layer in DENSE mode, and the cache contents are its K, V and summaries
    w = small_workload(dtype=dtype, seq_len=70, segments=(("img", 30), ("txt", 40)), block_size=16)
    x = f64(inputs.embeddings(w))
    W = {k: (None if v is None else f64(v)) for k, v in inputs.layer_weights(w, selector_proj=True).items()}
    sp = spec_of(w, "dense")
    full = oracle.layer_forward(x, W, sp)
    for bi in range(w.batch):
        d = oracle.dense_prefill_layer(x[bi], W, sp)
        np.testing.assert_array_equal(d["K"], full["K"][bi])
        np.testing.assert_array_equal(d["V"], full["V"][bi])
        np.testing.assert_array_equal(d["k_summary"], full["k_summary"][bi])
        tol = 1e-12 * float(np.abs(full["y"][bi]).max())
        # roundings of O may differ where the two fp64 attention forms straddle a tie: compare h1/y loosely
        np.testing.assert_allclose(d["O_exact"], full["O_exact"][bi], rtol=0, atol=1e-12)
        np.testing.assert_allclose(d["y"], full["y"][bi], rtol=0, atol=max(tol, 4 * float(np.abs(d["y"]).max())
                                                                             * (2 ** -8 if dtype == "bf16" else 2 ** -23)))
