"""Pins of the oracle's SAS attention (Eq. ours_train; Alg. 2's sparse set;
Eq. fula for dense) against closed forms, torch's scaled_dot_product_attention
on the special cases that reduce to textbook attention, and causality."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle.layer import Spec


def bf16(rng, shape, scale=1.0):
    return oracle.round_bf16(rng.standard_normal(shape) * scale)


def run(Q, K, V, B, K_top, mode, dtype="bf16"):
    H, Hkv, dh = Q.shape[1], K.shape[1], Q.shape[2]
    spec = Spec(H, Hkv, dh, B, K_top, mode, dtype)
    return oracle.attention_prefill(Q[None], K[None], V[None], spec)


def sdpa(Q, K, V, mask=None, causal=False):
    """torch reference, fp64: Q[n,H,dh], K/V[n,Hkv,dh] -> O[n,H,dh], LSE[H,n]."""
    H, Hkv, dh = Q.shape[1], K.shape[1], Q.shape[2]
    G = H // Hkv
    q = torch.from_numpy(Q).permute(1, 0, 2)[None]
    k = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    v = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(G, dim=0)[None]
    sm = 1.0 / math.sqrt(dh)
    if causal:
        n = Q.shape[0]
        mask = torch.ones(n, n, dtype=torch.bool).tril()
    o = F.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=sm)
    logits = (q @ k.transpose(-1, -2)) * sm
    if mask is not None:
        logits = logits.masked_fill(~mask, -math.inf) if mask.dtype == torch.bool else logits + mask
    lse = torch.logsumexp(logits, dim=-1)
    return o[0].permute(1, 0, 2).numpy(), lse[0].numpy()


@pytest.mark.parametrize("mode", ["gated", "sparse", "dense"])
def test_single_block_reduces_to_causal_attention(mode):
    rng = np.random.default_rng(20)
    n, H, Hkv, dh = 40, 4, 2, 16
    Q, K, V = bf16(rng, (n, H, dh)), bf16(rng, (n, Hkv, dh)), bf16(rng, (n, Hkv, dh))
    out = run(Q, K, V, 64, 3, mode)          # B >= n: only the current block
    o, lse = sdpa(Q, K, V, causal=True)
    np.testing.assert_allclose(out["O_exact"][0], o, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out["LSE"][0], lse, rtol=1e-12, atol=1e-12)


def test_sparse_with_budget_covering_all_blocks_is_dense():
    rng = np.random.default_rng(21)
    n, H, Hkv, dh, B = 100, 3, 1, 8, 16
    Q, K, V = bf16(rng, (n, H, dh)), bf16(rng, (n, Hkv, dh)), bf16(rng, (n, Hkv, dh))
    out = run(Q, K, V, B, n // B + 1, "sparse")
    o, lse = sdpa(Q, K, V, causal=True)
    np.testing.assert_allclose(out["O_exact"][0], o, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out["LSE"][0], lse, rtol=1e-12, atol=1e-12)
    dense = run(Q, K, V, B, 0, "dense")
    np.testing.assert_array_equal(dense["O"][0], out["O"][0])


@pytest.mark.parametrize("mode", ["gated", "sparse"])
def test_zero_budget_is_block_local_causal_attention(mode):
    rng = np.random.default_rng(22)
    n, H, Hkv, dh, B = 70, 2, 2, 8, 16
    Q, K, V = bf16(rng, (n, H, dh)), bf16(rng, (n, Hkv, dh)), bf16(rng, (n, Hkv, dh))
    out = run(Q, K, V, B, 0, mode)
    i = torch.arange(n)
    mask = (i[:, None] >= i[None, :]) & ((i[:, None] // B) == (i[None, :] // B))
    o, lse = sdpa(Q, K, V, mask=mask)
    np.testing.assert_allclose(out["O_exact"][0], o, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out["LSE"][0], lse, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("mode", ["gated", "sparse", "dense"])
@pytest.mark.parametrize("K_top", [0, 2, 5])
def test_zero_query_closed_form(mode, K_top):
    # q = 0: every logit and every selector score is 0, so the lowest
    # min(K, C_t) blocks are selected (tie rule) and g = 1/C_t for all blocks.
    rng = np.random.default_rng(23)
    n, H, Hkv, dh, B = 75, 2, 1, 8, 8
    Q = np.zeros((n, H, dh))
    K, V = bf16(rng, (n, Hkv, dh)), bf16(rng, (n, Hkv, dh))
    out = run(Q, K, V, B, K_top, mode)
    for t in range(n):
        c = t // B
        kk = min(K_top, c)
        b0 = c * B
        rt = t - b0 + 1
        v_cur = V[b0:t + 1, 0].sum(axis=0)
        v_sel = V[:kk * B, 0].sum(axis=0)
        if mode == "dense":
            o, l = V[:t + 1, 0].sum(axis=0) / (t + 1), math.log(t + 1)
        elif c == 0:
            o, l = v_cur / rt, math.log(rt)
        elif mode == "gated":
            o = (v_cur + v_sel / c) / (rt + B * kk / c)
            l = math.log(rt + B * kk / c)
        else:
            o, l = (v_cur + v_sel) / (rt + B * kk), math.log(rt + B * kk)
        for h in range(H):
            np.testing.assert_allclose(out["O_exact"][0, t, h], o, rtol=1e-12, atol=1e-13)
            assert abs(out["LSE"][0, h, t] - l) < 1e-12
        if mode != "dense":
            assert [int(m) for m in out["sel"][0, 0, t] if m >= 0] == list(range(kk))
            if c:
                np.testing.assert_allclose(out["log_gate"][0, 0, t, :c], -math.log(c), atol=1e-13)


@pytest.mark.parametrize("mode", ["gated", "sparse", "dense"])
def test_constant_values_give_constant_output(mode):
    rng = np.random.default_rng(24)
    n, H, Hkv, dh, B = 90, 4, 2, 8, 16
    Q, K = bf16(rng, (n, H, dh), 2.0), bf16(rng, (n, Hkv, dh), 2.0)
    V = np.full((n, Hkv, dh), 1.5)
    out = run(Q, K, V, B, 2, mode)
    np.testing.assert_array_equal(out["O"][0], 1.5)


def test_gated_equals_dense_masked_matrix_with_log_gate_bias():
    # naive materialised form: a dense logit matrix with the gate bias added on
    # selected historical blocks, 0 on the current block and -inf elsewhere
    rng = np.random.default_rng(25)
    n, H, Hkv, dh, B, Kt = 130, 4, 2, 16, 16, 3
    Q, K, V = bf16(rng, (n, H, dh)), bf16(rng, (n, Hkv, dh)), bf16(rng, (n, Hkv, dh))
    out = run(Q, K, V, B, Kt, "gated")
    G = H // Hkv
    for g in range(Hkv):
        bias = torch.full((n, n), -math.inf, dtype=torch.float64)
        for t in range(n):
            b0 = (t // B) * B
            bias[t, b0:t + 1] = 0.0
            for m in out["sel"][0, g, t]:
                if m >= 0:
                    bias[t, m * B:(m + 1) * B] = float(out["log_gate"][0, g, t, m])
        hs = slice(g * G, (g + 1) * G)
        o, lse = sdpa(Q[:, hs], K[:, g:g + 1], V[:, g:g + 1], mask=bias)
        np.testing.assert_allclose(out["O_exact"][0][:, hs], o, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(out["LSE"][0][hs], lse, rtol=1e-12, atol=1e-12)


def test_gated_full_scope_soft_weights_are_bounded():
    # Eq. rank_unbounded: with every historical block kept, the gated weights
    # g_b(i) e^{z_i} / sum_j g_b(j) e^{z_j} are each <= 1 and sum to 1; the
    # oracle's LSE is that normaliser.
    rng = np.random.default_rng(26)
    n, H, Hkv, dh, B = 64, 1, 1, 8, 8
    Q, K, V = bf16(rng, (n, H, dh), 3.0), bf16(rng, (n, Hkv, dh), 3.0), bf16(rng, (n, Hkv, dh))
    out = run(Q, K, V, B, 100, "gated")
    sm = 1.0 / math.sqrt(dh)
    for t in range(n):
        c = t // B
        z = sm * (K[:t + 1, 0] @ Q[t, 0])
        logg = np.zeros(t + 1)
        for i in range(c * B):
            logg[i] = out["log_gate"][0, 0, t, i // B]
        w = np.exp(z + logg - out["LSE"][0, 0, t])
        assert np.all(w <= 1.0 + 1e-12)
        assert abs(w.sum() - 1.0) < 1e-12
        np.testing.assert_allclose(w @ V[:t + 1, 0], out["O_exact"][0, t, 0], rtol=1e-11, atol=1e-12)


def test_causality_of_outputs_and_selection():
    rng = np.random.default_rng(27)
    n, H, Hkv, dh, B, t0 = 96, 2, 1, 8, 8, 50
    Q, K, V = bf16(rng, (n, H, dh)), bf16(rng, (n, Hkv, dh)), bf16(rng, (n, Hkv, dh))
    a = run(Q, K, V, B, 2, "gated")
    Q2, K2, V2 = Q.copy(), K.copy(), V.copy()
    Q2[t0 + 1:] = bf16(rng, Q2[t0 + 1:].shape)
    K2[t0 + 1:] = bf16(rng, K2[t0 + 1:].shape)
    V2[t0 + 1:] = bf16(rng, V2[t0 + 1:].shape)
    b = run(Q2, K2, V2, B, 2, "gated")
    np.testing.assert_array_equal(a["O"][0, :t0 + 1], b["O"][0, :t0 + 1])
    np.testing.assert_array_equal(a["sel"][0, :, :t0 + 1], b["sel"][0, :, :t0 + 1])
    np.testing.assert_array_equal(a["LSE"][0, :, :t0 + 1], b["LSE"][0, :, :t0 + 1])
    assert not np.array_equal(a["O"][0, t0 + 1:], b["O"][0, t0 + 1:])


def test_gate_shift_leaves_attention_unchanged():
    # Eq. normalized_log_gate: adding the same constant to every score of a
    # query changes neither the gates nor the output
    rng = np.random.default_rng(28)
    n, H, Hkv, dh, B = 80, 2, 1, 8, 8
    Q, K, V = bf16(rng, (n, H, dh)), bf16(rng, (n, Hkv, dh)), bf16(rng, (n, Hkv, dh))
    st = oracle.select(Q, K, B, 3, "bf16")
    G = H // Hkv
    lg2 = oracle.normalized_log_gate(st["r"] + 5.0 * G * math.sqrt(dh), st["ct"], G, dh)
    lg2f = np.full_like(st["log_gate"], -np.inf)
    lg2f[:, :, :lg2.shape[2]] = lg2
    o1, oe1, l1 = oracle.sas_attention(Q, K, V, B, "gated", "bf16", sel=st["sel"], log_gate=st["log_gate"])
    o2, oe2, l2 = oracle.sas_attention(Q, K, V, B, "gated", "bf16", sel=st["sel"], log_gate=lg2f)
    np.testing.assert_allclose(oe2, oe1, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(l2, l1, rtol=1e-11, atol=1e-12)


def test_rows_subset_matches_full():
    rng = np.random.default_rng(29)
    n, H, Hkv, dh, B = 77, 4, 2, 8, 8
    Q, K, V = bf16(rng, (n, H, dh)), bf16(rng, (n, Hkv, dh)), bf16(rng, (n, Hkv, dh))
    spec = Spec(H, Hkv, dh, B, 2, "gated", "bf16")
    full = oracle.attention_prefill(Q[None], K[None], V[None], spec)
    rows = np.array([0, 9, 40, 76])
    part = oracle.attention_prefill(Q[None][:, rows], K[None], V[None], spec, rows=rows)
    np.testing.assert_array_equal(part["O"][0], full["O"][0][rows])
    np.testing.assert_array_equal(part["sel"][0], full["sel"][0][:, rows])
    np.testing.assert_array_equal(part["LSE"][0], full["LSE"][0][:, rows])


@pytest.mark.parametrize("H,Hkv", [(4, 2), (3, 3), (6, 1)])
def test_causal_attention_matches_sdpa_and_the_gather_form(H, Hkv):
    # the masked-matrix form of Eq. fula equals torch's causal attention and the
    # oracle's per-row gather form in DENSE mode, over many blocks
    rng = np.random.default_rng(30 + H)
    n, dh = 150, 16
    Q, K, V = bf16(rng, (n, H, dh)), bf16(rng, (n, Hkv, dh)), bf16(rng, (n, Hkv, dh))
    O, Oe, LSE = oracle.causal_attention(Q, K, V, "bf16")
    o, lse = sdpa(Q, K, V, causal=True)
    np.testing.assert_allclose(Oe, o, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(LSE, lse, rtol=1e-12, atol=1e-12)
    out = run(Q, K, V, 16, 2, "dense")
    np.testing.assert_allclose(Oe, out["O_exact"][0], rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(O, oracle.round_bf16(Oe))
