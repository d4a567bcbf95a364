"""Pins of the oracle's selector: exact rational brute force, planted
rankings, the gate's invariants (Eq. normalized_log_gate: softmax gates sum to
one and are invariant to a global shift of the scores) and monotonicity of
the Top-K (Alg. 1 ranks g, Alg. 2 ranks s: the same blocks)."""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle.selector import project_summaries


def bf16_values(rng, shape, scale=1.0):
    return oracle.round_bf16(rng.standard_normal(shape) * scale)


def frac_round_bf16(fr):
    return Fraction(oracle.round_bf16(np.array([float(fr)]))[0]) if _exact_double(fr) else None


def _exact_double(fr):
    return Fraction(float(fr)) == fr


def test_summaries_and_scores_equal_exact_rationals():
    rng = np.random.default_rng(10)
    n, H, Hkv, dh, B = 48, 4, 2, 16, 8
    Q = bf16_values(rng, (n, H, dh))
    K = bf16_values(rng, (n, Hkv, dh))
    st = oracle.select(Q, K, B, 3, "bf16")
    G = H // Hkv
    for g in range(Hkv):
        for m in range(n // B):
            for j in range(dh):
                ex = sum(Fraction(K[i, g, j]) for i in range(m * B, (m + 1) * B)) / B
                assert _exact_double(ex)                      # mean of B bf16 values is exact in fp64
                assert Fraction(st["kbar"][g, m, j]) == Fraction(oracle.round_bf16(np.array([float(ex)]))[0])
        for t in range(n):
            qs = [sum(Fraction(Q[t, h, j]) for h in range(g * G, (g + 1) * G)) for j in range(dh)]
            qh = [Fraction(oracle.round_bf16(np.array([float(v)]))[0]) for v in qs]
            assert [Fraction(v) for v in st["qhat"][g, t]] == qh
            for m in range(n // B):
                ex = sum(qh[j] * Fraction(st["kbar"][g, m, j]) for j in range(dh))
                assert Fraction(st["r"][g, t, m]) == ex           # bf16 dot products are exact in fp64


def test_topk_brute_force_with_exact_keys():
    rng = np.random.default_rng(11)
    n, H, Hkv, dh, B, K = 96, 2, 1, 8, 8, 4
    Q = bf16_values(rng, (n, H, dh))
    Kk = bf16_values(rng, (n, Hkv, dh))
    # duplicate a block so that exact ties occur and the tie rule is exercised
    Kk[8:16] = Kk[0:8]
    st = oracle.select(Q, Kk, B, K, "bf16")
    ties_seen = 0
    for t in range(n):
        c = t // B
        keys = []
        for m in range(c):
            ex = sum(Fraction(st["qhat"][0, t, j]) * Fraction(st["kbar"][0, m, j]) for j in range(dh))
            keys.append((ex, m))
        ranked = sorted(keys, key=lambda km: (-km[0], km[1]))
        want = sorted(m for _, m in ranked[:min(K, c)])
        got = [int(m) for m in st["sel"][0, t] if m >= 0]
        assert got == want, (t, got, want)
        assert all(m == -1 for m in st["sel"][0, t][len(want):])
        if c >= 2 and keys[0][0] == keys[1][0]:
            ties_seen += 1
    assert ties_seen > 0


def test_planted_ranking():
    n, H, Hkv, dh, B, K = 128, 1, 1, 4, 16, 3
    alphas = [0.5, 4.0, -1.0, 2.0, 3.0, 0.25, 1.0, 8.0]
    Kk = np.zeros((n, Hkv, dh))
    for m, a in enumerate(alphas):
        Kk[m * B:(m + 1) * B, 0, 0] = a
    Q = np.zeros((n, H, dh))
    Q[:, 0, 0] = 1.0
    st = oracle.select(Q, Kk, B, K, "bf16")
    for t in range(n):
        c = t // B
        want = sorted(sorted(range(c), key=lambda m: (-alphas[m], m))[:min(K, c)])
        assert [int(m) for m in st["sel"][0, t] if m >= 0] == want
    # t = 127 (c = 7): blocks 1 (4.0), 4 (3.0), 3 (2.0)
    assert list(st["sel"][0, 127]) == [1, 3, 4]


def test_log_gate_sums_to_one_shift_invariant_and_tau():
    rng = np.random.default_rng(12)
    n, H, Hkv, dh, B, K = 200, 4, 2, 32, 16, 4
    Q = bf16_values(rng, (n, H, dh))
    Kk = bf16_values(rng, (n, Hkv, dh))
    st = oracle.select(Q, Kk, B, K, "bf16")
    lg, ct = st["log_gate"], st["ct"]
    G = H // Hkv
    for t in range(n):
        c = int(ct[t])
        if c == 0:
            assert np.all(np.isneginf(lg[:, t]))
            continue
        np.testing.assert_allclose(np.exp(lg[:, t, :c]).sum(axis=1), 1.0, rtol=1e-13)
        assert np.all(np.isneginf(lg[:, t, c:]))
        for g in range(Hkv):
            chosen = [int(m) for m in st["sel"][g, t] if m >= 0]
            # Top-K of g equals Top-K of r (softmax is monotone)
            by_gate = sorted(np.lexsort((np.arange(c), -lg[g, t, :c]))[:min(K, c)].tolist())
            assert by_gate == chosen
            tau = st["tau"][g, t]
            if c <= K:
                assert tau == -np.inf
            else:
                assert set(np.nonzero(lg[g, t, :c] >= tau)[0].tolist()) == set(chosen)
    # s -> s + const leaves the normalized log gate unchanged (Eq. normalized_log_gate)
    shift = 3.7 * G * math.sqrt(dh)
    lg2 = oracle.normalized_log_gate(st["r"] + shift, ct, G, dh)
    lg1 = lg[:, :, :lg2.shape[2]]
    fin = np.isfinite(lg1)
    assert np.array_equal(fin, np.isfinite(lg2))
    np.testing.assert_allclose(lg2[fin], lg1[fin], rtol=0, atol=1e-12)


def test_k_zero_and_k_at_least_c():
    rng = np.random.default_rng(13)
    n, H, Hkv, dh, B = 64, 2, 2, 8, 8
    Q = bf16_values(rng, (n, H, dh))
    Kk = bf16_values(rng, (n, Hkv, dh))
    st0 = oracle.select(Q, Kk, B, 0, "bf16")
    assert st0["sel"].shape == (Hkv, n, 0)
    assert np.all(st0["tau"][:, B:] == np.inf) and np.all(st0["tau"][:, :B] == -np.inf)
    stall = oracle.select(Q, Kk, B, 100, "bf16")
    for t in range(n):
        c = t // B
        for g in range(Hkv):
            assert [int(m) for m in stall["sel"][g, t] if m >= 0] == list(range(c))


def test_gate_query_projection_is_exact_matvec():
    rng = np.random.default_rng(14)
    n, H, Hkv, dh, B = 32, 4, 2, 8, 8
    Q = bf16_values(rng, (n, H, dh))
    Kk = bf16_values(rng, (n, Hkv, dh))
    W = bf16_values(rng, (Hkv, dh, dh), 0.3)
    st = oracle.select(Q, Kk, B, 2, "bf16", w_gq=W, w_gk=W)
    plain = oracle.select(Q, Kk, B, 2, "bf16")
    for g in range(Hkv):
        for t in range(0, n, 5):
            for k in range(dh):
                ex = sum(Fraction(W[g, k, j]) * Fraction(plain["qhat"][g, t, j]) for j in range(dh))
                assert Fraction(st["qhat"][g, t, k]) == Fraction(oracle.round_bf16(np.array([float(ex)]))[0])
    kb = project_summaries(plain["kbar"], W, "bf16")
    np.testing.assert_array_equal(st["kbar_proj"], kb)


def test_f32_selector_is_sequential_fp64():
    # fp32 inputs: products are exact in fp64 but sums are not; the contract
    # is the ascending-index sequential fp64 sum
    rng = np.random.default_rng(15)
    n, H, Hkv, dh, B = 32, 2, 1, 16, 8
    Q = oracle.round_f32(rng.standard_normal((n, H, dh)))
    Kk = oracle.round_f32(rng.standard_normal((n, Hkv, dh)))
    st = oracle.select(Q, Kk, B, 2, "f32")
    for m in range(n // B):
        acc = np.zeros(dh)
        for i in range(m * B, (m + 1) * B):
            acc = acc + Kk[i, 0]
        np.testing.assert_array_equal(st["kbar"][0, m], oracle.round_f32(acc / B))
    t = 30
    acc = 0.0
    for j in range(dh):
        acc = acc + float(st["qhat"][0, t, j]) * float(st["kbar"][0, 2, j])
    assert st["r"][0, t, 2] == acc


def test_decode_select_brute_force_with_exact_keys():
    # Alg. 2's selection alone: gate query of the group's heads against the
    # cached summaries of the floor(pos/B) complete blocks, Top-K under
    # (r desc, m asc), ascending output, -1 padding; positions past the cache
    # capacity see only the cached blocks
    rng = np.random.default_rng(12)
    b, H, Hkv, dh, B, K, M = 3, 4, 2, 8, 16, 5, 40
    q = bf16_values(rng, (b, H, dh))
    kbar = bf16_values(rng, (b, Hkv, M, dh))
    kbar[:, :, 7] = kbar[:, :, 3]          # exact ties: the lower block must win
    kbar[:, :, 20] = kbar[:, :, 3]
    spec = oracle.Spec(H, Hkv, dh, B, K, "sparse", "bf16", 10000.0, 1e-6)
    G = H // Hkv
    for pos in ([0, 15, 16], [4 * B + 3, 5 * B, 6 * B - 1], [21 * B + 2, M * B + 70, -1]):
        sel, _ = oracle.decode_select(q, np.array(pos), kbar, spec)
        for bi in range(b):
            c = 0 if pos[bi] < 0 else min(pos[bi] // B, M)
            for g in range(Hkv):
                qs = [sum(Fraction(q[bi, h, j]) for h in range(g * G, (g + 1) * G)) for j in range(dh)]
                qh = [Fraction(oracle.round_bf16(np.array([float(v)]))[0]) for v in qs]
                keys = [(sum(qh[j] * Fraction(kbar[bi, g, m, j]) for j in range(dh)), m) for m in range(c)]
                ranked = sorted(keys, key=lambda km: (-km[0], km[1]))
                want = sorted(m for _, m in ranked[:min(K, c)])
                got = [int(m) for m in sel[bi, g] if m >= 0]
                assert got == want, (pos[bi], g, got, want)
                assert all(m == -1 for m in sel[bi, g][len(want):])
