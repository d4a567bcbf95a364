"""Pins of the selection statistics (Sec. 6.1: Eq. mass_coverage, Eq.
overlap_recall): torch softmax masses, closed forms (q = 0, every block
kept, equal value norms), torch.topk of block masses, and hand-worked
majority votes and recalls."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle.stats import block_mass_topk, majority_vote, mass_coverage, overlap_recall, selection_sets


def _problem(seed, n=48, B=8, H=4, Hkv=2, dh=8, K=2):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((n, H, dh))
    Kk = rng.standard_normal((n, Hkv, dh))
    V = rng.standard_normal((n, Hkv, dh))
    sel = oracle.select(Q, Kk, B, K, "f32")["sel"]
    return Q, Kk, V, sel


def test_coverage_matches_torch_softmax_mass():
    Q, Kk, V, sel = _problem(60)
    cov, cov_v = mass_coverage(Q, Kk, V, 8, sel)
    n, H, dh = Q.shape
    G = H // Kk.shape[1]
    vn = torch.linalg.vector_norm(torch.tensor(V), dim=2)
    for t in range(n):
        for h in range(H):
            g = h // G
            z = torch.tensor(Kk[:t + 1, g] @ Q[t, h]) / math.sqrt(dh)
            mask = torch.zeros(t + 1, dtype=torch.bool)
            mask[(t // 8) * 8:] = True
            for m in sel[g, t]:
                if m >= 0:
                    mask[m * 8:(m + 1) * 8] = True
            p = torch.softmax(z, 0)
            pv = p * vn[:t + 1, g]
            assert cov[h, t] == pytest.approx(float(p[mask].sum()), rel=1e-12, abs=1e-14)
            assert cov_v[h, t] == pytest.approx(float(pv[mask].sum() / pv.sum()), rel=1e-12, abs=1e-14)


def test_coverage_closed_forms():
    Q, Kk, V, sel = _problem(61)
    n = Q.shape[0]
    # q = 0: uniform weights, Cov = |S| / (t + 1)
    cov, cov_v = mass_coverage(np.zeros_like(Q), Kk, V, 8, sel)
    vn = np.linalg.norm(V, axis=2)
    for t in range(n):
        for h in range(Q.shape[1]):
            g = h // 2
            S = set(range((t // 8) * 8, t + 1)) | {i for m in sel[g, t] if m >= 0 for i in range(m * 8, m * 8 + 8)}
            assert cov[h, t] == pytest.approx(len(S) / (t + 1), rel=1e-12)
            assert cov_v[h, t] == pytest.approx(vn[list(S), g].sum() / vn[:t + 1, g].sum(), rel=1e-12)
    # every historical block kept: Cov = 1
    sel_all = oracle.select(Q, Kk, 8, 6, "f32")["sel"]
    cov, cov_v = mass_coverage(Q, Kk, V, 8, sel_all)
    np.testing.assert_allclose(cov, 1.0, rtol=1e-12)
    np.testing.assert_allclose(cov_v, 1.0, rtol=1e-12)
    # equal value norms: the value-aware weights are the raw weights
    Vn = V / np.linalg.norm(V, axis=2, keepdims=True) * 3.0
    cov, cov_v = mass_coverage(Q, Kk, Vn, 8, sel)
    np.testing.assert_allclose(cov_v, cov, rtol=1e-12)


def test_block_mass_topk_matches_torch_topk():
    Q, Kk, V, sel = _problem(62, n=64, K=3)
    sets, lmass = block_mass_topk(Q, Kk, 8, 3)
    n, H, dh = Q.shape
    G = H // Kk.shape[1]
    for t in range(n):
        c = t // 8
        for h in range(H):
            g = h // G
            z = torch.tensor(Kk[:c * 8, g] @ Q[t, h]) / math.sqrt(dh)
            if c == 0:
                assert not sets[h, t].any()
                continue
            mass = torch.softmax(torch.cat([z, torch.tensor(Kk[c * 8:t + 1, g] @ Q[t, h]) / math.sqrt(dh)]), 0)
            bm = mass[:c * 8].reshape(c, 8).sum(1)
            top = set(torch.topk(bm, min(3, c)).indices.tolist())
            assert set(np.nonzero(sets[h, t])[0].tolist()) == top


def test_majority_vote_by_hand():
    # 2 groups: G = 3 (2 of 3 is a majority) and, separately, G = 2 (1 of 2 is not)
    hs = np.zeros((6, 1, 4), dtype=bool)
    hs[0, 0, [0, 1]] = True
    hs[1, 0, [1, 2]] = True
    hs[2, 0, [1, 3]] = True
    hs[3, 0, [0]] = True
    hs[4, 0, [0, 3]] = True
    hs[5, 0, [2]] = True
    v = majority_vote(hs, 3)
    assert v[0, 0].tolist() == [False, True, False, False]
    assert v[1, 0].tolist() == [True, False, False, False]
    h2 = np.array([[[True, True, False]], [[True, False, False]]])
    assert majority_vote(h2, 2)[0, 0].tolist() == [True, False, False]


def test_overlap_recall_by_hand():
    NB = 4
    sel1 = np.array([[[0, 1]]])          # layer 1: blocks {0, 1}
    sel2 = np.array([[[2, -1]]])         # layer 2: block {2}
    m = [selection_sets(sel1, NB), selection_sets(sel2, NB)]
    o1 = np.zeros((1, 1, NB), dtype=bool)
    o1[0, 0, [1, 3]] = True
    o2 = np.zeros((1, 1, NB), dtype=bool)
    o2[0, 0, [2]] = True
    inter, tot, rec = overlap_recall(m, [o1, o2])
    assert (inter, tot) == (2, 3) and rec == pytest.approx(2 / 3)
    # a method that keeps the reference's sets recalls everything
    assert overlap_recall([o1, o2], [o1, o2])[2] == 1.0
