"""Selection-analysis statistics of Sec. 6.1, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

* Attention mass coverage (Eq. mass_coverage): for head h and query t,
  Cov(S) = sum_{i in S} w_i / sum_{j <= t} w_j over the causal context,
  with w_i = exp(z_i) or w_i = exp(z_i + log ||v_i||_2), z_i = sm q.k_i the
  attention logit (unbiased: the gate is not part of the mass).  S is the
  query's attended set: its current block and its selected blocks.
* Full-attention reference set and overlap recall (Eq. overlap_recall): per
  head, the Top-K historical blocks by full-attention mass (sum of exp(z_i)
  over the block's tokens; descending, lower block first on ties); per KV
  group, a block is in the group's set when a strict majority of the group's
  heads selected it.  Sets are unioned over layers per (query, KV group);
  Recall = |I_all n I*_all| / |I*_all| summed over every (query, group).
"""
import math

import numpy as np


def _sm(dh, sm_scale):
    return (1.0 / math.sqrt(dh)) if (sm_scale is None or sm_scale <= 0) else float(sm_scale)


def _lse(x):
    m = x.max()
    return m + math.log(np.exp(x - m).sum())


def mass_coverage(Q, K, V, B, sel, sm_scale=None):
    """One sequence: Q[n, H, dh], K/V[n, Hkv, dh], sel[Hkv, n, K] (ascending,
    -1 padded).  Returns cov[H, n] and cov_v[H, n]."""
    Q, K, V = (np.asarray(a, dtype=np.float64) for a in (Q, K, V))
    n, Hkv, dh = K.shape
    H = Q.shape[1]
    G = H // Hkv
    sm = _sm(dh, sm_scale)
    lvn = np.log(np.linalg.norm(V, axis=2))          # [n, Hkv]
    cov = np.zeros((H, n))
    cov_v = np.zeros((H, n))
    for t in range(n):
        b0 = (t // B) * B
        for g in range(Hkv):
            inS = np.zeros(t + 1, dtype=bool)
            inS[b0:] = True
            for m in sel[g, t]:
                if m >= 0:
                    inS[m * B:(m + 1) * B] = True
            for h in range(g * G, (g + 1) * G):
                z = sm * (K[:t + 1, g] @ Q[t, h])
                zv = z + lvn[:t + 1, g]
                cov[h, t] = math.exp(_lse(z[inS]) - _lse(z))
                cov_v[h, t] = math.exp(_lse(zv[inS]) - _lse(zv))
    return cov, cov_v


def block_mass_topk(Q, K, B, top_k, sm_scale=None):
    """Per-head Top-K historical blocks by full-attention mass.  Returns
    sets[H, n, NB] (bool) and the per-head block masses (log-sum-exp of the
    block's logits; -inf for non-historical blocks)."""
    Q, K = (np.asarray(a, dtype=np.float64) for a in (Q, K))
    n, Hkv, dh = K.shape
    H = Q.shape[1]
    G = H // Hkv
    NB = -(-n // B)
    sm = _sm(dh, sm_scale)
    lmass = np.full((H, n, NB), -np.inf)
    sets = np.zeros((H, n, NB), dtype=bool)
    for t in range(n):
        c = t // B
        for h in range(H):
            g = h // G
            for m in range(c):
                lmass[h, t, m] = _lse(sm * (K[m * B:(m + 1) * B, g] @ Q[t, h]))
            if c == 0 or top_k <= 0:
                continue
            order = np.lexsort((np.arange(c), -lmass[h, t, :c]))
            sets[h, t, order[:min(top_k, c)]] = True
    return sets, lmass


def majority_vote(head_sets, G):
    """head_sets[H, n, NB] -> group sets[Hkv, n, NB]: selected by more than
    half of the group's heads."""
    H, n, NB = head_sets.shape
    counts = head_sets.reshape(H // G, G, n, NB).sum(axis=1)
    return counts * 2 > G


def selection_sets(sel, NB):
    """sel[Hkv, n, K] (ascending, -1 padded) -> sets[Hkv, n, NB] (bool)."""
    Hkv, n, _ = sel.shape
    sets = np.zeros((Hkv, n, NB), dtype=bool)
    for g in range(Hkv):
        for t in range(n):
            for m in sel[g, t]:
                if m >= 0:
                    sets[g, t, m] = True
    return sets


def overlap_recall(method_sets, oracle_sets):
    """Lists over layers of sets[Hkv, n, NB] -> (|I_all n I*_all|, |I*_all|, recall)."""
    I = np.zeros_like(method_sets[0], dtype=bool)
    Istar = np.zeros_like(oracle_sets[0], dtype=bool)
    for s in method_sets:
        I |= s
    for s in oracle_sets:
        Istar |= s
    inter = int((I & Istar).sum())
    tot = int(Istar.sum())
    return inter, tot, (inter / tot if tot else float("nan"))
