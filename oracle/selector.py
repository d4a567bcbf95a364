"""SAS block selector: block summaries, gate query, scores, normalized log
gate and Top-K selection, in float64.

Sec. 3 (block sparse attention): the context is cut into contiguous blocks of
B tokens and a selector scores them; Eq. selected_context keeps the Top-K.
Sec. 4.1: the block holding the query is the always-retained current block
B_0; the selector ranks only the earlier (historical) blocks.  For query t
those are m = 0 .. C_t - 1 with C_t = floor(t / B), all complete.

The selector's architecture is not given in the paper (it reuses an existing
gate module).  Its clues are: a gate query projected and dot-multiplied with
block summaries (Sec. 6.3, decode step cost breakdown), pooling of keys, and
one selection shared by all query heads of a KV group (Sec. 5.1, inference;
Sec. 5.3).  The reading implemented here:

* summary  kbar[g, m] = rho( (sum_{i in B_m} K[i, g]) / B ), sum in fp64 over
  ascending i;
* gate query  qhat[g, t] = rho( sum_{h in group g} Q[t, h] ), ascending h;
* optional per-group projections qhat <- rho(W_gq[g] qhat),
  kbar <- rho(W_gk[g] kbar) (identity when absent);
* score r[g, t, m] = sum_j qhat[g,t,j] * kbar[g,m,j], sequential fp64 sum over
  ascending j (each product of two bf16/fp32 values is exact in fp64);
* s = r / (G * sqrt(dh)); log g = s - LSE(s) over the C_t historical blocks
  (Eq. normalized_log_gate);
* selection: the min(K, C_t) blocks that are largest under the total order
  (r descending, m ascending) -- Top-K of g equals Top-K of s equals Top-K of
  r because softmax and the positive scaling are monotone (Alg. 1 ranks g,
  Alg. 2 ranks s).

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import math

import numpy as np

from .numerics import rho


def block_summaries(K, B, dtype):
    """K[n, Hkv, dh] -> kbar[Hkv, n // B, dh]: mean-pooled keys of every
    complete block, summed in fp64 over ascending token index."""
    K = np.asarray(K, dtype=np.float64)
    n, Hkv, dh = K.shape
    nf = n // B
    kbar = np.zeros((Hkv, nf, dh))
    for m in range(nf):
        acc = np.zeros((Hkv, dh))
        for i in range(m * B, (m + 1) * B):
            acc = acc + K[i]
        kbar[:, m, :] = rho(acc / B, dtype)
    return kbar


def _project(v, W, dtype):
    """out[g, r, k] = rho( sum_j W[g, k, j] * v[g, r, j] ), ascending j."""
    Hkv, R, dh = v.shape
    acc = np.zeros((Hkv, R, W.shape[1]))
    for j in range(dh):
        acc = acc + v[:, :, j:j + 1] * W[:, None, :, j]
    return rho(acc, dtype)


def gate_query(Q, G, dtype, w_gq=None):
    """Q[n, H, dh] -> qhat[Hkv, n, dh]: the group's query heads summed in
    fp64 over ascending head index, then optionally projected by W_gq."""
    Q = np.asarray(Q, dtype=np.float64)
    n, H, dh = Q.shape
    Hkv = H // G
    qh = np.zeros((Hkv, n, dh))
    for g in range(Hkv):
        acc = np.zeros((n, dh))
        for h in range(g * G, (g + 1) * G):
            acc = acc + Q[:, h, :]
        qh[g] = rho(acc, dtype)
    if w_gq is not None:
        qh = _project(qh, np.asarray(w_gq, dtype=np.float64), dtype)
    return qh


def project_summaries(kbar, w_gk, dtype):
    if w_gk is None:
        return kbar
    return _project(kbar, np.asarray(w_gk, dtype=np.float64), dtype)


def selector_scores(qhat, kbar):
    """r[g, t, m] = sum_j qhat[g,t,j] kbar[g,m,j], sequential fp64 sum."""
    Hkv, n, dh = qhat.shape
    nf = kbar.shape[1]
    r = np.zeros((Hkv, n, nf))
    for j in range(dh):
        r = r + qhat[:, :, j, None] * kbar[:, None, :, j]
    return r


def normalized_log_gate(r, ct, G, dh):
    """Eq. normalized_log_gate: log g_m = s_m - LSE_{m' < C_t}(s_m'), with
    s = r / (G sqrt(dh)).  r[Hkv, R, nf]; ct[R] = historical block count of
    each row.  Entries m >= C_t are -inf (not historical for that query)."""
    s = r / (G * math.sqrt(dh))
    R = r.shape[1]
    lg = np.full(r.shape, -np.inf)
    for row in range(R):
        c = int(ct[row])
        if c == 0:
            continue
        srow = s[:, row, :c]                                          # [Hkv, c]
        mx = srow.max(axis=1, keepdims=True)
        lse = mx + np.log(np.exp(srow - mx).sum(axis=1, keepdims=True))
        lg[:, row, :c] = srow - lse
    return lg


def topk_blocks(r_row, c, K):
    """Selected historical blocks of one query: the min(K, c) indices m < c
    largest under (r desc, m asc), returned ascending, plus the rank order."""
    kk = min(K, c)
    if kk == 0:
        return np.zeros(0, dtype=np.int64), np.zeros(0, dtype=np.int64)
    cand = np.arange(c)
    order = np.lexsort((cand, -np.asarray(r_row[:c], dtype=np.float64)))
    top = order[:kk]
    return np.sort(top), top


def select(Q, K, B, top_k, dtype, rows=None, w_gq=None, w_gk=None):
    """Full selector for one sequence.  K[n,Hkv,dh]; Q[R,H,dh] holds the
    query rows listed in ``rows`` (all n rows, in order, when it is None).

    Returns a dict with kbar[Hkv, n//B, dh], qhat[Hkv, R, dh], r[Hkv, R, nf],
    log_gate[Hkv, R, NB] (NB = ceil(n/B), -inf where undefined),
    sel[Hkv, R, K] (ascending, -1 padded), tau[Hkv, R] and the row indices.
    tau is the log gate of the lowest-ranked selected block when C_t > K >= 1
    (so that "log g >= tau" marks the selected blocks, up to ties), +inf when
    K = 0 < C_t, and -inf when C_t <= K (every historical block is kept).
    """
    n, Hkv, dh = K.shape
    H = Q.shape[1]
    G = H // Hkv
    rows = np.arange(n) if rows is None else np.asarray(rows)
    R = len(rows)
    assert Q.shape[0] == R
    NB = -(-n // B)
    kbar = block_summaries(K, B, dtype)
    kb = project_summaries(kbar, w_gk, dtype)
    qhat = gate_query(Q, G, dtype, w_gq)
    r = selector_scores(qhat, kb)                                     # [Hkv, R, nf]
    ct = rows // B
    lg_f = normalized_log_gate(r, ct, G, dh)
    log_gate = np.full((Hkv, R, NB), -np.inf)
    log_gate[:, :, :lg_f.shape[2]] = lg_f
    sel = np.full((Hkv, R, max(top_k, 0)), -1, dtype=np.int64)
    tau = np.full((Hkv, R), -np.inf)
    for g in range(Hkv):
        for ri in range(R):
            c = int(ct[ri])
            chosen, order = topk_blocks(r[g, ri], c, top_k)
            sel[g, ri, :len(chosen)] = chosen
            if c > top_k:
                # lowest-ranked selected block; nothing selected (K = 0): +inf
                tau[g, ri] = log_gate[g, ri, order[-1]] if len(order) else np.inf
    return {"kbar": kbar, "kbar_proj": kb, "qhat": qhat, "r": r, "log_gate": log_gate,
            "sel": sel, "tau": tau, "rows": rows, "ct": ct}
