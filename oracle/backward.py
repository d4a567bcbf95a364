"""Backward of SAS attention and of its selector, in float64, gather form.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Attention (Sec. 4.3, Eq. ours_train; App. E, the recomputation-based
backward).  For head h of group g and query t, with the forward's set S,
bias and z_i = sm q.k_i + bias_i, p = softmax(z) over S, o = sum p_i v_i,
and an upstream gradient dO:

  dp_i = dO . v_i,   Delta = dO . o,   ds_i = p_i (dp_i - Delta)
  dq = sm sum_i ds_i k_i,   dk_i += sm ds_i q,   dv_i += p_i dO
  dlog g[g, t, m] = sum_{h in g} sum_{i in B_m} ds_i   (selected blocks, GATED)

The last line is Eq. gate_posi's inner-gate gradient expressed for the log
gate (dlog g_m = g_m dg_m = sum_{i in B_m} p_i dO.(v_i - o)).

Gate (Eq. normalized_log_gate).  log g_m = s_m - LSE_{m' < C_t}(s), so
ds_m = dlog g_m - g_m sum_{m' < C_t} dlog g_{m'} with g = softmax(s) over the
historical blocks.  Only selected blocks carry a bias, so dlog g is zero on
the others; the Top-K set is piecewise constant and passes no gradient.

Selector (this implementation's reading of the paper's undefined selector): s =
r / (G sqrt(dh)), r = qhat . kbar, qhat = rho(qhat0 W_gq^T) and kbar =
rho(kbar0 W_gk^T) when the projections exist (qhat0 = rho(sum of the group's
query heads), kbar0 = rho(mean pooled keys)).  The backward treats the
roundings as identities and stops at the selector parameters: Alg. 1 updates
theta (W_gq, W_gk) only.
"""
import math

import numpy as np


def _sets(t, g, B, mode, sel_row, log_gate_row):
    """Key indices of query t in group g and the bias of each, plus the block
    of each key when it is a selected historical block (else -1)."""
    b0 = (t // B) * B
    if mode == "dense":
        idx = np.arange(0, t + 1)
        return idx, np.zeros(t + 1), np.full(t + 1, -1)
    blocks = [int(m) for m in sel_row if m >= 0]
    idx = np.concatenate([np.arange(m * B, (m + 1) * B) for m in blocks] + [np.arange(b0, t + 1)])
    blk = np.concatenate([np.full(B, m) for m in blocks] + [np.full(t + 1 - b0, -1)])
    if mode == "gated":
        bias = np.concatenate([np.full(B, log_gate_row[m]) for m in blocks] + [np.zeros(t + 1 - b0)])
    else:
        bias = np.zeros(len(idx))
    return idx, bias, blk


def sas_attention_backward(Q, K, V, dO, B, mode, sel=None, log_gate=None, sm_scale=None):
    """One sequence: Q, dO[n, H, dh]; K, V[n, Hkv, dh]; sel[Hkv, n, K];
    log_gate[Hkv, n, NB].  Returns dQ[n, H, dh], dK, dV[n, Hkv, dh] and
    dLogG[Hkv, n, NB] (zero outside the selected blocks; GATED only)."""
    Q, K, V, dO = (np.asarray(a, dtype=np.float64) for a in (Q, K, V, dO))
    n, Hkv, dh = K.shape
    H = Q.shape[1]
    G = H // Hkv
    sm = (1.0 / math.sqrt(dh)) if (sm_scale is None or sm_scale <= 0) else float(sm_scale)
    NB = -(-n // B)
    dQ = np.zeros_like(Q)
    dK = np.zeros_like(K)
    dV = np.zeros_like(V)
    dL = np.zeros((Hkv, n, NB))
    for t in range(n):
        for g in range(Hkv):
            idx, bias, blk = _sets(t, g, B, mode, None if sel is None else sel[g, t],
                                   None if log_gate is None else log_gate[g, t])
            Kg, Vg = K[idx, g, :], V[idx, g, :]
            for h in range(g * G, (g + 1) * G):
                q, do = Q[t, h], dO[t, h]
                z = sm * (Kg @ q) + bias
                p = np.exp(z - z.max())
                p /= p.sum()
                o = p @ Vg
                ds = p * (Vg @ do - do @ o)
                dQ[t, h] = sm * (ds @ Kg)
                # the attended keys of one query are distinct (disjoint blocks), so
                # indexed accumulation adds each contribution once
                dK[idx, g, :] += sm * ds[:, None] * q[None, :]
                dV[idx, g, :] += p[:, None] * do[None, :]
                if mode == "gated":
                    for m in np.unique(blk[blk >= 0]):
                        dL[g, t, m] += ds[blk == m].sum()
    return dQ, dK, dV, dL


def gate_backward(dlog_gate, r, ct, G, dh):
    """ds[Hkv, R, nf] from dlog g[Hkv, R, >= nf] through log g = s - LSE(s) over
    the C_t historical blocks of each row (s = r / (G sqrt(dh)))."""
    r = np.asarray(r, dtype=np.float64)
    s = r / (G * math.sqrt(dh))
    ds = np.zeros_like(s)
    for ri, c in enumerate(ct):
        c = int(c)
        if c == 0:
            continue
        sr = s[:, ri, :c]
        g = np.exp(sr - sr.max(axis=1, keepdims=True))
        g /= g.sum(axis=1, keepdims=True)
        dl = np.asarray(dlog_gate[:, ri, :c], dtype=np.float64)
        ds[:, ri, :c] = dl - g * dl.sum(axis=1, keepdims=True)
    return ds


def selector_backward(ds, qhat, kbar, G, dh, qhat0=None, kbar0=None):
    """Gradients of the selector parameters from ds[Hkv, R, nf]:
    dr = ds / (G sqrt(dh)); dqhat[g, t] = sum_m dr kbar[g, m];
    dkbar[g, m] = sum_t dr qhat[g, t]; with the projections qhat = qhat0 W_gq^T,
    kbar = kbar0 W_gk^T: dW_gq[g] = dqhat^T qhat0, dW_gk[g] = dkbar^T kbar0."""
    dr = np.asarray(ds, dtype=np.float64) / (G * math.sqrt(dh))
    qhat = np.asarray(qhat, dtype=np.float64)
    kbar = np.asarray(kbar, dtype=np.float64)
    nf = dr.shape[2]
    dq = np.einsum("gtm,gmj->gtj", dr, kbar[:, :nf])
    dk = np.einsum("gtm,gtj->gmj", dr, qhat)
    out = {"dqhat": dq, "dkbar": dk}
    if qhat0 is not None:
        out["dw_gq"] = np.einsum("gtk,gtj->gkj", dq, np.asarray(qhat0, dtype=np.float64))
    if kbar0 is not None:
        out["dw_gk"] = np.einsum("gmk,gmj->gkj", dk, np.asarray(kbar0, dtype=np.float64)[:, :nf])
    return out
