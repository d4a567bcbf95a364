"""The gating formulations compared in Table 1 (Sec. 4.1-4.2; the gradients
of App. D), in float64, gather form.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A formulation is (pos, act, scope, ste) plus optional score noise:

* act (gate activation, Sec. 4.1): the log gate of historical block m of a
  query with C historical blocks is
    softmax: log g_m = s_m - LSE_{m' < C}(s)       (Eq. normalized_log_gate)
    sigmoid: log g_m = log sigmoid(s_m)
    raw:     log g_m = s_m                          (s added to the logits)
  The current block always has g = 1.
* noise (full*, Table 1 row 11): the scores are s + eps before the
  activation and before Top-K; eps is an input.
* scope: "sparse" attends the current block and the Top-K blocks (Eq.
  ours_train); "full" attends every token up to the query, each historical
  block with its gate.
* pos (gate position): "inner" adds log g to the logits; "outer" keeps the
  logits unbiased and weights each value by its block's gate,
  o = sum_i p_i g_{b(i)} v_i.
* ste (ranking preservation, hard): the forward uses the hard gate g^hard
  (1 on the Top-K blocks, 0 elsewhere), i.e. attends the current block and
  the Top-K blocks with no bias; the backward passes the gradient of
  g^hard straight to the soft gate g.  A block outside the Top-K then gets
  dg_m = sum_{i in B_m} exp(z_i - LSE_S) dO.(v_i - o) (the limit of the
  inner-gate gradient at g_m -> 0, App. D.2); scope decides which blocks
  receive it (the Top-K set for "sparse", every historical block for "full").

Gradients are returned for the log gate: dL/dlog g_m = g_m dL/dg_m (with
STE, g_m times the straight-through gradient), for every historical block
(zero where a block receives none), so one selector backward serves every
formulation: ds = gate_backward_act(dlog g, s, act).
"""
import math

import numpy as np

from .numerics import rho
from .selector import select, topk_blocks

ACTS = ("softmax", "sigmoid", "raw")


def log_gates(s, ct, act):
    """s[Hkv, R, nf] scores (noise included); ct[R] historical block counts.
    Returns log g[Hkv, R, nf], -inf for m >= C_t."""
    s = np.asarray(s, dtype=np.float64)
    out = np.full(s.shape, -np.inf)
    for ri, c in enumerate(ct):
        c = int(c)
        if c == 0:
            continue
        sr = s[:, ri, :c]
        if act == "softmax":
            mx = sr.max(axis=1, keepdims=True)
            out[:, ri, :c] = sr - (mx + np.log(np.exp(sr - mx).sum(axis=1, keepdims=True)))
        elif act == "sigmoid":
            # log sigmoid(x) = -log(1 + e^-x), evaluated without overflow
            out[:, ri, :c] = np.where(sr >= 0, -np.log1p(np.exp(-np.abs(sr))),
                                      sr - np.log1p(np.exp(-np.abs(sr))))
        elif act == "raw":
            out[:, ri, :c] = sr
        else:
            raise ValueError(act)
    return out


def select_variant(Q, K, B, top_k, dtype, act="softmax", noise=None, w_gq=None, w_gk=None):
    """The selector of ``select`` with an activation and optional score noise
    noise[Hkv, n, >= nf].  Without noise the Top-K ranks r = qhat.kbar (as
    ``select``); with noise it ranks s + eps (descending, lower block first on
    ties).  Returns sel, log_gate[Hkv, n, NB] (-inf where undefined), the
    scores s (noise included), ct and the selector intermediates."""
    st = select(Q, K, B, top_k, dtype, w_gq=w_gq, w_gk=w_gk)
    n, Hkv, dh = np.asarray(K).shape
    G = np.asarray(Q).shape[1] // Hkv
    NB = -(-n // B)
    r, ct = st["r"], st["ct"]
    nf = r.shape[2]
    s = r / (G * math.sqrt(dh))
    if noise is not None:
        s = s + np.asarray(noise, dtype=np.float64)[:, :, :nf]
    lg = np.full((Hkv, n, NB), -np.inf)
    lg[:, :, :nf] = log_gates(s, ct, act)
    sel = st["sel"].copy()
    if noise is not None:
        sel[:] = -1
        for g in range(Hkv):
            for t in range(n):
                chosen, _ = topk_blocks(s[g, t], int(ct[t]), top_k)
                sel[g, t, :len(chosen)] = chosen
    out = dict(st)
    out.update({"sel": sel, "log_gate": lg, "s": s})
    return out


def _sets(t, g, B, sel_row, lg_row, pos, scope, ste):
    """Attended token indices of query t in group g, their logit bias, their
    value weight and their block (-1 for the current block)."""
    b0 = (t // B) * B
    beta = t // B
    if scope == "full" and not ste:
        blocks = list(range(beta))
    else:
        blocks = [int(m) for m in sel_row if m >= 0]
    idx = np.concatenate([np.arange(m * B, (m + 1) * B) for m in blocks] + [np.arange(b0, t + 1)])
    blk = np.concatenate([np.full(B, m) for m in blocks] + [np.full(t + 1 - b0, -1)]).astype(np.int64)
    lgv = np.array([lg_row[m] if m >= 0 else 0.0 for m in blk])
    if ste:
        bias, w = np.zeros(len(idx)), np.ones(len(idx))
    elif pos == "inner":
        bias, w = lgv, np.ones(len(idx))
    elif pos == "outer":
        bias, w = np.zeros(len(idx)), np.exp(lgv)
    else:
        raise ValueError(pos)
    return idx, bias, w, blk


def _sm(dh, sm_scale):
    return (1.0 / math.sqrt(dh)) if (sm_scale is None or sm_scale <= 0) else float(sm_scale)


def variant_attention(Q, K, V, B, dtype, sel, log_gate, pos="inner", scope="sparse", ste=False, sm_scale=None):
    """One sequence: Q[n, H, dh], K/V[n, Hkv, dh], sel[Hkv, n, K],
    log_gate[Hkv, n, NB].  Returns O (rounded), O_exact and LSE[H, n]: the
    log-sum-exp of the logits the softmax normalizes (bias included for the
    inner gate, unbiased for the outer gate)."""
    Q, K, V = (np.asarray(a, dtype=np.float64) for a in (Q, K, V))
    n, Hkv, dh = K.shape
    H = Q.shape[1]
    G = H // Hkv
    sm = _sm(dh, sm_scale)
    O = np.zeros((n, H, dh))
    LSE = np.zeros((H, n))
    for t in range(n):
        for g in range(Hkv):
            idx, bias, w, _ = _sets(t, g, B, sel[g, t], log_gate[g, t], pos, scope, ste)
            z = sm * (Q[t, g * G:(g + 1) * G] @ K[idx, g].T) + bias[None, :]
            zmax = z.max(axis=1, keepdims=True)
            e = np.exp(z - zmax)
            l = e.sum(axis=1, keepdims=True)
            O[t, g * G:(g + 1) * G] = ((e * w[None, :]) @ V[idx, g]) / l
            LSE[g * G:(g + 1) * G, t] = (zmax + np.log(l))[:, 0]
    return rho(O, dtype), O, LSE


def variant_attention_backward(Q, K, V, dO, B, sel, log_gate, pos="inner", scope="sparse", ste=False,
                               sm_scale=None):
    """Gradients of sum(O * dO) for one sequence: dQ, dK, dV and
    dLG[Hkv, n, NB] = dL/dlog g of every historical block (summed over the
    group's heads; zero for blocks that receive none)."""
    Q, K, V, dO = (np.asarray(a, dtype=np.float64) for a in (Q, K, V, dO))
    n, Hkv, dh = K.shape
    H = Q.shape[1]
    G = H // Hkv
    sm = _sm(dh, sm_scale)
    NB = -(-n // B)
    dQ, dK, dV = np.zeros_like(Q), np.zeros_like(K), np.zeros_like(V)
    dLG = np.zeros((Hkv, n, NB))
    for t in range(n):
        beta = t // B
        for g in range(Hkv):
            idx, bias, w, blk = _sets(t, g, B, sel[g, t], log_gate[g, t], pos, scope, ste)
            Kg, Vg = K[idx, g], V[idx, g]
            for h in range(g * G, (g + 1) * G):
                q, do = Q[t, h], dO[t, h]
                z = sm * (Kg @ q) + bias
                zmax = z.max()
                lse = zmax + math.log(np.exp(z - zmax).sum())
                p = np.exp(z - lse)
                o = (p * w) @ Vg
                dp = w * (Vg @ do)
                delta = do @ o
                ds = p * (dp - delta)
                dQ[t, h] += sm * (ds @ Kg)
                dK[idx, g] += sm * ds[:, None] * q[None, :]
                dV[idx, g] += (p * w)[:, None] * do[None, :]
                if ste:
                    # straight-through: every block in the gradient scope, unit forward gate
                    scope_blocks = range(beta) if scope == "full" else [int(m) for m in sel[g, t] if m >= 0]
                    for m in scope_blocks:
                        ii = np.arange(m * B, (m + 1) * B)
                        pv = np.exp(sm * (K[ii, g] @ q) - lse)
                        dLG[g, t, m] += math.exp(log_gate[g, t, m]) * (pv @ (V[ii, g] @ do - delta))
                else:
                    for m in np.unique(blk[blk >= 0]):
                        sel_m = blk == m
                        if pos == "inner":
                            dLG[g, t, m] += ds[sel_m].sum()
                        else:
                            dLG[g, t, m] += (p[sel_m] * dp[sel_m]).sum()
    return dQ, dK, dV, dLG


def gate_backward_act(dlog_gate, s, ct, act):
    """ds[Hkv, R, nf] from dL/dlog g[Hkv, R, >= nf] through the activation:
    softmax: ds = dlg - g sum_{m < C} dlg (the softmax backward of App. D.3
    written for log g); sigmoid: ds = dlg (1 - sigmoid(s)); raw: ds = dlg."""
    s = np.asarray(s, dtype=np.float64)
    ds = np.zeros_like(s)
    for ri, c in enumerate(ct):
        c = int(c)
        if c == 0:
            continue
        dl = np.asarray(dlog_gate[:, ri, :c], dtype=np.float64)
        sr = s[:, ri, :c]
        if act == "softmax":
            g = np.exp(sr - sr.max(axis=1, keepdims=True))
            g /= g.sum(axis=1, keepdims=True)
            ds[:, ri, :c] = dl - g * dl.sum(axis=1, keepdims=True)
        elif act == "sigmoid":
            ds[:, ri, :c] = dl / (1.0 + np.exp(sr))
        elif act == "raw":
            ds[:, ri, :c] = dl
        else:
            raise ValueError(act)
    return ds
