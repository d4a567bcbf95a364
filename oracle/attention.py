"""SAS attention in float64, gather form.

For head h of KV group g = h // G and query t (0-based):

* DENSE  (Eq. fula, causal): S = {0..t}, no bias.
* SPARSE (Eq. spa with Alg. 2's set): S = B_0(t) u (union of the selected
  historical blocks), no bias -- the inference-time attention.
* GATED  (Eq. ours_train, Sec. 4.3): same S; every token of a selected
  historical block m carries the bias log g[g, t, m]; the current block
  B_0(t) = [B*floor(t/B), t] carries bias 0 (unit gate g_0 = 1).

z_i = sm * q . k_i with sm = 1/sqrt(dh) by default (the paper omits the scale
in its notation and scales q k^T before adding the gate in its kernel
description, App. E); p = softmax(z + bias) over S; o = sum_i p_i v_i;
LSE = log sum_{j in S} exp(z_j + bias_j) (natural log, scale and bias
included).  o is materialised in the activation dtype.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import math

import numpy as np

from .numerics import _POOL, rho


def sas_attention(Q, K, V, B, mode, dtype, sel=None, log_gate=None,
                  sm_scale=None, rows=None):
    """One sequence.  K/V[n, Hkv, dh]; Q[R, H, dh] holds the query rows
    listed in ``rows`` (all n rows, in order, when it is None); sel[Hkv, R, K]
    and log_gate[Hkv, R, NB] are indexed the same way.  Returns O[R, H, dh] (rounded),
    O_exact[R, H, dh] (fp64) and LSE[H, R]."""
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    n, Hkv, dh = K.shape
    H = Q.shape[1]
    G = H // Hkv
    sm = (1.0 / math.sqrt(dh)) if (sm_scale is None or sm_scale <= 0) else float(sm_scale)
    rows = np.arange(n) if rows is None else np.asarray(rows)
    R = len(rows)
    assert Q.shape[0] == R
    O = np.zeros((R, H, dh))
    LSE = np.zeros((H, R))
    for ri, t in enumerate(rows):
        t = int(t)
        b0 = (t // B) * B
        for g in range(Hkv):
            if mode == "dense":
                idx = np.arange(0, t + 1)
                bias = np.zeros(t + 1)
            else:
                blocks = [int(m) for m in sel[g, ri] if m >= 0]
                parts = [np.arange(m * B, (m + 1) * B) for m in blocks]
                parts.append(np.arange(b0, t + 1))
                idx = np.concatenate(parts)
                if mode == "gated":
                    bparts = [np.full(B, log_gate[g, ri, m]) for m in blocks]
                elif mode == "sparse":
                    bparts = [np.zeros(B) for _ in blocks]
                else:
                    raise ValueError(mode)
                bparts.append(np.zeros(t + 1 - b0))
                bias = np.concatenate(bparts)
            q = Q[ri, g * G:(g + 1) * G, :]                    # [G, dh]
            z = sm * (q @ K[idx, g, :].T) + bias[None, :]     # [G, |S|]
            zmax = z.max(axis=1, keepdims=True)
            e = np.exp(z - zmax)
            l = e.sum(axis=1, keepdims=True)
            O[ri, g * G:(g + 1) * G, :] = (e @ V[idx, g, :]) / l
            LSE[g * G:(g + 1) * G, ri] = (zmax + np.log(l))[:, 0]
    return rho(O, dtype), O, LSE


def causal_attention(Q, K, V, dtype, sm_scale=None):
    """Standard causal softmax attention (Eq. fula with the causal mask) of
    one sequence, written as masked score matrices: for query head h (KV
    head h // G), Z = sm * Q_h K_g^T with Z[t, i] = -inf for i > t,
    P = softmax over each row, O = P V_g, LSE = log sum_i exp(Z[t, i]).
    Q[n, H, dh], K/V[n, Hkv, dh] -> O[n, H, dh] (rounded), O_exact (fp64),
    LSE[H, n].  This is the DENSE mode of ``sas_attention`` for every row at
    once (the serving prefill of Sec. 5.1 attends densely)."""
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    n, H, dh = Q.shape
    Hkv = K.shape[1]
    G = H // Hkv
    sm = (1.0 / math.sqrt(dh)) if (sm_scale is None or sm_scale <= 0) else float(sm_scale)
    future = np.triu(np.ones((n, n), dtype=bool), k=1)        # key i after query t
    O = np.zeros((n, H, dh))
    LSE = np.zeros((H, n))

    def head(h):
        g = h // G
        Z = sm * (Q[:, h, :] @ K[:, g, :].T)
        Z[future] = -np.inf
        zmax = Z.max(axis=1, keepdims=True)
        E = np.exp(Z - zmax)
        L = E.sum(axis=1, keepdims=True)
        O[:, h, :] = (E @ V[:, g, :]) / L
        LSE[h] = (zmax + np.log(L))[:, 0]
    # heads are independent: computed on threads when the sequence is long
    if n >= 512:
        list(_POOL.map(head, range(H)))
    else:
        for h in range(H):
            head(h)
    return rho(O, dtype), O, LSE
