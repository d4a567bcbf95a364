"""Pins of the oracle's backward (App. E, the recomputation-based backward;
Eq. gate_posi; Eq. normalized_log_gate): torch autograd on a dense masked
formulation of the same attention (an independent library computation),
central finite differences of the fp64 forward, and the paper's inner-gate
gradient written out directly."""
import math

import numpy as np
import pytest
import torch

import oracle


def _problem(seed, n=40, B=8, H=4, Hkv=2, dh=8, K=2, dtype="f32"):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((n, H, dh))
    Kk = rng.standard_normal((n, Hkv, dh))
    V = rng.standard_normal((n, Hkv, dh))
    dO = rng.standard_normal((n, H, dh))
    st = oracle.select(Q, Kk, B, K, dtype)
    return Q, Kk, V, dO, st["sel"], st["log_gate"]


def _torch_masked(Q, Kk, V, dO, B, mode, sel, log_gate):
    """Dense masked attention with autograd: mask and bias per (t, i) built
    from the selection; loss = sum O * dO."""
    n, H, dh = Q.shape
    Hkv = Kk.shape[1]
    G = H // Hkv
    NB = -(-n // B)
    q = torch.tensor(Q, requires_grad=True)
    k = torch.tensor(Kk, requires_grad=True)
    v = torch.tensor(V, requires_grad=True)
    lg = torch.tensor(np.nan_to_num(log_gate, neginf=0.0), requires_grad=True)   # [Hkv, n, NB]
    t_idx = torch.arange(n)[:, None]
    i_idx = torch.arange(n)[None, :]
    blk = (i_idx // B).expand(n, n)
    loss = 0.0
    for g in range(Hkv):
        causal = i_idx <= t_idx
        cur = (i_idx >= (t_idx // B) * B) & causal
        if mode == "dense":
            allow, hist = causal, torch.zeros(n, n, dtype=torch.bool)
        else:
            s = torch.zeros(n, NB, dtype=torch.bool)
            for t in range(n):
                for m in sel[g, t]:
                    if m >= 0:
                        s[t, m] = True
            hist = torch.gather(s, 1, blk) & ~cur
            allow = cur | hist
        bias = torch.zeros(n, n, dtype=torch.float64)
        if mode == "gated":
            bias = torch.where(hist, torch.gather(lg[g], 1, blk), bias)
        for h in range(g * G, (g + 1) * G):
            z = (q[:, h] @ k[:, g].T) / math.sqrt(dh) + bias
            z = z.masked_fill(~allow, float("-inf"))
            p = torch.softmax(z, dim=1)
            o = p @ v[:, g]
            loss = loss + (o * torch.tensor(dO[:, h])).sum()
    loss.backward()
    tl = lg.grad.numpy() if lg.grad is not None else np.zeros(lg.shape)
    return q.grad.numpy(), k.grad.numpy(), v.grad.numpy(), tl


@pytest.mark.parametrize("mode", ["gated", "sparse", "dense"])
def test_attention_backward_matches_torch_autograd(mode):
    Q, Kk, V, dO, sel, lg = _problem(20)
    dQ, dK, dV, dL = oracle.sas_attention_backward(Q, Kk, V, dO, 8, mode, sel, lg)
    tq, tk, tv, tl = _torch_masked(Q, Kk, V, dO, 8, mode, sel, lg)
    np.testing.assert_allclose(dQ, tq, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dK, tk, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dV, tv, rtol=1e-10, atol=1e-12)
    if mode == "gated":
        np.testing.assert_allclose(dL, tl, rtol=1e-10, atol=1e-12)
        assert np.abs(dL).max() > 0
    else:
        assert np.all(dL == 0)


def test_attention_backward_finite_differences():
    Q, Kk, V, dO, sel, lg = _problem(21, n=20, B=4, H=2, Hkv=1, dh=4, K=2)
    B = 4
    dQ, dK, dV, dL = oracle.sas_attention_backward(Q, Kk, V, dO, B, "gated", sel, lg)

    def loss(Q_, K_, V_, lg_):
        _, O, _ = oracle.sas_attention(Q_, K_, V_, B, "gated", "f32", sel=sel, log_gate=lg_)
        return float((O * dO).sum())

    eps = 1e-6
    rng = np.random.default_rng(3)
    for arr, grad, name in ((Q, dQ, "Q"), (Kk, dK, "K"), (V, dV, "V")):
        for _ in range(6):
            ix = tuple(int(rng.integers(0, s)) for s in arr.shape)
            a, b = arr.copy(), arr.copy()
            a[ix] += eps
            b[ix] -= eps
            args_a = [Q, Kk, V, lg]
            args_b = [Q, Kk, V, lg]
            pos = {"Q": 0, "K": 1, "V": 2}[name]
            args_a[pos], args_b[pos] = a, b
            fd = (loss(*args_a) - loss(*args_b)) / (2 * eps)
            assert abs(fd - grad[ix]) < 1e-6 * max(1.0, abs(fd)), (name, ix, fd, grad[ix])
    # the gate of selected blocks
    checked = 0
    for t in range(20):
        for m in sel[0, t]:
            if m < 0 or checked >= 8:
                continue
            a, b = lg.copy(), lg.copy()
            a[0, t, m] += eps
            b[0, t, m] -= eps
            fd = (loss(Q, Kk, V, a) - loss(Q, Kk, V, b)) / (2 * eps)
            assert abs(fd - dL[0, t, m]) < 1e-6 * max(1.0, abs(fd)), (t, m, fd, dL[0, t, m])
            checked += 1
    assert checked == 8


def test_log_gate_gradient_is_eq_gate_posi():
    # dlog g_m = g_m dg_m^inner = sum_{h in g} sum_{i in B_m} p_i dO.(v_i - o)
    Q, Kk, V, dO, sel, lg = _problem(22)
    B, n, H, Hkv, dh = 8, 40, 4, 2, 8
    G = H // Hkv
    _, _, _, dL = oracle.sas_attention_backward(Q, Kk, V, dO, B, "gated", sel, lg)
    _, O, _ = oracle.sas_attention(Q, Kk, V, B, "gated", "f32", sel=sel, log_gate=lg)
    for t in range(n):
        b0 = (t // B) * B
        for g in range(Hkv):
            blocks = [int(m) for m in sel[g, t] if m >= 0]
            idx = np.concatenate([np.arange(m * B, (m + 1) * B) for m in blocks] + [np.arange(b0, t + 1)])
            bias = np.concatenate([np.full(B, lg[g, t, m]) for m in blocks] + [np.zeros(t + 1 - b0)])
            for m in blocks:
                want = 0.0
                for h in range(g * G, (g + 1) * G):
                    z = Q[t, h] @ Kk[idx, g].T / math.sqrt(dh) + bias
                    p = np.exp(z - z.max())
                    p /= p.sum()
                    inb = (idx >= m * B) & (idx < (m + 1) * B)
                    want += float((p[inb] * ((V[idx[inb], g] - O[t, h]) @ dO[t, h])).sum())
                assert abs(dL[g, t, m] - want) < 1e-10 * max(1.0, abs(want))


def test_gate_and_selector_backward_match_autograd():
    # s = (qhat0 W_gq^T) . (kbar0 W_gk^T) / (G sqrt dh); log g = log_softmax over
    # the C_t historical blocks; loss = sum dlog g * log g
    rng = np.random.default_rng(23)
    Hkv, R, nf, dh, G = 2, 9, 6, 8, 3
    qhat0 = rng.standard_normal((Hkv, R, dh))
    kbar0 = rng.standard_normal((Hkv, nf, dh))
    Wq = rng.standard_normal((Hkv, dh, dh)) * 0.3
    Wk = rng.standard_normal((Hkv, dh, dh)) * 0.3
    dl = rng.standard_normal((Hkv, R, nf))
    ct = np.array([0, 1, 2, 3, 4, 5, 6, 6, 2])
    wq = torch.tensor(Wq, requires_grad=True)
    wk = torch.tensor(Wk, requires_grad=True)
    qh = torch.tensor(qhat0) @ wq.transpose(1, 2)
    kb = torch.tensor(kbar0) @ wk.transpose(1, 2)
    s = (qh @ kb.transpose(1, 2)) / (G * math.sqrt(dh))
    loss = 0.0
    for ri, c in enumerate(ct):
        if c:
            loss = loss + (torch.tensor(dl[:, ri, :c]) * torch.log_softmax(s[:, ri, :c], dim=1)).sum()
    loss.backward()
    qhat = np.einsum("gtj,gkj->gtk", qhat0, Wq)
    kbar = np.einsum("gmj,gkj->gmk", kbar0, Wk)
    r = np.einsum("gtj,gmj->gtm", qhat, kbar)
    ds = oracle.gate_backward(dl, r, ct, G, dh)
    out = oracle.selector_backward(ds, qhat, kbar, G, dh, qhat0=qhat0, kbar0=kbar0)
    np.testing.assert_allclose(out["dw_gq"], wq.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(out["dw_gk"], wk.grad.numpy(), rtol=1e-10, atol=1e-12)
    # gate gradient alone: rows of ds sum to zero (shift invariance of the normalized gate)
    np.testing.assert_allclose(ds.sum(axis=2), 0.0, atol=1e-12)
