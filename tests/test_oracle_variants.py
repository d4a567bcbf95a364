"""Pins of the oracle's gating formulations (Table 1; Sec. 4.1-4.2; App. D):
torch autograd on dense masked formulations written independently of the
oracle's gather form (the straight-through gate in its multiplicative form,
where dropped blocks carry a zero gate), torch's log_softmax / logsigmoid,
Top-K ordering properties, and reductions to the plain modes."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle.variants import (gate_backward_act, log_gates, select_variant, variant_attention,
                             variant_attention_backward)


def _problem(seed, n=40, B=8, H=4, Hkv=2, dh=8, K=2, act="softmax", noise=False):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((n, H, dh))
    Kk = rng.standard_normal((n, Hkv, dh))
    V = rng.standard_normal((n, Hkv, dh))
    dO = rng.standard_normal((n, H, dh))
    eps = rng.gumbel(size=(Hkv, n, -(-n // B))) if noise else None
    st = select_variant(Q, Kk, B, K, "f32", act=act, noise=eps)
    return Q, Kk, V, dO, st


def _torch_variant(Q, Kk, V, dO, B, sel, log_gate, pos, scope, ste):
    """sum(O * dO) of a dense masked formulation, with autograd."""
    n, H, dh = Q.shape
    Hkv = Kk.shape[1]
    G = H // Hkv
    NB = -(-n // B)
    q = torch.tensor(Q, requires_grad=True)
    k = torch.tensor(Kk, requires_grad=True)
    v = torch.tensor(V, requires_grad=True)
    lg = torch.tensor(np.where(np.isfinite(log_gate), log_gate, 0.0), requires_grad=True)
    ti = torch.arange(n)[:, None].expand(n, n)
    ii = torch.arange(n)[None, :].expand(n, n)
    blk = ii // B
    cur = (blk == ti // B) & (ii <= ti)
    hist = blk < ti // B
    loss = 0.0
    for g in range(Hkv):
        selm = torch.zeros(n, NB, dtype=torch.bool)
        for t in range(n):
            for m in sel[g, t]:
                if m >= 0:
                    selm[t, m] = True
        chosen = torch.gather(selm, 1, blk) & hist
        gate = torch.exp(torch.gather(lg[g], 1, blk))          # g_{b(i)} for row t
        if ste:
            scope_m = hist if scope == "full" else chosen
            hard = chosen.double()
            gh = (hard - gate).detach() + gate                 # straight-through gate
            wgt = torch.where(cur, torch.ones_like(gate), torch.where(scope_m, gh, torch.zeros_like(gate)))
            allow = cur | scope_m
        else:
            allow = cur | (hist if scope == "full" else chosen)
            wgt = torch.where(cur, torch.ones_like(gate), gate)
        for h in range(g * G, (g + 1) * G):
            z = (q[:, h] @ k[:, g].T) / math.sqrt(dh)
            z = z.masked_fill(~allow, float("-inf"))
            if ste:
                # o = sum_i g_i e^{z_i} v_i / sum_j g_j e^{z_j}: zero gates drop blocks
                e = torch.exp(z - z.max(dim=1, keepdim=True).values.detach()) * wgt
                o = (e @ v[:, g]) / e.sum(dim=1, keepdim=True)
            elif pos == "inner":
                p = torch.softmax(z + torch.log(torch.where(allow, wgt, torch.ones_like(wgt))), dim=1)
                o = p @ v[:, g]
            else:
                p = torch.softmax(z, dim=1)
                o = (p * wgt) @ v[:, g]
            loss = loss + (o * torch.tensor(dO[:, h])).sum()
    loss.backward()
    return q.grad.numpy(), k.grad.numpy(), v.grad.numpy(), lg.grad.numpy()


# Table 1's formulations: (pos, act, scope, ste, noise)
TABLE1 = [
    ("inner", "softmax", "full", False, False),   # rows 2, 4, 7, 9
    ("outer", "softmax", "full", False, False),   # row 3
    ("inner", "sigmoid", "full", False, False),   # row 5
    ("inner", "raw", "full", False, False),       # row 6
    ("inner", "softmax", "full", True, False),    # row 8 (STE)
    ("inner", "softmax", "sparse", False, False),  # row 10 (SAS)
    ("inner", "softmax", "sparse", False, True),  # row 11 (full*: noise)
    ("outer", "softmax", "sparse", False, False),
    ("inner", "softmax", "sparse", True, False),
    ("inner", "sigmoid", "sparse", False, False),
]


@pytest.mark.parametrize("pos,act,scope,ste,noise", TABLE1)
def test_variant_backward_matches_torch_autograd(pos, act, scope, ste, noise):
    Q, Kk, V, dO, st = _problem(31, act=act, noise=noise)
    dQ, dK, dV, dLG = variant_attention_backward(Q, Kk, V, dO, 8, st["sel"], st["log_gate"], pos, scope, ste)
    tq, tk, tv, tl = _torch_variant(Q, Kk, V, dO, 8, st["sel"], st["log_gate"], pos, scope, ste)
    np.testing.assert_allclose(dQ, tq, rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(dK, tk, rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(dV, tv, rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(dLG, tl, rtol=1e-9, atol=1e-11)
    assert np.abs(dLG).max() > 0


@pytest.mark.parametrize("pos,act,scope,ste,noise", TABLE1)
def test_variant_forward_matches_torch(pos, act, scope, ste, noise):
    Q, Kk, V, dO, st = _problem(32, act=act, noise=noise)
    _, O, _ = variant_attention(Q, Kk, V, 8, "f32", st["sel"], st["log_gate"], pos, scope, ste)
    # the dense masked formulation's output, head by head
    n, H, dh = Q.shape
    q = torch.tensor(Q)
    k = torch.tensor(Kk)
    v = torch.tensor(V)
    Hkv = Kk.shape[1]
    G = H // Hkv
    B = 8
    NB = -(-n // B)
    lgt = torch.tensor(np.where(np.isfinite(st["log_gate"]), st["log_gate"], 0.0))
    ti = torch.arange(n)[:, None].expand(n, n)
    ii = torch.arange(n)[None, :].expand(n, n)
    blk = ii // B
    cur = (blk == ti // B) & (ii <= ti)
    hist = blk < ti // B
    for g in range(Hkv):
        selm = torch.zeros(n, NB, dtype=torch.bool)
        for t in range(n):
            for m in st["sel"][g, t]:
                if m >= 0:
                    selm[t, m] = True
        chosen = torch.gather(selm, 1, blk) & hist
        gate = torch.exp(torch.gather(lgt[g], 1, blk))
        allow = cur | (hist if (scope == "full" and not ste) else chosen)
        for h in range(g * G, (g + 1) * G):
            z = ((q[:, h] @ k[:, g].T) / math.sqrt(dh)).masked_fill(~allow, float("-inf"))
            if ste:
                o = torch.softmax(z, dim=1) @ v[:, g]
            elif pos == "inner":
                o = torch.softmax(z + torch.where(hist & allow, torch.log(gate), torch.zeros_like(gate)), 1) @ v[:, g]
            else:
                o = (torch.softmax(z, dim=1) * torch.where(hist, gate, torch.ones_like(gate))) @ v[:, g]
            np.testing.assert_allclose(O[:, h], o.numpy(), rtol=1e-11, atol=1e-12)


def test_variants_reduce_to_plain_modes():
    Q, Kk, V, dO, st = _problem(33, K=2)
    sel, lg = st["sel"], st["log_gate"]
    _, gated, lse_g = oracle.sas_attention(Q, Kk, V, 8, "gated", "f32", sel=sel, log_gate=lg)[:3]
    _, sparse, lse_s = oracle.sas_attention(Q, Kk, V, 8, "sparse", "f32", sel=sel)[:3]
    _, o, l = variant_attention(Q, Kk, V, 8, "f32", sel, lg, "inner", "sparse", False)
    np.testing.assert_allclose(o, gated, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l, lse_g, rtol=1e-12, atol=1e-13)
    # the hard (STE) forward is the sparse forward
    _, o, l = variant_attention(Q, Kk, V, 8, "f32", sel, lg, "inner", "full", True)
    np.testing.assert_allclose(o, sparse, rtol=1e-12, atol=1e-13)
    # unit gates: outer gating is the ungated attention over the same set
    zero = np.where(np.isfinite(lg), 0.0, lg)
    _, o, _ = variant_attention(Q, Kk, V, 8, "f32", sel, zero, "outer", "sparse", False)
    np.testing.assert_allclose(o, sparse, rtol=1e-12, atol=1e-13)
    # K >= C: the sparse scope keeps every block, so it is the full scope
    stk = select_variant(Q, Kk, 8, 5, "f32")
    _, a, _ = variant_attention(Q, Kk, V, 8, "f32", stk["sel"], stk["log_gate"], "inner", "sparse", False)
    _, b, _ = variant_attention(Q, Kk, V, 8, "f32", stk["sel"], stk["log_gate"], "inner", "full", False)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)
    # the sparse-scope inner-softmax gradients are the plain SAS backward's
    dQ, dK, dV, dLG = variant_attention_backward(Q, Kk, V, dO, 8, sel, lg, "inner", "sparse", False)
    rQ, rK, rV, rL = oracle.sas_attention_backward(Q, Kk, V, dO, 8, "gated", sel, lg)
    for x, y in ((dQ, rQ), (dK, rK), (dV, rV), (dLG, rL)):
        np.testing.assert_allclose(x, y, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("act", ["softmax", "sigmoid", "raw"])
def test_log_gates_match_torch(act):
    rng = np.random.default_rng(40)
    s = rng.standard_normal((3, 6, 5)) * 4
    ct = np.array([0, 1, 2, 3, 5, 5])
    got = log_gates(s, ct, act)
    for ri, c in enumerate(ct):
        assert np.all(np.isneginf(got[:, ri, c:]))
        if c == 0:
            continue
        x = torch.tensor(s[:, ri, :c])
        ref = {"softmax": torch.log_softmax(x, dim=1), "sigmoid": torch.nn.functional.logsigmoid(x),
               "raw": x}[act].numpy()
        np.testing.assert_allclose(got[:, ri, :c], ref, rtol=1e-13, atol=1e-14)
    if act == "softmax":  # invariant to a shift of the scores
        np.testing.assert_allclose(log_gates(s + 3.5, ct, act), got, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("act", ["softmax", "sigmoid", "raw"])
def test_gate_backward_act_matches_autograd(act):
    rng = np.random.default_rng(41)
    s = rng.standard_normal((2, 7, 6))
    ct = np.array([0, 1, 3, 4, 6, 6, 2])
    dl = rng.standard_normal(s.shape)
    st = torch.tensor(s, requires_grad=True)
    loss = 0.0
    for ri, c in enumerate(ct):
        if c == 0:
            continue
        x = st[:, ri, :c]
        lg = {"softmax": torch.log_softmax(x, dim=1), "sigmoid": torch.nn.functional.logsigmoid(x), "raw": x}[act]
        loss = loss + (lg * torch.tensor(dl[:, ri, :c])).sum()
    loss.backward()
    got = gate_backward_act(dl, s, ct, act)
    np.testing.assert_allclose(got, st.grad.numpy(), rtol=1e-12, atol=1e-13)
    if act == "softmax":  # agrees with the plain gate backward (r = s G sqrt(dh))
        np.testing.assert_allclose(got, oracle.gate_backward(dl, s * 2 * math.sqrt(4), ct, 2, 4),
                                   rtol=1e-12, atol=1e-13)


def test_noisy_topk_orders_by_noisy_scores():
    Q, Kk, V, dO, st = _problem(42, n=96, B=8, K=3, noise=True)
    s, ct, sel = st["s"], st["ct"], st["sel"]
    for g in range(s.shape[0]):
        for t in range(s.shape[1]):
            c = int(ct[t])
            chosen = [int(m) for m in sel[g, t] if m >= 0]
            assert chosen == sorted(chosen) and len(chosen) == min(3, c)
            rest = [m for m in range(c) if m not in chosen]
            for a in chosen:
                for b in rest:
                    assert s[g, t, a] > s[g, t, b] or (s[g, t, a] == s[g, t, b] and a < b)
    # without noise the selection is the plain selector's
    st0 = select_variant(Q, Kk, 8, 3, "f32")
    np.testing.assert_array_equal(st0["sel"], oracle.select(Q, Kk, 8, 3, "f32")["sel"])
