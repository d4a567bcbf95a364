"""Pins of the packed-document oracle: a one-document table reproduces the
unpacked oracle, and a packed row matches torch autograd on a dense masked
formulation whose mask is block-diagonal over documents (an independent
computation of the same attention and gradients)."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle.varlen import attention_packed, backward_packed, coverage_packed, doc_spans, select_packed


def _doc_row(lengths, B):
    row = []
    first = 0
    for L in lengths:
        nb = -(-L // B)
        row += [first] * nb
        first += nb
    return np.array(row)


def _problem(seed, lengths=(24, 16, 29), B=8, H=4, Hkv=2, dh=8):
    rng = np.random.default_rng(seed)
    n = sum(lengths)
    Q = rng.standard_normal((n, H, dh))
    K = rng.standard_normal((n, Hkv, dh))
    V = rng.standard_normal((n, Hkv, dh))
    dO = rng.standard_normal((n, H, dh))
    return Q, K, V, dO, _doc_row(lengths, B)


def test_doc_spans():
    assert doc_spans(np.array([0, 0, 2, 2, 2, 5]), 44, 8) == [(0, 16, 0), (16, 40, 2), (40, 44, 5)]
    with pytest.raises(ValueError):
        doc_spans(np.array([0, 0, 1]), 24, 8)


def test_one_document_is_the_unpacked_oracle():
    Q, K, V, dO, _ = _problem(70, lengths=(69,))
    doc = np.zeros(-(-69 // 8), dtype=np.int64)
    st = select_packed(Q, K, 8, 2, "f32", doc)
    ref = oracle.select(Q, K, 8, 2, "f32")
    np.testing.assert_array_equal(st["sel"], ref["sel"])
    np.testing.assert_array_equal(st["log_gate"], ref["log_gate"])
    _, O, L = attention_packed(Q, K, V, 8, "f32", "gated", doc, st["sel"], st["log_gate"])
    _, O2, L2 = oracle.sas_attention(Q, K, V, 8, "gated", "f32", sel=ref["sel"], log_gate=ref["log_gate"])
    np.testing.assert_array_equal(O, O2)
    np.testing.assert_array_equal(L, L2)


@pytest.mark.parametrize("mode", ["gated", "sparse", "dense"])
def test_packed_matches_torch_document_mask(mode):
    Q, K, V, dO, doc = _problem(71)
    n, H, dh = Q.shape
    Hkv, G, B = K.shape[1], H // K.shape[1], 8
    NB = -(-n // B)
    st = select_packed(Q, K, B, 2, "f32", doc)
    sel, lg = st["sel"], st["log_gate"]
    _, O, _ = attention_packed(Q, K, V, B, "f32", mode, doc, sel, lg)
    dQ, dK, dV, dLG = backward_packed(Q, K, V, dO, B, mode, doc, sel, lg)
    q = torch.tensor(Q, requires_grad=True)
    k = torch.tensor(K, requires_grad=True)
    v = torch.tensor(V, requires_grad=True)
    lgt = torch.tensor(np.where(np.isfinite(lg), lg, 0.0), requires_grad=True)
    ti = torch.arange(n)[:, None].expand(n, n)
    ii = torch.arange(n)[None, :].expand(n, n)
    blk = ii // B
    docb = torch.tensor(doc)
    same = docb[ti // B] == docb[blk]                      # same document
    cur = (blk == ti // B) & (ii <= ti)
    hist = (blk < ti // B) & same
    loss = 0.0
    for g in range(Hkv):
        selm = torch.zeros(n, NB, dtype=torch.bool)
        for t in range(n):
            for m in sel[g, t]:
                if m >= 0:
                    selm[t, m] = True
        chosen = torch.gather(selm, 1, blk) & hist
        allow = cur | (hist if mode == "dense" else chosen)
        bias = torch.where(chosen, torch.gather(lgt[g], 1, blk), torch.zeros(n, n, dtype=torch.float64))
        for h in range(g * G, (g + 1) * G):
            z = (q[:, h] @ k[:, g].T) / math.sqrt(dh) + (bias if mode == "gated" else 0.0)
            p = torch.softmax(z.masked_fill(~allow, float("-inf")), dim=1)
            o = p @ v[:, g]
            np.testing.assert_allclose(O[:, h], o.detach().numpy(), rtol=1e-11, atol=1e-12)
            loss = loss + (o * torch.tensor(dO[:, h])).sum()
    loss.backward()
    np.testing.assert_allclose(dQ, q.grad.numpy(), rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(dK, k.grad.numpy(), rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(dV, v.grad.numpy(), rtol=1e-9, atol=1e-11)
    if mode == "gated":
        np.testing.assert_allclose(dLG, lgt.grad.numpy(), rtol=1e-9, atol=1e-11)


def test_packed_documents_are_independent():
    Q, K, V, dO, doc = _problem(72)
    st = select_packed(Q, K, 8, 2, "f32", doc)
    Q2, K2 = Q.copy(), K.copy()
    Q2[24:40] += 1.0
    K2[24:40] -= 2.0                                         # the second document only
    st2 = select_packed(Q2, K2, 8, 2, "f32", doc)
    for a, b in ((st["sel"], st2["sel"]), (st["log_gate"], st2["log_gate"])):
        np.testing.assert_array_equal(a[:, :24], b[:, :24])
        np.testing.assert_array_equal(a[:, 40:], b[:, 40:])
    cov, _ = coverage_packed(Q, K, V, 8, doc, st["sel"])
    cov2, _ = coverage_packed(Q2, K2, V, 8, doc, st2["sel"])
    np.testing.assert_array_equal(cov[:, 40:], cov2[:, 40:])
