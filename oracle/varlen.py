"""Variable-length packing: several documents in one row (App. E notes that
the training kernel supports packed sequences; the paper gives no layout).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Reading: documents start on block boundaries (every document but a row's
last is a whole number of blocks long); doc_row[m] is the first block of
the document that block m belongs to.  A packed row is the concatenation of
independent documents: each document's results are those of the document
alone, with block indices offset by its first block.
"""
import numpy as np

from . import attention as _att
from . import backward as _bwd
from .stats import mass_coverage
from .variants import select_variant, variant_attention, variant_attention_backward


def doc_spans(doc_row, n, B):
    """doc_row[NB] -> [(t0, t1, fb)]: token range and first block of each document."""
    NB = -(-n // B)
    spans, m = [], 0
    while m < NB:
        fb = int(doc_row[m])
        if fb != m:
            raise ValueError(f"block {m} starts no document (first block {fb})")
        e = m + 1
        while e < NB and int(doc_row[e]) == fb:
            e += 1
        spans.append((fb * B, min(n, e * B), fb))
        m = e
    return spans


def select_packed(Q, K, B, top_k, dtype, doc_row, act="softmax", noise=None, w_gq=None, w_gk=None):
    """The selector of each document; sel[Hkv, n, K] (global block ids, -1
    padded), log_gate[Hkv, n, NB] (-inf outside the document's history)."""
    Q, K = np.asarray(Q, dtype=np.float64), np.asarray(K, dtype=np.float64)
    n, Hkv, dh = K.shape
    NB = -(-n // B)
    sel = np.full((Hkv, n, max(top_k, 0)), -1, dtype=np.int64)
    lg = np.full((Hkv, n, NB), -np.inf)
    for t0, t1, fb in doc_spans(doc_row, n, B):
        st = select_variant(Q[t0:t1], K[t0:t1], B, top_k, dtype, act=act,
                            noise=None if noise is None else np.asarray(noise)[:, t0:t1, fb:],
                            w_gq=w_gq, w_gk=w_gk)
        sd = st["sel"]
        sel[:, t0:t1] = np.where(sd >= 0, sd + fb, -1)
        nbd = st["log_gate"].shape[2]
        lg[:, t0:t1, fb:fb + nbd] = st["log_gate"]
    return {"sel": sel, "log_gate": lg}


def _local(sel, log_gate, t0, t1, fb):
    sl = None if sel is None else np.where(sel[:, t0:t1] >= 0, sel[:, t0:t1] - fb, -1)
    lgl = None if log_gate is None else log_gate[:, t0:t1, fb:]
    return sl, lgl


def attention_packed(Q, K, V, B, dtype, mode, doc_row, sel=None, log_gate=None, pos="inner", scope="sparse",
                     ste=False):
    """O (rounded), O_exact [n, H, dh] and LSE [H, n] of a packed row."""
    Q, K, V = (np.asarray(a, dtype=np.float64) for a in (Q, K, V))
    n, H, dh = Q.shape
    O, Oex, LSE = np.zeros((n, H, dh)), np.zeros((n, H, dh)), np.zeros((H, n))
    for t0, t1, fb in doc_spans(doc_row, n, B):
        sl, lgl = _local(sel, log_gate, t0, t1, fb)
        if mode == "gated":
            o, oe, l = variant_attention(Q[t0:t1], K[t0:t1], V[t0:t1], B, dtype, sl, lgl, pos, scope, ste)
        else:
            o, oe, l = _att.sas_attention(Q[t0:t1], K[t0:t1], V[t0:t1], B, mode, dtype, sel=sl, log_gate=lgl)
        O[t0:t1], Oex[t0:t1], LSE[:, t0:t1] = o, oe, l
    return O, Oex, LSE


def backward_packed(Q, K, V, dO, B, mode, doc_row, sel=None, log_gate=None, pos="inner", scope="sparse",
                    ste=False):
    """dQ, dK, dV and dLG[Hkv, n, NB] of a packed row."""
    Q, K, V, dO = (np.asarray(a, dtype=np.float64) for a in (Q, K, V, dO))
    n, Hkv, dh = K.shape
    NB = -(-n // B)
    dQ, dK, dV = np.zeros_like(Q), np.zeros_like(K), np.zeros_like(V)
    dLG = np.zeros((Hkv, n, NB))
    for t0, t1, fb in doc_spans(doc_row, n, B):
        sl, lgl = _local(sel, log_gate, t0, t1, fb)
        if mode == "gated":
            r = variant_attention_backward(Q[t0:t1], K[t0:t1], V[t0:t1], dO[t0:t1], B, sl, lgl, pos, scope, ste)
        else:
            r = _bwd.sas_attention_backward(Q[t0:t1], K[t0:t1], V[t0:t1], dO[t0:t1], B, mode, sl, lgl)
        dQ[t0:t1], dK[t0:t1], dV[t0:t1] = r[0], r[1], r[2]
        dLG[:, t0:t1, fb:fb + r[3].shape[2]] = r[3]
    return dQ, dK, dV, dLG


def coverage_packed(Q, K, V, B, doc_row, sel):
    """Eq. mass_coverage per document (cov, cov_v [H, n])."""
    n = np.asarray(K).shape[0]
    H = np.asarray(Q).shape[1]
    cov, cov_v = np.zeros((H, n)), np.zeros((H, n))
    for t0, t1, fb in doc_spans(doc_row, n, B):
        sl, _ = _local(sel, None, t0, t1, fb)
        c, cv = mass_coverage(np.asarray(Q)[t0:t1], np.asarray(K)[t0:t1], np.asarray(V)[t0:t1], B, sl)
        cov[:, t0:t1], cov_v[:, t0:t1] = c, cv
    return cov, cov_v
