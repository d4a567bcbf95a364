"""GPU parity of variable-length packing (several block-aligned documents in
one row, a per-block table of document starts) against the packed oracle:
selection (bit-exact) and log gates, attention forward, attention backward
with the per-block log-gate gradient, the selector's score gradient, and
the coverage statistics."""
import numpy as np
import pytest
import torch

from oracle.variants import gate_backward_act, select_variant
from oracle.varlen import attention_packed, backward_packed, coverage_packed, doc_spans, select_packed
from paper_2609_13141_amd import configs, inputs, sas

from helpers import assert_close, f64

pytestmark = pytest.mark.gpu


def _doc_row(lengths, B):
    row, first = [], 0
    for L in lengths:
        nb = -(-L // B)
        row += [first] * nb
        first += nb
    return np.array(row, dtype=np.int32)


def W(dtype="bf16", n=213, H=4, Hkv=2, dh=64, B=16, K=2, index=180):
    return configs.Workload(name="varlen", dtype=dtype, batch=2, seq_len=n, d_model=256, n_heads=H, n_kv_heads=Hkv,
                            head_dim=dh, d_ff=512, block_size=B, top_k=K, mode="gated",
                            segments=(("txt", n),), index=index)


# (workload, per-row document lengths, mode, scope)
CASES = [
    (W(), ([64, 32, 80, 37], [16, 197]), "gated", "sparse"),
    (W(dtype="f32", index=181), ([64, 32, 80, 37], [213]), "gated", "sparse"),
    (W(index=182), ([48, 48, 117], [96, 117]), "sparse", "sparse"),
    (W(index=183), ([48, 48, 117], [32, 64, 117]), "dense", "sparse"),
    (W(index=184), ([64, 32, 80, 37], [112, 101]), "gated", "full"),
    (W(dh=128, B=64, K=2, n=470, H=4, Hkv=1, index=185), ([192, 64, 214], [320, 150]), "gated", "sparse"),
]
IDS = [f"{w.dtype}-{mode}-{scope}-B{w.block_size}-dh{w.head_dim}" for w, _, mode, scope in CASES]


@pytest.mark.parametrize("case", CASES, ids=IDS)
def test_packed_documents_match_oracle(case):
    w, lengths, mode, scope = case
    print(f"\n[case] packed {IDS[CASES.index(case)]}", flush=True)
    B, n, dt = w.block_size, w.seq_len, w.dtype
    docs = np.stack([_doc_row(L, B) for L in lengths])
    q, k, v = inputs.qkv(w)
    d_o = inputs.normal(w, "d_o", q.shape, 1.0)
    cfg = sas.make_config(w, mode, scope=scope)
    qd, kd, vd, dod = (sas.to_device(a, dt) for a in (q, k, v, d_o))
    docd = torch.from_numpy(docs).cuda()
    fw = sas.attention_prefill(cfg, qd, kd, vd, log_gate=True, doc=docd)
    bw = sas.attention_backward(cfg, qd, kd, vd, fw["o"], dod, fw["lse"], fw["sel_idx"], fw["log_gate"],
                                dlog_gate=False, dlog_gate_full=True, doc=docd)
    sb = sas.selector_backward(cfg, qd, kd, None, fw["log_gate"], None, dlog_gate_full=bw["dlog_gate_full"],
                               doc=docd) if mode == "gated" else None
    st_gpu = sas.selection_stats(cfg, qd, kd, vd, fw["sel_idx"], doc=docd)
    torch.cuda.synchronize()
    tol = 2e-2 if dt == "bf16" else 2e-5
    for bi in range(w.batch):
        doc = docs[bi]
        st = select_packed(f64(q[bi]), f64(k[bi]), B, w.top_k, dt, doc)
        sel, lg = st["sel"], st["log_gate"]
        np.testing.assert_array_equal(fw["sel_idx"][bi].cpu().numpy(), sel)
        glg = fw["log_gate"][bi].cpu().numpy()
        fin = np.isfinite(lg)
        np.testing.assert_array_equal(np.isfinite(glg), fin)
        assert_close(glg[fin], lg[fin], dt, "log_gate", tol=1e-5)
        _, O, LSE = attention_packed(f64(q[bi]), f64(k[bi]), f64(v[bi]), B, dt, mode, doc, sel, lg, scope=scope)
        assert_close(fw["o"][bi].float().cpu().numpy(), O, dt, f"O b={bi}")
        assert_close(fw["lse"][bi].cpu().numpy(), LSE, dt, f"LSE b={bi}", tol=1e-3 if dt == "bf16" else 1e-5)
        dQ, dK, dV, dLG = backward_packed(f64(q[bi]), f64(k[bi]), f64(v[bi]), f64(d_o[bi]), B, mode, doc, sel, lg,
                                          scope=scope)
        assert_close(bw["dq"][bi].float().cpu().numpy(), dQ, dt, f"dQ b={bi}", tol=tol)
        assert_close(bw["dk"][bi].float().cpu().numpy(), dK, dt, f"dK b={bi}", tol=tol)
        assert_close(bw["dv"][bi].float().cpu().numpy(), dV, dt, f"dV b={bi}", tol=tol)
        if mode == "gated":
            assert_close(bw["dlog_gate_full"][bi].cpu().numpy(), dLG, dt, f"dLogG b={bi}", tol=tol)
            ds = np.zeros(dLG.shape)
            for t0, t1, fb in doc_spans(doc, n, B):
                sv = select_variant(f64(q[bi][t0:t1]), f64(k[bi][t0:t1]), B, w.top_k, dt)
                nf = sv["s"].shape[2]
                ds[:, t0:t1, fb:fb + nf] = gate_backward_act(dLG[:, t0:t1, fb:fb + nf], sv["s"], sv["ct"], "softmax")
            assert_close(sb["ds"][bi].cpu().numpy(), ds, dt, f"ds b={bi}", tol=tol)
        cov, cov_v = coverage_packed(f64(q[bi]), f64(k[bi]), f64(v[bi]), B, doc,
                                     sel if mode != "dense" else np.full_like(sel, -1))
        if mode != "dense":
            assert_close(st_gpu["cov"][bi].cpu().numpy(), cov, dt, "cov", tol=1e-4)
            assert_close(st_gpu["cov_v"][bi].cpu().numpy(), cov_v, dt, "cov_v", tol=1e-4)
        else:
            assert np.allclose(st_gpu["cov"][bi].cpu().numpy(), 1.0, atol=1e-5)
