"""GPU parity of the selector backward (Alg. 1's selector update): the score
gradient through the normalized log gate (Eq. normalized_log_gate; the
softmax backward of App. D.3) and the gradients of the gate queries, block
summaries and the optional W_gq / W_gk, against the fp64 oracle.

The library's selection is bit-exact with the oracle's and its gate queries
and summaries carry the same roundings, so the only differences are fp32
accumulation: the bar here is 1e-4 of each tensor's largest magnitude in
both dtypes (the arithmetic is fp32 throughout)."""
import numpy as np
import pytest
import torch

import oracle
from oracle.selector import block_summaries, gate_query
from paper_2609_13141_amd import configs, inputs, sas

from helpers import assert_close, f64

pytestmark = pytest.mark.gpu
TOL = 1e-4


def W(dtype="bf16", n=200, H=4, Hkv=2, dh=64, B=16, K=2, b=2, index=120):
    return configs.Workload(name="selbwd", dtype=dtype, batch=b, seq_len=n, d_model=256, n_heads=H,
                            n_kv_heads=Hkv, head_dim=dh, d_ff=512, block_size=B, top_k=K, mode="gated",
                            segments=(("img", n // 2), ("txt", n - n // 2)), index=index)


CASES = [
    (W(), False),
    (W(), True),
    (W(dtype="f32", index=121), True),
    (W(dh=128, B=32, K=3, n=300, H=4, Hkv=1, index=122), True),
    (W(dh=128, B=64, K=4, n=1100, H=8, Hkv=2, b=1, index=123), False),
    (W(dh=64, B=16, K=8, n=700, H=2, Hkv=2, b=3, index=124), True),
]
IDS = [f"{w.dtype}-dh{w.head_dim}-B{w.block_size}-K{w.top_k}-n{w.seq_len}-b{w.batch}-{'proj' if p else 'plain'}"
       for w, p in CASES]


@pytest.mark.parametrize("w,proj", CASES, ids=IDS)
def test_selector_backward_matches_oracle(w, proj):
    print(f"\n[case] selector backward {IDS[CASES.index((w, proj))]}", flush=True)
    q, k, v = inputs.qkv(w)
    Wl = inputs.layer_weights(w, selector_proj=proj)
    wgq, wgk = Wl["w_gq"], Wl["w_gk"]
    cfg = sas.make_config(w)
    dt = w.dtype
    qd, kd, vd = (sas.to_device(a, dt) for a in (q, k, v))
    wgq_d = None if wgq is None else sas.to_device(wgq, dt)
    wgk_d = None if wgk is None else sas.to_device(wgk, dt)
    fw = sas.attention_prefill(cfg, qd, kd, vd, wgq_d, wgk_d, log_gate=True)
    dlg = inputs.normal(w, "dlog_gate", (w.batch, w.n_kv_heads, w.seq_len, w.top_k), 1.0, dtype="f32")
    bw = sas.selector_backward(cfg, qd, kd, fw["sel_idx"], fw["log_gate"], torch.from_numpy(dlg).cuda(),
                               wgq_d, wgk_d)
    torch.cuda.synchronize()
    G, dh, B, n = w.group, w.head_dim, w.block_size, w.seq_len
    nf = n // B
    dwq = np.zeros((w.n_kv_heads, dh, dh))
    dwk = np.zeros((w.n_kv_heads, dh, dh))
    for bi in range(w.batch):
        st = oracle.select(f64(q[bi]), f64(k[bi]), B, w.top_k, dt,
                           w_gq=None if wgq is None else f64(wgq), w_gk=None if wgk is None else f64(wgk))
        sel = st["sel"]
        np.testing.assert_array_equal(fw["sel_idx"][bi].cpu().numpy(), sel)
        table = np.zeros((w.n_kv_heads, n, nf))
        for g in range(w.n_kv_heads):
            for t in range(n):
                for s_ in range(w.top_k):
                    if sel[g, t, s_] >= 0:
                        table[g, t, sel[g, t, s_]] = dlg[bi, g, t, s_]
        ds = oracle.gate_backward(table, st["r"], st["ct"], G, dh)
        q0 = gate_query(f64(q[bi]), G, dt) if wgq is not None else None
        k0 = block_summaries(f64(k[bi]), B, dt) if wgk is not None else None
        ref = oracle.selector_backward(ds, st["qhat"], st["kbar_proj"], G, dh, q0, k0)
        got_ds = bw["ds"][bi].cpu().numpy()
        assert_close(got_ds[:, :, :nf], ds, dt, f"ds b={bi}", tol=TOL)
        assert np.all(got_ds[:, :, nf:] == 0)
        assert_close(bw["dqhat"][bi].cpu().numpy(), ref["dqhat"], dt, f"dqhat b={bi}", tol=TOL)
        got_dk = bw["dkbar"][bi].cpu().numpy()
        assert_close(got_dk[:, :nf], ref["dkbar"], dt, f"dkbar b={bi}", tol=TOL)
        assert np.all(got_dk[:, nf:] == 0)
        if wgq is not None:
            dwq += ref["dw_gq"]
            dwk += ref["dw_gk"]
    if wgq is not None:
        assert_close(bw["dw_gq"].cpu().numpy(), dwq, dt, "dW_gq", tol=TOL)
        assert_close(bw["dw_gk"].cpu().numpy(), dwk, dt, "dW_gk", tol=TOL)


def test_selector_backward_k0_is_zero():
    w = W(K=0, index=125)
    q, k, v = inputs.qkv(w)
    cfg = sas.make_config(w)
    qd, kd = sas.to_device(q, "bf16"), sas.to_device(k, "bf16")
    bw = sas.selector_backward(cfg, qd, kd, None, None, None)
    torch.cuda.synchronize()
    for name in ("ds", "dqhat", "dkbar"):
        assert torch.all(bw[name] == 0), name


def test_training_chain_at_benchmark_shape():
    """Attention backward then selector backward at the 7B 1024-token shape
    (32 groups of 1 head, dh 128, B 64, K 8): the library's dlog_gate feeds
    its own selector backward; the oracle chains its own gradients.  dlog_gate
    carries the bf16 attention backward's error, so the bar is bf16's."""
    w = configs.L7B_1K.with_(index=126)
    print("\n[case] attention + selector backward at the 7B 1024-token shape", flush=True)
    q, k, v = inputs.qkv(w)
    d_o = inputs.normal(w, "d_o", q.shape, 1.0)
    cfg = sas.make_config(w)
    qd, kd, vd, dod = (sas.to_device(a, "bf16") for a in (q, k, v, d_o))
    fw = sas.attention_prefill(cfg, qd, kd, vd, log_gate=True)
    ab = sas.attention_backward(cfg, qd, kd, vd, fw["o"], dod, fw["lse"], fw["sel_idx"], fw["log_gate"])
    bw = sas.selector_backward(cfg, qd, kd, fw["sel_idx"], fw["log_gate"], ab["dlog_gate"])
    torch.cuda.synchronize()
    st = oracle.select(f64(q[0]), f64(k[0]), w.block_size, w.top_k, "bf16")
    _, _, _, dL = oracle.sas_attention_backward(f64(q[0]), f64(k[0]), f64(v[0]), f64(d_o[0]), w.block_size,
                                                "gated", st["sel"], st["log_gate"])
    nf = w.seq_len // w.block_size
    ds = oracle.gate_backward(dL[:, :, :nf], st["r"], st["ct"], w.group, w.head_dim)
    ref = oracle.selector_backward(ds, st["qhat"], st["kbar_proj"], w.group, w.head_dim)
    assert_close(bw["ds"][0, :, :, :nf].cpu().numpy(), ds, "bf16", "ds")
    assert_close(bw["dqhat"][0].cpu().numpy(), ref["dqhat"], "bf16", "dqhat")
    assert_close(bw["dkbar"][0, :, :nf].cpu().numpy(), ref["dkbar"], "bf16", "dkbar")
