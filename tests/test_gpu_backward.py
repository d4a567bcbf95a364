"""GPU parity of the SAS attention backward (Sec. 4.3; App. E's
recomputation backward, Alg. 1's training step): dQ, dK, dV and the block
log-gate gradient from the library, on its own forward's outputs, against
the fp64 oracle's backward on the oracle's own selection and gates (the
selections are bit-exact, so both attend the same sets)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_13141_amd import configs, inputs, sas

from helpers import assert_close, f64

pytestmark = pytest.mark.gpu


def W(dtype="bf16", n=200, H=4, Hkv=2, dh=64, B=16, K=2, mode="gated", b=2, index=100):
    return configs.Workload(name="bwd", dtype=dtype, batch=b, seq_len=n, d_model=256, n_heads=H, n_kv_heads=Hkv,
                            head_dim=dh, d_ff=512, block_size=B, top_k=K, mode=mode,
                            segments=(("img", n // 2), ("txt", n - n // 2)), index=index)


CASES = [
    W(),
    W(dtype="f32", index=101),
    W(mode="sparse", index=102),
    W(mode="dense", n=130, index=103),
    W(dh=128, B=32, K=3, n=256, index=104),
    W(dh=128, B=64, K=2, n=300, H=4, Hkv=4, index=105),
    W(dh=64, B=128, K=1, n=400, H=2, Hkv=1, index=106),
    W(dtype="f32", dh=128, B=64, K=2, n=200, H=2, Hkv=1, index=107),
    W(K=0, index=108),
    W(dh=128, B=128, K=2, n=520, H=4, Hkv=2, index=111),
]
IDS = [f"{w.dtype}-{w.mode}-dh{w.head_dim}-B{w.block_size}-K{w.top_k}-n{w.seq_len}-G{w.n_heads // w.n_kv_heads}"
       for w in CASES]


def _run(w):
    q, k, v = inputs.qkv(w)
    d_o = inputs.normal(w, "d_o", q.shape, 1.0)
    cfg = sas.make_config(w)
    dt = w.dtype
    qd, kd, vd, dod = (sas.to_device(a, dt) for a in (q, k, v, d_o))
    fw = sas.attention_prefill(cfg, qd, kd, vd, log_gate=True)
    bw = sas.attention_backward(cfg, qd, kd, vd, fw["o"], dod, fw["lse"], fw["sel_idx"], fw["log_gate"])
    torch.cuda.synchronize()
    return q, k, v, d_o, fw, bw


@pytest.mark.parametrize("w", CASES, ids=IDS)
def test_attention_backward_matches_oracle(w):
    print(f"\n[case] backward {w.dtype} {w.mode} dh={w.head_dim} B={w.block_size} K={w.top_k} n={w.seq_len}",
          flush=True)
    q, k, v, d_o, fw, bw = _run(w)
    tol = 2e-2 if w.dtype == "bf16" else 2e-5
    for bi in range(w.batch):
        if w.mode == "dense":
            sel = lg = None
        else:
            st = oracle.select(f64(q[bi]), f64(k[bi]), w.block_size, w.top_k, w.dtype)
            sel, lg = st["sel"], st["log_gate"]
            np.testing.assert_array_equal(fw["sel_idx"][bi].cpu().numpy(), sel)
        dQ, dK, dV, dL = oracle.sas_attention_backward(f64(q[bi]), f64(k[bi]), f64(v[bi]), f64(d_o[bi]),
                                                       w.block_size, w.mode, sel, lg)
        assert_close(bw["dq"][bi].float().cpu().numpy(), dQ, w.dtype, f"dQ b={bi}", tol=tol)
        assert_close(bw["dk"][bi].float().cpu().numpy(), dK, w.dtype, f"dK b={bi}", tol=tol)
        assert_close(bw["dv"][bi].float().cpu().numpy(), dV, w.dtype, f"dV b={bi}", tol=tol)
        got = bw["dlog_gate"][bi].cpu().numpy()
        if w.mode == "gated" and w.top_k > 0:
            want = np.zeros(got.shape)
            for g in range(w.n_kv_heads):
                for t in range(w.seq_len):
                    for s_ in range(w.top_k):
                        if sel[g, t, s_] >= 0:
                            want[g, t, s_] = dL[g, t, sel[g, t, s_]]
            assert_close(got, want, w.dtype, f"dlog_gate b={bi}", tol=tol)
        else:
            assert np.all(got == 0)


def test_attention_backward_benchmark_shape():
    # the benchmark workload's attention (1024 tokens, 32 heads, dh 128, B 64, K 8), every row
    w = configs.L7B_1K
    print("\n[case] backward at the 7B 1024-token shape", flush=True)
    q, k, v, d_o, fw, bw = _run(w.with_(index=109))
    st = oracle.select(f64(q[0]), f64(k[0]), w.block_size, w.top_k, "bf16")
    dQ, dK, dV, dL = oracle.sas_attention_backward(f64(q[0]), f64(k[0]), f64(v[0]), f64(d_o[0]), w.block_size,
                                                   "gated", st["sel"], st["log_gate"])
    assert_close(bw["dq"][0].float().cpu().numpy(), dQ, "bf16", "dQ")
    assert_close(bw["dk"][0].float().cpu().numpy(), dK, "bf16", "dK")
    assert_close(bw["dv"][0].float().cpu().numpy(), dV, "bf16", "dV")


def test_attention_backward_4k_b4_work_queue():
    # 4 x 4096 tokens, 32/32 heads, K = 16: more jobs than resident workgroups, so both passes
    # run as work queues, and dK/dV walks the per-tile lists of attending rows.  The oracle
    # checks every row of two heads of the second sequence (one head per KV group: a head's
    # gradients depend on that head and its group alone, so the oracle runs on the slice).
    w = configs.BY_NAME["7b_layer_4k_b4"].with_(index=110)
    print("\n[case] backward at 4 x 4096 (work queues, row lists)", flush=True)
    q, k, v, d_o, fw, bw = _run(w)
    bi, heads = 1, [0, 31]
    st = oracle.select(f64(q[bi][:, heads]), f64(k[bi][:, heads]), w.block_size, w.top_k, "bf16")
    np.testing.assert_array_equal(fw["sel_idx"][bi][heads].cpu().numpy(), st["sel"])
    for j, h in enumerate(heads):
        sl = slice(h, h + 1)
        dQ, dK, dV, dL = oracle.sas_attention_backward(f64(q[bi][:, sl]), f64(k[bi][:, sl]), f64(v[bi][:, sl]),
                                                       f64(d_o[bi][:, sl]), w.block_size, "gated",
                                                       st["sel"][j:j + 1], st["log_gate"][j:j + 1])
        assert_close(bw["dq"][bi][:, sl].float().cpu().numpy(), dQ, "bf16", f"dQ h={h}")
        assert_close(bw["dk"][bi][:, sl].float().cpu().numpy(), dK, "bf16", f"dK h={h}")
        assert_close(bw["dv"][bi][:, sl].float().cpu().numpy(), dV, "bf16", f"dV h={h}")
        sel = st["sel"][j]
        want = np.where(sel >= 0, np.take_along_axis(dL[0], np.maximum(sel, 0), axis=1), 0.0)
        assert_close(bw["dlog_gate"][bi][h].cpu().numpy(), want, "bf16", f"dlog_gate h={h}")
