"""GPU parity of the selection statistics (Sec. 6.1): mass coverage with both
weightings against the fp64 oracle, the full-attention reference sets
(per-head Top-K by block mass, group majority vote) against the oracle's
sets on every (query, group) whose per-head rankings have no near-tie at
the K-th place, the selection bitmasks exactly, and the overlap-recall
counts exactly from the bitmasks."""
import numpy as np
import pytest
import torch

import oracle
from oracle.stats import block_mass_topk, majority_vote, mass_coverage, overlap_recall, selection_sets
from paper_2609_13141_amd import configs, inputs, sas

from helpers import assert_close, f64

pytestmark = pytest.mark.gpu


def W(dtype="bf16", n=200, H=4, Hkv=2, dh=64, B=16, K=2, b=2, index=160):
    return configs.Workload(name="stats", dtype=dtype, batch=b, seq_len=n, d_model=256, n_heads=H,
                            n_kv_heads=Hkv, head_dim=dh, d_ff=512, block_size=B, top_k=K, mode="gated",
                            segments=(("img", n // 2), ("txt", n - n // 2)), index=index)


CASES = [
    W(),
    W(dtype="f32", index=161),
    W(dh=128, B=32, K=3, n=300, H=6, Hkv=2, b=1, index=162),
    W(dh=128, B=64, K=2, n=333, H=4, Hkv=4, b=1, index=163),
    W(dh=64, B=128, K=1, n=400, H=3, Hkv=1, b=1, index=164),
]
IDS = [f"{w.dtype}-dh{w.head_dim}-B{w.block_size}-K{w.top_k}-n{w.seq_len}-G{w.group}" for w in CASES]


def _bits(mask_t, NB):
    """int32 bitmask tensor [b, Hkv, n, W] -> bool [b, Hkv, n, NB]."""
    w = mask_t.cpu().numpy().view(np.uint32)
    bits = (w[..., :, None] >> np.arange(32, dtype=np.uint32)) & 1
    return bits.reshape(*w.shape[:-1], -1)[..., :NB].astype(bool)


def _clear_rows(lmass, top_k, G, margin=1e-4):
    """(Hkv, n) rows whose every head has a gap above `margin` (relative, in
    block log-mass) between its K-th and (K+1)-th block: there the Top-K is
    unique at the kernel's precision."""
    H, n, NB = lmass.shape
    ok = np.ones((H // G, n), dtype=bool)
    for h in range(H):
        for t in range(n):
            row = np.sort(lmass[h, t][np.isfinite(lmass[h, t])])[::-1]
            if top_k < len(row) and top_k > 0:
                if row[top_k - 1] - row[top_k] <= margin * max(1.0, abs(row[top_k - 1])):
                    ok[h // G, t] = False
    return ok


@pytest.mark.parametrize("w", CASES, ids=IDS)
def test_stats_match_oracle(w):
    print(f"\n[case] stats {w.dtype} dh={w.head_dim} B={w.block_size} K={w.top_k} n={w.seq_len}", flush=True)
    q, k, v = inputs.qkv(w)
    cfg = sas.make_config(w)
    dt = w.dtype
    qd, kd, vd = (sas.to_device(a, dt) for a in (q, k, v))
    fw = sas.attention_prefill(cfg, qd, kd, vd)
    su, ru = sas.alloc_union(cfg, w.batch, w.seq_len), sas.alloc_union(cfg, w.batch, w.seq_len)
    st = sas.selection_stats(cfg, qd, kd, vd, fw["sel_idx"], sel_union=su, ref_union=ru)
    torch.cuda.synchronize()
    NB = -(-w.seq_len // w.block_size)
    gsel, gref = _bits(su, NB), _bits(ru, NB)
    for bi in range(w.batch):
        sel = oracle.select(f64(q[bi]), f64(k[bi]), w.block_size, w.top_k, dt)["sel"]
        np.testing.assert_array_equal(fw["sel_idx"][bi].cpu().numpy(), sel)
        cov, cov_v = mass_coverage(f64(q[bi]), f64(k[bi]), f64(v[bi]), w.block_size, sel)
        assert_close(st["cov"][bi].cpu().numpy(), cov, dt, "cov", tol=1e-4)
        assert_close(st["cov_v"][bi].cpu().numpy(), cov_v, dt, "cov_v", tol=1e-4)
        np.testing.assert_array_equal(gsel[bi], selection_sets(sel, NB))
        hs, lmass = block_mass_topk(f64(q[bi]), f64(k[bi]), w.block_size, w.top_k)
        ref = majority_vote(hs, w.group)
        ok = _clear_rows(lmass, w.top_k, w.group)
        assert ok.mean() > 0.9
        np.testing.assert_array_equal(gref[bi][ok], ref[ok])


def test_overlap_recall_over_layers():
    """Two layers' sets accumulated on the GPU: the recall counts are exact
    for the GPU's bitmasks; the union equals the oracle's on every (query,
    group) without a near-tie in either layer, and the recall is within the
    bound the remaining rows allow."""
    w = W(b=1, n=256, B=16, K=3, index=170)
    cfg = sas.make_config(w)
    su, ru = sas.alloc_union(cfg, 1, w.seq_len), sas.alloc_union(cfg, 1, w.seq_len)
    NB = -(-w.seq_len // w.block_size)
    msets, osets = [], []
    clear = np.ones((w.n_kv_heads, w.seq_len), dtype=bool)
    for layer in range(2):
        q, k, v = inputs.qkv(w, seed=layer)
        qd, kd, vd = (sas.to_device(a, "bf16") for a in (q, k, v))
        fw = sas.attention_prefill(cfg, qd, kd, vd)
        sas.selection_stats(cfg, qd, kd, vd, fw["sel_idx"], cov=False, cov_v=False, sel_union=su, ref_union=ru)
        sel = oracle.select(f64(q[0]), f64(k[0]), w.block_size, w.top_k, "bf16")["sel"]
        msets.append(selection_sets(sel, NB))
        hs, lmass = block_mass_topk(f64(q[0]), f64(k[0]), w.block_size, w.top_k)
        clear &= _clear_rows(lmass, w.top_k, w.group)
        osets.append(majority_vote(hs, w.group))
    inter, tot, rec = sas.overlap_recall(su, ru)
    a, b = _bits(su, NB)[0], _bits(ru, NB)[0]
    assert inter == int((a & b).sum()) and tot == int(b.sum())
    np.testing.assert_array_equal(a, msets[0] | msets[1])
    ustar = osets[0] | osets[1]
    np.testing.assert_array_equal(b[clear], ustar[clear])
    assert clear.mean() > 0.95
    gi, gt, grec = overlap_recall(msets, osets)
    slack = int((~clear).sum()) * 2 * w.top_k  # blocks the unclear rows can change
    assert abs(inter - gi) <= slack and abs(tot - gt) <= slack
    assert 0.0 < rec <= 1.0


def test_stats_benchmark_shape_every_row():
    """The 7B 1024-token layer shape: coverage of every row against the oracle."""
    w = configs.L7B_1K.with_(index=171)
    print("\n[case] stats at the 7B 1024-token shape", flush=True)
    q, k, v = inputs.qkv(w)
    cfg = sas.make_config(w)
    qd, kd, vd = (sas.to_device(a, "bf16") for a in (q, k, v))
    fw = sas.attention_prefill(cfg, qd, kd, vd)
    st = sas.selection_stats(cfg, qd, kd, vd, fw["sel_idx"])
    torch.cuda.synchronize()
    sel = oracle.select(f64(q[0]), f64(k[0]), w.block_size, w.top_k, "bf16")["sel"]
    np.testing.assert_array_equal(fw["sel_idx"][0].cpu().numpy(), sel)
    cov, cov_v = mass_coverage(f64(q[0]), f64(k[0]), f64(v[0]), w.block_size, sel)
    assert_close(st["cov"][0].cpu().numpy(), cov, "bf16", "cov", tol=1e-4)
    assert_close(st["cov_v"][0].cpu().numpy(), cov_v, "bf16", "cov_v", tol=1e-4)


def test_stats_4k_b4_work_queue():
    # 4 x 4096 tokens, 32/32 heads: more jobs than resident workgroups (work queue); every row
    # of one head of the last sequence (one head per group: its coverage depends on it alone)
    w = configs.BY_NAME["7b_layer_4k_b4"].with_(index=172)
    print("\n[case] stats at 4 x 4096 (work queue)", flush=True)
    q, k, v = inputs.qkv(w)
    cfg = sas.make_config(w)
    qd, kd, vd = (sas.to_device(a, "bf16") for a in (q, k, v))
    fw = sas.attention_prefill(cfg, qd, kd, vd)
    st = sas.selection_stats(cfg, qd, kd, vd, fw["sel_idx"])
    torch.cuda.synchronize()
    bi, h = 3, 17
    sl = slice(h, h + 1)
    sel = oracle.select(f64(q[bi][:, sl]), f64(k[bi][:, sl]), w.block_size, w.top_k, "bf16")["sel"]
    np.testing.assert_array_equal(fw["sel_idx"][bi][sl].cpu().numpy(), sel)
    cov, cov_v = mass_coverage(f64(q[bi][:, sl]), f64(k[bi][:, sl]), f64(v[bi][:, sl]), w.block_size, sel)
    assert_close(st["cov"][bi][sl].cpu().numpy(), cov, "bf16", "cov", tol=1e-4)
    assert_close(st["cov_v"][bi][sl].cpu().numpy(), cov_v, "bf16", "cov_v", tol=1e-4)
