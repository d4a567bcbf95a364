"""The no-allocation decode step (sas_decode_step_noalloc) against the
workspace entry point (sas_decode_step): the same kernels, so the same
outputs bit for bit, on two calls in a row (the second with a smaller
input), each on its own copy of the same prefilled cache."""
import numpy as np
import pytest
import torch

from paper_2609_13141_amd import configs, inputs, sas

pytestmark = pytest.mark.gpu


def _prefilled_pair(w, n0, max_len):
    x = inputs.embeddings(w.with_(seq_len=n0 + 1, segments=(("img", n0 // 2), ("txt", n0 + 1 - n0 // 2))))
    Wd = sas.weights_to_device(inputs.layer_weights(w), "bf16")
    xd = sas.to_device(x, "bf16")
    cfg_p, cfg_d = sas.make_config(w, "dense"), sas.make_config(w, "sparse")
    caches = []
    for _ in range(2):
        c = sas.alloc_cache(cfg_d, w.batch, max_len, page_size=16, seed=1)
        sas.layer_forward(cfg_p, xd[:, :n0].contiguous(), Wd, stats=False, cache=c)
        caches.append(c)
    return cfg_d, Wd, xd[:, n0].contiguous(), caches


def _compare(w, n0, max_len):
    print(f"\n[case] no-alloc decode b={w.batch} d={w.d_model} ctx={n0}", flush=True)
    cfg, Wd, x, (ca, cb) = _prefilled_pair(w, n0, max_len)
    pos = torch.full((w.batch,), n0, dtype=torch.int32, device="cuda")
    ya, sa = sas.decode_step(cfg, x, pos, Wd, ca)
    yb, sb = sas.decode_step_noalloc(cfg, x, pos, Wd, cb)
    torch.cuda.synchronize()
    assert torch.equal(ya, yb)
    assert torch.equal(sa, sb)
    assert torch.equal(ca.k_pages, cb.k_pages) and torch.equal(ca.v_pages, cb.v_pages)
    assert torch.equal(ca.k_summary, cb.k_summary)
    assert bool(torch.isfinite(yb.float()).all())


def test_noalloc_decode_step_matches_workspace_entry_point_twice():
    # first: one layer of the 7B serving shape, 8 sequences after a 2048-token prefill
    _compare(configs.STACK_DECODE, 2048, 2304)
    # second, smaller: 3 sequences of a narrow GQA layer after 100 tokens
    small = configs.Workload(name="noalloc_small", dtype="bf16", batch=3, seq_len=101, d_model=256, n_heads=4,
                             n_kv_heads=2, head_dim=64, d_ff=512, block_size=16, top_k=2, mode="sparse",
                             segments=(("img", 50), ("txt", 51)), index=190)
    _compare(small, 100, 160)
