"""The decode step over the packed copy of the layer's weights
(sas_pack_decode_weights) gives the same bits as over the row-major
weights: outputs, selections and the q/k/v/h1 taps, over several steps,
at small shapes, the 7B stack layer and the 28/4 GQA layer.  Both runs start
from caches filled by the same prefill."""
import pytest
import torch

from paper_2609_13141_amd import configs, inputs, sas

pytestmark = pytest.mark.gpu


def W_(**kw):
    base = dict(name="decpk", dtype="bf16", batch=3, seq_len=72, d_model=256, n_heads=4, n_kv_heads=2,
                head_dim=64, d_ff=512, block_size=16, top_k=2, mode="sparse", segments=(), index=90)
    base.update(kw)
    n = base["seq_len"]
    base["segments"] = (("img", n // 2), ("txt", n - n // 2))
    return configs.Workload(**base)


CASES = {
    "small-dh64": (W_(), 51),
    "small-dh128-G7": (W_(head_dim=128, n_heads=7, n_kv_heads=1, d_model=896, d_ff=1280, index=91), 51),
    "7b-layer-b8": (configs.STACK_DECODE.with_(seq_len=140, segments=(("img", 64), ("txt", 76))), 127),
    "gqa28x4-layer-b2": (configs.BY_NAME["gqa28x4_layer_16k"].with_(batch=2, seq_len=140, mode="sparse",
                                                                     segments=(("img", 64), ("txt", 76))), 127),
}


@pytest.mark.parametrize("name", list(CASES))
def test_packed_decode_is_bit_identical(name):
    w, n0 = CASES[name]
    print(f"\n[case] packed decode {name}: b={w.batch} d={w.d_model} H={w.n_heads}/{w.n_kv_heads} "
          f"dh={w.head_dim} d_ff={w.d_ff} prefill {n0}", flush=True)
    x = sas.to_device(inputs.embeddings(w), "bf16")
    Wd = sas.weights_to_device(inputs.layer_weights(w), "bf16")
    cfg_p, cfg_d = sas.make_config(w, "dense"), sas.make_config(w, "sparse")
    Wp = sas.pack_decode_weights(cfg_d, Wd)
    caches = []
    for _ in range(2):
        cache = sas.alloc_cache(cfg_d, w.batch, w.seq_len, page_size=16)
        sas.layer_forward(cfg_p, x[:, :n0].contiguous(), Wd, stats=False, cache=cache)
        caches.append(cache)
    for t in range(n0, w.seq_len):
        pos = torch.full((w.batch,), t, dtype=torch.int32, device="cuda")
        xt = x[:, t].contiguous()
        y0, s0, tp0 = sas.decode_step(cfg_d, xt, pos, Wd, caches[0], taps=True)
        y1, s1, tp1 = sas.decode_step(cfg_d, xt, pos, Wp, caches[1], taps=True)
        torch.cuda.synchronize()
        assert torch.equal(y0, y1), (name, t, "y")
        assert torch.equal(s0, s1), (name, t, "sel")
        for k in ("q", "k", "v", "h1"):
            assert torch.equal(tp0[k], tp1[k]), (name, t, k)
    for a, b in zip((caches[0].k_pages, caches[0].v_pages, caches[0].k_summary),
                    (caches[1].k_pages, caches[1].v_pages, caches[1].k_summary)):
        assert torch.equal(a, b)
