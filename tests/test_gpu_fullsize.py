"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times, on sampled rows the oracle computes one by one (K/V of
every earlier token are computed by the oracle, so each sampled row is
exact): the 7B layer over 1024 tokens (the benchmark workload), the 7B layer
over 4 x 4096 tokens (one sequence), the GQA 28/4 layer over 16384 tokens,
and attention-only checks with bit-exact selections at those shapes."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_13141_amd import configs, inputs, sas

from oracle.selector import select
from helpers import assert_close, assert_selection_near_ties, check_decode_selection, f64, score_bounds, spec_of

pytestmark = pytest.mark.gpu


def sample_rows(n, B, extra=(), k=20, seed=0):
    rng = np.random.default_rng(seed)
    rows = {0, 1, B - 1, B, n - 1, n // 2}
    rows |= {r for r in extra if 0 <= r < n}
    rows |= set(rng.integers(0, n, size=k).tolist())
    return np.array(sorted(rows))


def _oracle_W(Wl):
    return {k: (None if a is None else f64(a)) for k, a in Wl.items()}


def _check_layer_selection(w, sel_gpu, q_gpu, k_gpu, ref, rows):
    """sel_gpu [b, Hkv, R, K] at `rows`; q_gpu [b, R, H, dh] and k_gpu [b, n, Hkv, dh] the GPU's taps."""
    for bi in range(sel_gpu.shape[0]):
        # the oracle's selector on the GPU's own materialised Q/K: bit-exact
        st = select(f64(q_gpu[bi]), f64(k_gpu[bi]), w.block_size, w.top_k, "bf16", rows=rows)
        np.testing.assert_array_equal(sel_gpu[bi], st["sel"])
        # against the oracle's own Q/K: rows may differ only at near-ties within one ulp of Q/K
        r, bd = score_bounds(ref["Q"][bi], ref["K"][bi], w.block_size, w.group, "bf16")
        nf = r.shape[2]
        np.testing.assert_array_equal(r, ref["r"][bi][..., :nf])
        nd = assert_selection_near_ties(sel_gpu[bi], ref["sel"][bi], r, bd, "layer")
        print(f"  sequence {bi}: {nd} of {sel_gpu.shape[1] * sel_gpu.shape[2]} sampled rows differ from the "
              f"oracle's own selection, each at a near-tie", flush=True)


@pytest.mark.parametrize("name,batch_sel", [("7b_layer_1k", None), ("7b_layer_4k_b4", 0), ("gqa28x4_layer_16k", None)])
def test_layer_forward_fullsize_sampled_rows(name, batch_sel):
    w = configs.BY_NAME[name]
    print(f"\n[case] full-size layer {name} b={w.batch} n={w.seq_len}", flush=True)
    x = inputs.embeddings(w)
    Wl = inputs.layer_weights(w)
    cfg = sas.make_config(w)
    out = sas.layer_forward(cfg, sas.to_device(x, "bf16"), sas.weights_to_device(Wl, "bf16"), taps=True)
    torch.cuda.synchronize()
    bsel = [batch_sel] if batch_sel is not None else list(range(w.batch))
    rows = sample_rows(w.seq_len, w.block_size, extra=(575, 576, 577, 4095, 4096, 15871, 15872), k=16)
    ref = oracle.layer_forward(f64(x[bsel]), _oracle_W(Wl), spec_of(w), rows=rows)
    g = {k: out[k][bsel].float().cpu().numpy() if out[k].dtype != torch.int32 else out[k][bsel].cpu().numpy()
         for k in ("y", "q", "k", "v", "o", "h1", "sel_idx", "lse")}
    assert_close(g["k"], ref["K"], "bf16", "K (all rows)")
    assert_close(g["v"], ref["V"], "bf16", "V (all rows)")
    assert_close(g["q"][:, rows], ref["Q"], "bf16", "Q rows")
    assert_close(g["o"][:, rows], ref["O"], "bf16", "O rows")
    assert_close(g["h1"][:, rows], ref["h1"], "bf16", "h1 rows")
    assert_close(g["y"][:, rows], ref["y"], "bf16", "y rows")
    assert_close(g["lse"][:, :, rows], ref["LSE"], "bf16", "LSE rows", tol=1e-3)
    _check_layer_selection(w, g["sel_idx"][:, :, rows], g["q"][:, rows], g["k"], ref, rows)


@pytest.mark.parametrize("name,mode", [("7b_layer_1k", "gated"), ("7b_layer_4k_b4", "gated"),
                                       ("7b_stack32_prefill2k_decode256_b8", "dense"),
                                       ("gqa28x4_layer_16k", "gated"), ("gqa28x4_layer_16k", "sparse")])
def test_attention_fullsize_exact_selection(name, mode):
    w = configs.BY_NAME[name]
    print(f"\n[case] full-size attention {name} mode={mode}", flush=True)
    q, k, v = inputs.qkv(w)
    cfg = sas.make_config(w, mode)
    out = sas.attention_prefill(cfg, *(sas.to_device(a, "bf16") for a in (q, k, v)), tau=True)
    torch.cuda.synchronize()
    bsel = list(range(min(w.batch, 2)))
    rows = sample_rows(w.seq_len, w.block_size, extra=(575, 576, 15872), k=12, seed=1)
    ref = oracle.attention_prefill(f64(q[bsel][:, rows]), f64(k[bsel]), f64(v[bsel]), spec_of(w, mode), rows=rows)
    # identical Q/K bits on both sides: selections are bit-exact
    np.testing.assert_array_equal(out["sel_idx"][bsel][:, :, rows].cpu().numpy(), ref["sel"])
    nfull = w.seq_len // w.block_size
    np.testing.assert_array_equal(out["k_summary"][bsel][:, :, :nfull].float().cpu().numpy(),
                                  ref["k_summary"][:, :, :nfull])
    assert_close(out["o"][bsel][:, rows].float().cpu().numpy(), ref["O_exact"], "bf16", "O rows")
    assert_close(out["lse"][bsel][:, :, rows].cpu().numpy(), ref["LSE"], "bf16", "LSE rows", tol=1e-3)
    tau = out["tau"][bsel][:, :, rows].cpu().numpy()
    fin = np.isfinite(ref["tau"])
    np.testing.assert_array_equal(np.isfinite(tau), fin)
    if fin.any():
        assert_close(tau[fin], ref["tau"][fin], "bf16", "tau", tol=1e-5)


def test_attention_7b_1k_every_row_selection():
    # every row of the benchmark workload's selection, against the oracle's
    w = configs.L7B_1K
    q, k, v = inputs.qkv(w)
    cfg = sas.make_config(w)
    out = sas.attention_prefill(cfg, *(sas.to_device(a, "bf16") for a in (q, k, v)), log_gate=True)
    torch.cuda.synchronize()
    from oracle.selector import select
    st = select(f64(q[0]), f64(k[0]), w.block_size, w.top_k, "bf16")
    np.testing.assert_array_equal(out["sel_idx"][0].cpu().numpy(), st["sel"])
    lg = out["log_gate"][0].cpu().numpy()
    fin = np.isfinite(st["log_gate"])
    np.testing.assert_array_equal(np.isfinite(lg), fin)
    np.testing.assert_allclose(lg[fin], st["log_gate"][fin], rtol=0, atol=1e-5 * np.abs(st["log_gate"][fin]).max())


def test_decode_step_at_stack_shape_matches_oracle():
    # one layer of the 32-layer serving workload: dense prefill of 2048 tokens
    # for 8 sequences into 16-token pages, then decode steps at 2048..2050
    # (the first step closes no block; positions 2111 would)
    w = configs.STACK_DECODE
    print("\n[case] decode at the stack shape (one layer, b=8, ctx 2048)", flush=True)
    x_all = inputs.embeddings(w.with_(seq_len=2051, segments=(("img", 576), ("txt", 1475))))
    Wl = inputs.layer_weights(w)
    Wd = sas.weights_to_device(Wl, "bf16")
    xd = sas.to_device(x_all, "bf16")
    cfg_p, cfg_d = sas.make_config(w, "dense"), sas.make_config(w, "sparse")
    cache = sas.alloc_cache(cfg_d, w.batch, 2304, page_size=16)
    n0 = 2048
    sas.layer_forward(cfg_p, xd[:, :n0].contiguous(), Wd, stats=False, cache=cache)
    sp = spec_of(w, "sparse")
    bsel = [0, 5]
    ocache = oracle.DecodeCache(len(bsel), 2304, sp)
    from oracle.layer import qkv_projection
    from oracle.selector import block_summaries
    Q, K, V = qkv_projection(f64(x_all[bsel, :n0]), _oracle_W(Wl), sp, np.arange(0))
    for j in range(len(bsel)):
        ocache.fill_prefill(j, K[j], V[j], block_summaries(K[j], w.block_size, "bf16"))
    for t in range(n0, n0 + 3):
        pos = torch.full((w.batch,), t, dtype=torch.int32, device="cuda")
        y, sel, tp = sas.decode_step(cfg_d, xd[:, t].contiguous(), pos, Wd, cache, taps=True)
        torch.cuda.synchronize()
        # (the oracle's cache is filled in place by its decode step)
        yo, selo, qo = oracle.decode_step(f64(x_all[bsel, t]), np.full(len(bsel), t), _oracle_W(Wl), ocache, sp,
                                          taps=True)
        assert_close(y[bsel].float().cpu().numpy(), yo, "bf16", f"y t={t}")
        nd = check_decode_selection(sel.cpu().numpy(), tp["q"], cache, t, sp, ocache, bsel, q_ref=qo)
        print(f"  t={t}: {nd} of {len(bsel) * w.n_kv_heads} rows differ from the oracle's own selection, "
              f"each at a near-tie", flush=True)


def test_attention_7b_1k_every_row_output():
    # the benchmark workload's attention (1024 tokens, 32 heads): fewer (query tile, head) jobs
    # than resident workgroups, so the long query tiles run split and are merged; O and LSE of
    # every row of the first sequence against the oracle
    w = configs.L7B_1K.with_(index=173)
    print("\n[case] attention at the 7B 1024-token shape, every row", flush=True)
    q, k, v = inputs.qkv(w)
    cfg = sas.make_config(w)
    out = sas.attention_prefill(cfg, *(sas.to_device(a, "bf16") for a in (q, k, v)), log_gate=True)
    torch.cuda.synchronize()
    from oracle.selector import select
    st = select(f64(q[0]), f64(k[0]), w.block_size, w.top_k, "bf16")
    np.testing.assert_array_equal(out["sel_idx"][0].cpu().numpy(), st["sel"])
    _, O, LSE = oracle.sas_attention(f64(q[0]), f64(k[0]), f64(v[0]), w.block_size, "gated", "bf16",
                                     st["sel"], st["log_gate"])
    assert_close(out["o"][0].float().cpu().numpy(), O, "bf16", "O")
    assert_close(out["lse"][0].cpu().numpy(), LSE, "bf16", "LSE", tol=1e-3)
