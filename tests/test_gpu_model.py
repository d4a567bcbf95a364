"""GPU parity of the served stack (Sec. 5.1, Alg. 2): embedding, a dense
prefill through every layer into paged caches, then greedy SAS decode steps
(embed -> each layer's decode step -> final RMSNorm + LM head + argmax),
against the fp64 oracle teacher-forced on the GPU's tokens."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_13141_amd import configs, inputs, model, sas

from helpers import assert_close, check_decode_selection, f64, spec_of

pytestmark = pytest.mark.gpu

W = configs.Workload(name="stack_small", dtype="bf16", batch=2, seq_len=40, d_model=256, n_heads=4, n_kv_heads=2,
                     head_dim=64, d_ff=512, block_size=16, top_k=2, mode="sparse",
                     segments=(("img", 16), ("txt", 24)), n_layers=2, vocab=300, decode_steps=6, page_size=8,
                     index=81)


def _check_tokens(tok, ref_tok, logits, ref_logits):
    # where the oracle's top two logits are apart by more than the logit error, the argmax must agree
    err = np.max(np.abs(logits - ref_logits))
    srt = np.sort(ref_logits, axis=1)
    for r in range(len(tok)):
        if srt[r, -1] - srt[r, -2] > 2 * err:
            assert tok[r] == ref_tok[r], (r, tok[r], ref_tok[r])


def test_stack_prefill_and_greedy_decode_match_oracle():
    print("\n[case] 2-layer stack: prefill 40 tokens, 6 greedy decode steps", flush=True)
    ends = inputs.model_ends(W)
    layers = [inputs.layer_weights(W, layer=l) for l in range(W.n_layers)]
    dev_ends = {k: sas.to_device(ends[k], "bf16") for k in ("embed", "w_lm", "rms_final")}
    max_len = W.seq_len + W.decode_steps + 2
    st = model.Stack(W, [sas.weights_to_device(L, "bf16") for L in layers], dev_ends, max_len=max_len)
    ids = torch.from_numpy(ends["token_ids"]).cuda()
    tok, lg0 = st.prefill(ids, sas.to_device(ends["img_embed"], "bf16"), logits=True)
    torch.cuda.synchronize()

    sp_dense, sp = spec_of(W, "dense"), spec_of(W, "sparse")
    Wo = [{k: (None if a is None else f64(a)) for k, a in L.items()} for L in layers]
    x = oracle.embed_tokens(ends["token_ids"], f64(ends["embed"]), f64(ends["img_embed"]))
    caches = []
    for l in range(W.n_layers):
        pre = oracle.layer_forward(x, Wo[l], sp_dense)
        c = oracle.DecodeCache(W.batch, max_len, sp)
        for bi in range(W.batch):
            c.fill_prefill(bi, pre["K"][bi], pre["V"][bi], pre["k_summary"][bi])
        caches.append(c)
        x = pre["y"]
    otok, olog = oracle.lm_head_argmax(x[:, -1], f64(ends["rms_final"]), f64(ends["w_lm"]), W.rms_eps, "bf16")
    assert_close(lg0.cpu().numpy(), olog, "bf16", "prefill logits")
    _check_tokens(tok.cpu().numpy(), otok, lg0.cpu().numpy(), olog)

    for s, pos in enumerate(st.positions(W.decode_steps)):
        t = W.seq_len + s
        nxt, lg, sels, taps = st.step(tok, pos, logits=True, sel_idx=True, taps=True)
        torch.cuda.synchronize()
        tk = tok.cpu().numpy()
        xo = oracle.embed_tokens(tk[:, None], f64(ends["embed"]))[:, 0]
        for l in range(W.n_layers):
            xo, _ = oracle.decode_step(xo, np.full(W.batch, t), Wo[l], caches[l], sp)
            # every layer's selection equals the oracle's on the layer's own query heads and cache: bit-exact
            check_decode_selection(sels[l].cpu().numpy(), taps[l]["q"], st.caches[l], t, sp)
        otk, olg = oracle.lm_head_argmax(xo, f64(ends["rms_final"]), f64(ends["w_lm"]), W.rms_eps, "bf16")
        lgn = lg.cpu().numpy()
        assert_close(lgn, olg, "bf16", f"logits at t={t}")
        assert list(nxt.cpu().numpy()) == list(np.argmax(lgn, axis=1))   # argmax of the GPU's own logits
        _check_tokens(nxt.cpu().numpy(), otk, lgn, olg)
        tok = nxt


def test_stack_generate_is_deterministic():
    ends = inputs.model_ends(W)
    layers = [sas.weights_to_device(inputs.layer_weights(W, layer=l), "bf16") for l in range(W.n_layers)]
    dev_ends = {k: sas.to_device(ends[k], "bf16") for k in ("embed", "w_lm", "rms_final")}
    ids = torch.from_numpy(ends["token_ids"]).cuda()
    img = sas.to_device(ends["img_embed"], "bf16")
    outs = []
    for _ in range(2):
        st = model.Stack(W, layers, dev_ends, max_len=W.seq_len + W.decode_steps + 2)
        outs.append(st.generate(ids, img, W.decode_steps).cpu().numpy())
    assert outs[0].shape == (W.batch, W.decode_steps + 1)
    np.testing.assert_array_equal(outs[0], outs[1])
    assert outs[0].min() >= 0 and outs[0].max() < W.vocab
