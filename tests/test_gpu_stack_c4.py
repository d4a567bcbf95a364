"""Full-shape parity of the 32-layer serving workload (Sec. 5.1, Alg. 2):
8 sequences of 576 image + 1472 text tokens prefilled densely through 32
7B-shape layers into 16-token pages, then greedy SAS decode steps
(B = 64, K = 16), against the fp64 oracle for sequence 0.

The weights, embedding table and LM head are the ones the benchmark draws
on the GPU; the oracle receives them by copying them to the host, layer by
layer.  An fp64 chain run independently through the stack drifts from any
bf16 one by about 2e-3 (relative) per layer -- 4e-3 after the first layer,
2.2e-2 after the eighth, measured against this implementation -- so every
layer is checked on the GPU's own input to that layer (the oracle computes
the layer from it, prefill rows and decode rows alike; decode is
teacher-forced on the GPU's generated tokens):
* every layer's output of the prefill (all 2048 rows of sequence 0) and of
  each decode step is within the bf16 tolerance of the GPU's;
* the logits of the prefill's last row and of every decode step, computed by
  the oracle from the GPU's final hidden states, are within tolerance, and the
  greedy token agrees wherever the oracle's top two logits are further apart
  than twice the observed logit error;
* every layer's decode selection of every sequence equals the oracle's
  selector on the layer's own query heads and cached summaries, and the
  cached summaries equal the oracle's pooling of the cached keys (both
  bit-exact)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_13141_amd import configs, inputs, model, sas

from helpers import assert_close, check_decode_selection, f64, rel_err, spec_of

pytestmark = pytest.mark.gpu

W = configs.STACK_DECODE
STEPS = 3          # teacher-forced decode steps checked
SEQ = 0            # the sequence the oracle follows
PARTS = 4          # the 32 layers are checked in 4 tests of 8 layers
TOL = 2e-2


@pytest.fixture(scope="module")
def run():
    dev = "cuda"
    print(f"\n[case] C4 stack on the GPU: {W.n_layers} layers, b={W.batch}, n={W.seq_len}, "
          f"{STEPS} decode steps", flush=True)
    layers = [inputs.layer_weights_device(W, layer=l, device=dev) for l in range(W.n_layers)]
    ends = inputs.model_ends_device(W, device=dev)
    st = model.Stack(W, layers, ends, max_len=W.seq_len + STEPS + 8, device=dev)
    hid = {}

    def keep(l, x):
        hid[l] = x[SEQ].float().cpu().numpy()
    tok, lg0 = st.prefill(ends["token_ids"], ends["img_embed"], logits=True, on_layer=keep)
    torch.cuda.synchronize()
    sp = spec_of(W, "sparse")
    toks, logits, dec = [tok.cpu().numpy()], [lg0[SEQ].cpu().numpy()], []
    for s, pos in enumerate(st.positions(STEPS)):
        t = W.seq_len + s
        nxt, lg, sels, taps = st.step(tok, pos, logits=True, sel_idx=True, taps=True)
        torch.cuda.synchronize()
        for l in range(W.n_layers):
            # bit-exact: each layer's selection on its own query heads and cache (and, at the
            # first step, the cached summaries against the pooling of the cached keys)
            check_decode_selection(sels[l].cpu().numpy(), taps[l]["q"], st.caches[l], t, sp,
                                   summaries_from_keys=(s == 0))
        dec.append([taps[l]["x"][SEQ].float().cpu().numpy() for l in range(W.n_layers)]
                   + [taps[-1]["y"][SEQ].float().cpu().numpy()])
        toks.append(nxt.cpu().numpy())
        logits.append(lg[SEQ].cpu().numpy())
        tok = nxt
    print(f"  GPU run done; first tokens of sequence {SEQ}: {[int(t[SEQ]) for t in toks]}", flush=True)
    # the embeddings: the oracle's gather of the prompt (image rows in order) and of the GPU's tokens
    ids = ends["token_ids"][SEQ:SEQ + 1].cpu().numpy()
    n_img = int((ids < 0).sum())
    img = ends["img_embed"][SEQ:SEQ + 1, :n_img].float().cpu().numpy()
    table = ends["embed"].float().cpu().numpy()
    np.testing.assert_array_equal(hid[0], oracle.embed_tokens(ids, table, img)[0])
    for s in range(STEPS):
        np.testing.assert_array_equal(dec[s][0], table[int(toks[s][SEQ])])
    return {"st": st, "layers": layers, "ends": ends, "hid": hid, "dec": dec, "toks": toks, "logits": logits,
            "done": 0}


def _host_weights(Wd):
    return {k: (None if v is None else f64(v.float().cpu().numpy())) for k, v in Wd.items()}


def _check_layers(r, lo, hi):
    """Layers lo..hi-1: the oracle computes each from the GPU's input to it
    (the 2048 prefill rows, then the decode rows in order, which attend to the
    oracle's own cache of that layer) and is compared with the GPU's output."""
    spd, sps = spec_of(W, "dense"), spec_of(W, "sparse")
    for l in range(lo, hi):
        Wl = _host_weights(r["layers"][l])
        pre = oracle.dense_prefill_layer(f64(r["hid"][l]), Wl, spd)
        cache = oracle.DecodeCache(1, W.seq_len + STEPS, sps)
        cache.fill_prefill(0, pre["K"], pre["V"], pre["k_summary"])
        e_pre = rel_err(r["hid"][l + 1], pre["y"])
        e_dec = 0.0
        for s in range(STEPS):
            y, _ = oracle.decode_step(f64(r["dec"][s][l])[None], np.array([W.seq_len + s]), Wl, cache, sps)
            e_dec = max(e_dec, rel_err(r["dec"][s][l + 1], y[0]))
        print(f"  layer {l:2d}: prefill rel err {e_pre:.2e}, decode rel err {e_dec:.2e}", flush=True)
        assert e_pre <= TOL, f"layer {l} prefill output: rel err {e_pre:.3e}"
        assert e_dec <= TOL, f"layer {l} decode output: rel err {e_dec:.3e}"
    r["done"] = max(r["done"], hi)


@pytest.mark.parametrize("part", range(PARTS))
def test_c4_stack_layers_match_oracle(run, part):
    per = W.n_layers // PARTS
    _check_layers(run, part * per, (part + 1) * per)


def test_c4_stack_logits_and_greedy_tokens(run):
    ends = run["ends"]
    gamma = f64(ends["rms_final"].float().cpu().numpy())
    w_lm = f64(ends["w_lm"].float().cpu().numpy())
    L = W.n_layers
    # the GPU's final hidden states: the prefill's last row, then each decode step's
    hs = np.concatenate([f64(run["hid"][L][-1:])] + [f64(run["dec"][s][L])[None] for s in range(STEPS)])
    otok, olog = oracle.lm_head_argmax(hs, gamma, w_lm, W.rms_eps, "bf16")
    glog = np.stack(run["logits"])
    gtok = np.array([t[SEQ] for t in run["toks"]])
    for s in range(STEPS + 1):
        assert_close(glog[s], olog[s], "bf16", f"logits {s}")
        err = np.max(np.abs(glog[s] - olog[s]))
        top = np.sort(olog[s])[-2:]
        if top[1] - top[0] > 2 * err:
            assert gtok[s] == otok[s], (s, gtok[s], otok[s])
        print(f"  step {s}: logits rel err {rel_err(glog[s], olog[s]):.2e}, token {gtok[s]} "
              f"(oracle {otok[s]}, top-2 gap {top[1] - top[0]:.3f}, error {err:.3f})", flush=True)
