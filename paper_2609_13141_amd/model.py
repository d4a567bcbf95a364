"""A decoder stack served with SAS (Sec. 5.1, Alg. 2), over the C ABI.

The prompt is prefilled densely through every layer, which fills each
layer's paged KV cache and block summaries; every generated token is then
embedded, runs the SAS decode step in each layer (Top-K blocks per KV group
by the selector, attention to them plus the current block without gate bias)
and the greedy LM head (final RMSNorm, logits in fp32, lowest id on ties).
Every step runs in the library's kernels; this module only sequences them.
"""
from __future__ import annotations

import torch

from . import sas
from .configs import Workload


class Stack:
    def __init__(self, w: Workload, layers: list, ends: dict, *, max_len: int, page_size: int | None = None,
                 device="cuda", packed: bool = True):
        """layers: per-layer device weight dicts; ends: device tensors
        'embed' [V, d], 'w_lm' [V, d], 'rms_final' [d].  packed: the decode
        steps stream a packed copy of each layer's linear weights (made here
        when the configuration has a packed layout; results are identical)."""
        self.w = w
        self.ends = ends
        self.device = device
        self.cfg_prefill = sas.make_config(w, "dense")
        self.cfg_decode = sas.make_config(w, "sparse")
        if packed and sas.lib().sas_decode_packed_bytes(sas.C.byref(self.cfg_decode)) > 0:
            layers = [sas.pack_decode_weights(self.cfg_decode, W) for W in layers]
        self.layers = layers
        ps = page_size or w.page_size
        self.caches = [sas.alloc_cache(self.cfg_decode, w.batch, max_len, page_size=ps, device=device, seed=l)
                       for l in range(len(layers))]
        self.ws = sas.Workspace(device)
        self.max_len = max_len
        self.pos = None

    def prefill(self, ids, img=None, *, logits: bool = False, on_layer=None):
        """ids [b, n] int32 on the device (-1 = next image embedding row);
        returns the first generated token of every sequence [b] int32 (and
        its fp32 logits when asked).  on_layer(l, x), when given, sees the
        input x [b, n, d] of every layer l and the last layer's output (l = L)."""
        x = sas.embed(self.cfg_prefill, ids, self.ends["embed"], img)
        for l, (W, cache) in enumerate(zip(self.layers, self.caches)):
            if on_layer is not None:
                on_layer(l, x)
            x = sas.layer_forward(self.cfg_prefill, x, W, stats=False, cache=cache, ws=self.ws)["y"]
        if on_layer is not None:
            on_layer(len(self.layers), x)
        self.pos = ids.shape[1]
        tok, lg = sas.lm_head_argmax(self.cfg_decode, x[:, -1].contiguous(), self.ends["rms_final"],
                                     self.ends["w_lm"], logits=logits, ws=self.ws)
        return (tok, lg) if logits else tok

    def positions(self, steps: int):
        """Device position vectors for the next `steps` decode steps."""
        b = self.w.batch
        return [torch.full((b,), self.pos + s, dtype=torch.int32, device=self.device) for s in range(steps)]

    def step(self, tok, pos, *, logits: bool = False, sel_idx: bool = False, taps: bool = False):
        """One generated token per sequence: tok [b] at positions pos [b]
        (device int32).  Returns the next tokens, the logits and per-layer
        selections when asked, and with taps a per-layer list of
        {"x": layer input, "q", "k", "v", "h1", "y": layer output}."""
        x = sas.embed(self.cfg_decode, tok.view(-1, 1), self.ends["embed"])[:, 0].contiguous()
        sels, tps = [], []
        for W, cache in zip(self.layers, self.caches):
            r = sas.decode_step(self.cfg_decode, x, pos, W, cache, sel_idx=sel_idx, taps=taps, ws=self.ws)
            if taps:
                r[2]["x"] = x
                r[2]["y"] = r[0]
                tps.append(r[2])
            x, sel = r[0], r[1]
            sels.append(sel)
        nxt, lg = sas.lm_head_argmax(self.cfg_decode, x, self.ends["rms_final"], self.ends["w_lm"], logits=logits,
                                     ws=self.ws)
        self.pos += 1
        out = (nxt, lg, (sels if sel_idx else None))
        return out + (tps,) if taps else out

    def generate(self, ids, img, steps: int):
        """Greedy generation: [b, steps + 1] tokens (the prefill's and `steps` more)."""
        tok = self.prefill(ids, img)
        out = [tok]
        for pos in self.positions(steps):
            tok, _, _ = self.step(tok, pos)
            out.append(tok)
        return torch.stack(out, 1)
