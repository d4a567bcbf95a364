"""Workload shapes for the SAS hot path.

Five synthetic workloads shaped like the paper's setting (a decoder layer of a
dense LLM whose attention is sparsified by SAS, block size 64 and a Top-K
budget of blocks, Sec. 4.2.1 and Sec. 5.1), with long mixed image/text
sequences.  SAS itself is modality-agnostic: image/video tokens are ordinary
context tokens drawn with a larger scale.

The SAS parameters (block size ``B``, budget ``K`` in blocks, mode) per
workload are chosen so that selection is actually exercised:

* ``tiny``: B=16, K=2 (with B=64 the 64-token sequence would be a single
  block and SAS the identity).
* ``7b_1k``: B=64, K=8; text queries (t >= 576) have 9..15 historical blocks.
* ``7b_4k_b4``: B=64, K=16 (a 1024-token budget, the tightest in Table 2).
* ``7b_stack_decode``: dense prefill then sparse decode, B=64, K=16 (the
  serving pipeline of Sec. 5.1: dense prefill, block-sparse decode).
* ``gqa_16k``: B=64, K=32 (the paper's default Top-K 32, Sec. 4.2.1).
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Tuple

MODES = ("dense", "sparse", "gated")


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                  # "bf16" or "f32": activations and weights
    batch: int
    seq_len: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    block_size: int             # B, tokens per SAS block
    top_k: int                  # K, historical blocks kept per query
    mode: str                   # "gated" | "sparse" | "dense" (prefill)
    # token order of every sequence: (kind, count) with kind in {"img", "txt"}
    segments: Tuple[Tuple[str, int], ...] = ()
    img_scale: float = 2.0      # image/video embeddings are N(0,1) * img_scale
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    weight_std: float = 0.02
    n_layers: int = 1
    vocab: int = 0
    decode_steps: int = 0
    page_size: int = 16
    index: int = 0              # position in the workload list; part of every seed

    @property
    def group(self) -> int:
        return self.n_heads // self.n_kv_heads

    @property
    def tokens(self) -> int:
        return self.batch * self.seq_len

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)

    def linear_params(self) -> int:
        """Parameters of the linear layers of one decoder layer."""
        qkv = (self.n_heads + 2 * self.n_kv_heads) * self.head_dim * self.d_model
        o = self.d_model * self.n_heads * self.head_dim
        mlp = 3 * self.d_model * self.d_ff
        return qkv + o + mlp

    def attended_pairs(self, mode: str | None = None) -> int:
        """sum over queries t of |S_t| for one sequence (independent of which
        blocks are selected: |S_t| = (t mod B) + 1 + B*min(K, floor(t/B)))."""
        mode = mode or self.mode
        n, B, K = self.seq_len, self.block_size, self.top_k
        if mode == "dense":
            return n * (n + 1) // 2
        tot = 0
        for t in range(n):
            tot += (t % B) + 1 + B * min(K, t // B)
        return tot

    def prefill_flops(self, mode: str | None = None) -> int:
        """Algorithmic FLOPs of one layer forward over the whole batch: the
        linear layers plus QK^T and PV over the attended pairs."""
        lin = 2 * self.tokens * self.linear_params()
        att = 4 * self.head_dim * self.n_heads * self.batch * self.attended_pairs(mode)
        return lin + att


def _img_txt(img: int, txt: int):
    return (("img", img), ("txt", txt))


TINY = Workload(
    name="tiny_1layer_f32", dtype="f32", batch=1, seq_len=64, d_model=256,
    n_heads=4, n_kv_heads=4, head_dim=64, d_ff=688, block_size=16, top_k=2,
    mode="gated", segments=_img_txt(48, 16), img_scale=1.0, index=0)

L7B_1K = Workload(
    name="7b_layer_1k", dtype="bf16", batch=1, seq_len=1024, d_model=4096,
    n_heads=32, n_kv_heads=32, head_dim=128, d_ff=11008, block_size=64, top_k=8,
    mode="gated", segments=_img_txt(576, 448), index=1)

L7B_4K_B4 = Workload(
    name="7b_layer_4k_b4", dtype="bf16", batch=4, seq_len=4096, d_model=4096,
    n_heads=32, n_kv_heads=32, head_dim=128, d_ff=11008, block_size=64, top_k=16,
    mode="gated", segments=_img_txt(576, 448) * 4, index=2)

STACK_DECODE = Workload(
    name="7b_stack32_prefill2k_decode256_b8", dtype="bf16", batch=8, seq_len=2048,
    d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128, d_ff=11008,
    block_size=64, top_k=16, mode="dense", segments=_img_txt(576, 1472),
    n_layers=32, vocab=32000, decode_steps=256, page_size=16, index=3)

GQA_16K = Workload(
    name="gqa28x4_layer_16k", dtype="bf16", batch=1, seq_len=16384, d_model=3584,
    n_heads=28, n_kv_heads=4, head_dim=128, d_ff=18944, block_size=64, top_k=32,
    mode="gated", segments=(("img", 64 * 248), ("txt", 512)), index=4)

# Long-context decode (the paper's measured regime): one 7B-shape layer's
# SAS decode step at contexts of 64K..512K tokens (seq_len = the context),
# the paper's default budget K = 32 blocks of 64; cache contents synthetic.
LONG_DECODE = Workload(
    name="7b_layer_decode_64k_512k", dtype="bf16", batch=8, seq_len=524288,
    d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128, d_ff=11008,
    block_size=64, top_k=32, mode="sparse", segments=(("txt", 524288),),
    page_size=16, index=5)

WORKLOADS = (TINY, L7B_1K, L7B_4K_B4, STACK_DECODE, GQA_16K, LONG_DECODE)
BY_NAME = {w.name: w for w in WORKLOADS}
