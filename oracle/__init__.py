"""Plain, slow fp64 CPU oracle of the SAS hot path.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import or run anything here; the product path (the HIP
library and its binding) never does, and this package imports nothing from
the product package.  Every function computes the paper's definitions
directly in float64 NumPy, rounding to the activation dtype only where the
GPU path materialises a tensor in HBM.

Sections and equations cited are those of the SAS paper (arXiv 2609.13141):
standard attention (Eq. fula), block-sparse attention (Eq. spa), the Top-K
block selection (Eq. selected_context), the normalized log gate
(Eq. normalized_log_gate, Sec. 4.2.2), SAS attention (Eq. ours_train,
Sec. 4.3), and the training/inference steps (Alg. 1, Alg. 2).

Parity status of each part (how it is pinned by the oracle self-tests):

* rounding ``rho``: pinned against torch's float32 -> bfloat16 conversion and
  hand-derived ties (a direct fp64 -> bf16 rounding, not via float32).
* RMSNorm, SiLU: pinned against torch.nn.functional.rms_norm / silu.
* RoPE: pinned by invariants (pair norms, identity at position 0, scores
  depending only on the relative position).
* selector (block summaries, gate query, scores): the paper names the
  selector but does not define its architecture; its arithmetic is pinned by
  exact rational brute force and planted rankings.  The architecture itself
  is "parity unpinned" by the paper (it is this implementation's reading).
* attention backward, gate backward, selector backward: pinned against
  torch autograd on a dense masked formulation and by central finite
  differences of the fp64 forward.
* gating formulations of Table 1 (inner/outer gate, softmax/sigmoid/raw
  activation, sparse/full scope, straight-through hard gate, score noise):
  pinned against torch autograd on dense masked formulations (the hard gate
  in its multiplicative form with zero gates), torch's log_softmax and
  logsigmoid, Top-K ordering properties and reductions to the plain modes.
* selection statistics (mass coverage, full-attention reference sets with
  the group majority vote, overlap recall): pinned against torch softmax
  masses and torch.topk, closed forms (q = 0, every block kept, equal value
  norms) and hand-worked votes and recalls.
* packed documents (varlen): a one-document table reproduces the unpacked
  oracle; packed rows match torch autograd on a dense masked formulation with
  a block-diagonal document mask; documents are independent.
* normalized log gate, Top-K, attention: pinned by closed forms (q = 0),
  V = const, reductions to textbook causal / block-local attention computed
  by torch's scaled_dot_product_attention, causality, shift invariance and
  the soft-reweighting identity of Eq. rank_unbounded.
"""
from .numerics import rho, round_bf16, round_f32, rmsnorm, rope, silu
from .selector import (block_summaries, gate_query, selector_scores,
                       normalized_log_gate, topk_blocks, select)
from .attention import causal_attention, sas_attention
from .backward import sas_attention_backward, gate_backward, selector_backward
from .variants import (log_gates, select_variant, variant_attention, variant_attention_backward,
                       gate_backward_act)
from .stats import mass_coverage, block_mass_topk, majority_vote, selection_sets, overlap_recall
from .varlen import doc_spans, select_packed, attention_packed, backward_packed, coverage_packed
from .layer import (Spec, layer_forward, mlp_forward, attention_prefill, dense_prefill_layer,
                    DecodeCache, decode_step, decode_select, embed_tokens, lm_head_argmax)

__all__ = [
    "rho", "round_bf16", "round_f32", "rmsnorm", "rope", "silu",
    "block_summaries", "gate_query", "selector_scores", "normalized_log_gate",
    "topk_blocks", "select", "sas_attention", "causal_attention", "Spec", "layer_forward",
    "dense_prefill_layer",
    "mlp_forward", "attention_prefill", "DecodeCache", "decode_step",
    "decode_select", "embed_tokens", "lm_head_argmax",
    "sas_attention_backward", "gate_backward", "selector_backward",
    "log_gates", "select_variant", "variant_attention", "variant_attention_backward",
    "gate_backward_act", "mass_coverage", "block_mass_topk", "majority_vote", "selection_sets",
    "overlap_recall", "doc_spans", "select_packed", "attention_packed", "backward_packed", "coverage_packed",
]
