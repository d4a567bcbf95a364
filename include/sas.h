/*
 * sas.h -- C ABI of the SAS (Simple Attention Sparsification) hot path for
 * AMD MI355X (gfx950).
 *
 * SAS (arXiv 2609.13141) splits the keys/values of every query into blocks of
 * B tokens (Sec. 3, Eq. selected_context).  The block holding the query is
 * the current block B_0 and is always attended with unit gate (Sec. 4.1).  A
 * selector scores the earlier ("historical") blocks, the scores become
 * normalized log gates log g = s - LSE(s) (Eq. normalized_log_gate), and the
 * Top-K historical blocks are kept.  Training-time attention adds log g to
 * the logits of the kept blocks (Eq. ours_train, Alg. 1); inference attends
 * to the kept blocks without the gate (Alg. 2).  The paper's serving
 * pipeline prefills densely and decodes block-sparsely (Sec. 5.1).
 *
 * Selector (the paper names one but does not define its architecture; this
 * library's reading, shared with the fp64 oracle): block summary = mean of the
 * block's post-RoPE keys, gate query = sum of the group's query heads, both
 * optionally projected by per-group [dh, dh] matrices, score = exact dot
 * product (fp64) scaled by 1/(G*sqrt(dh)).  Top-K ranks the exact score,
 * ties to the lower block index, so selected indices are exact integers.
 *
 * Conventions shared by every entry point:
 *  - All tensor pointers are caller-owned DEVICE memory, row-major and
 *    contiguous, 16-byte aligned; nothing is allocated by the library.
 *    Scratch memory comes from `ws` (size from sas_workspace_size).
 *  - Activations and weights share one dtype (SAS_F32 or SAS_BF16 storage);
 *    statistics are fp32, indices int32.  Accumulation is fp32; selector
 *    arithmetic is fp64.
 *  - Linear weights use the nn.Linear layout [out, in]; no biases.  Query
 *    head h reads KV head h / G with G = n_heads / n_kv_heads.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = default
 *    stream).  SAS_OK means "enqueued"; device faults surface at the
 *    caller's next synchronisation.
 *  - On any error nothing is enqueued, outputs are untouched and
 *    sas_last_error() returns a message (thread-local).
 *  - Optional outputs may be NULL; their writes are skipped.
 */
#ifndef SAS_H
#define SAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SAS_OK = 0,
  SAS_ERR_INVALID_ARGUMENT = -1, /* bad pointer, shape or config */
  SAS_ERR_UNSUPPORTED = -2,      /* valid but not implemented (e.g. head_dim 96) */
  SAS_ERR_WORKSPACE = -3,        /* ws NULL or smaller than sas_workspace_size */
  SAS_ERR_HIP = -4               /* a HIP launch or runtime call failed */
} sas_status;

typedef enum { SAS_F32 = 0, SAS_BF16 = 1 } sas_dtype;

/* Attention of the prefill entry points.
 *  DENSE : causal softmax attention over all earlier tokens (Eq. fula).
 *  SPARSE: current block + the Top-K historical blocks, no bias (Alg. 2).
 *  GATED : same set; every token of a kept historical block m carries the
 *          bias log g_m, the current block carries 0 (Eq. ours_train). */
typedef enum { SAS_MODE_DENSE = 0, SAS_MODE_SPARSE = 1, SAS_MODE_GATED = 2 } sas_mode;

/* Gating formulations of the training ablation (Sec. 4.1, Table 1); they
 * apply to GATED mode only and default to SAS's choices (all zero).
 *  gate_pos:  INNER adds log g_m to the logits (Eq. ours_train); OUTER keeps
 *             the logits unbiased and weights the values of block m by g_m,
 *             o = sum_i p_i g_b(i) v_i.
 *  gate_act:  log g_m = s_m - LSE over the historical blocks (SOFTMAX,
 *             Eq. normalized_log_gate), log sigmoid(s_m) (SIGMOID) or s_m
 *             itself added to the logits (RAW).
 *  scope:     SPARSE attends the current block and the Top-K blocks; FULL
 *             attends every earlier token, each historical block with its gate.
 *  gate_ste:  1 = straight-through hard gate: the forward attends the current
 *             block and the Top-K blocks with unit gates; the backward passes
 *             the hard gate's gradient to the soft gate (for a block outside
 *             the Top-K, the limit of the inner-gate gradient at g -> 0,
 *             App. D.2), to the Top-K blocks (scope SPARSE) or to every
 *             historical block (scope FULL).
 * OUTER supports SOFTMAX and SIGMOID and no straight-through gate (RAW
 * defines no gate value); other combinations return SAS_ERR_UNSUPPORTED. */
typedef enum { SAS_GATE_INNER = 0, SAS_GATE_OUTER = 1 } sas_gate_pos;
typedef enum { SAS_ACT_SOFTMAX = 0, SAS_ACT_SIGMOID = 1, SAS_ACT_RAW = 2 } sas_gate_act;
typedef enum { SAS_SCOPE_SPARSE = 0, SAS_SCOPE_FULL = 1 } sas_scope;

/* Operation codes for sas_workspace_size. */
typedef enum {
  SAS_OP_ATTENTION = 0, /* sas_attention_prefill: batch, seq_len */
  SAS_OP_MLP = 1,       /* sas_mlp_forward: batch = tokens, seq_len ignored */
  SAS_OP_LAYER = 2,     /* sas_layer_forward: batch, seq_len */
  SAS_OP_DECODE = 3,    /* sas_decode_step: batch, seq_len = max context (tokens) */
  SAS_OP_LM_HEAD = 4,   /* sas_lm_head_argmax: batch, seq_len = vocab */
  SAS_OP_DECODE_SELECT = 5, /* sas_decode_select: batch, seq_len = max context (tokens) */
  SAS_OP_ATTENTION_BACKWARD = 6, /* sas_attention_backward: batch, seq_len */
  SAS_OP_SELECTOR_BACKWARD = 7,  /* sas_selector_backward: batch, seq_len */
  SAS_OP_SELECTION_STATS = 8     /* sas_selection_stats: batch, seq_len */
} sas_op;

typedef struct {
  int32_t d_model;
  int32_t n_heads;
  int32_t n_kv_heads;  /* n_heads % n_kv_heads == 0 */
  int32_t head_dim;    /* 64 or 128 */
  int32_t d_ff;
  int32_t block_size;  /* B, tokens per SAS block: 16, 32, 64 or 128 */
  int32_t top_k;       /* K, historical blocks kept per query, 0..32 */
  float rope_base;     /* rotary base (rotate-half pairing i, i + head_dim/2) */
  float rms_eps;       /* RMSNorm epsilon */
  float sm_scale;      /* attention scale; <= 0 selects 1/sqrt(head_dim) */
  int32_t dtype;       /* sas_dtype */
  int32_t mode;        /* sas_mode (prefill only; decode always uses SPARSE) */
  int32_t gate_pos;    /* sas_gate_pos (GATED only) */
  int32_t gate_act;    /* sas_gate_act (GATED only) */
  int32_t scope;       /* sas_scope (GATED only) */
  int32_t gate_ste;    /* 0 or 1 (GATED only) */
} sas_config;

/* Attention inputs (post-RoPE), the paper's problem statement (Alg. 1/2):
 * q [b, n, H, dh], k and v [b, n, Hkv, dh]; optional selector projections
 * w_gq, w_gk [Hkv, dh, dh] ([out, in] per group; NULL = identity);
 * score_noise [b, Hkv, n, ceil(n/B)] fp32 or NULL: added to the selector
 * scores s before the gate activation and before Top-K (the noisy "full*"
 * scope of Table 1); with noise the Top-K ranks s + noise (s evaluated in
 * fp64 as r / (G sqrt(dh))), without it the raw scores r.
 * doc_first_block [b, ceil(n/B)] int32 or NULL: variable-length packing of
 * several documents into one row.  Entry m is the first block of the
 * document that block m belongs to (non-decreasing, <= m).  Documents start
 * on block boundaries (every document but a row's last is a whole number of
 * blocks long).  A query's context, historical blocks, selection and
 * normalizer are those of its own document; NULL = one document per row.
 * The table is not checked (it is device memory): entries outside [0, m]
 * are clamped into it, and a table that breaks the rules above gives
 * unspecified (but in-bounds) results. */
typedef struct {
  const void* q;
  const void* k;
  const void* v;
  const void* w_gq;
  const void* w_gk;
  const float* score_noise;
  const int32_t* doc_first_block;
} sas_attn_in;

/* Attention outputs.  NB = ceil(n / B).
 *  o         [b, n, H, dh]   attention output (activation dtype)
 *  lse       [b, H, n]       fp32 natural-log sum of exp of the scaled
 *                            logits (with the inner gate's bias) over the
 *                            attended set (optional)
 *  k_summary [b, Hkv, NB, dh] selector key summary of every complete block
 *                            (after w_gk); incomplete-block rows are zero
 *                            (optional)
 *  sel_idx   [b, Hkv, n, K]  int32 kept historical blocks, ascending, -1
 *                            padded (optional)
 *  log_gate  [b, Hkv, n, NB] fp32 log g of every historical block of every
 *                            query (per cfg->gate_act), -inf where
 *                            m >= floor(t / B) (optional)
 *  tau       [b, Hkv, n]     fp32 log gate of the lowest-ranked kept block
 *                            when floor(t/B) > K >= 1, +inf when K = 0 <
 *                            floor(t/B), -inf otherwise (optional)
 * The selector outputs are produced in every mode when requested; in DENSE
 * mode they do not influence attention. */
typedef struct {
  void* o;
  float* lse;
  void* k_summary;
  int32_t* sel_idx;
  float* log_gate;
  float* tau;
} sas_attn_out;

/* Decoder-layer weights (activation dtype).  rms1/rms2 [d]; wq [H*dh, d];
 * wk, wv [Hkv*dh, d]; wo [d, H*dh]; w_gate, w_up [d_ff, d]; w_down [d, d_ff];
 * w_gq, w_gk [Hkv, dh, dh] or NULL.  decode_packed: NULL, or the same
 * layer's linear weights repacked by sas_pack_decode_weights, which the
 * decode step then streams instead of wq..w_down (same results, bit for
 * bit); the other entry points ignore it. */
typedef struct {
  const void* rms1;
  const void* wq;
  const void* wk;
  const void* wv;
  const void* wo;
  const void* rms2;
  const void* w_gate;
  const void* w_up;
  const void* w_down;
  const void* w_gq;
  const void* w_gk;
  const void* decode_packed;
} sas_layer_weights;

/* Optional intermediate taps of sas_layer_forward (any field may be NULL):
 * q [b,n,H,dh], k, v [b,n,Hkv,dh] after RoPE, h1 = x + attention [b,n,d]. */
typedef struct {
  void* q;
  void* k;
  void* v;
  void* h1;
} sas_layer_taps;

/* Paged KV cache of one layer (Sec. 5.1's serving setting).
 *  k_pages, v_pages [num_pages, Hkv, page_size, dh] (activation dtype)
 *  block_table      [b, max_pages_per_seq] int32 page ids; logical
 *                   position p of sequence i lives in page
 *                   block_table[i][p / page_size], slot p % page_size
 *  k_summary        [b, Hkv, max_blocks, dh] selector key summaries of the
 *                   complete SAS blocks (after w_gk)
 *  block_size must be a multiple of page_size.  A page id outside
 *  [0, num_pages) (e.g. -1) marks an unmapped page: writes to its positions
 *  are dropped, they add zero to their block's summary, and the decode
 *  attention leaves their keys out (as if the selection had not kept them). */
typedef struct {
  void* k_pages;
  void* v_pages;
  const int32_t* block_table;
  void* k_summary;
  int32_t num_pages;
  int32_t page_size;
  int32_t max_pages_per_seq;
  int32_t max_blocks;
} sas_paged_kv;

/* Bytes of scratch memory an entry point needs (0 on invalid config). */
size_t sas_workspace_size(const sas_config* cfg, int32_t op, int32_t batch, int32_t seq_len);

/* Selector + SAS attention over given Q/K/V (the scoring, Top-K, gating
 * and attention steps of Alg. 1 / Alg. 2 applied to every query of a causal
 * prefill; App. E forward).
 * batch >= 1, seq_len >= 1. out->o is required. */
sas_status sas_attention_prefill(const sas_config* cfg, int32_t batch, int32_t seq_len,
                                 const sas_attn_in* in, sas_attn_out* out,
                                 void* ws, size_t ws_bytes, void* stream);

/* Inputs of sas_attention_backward: the forward's inputs and outputs.
 *  q [b,n,H,dh], k, v [b,n,Hkv,dh], o [b,n,H,dh] (sas_attention_prefill's
 *  output), d_o [b,n,H,dh] the upstream gradient (activation dtype);
 *  lse [b,H,n] fp32 (the forward's LSE); sel_idx [b,Hkv,n,K] and, in GATED
 *  mode, log_gate [b,Hkv,n,ceil(n/B)] fp32 (the forward's selection and
 *  log gates; unused in DENSE mode).  cfg must be the forward's, gating
 *  fields included. */
typedef struct {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const void* d_o;
  const float* lse;
  const int32_t* sel_idx;
  const float* log_gate;
  const int32_t* doc_first_block;  /* the forward's packing table or NULL */
} sas_bwd_in;

/* Outputs of sas_attention_backward: dq [b,n,H,dh], dk, dv [b,n,Hkv,dh]
 * (activation dtype), dlog_gate [b,Hkv,n,K] fp32 or NULL: the gradient of
 * each selected block's log gate (GATED), summed over the group's heads, at
 * the slots of sel_idx (0 in empty slots; scope SPARSE only);
 * dlog_gate_full [b,Hkv,n,ceil(n/B)] fp32 or NULL: the same gradient for
 * every block (0 where a block receives none), required in GATED mode with
 * scope FULL or the straight-through gate.  With the straight-through gate
 * the value is g_m times the gradient of the hard gate (the gradient of log g
 * under the straight-through rule). */
typedef struct {
  void* dq;
  void* dk;
  void* dv;
  float* dlog_gate;
  float* dlog_gate_full;
} sas_bwd_out;

/* Backward of the attention of sas_attention_prefill (Sec. 4.3, Eq.
 * ours_train; App. E's recomputation backward), the kernel of the training
 * step of Alg. 1: recomputes the attended sets and probabilities from the
 * forward's LSE and selection and writes dQ, dK, dV and the block log-gate
 * gradient dlog g_m = sum over the group's heads and the block's keys of
 * p_i (dO.v_i - dO.o) (the inner-gate gradient of Eq. gate_posi, for log g).
 * cfg->mode must be the forward's.  ws: sas_workspace_size(cfg,
 * SAS_OP_ATTENTION_BACKWARD, batch, seq_len). */
sas_status sas_attention_backward(const sas_config* cfg, int32_t batch, int32_t seq_len,
                                  const sas_bwd_in* in, sas_bwd_out* out,
                                  void* ws, size_t ws_bytes, void* stream);

/* Inputs of sas_selector_backward.  q [b,n,H,dh], k [b,n,Hkv,dh] (the
 * forward's post-RoPE queries and keys, activation dtype); w_gq, w_gk
 * [Hkv,dh,dh] or NULL (the selector's optional projections, as given to the
 * forward); sel_idx [b,Hkv,n,K] and log_gate [b,Hkv,n,ceil(n/B)] fp32 (the
 * forward's selection and normalized log gates); dlog_gate [b,Hkv,n,K] fp32
 * (sas_attention_backward's output, or any gradient of the selected blocks'
 * log gates at the slots of sel_idx); dlog_gate_full [b,Hkv,n,ceil(n/B)]
 * fp32 or NULL: when given, the gradient of every block's log gate, used
 * instead of sel_idx and dlog_gate (scope FULL, straight-through gate). */
typedef struct {
  const void* q;
  const void* k;
  const void* w_gq;
  const void* w_gk;
  const int32_t* sel_idx;
  const float* log_gate;
  const float* dlog_gate;
  const float* dlog_gate_full;
  const int32_t* doc_first_block;  /* the forward's packing table or NULL */
} sas_sel_bwd_in;

/* Outputs of sas_selector_backward, all fp32, each optional except as noted:
 *  ds [b,Hkv,n,ceil(n/B)]: gradient of the selector scores s (0 for blocks
 *    that are not historical for the row);
 *  dqhat [b,Hkv,n,dh]: gradient of the (projected) gate queries;
 *  dkbar [b,Hkv,ceil(n/B),dh]: gradient of the (projected) block summaries
 *    (0 for an incomplete last block);
 *  dw_gq, dw_gk [Hkv,dh,dh]: gradients of the projections, summed over the
 *    batch; required when the projection is given, ignored otherwise. */
typedef struct {
  float* ds;
  float* dqhat;
  float* dkbar;
  float* dw_gq;
  float* dw_gk;
} sas_sel_bwd_out;

/* Backward of the selector (Alg. 1's update of the selector parameters):
 * dlog g -> ds through the gate activation: for SOFTMAX, Eq.
 * normalized_log_gate's ds_m = dlog g_m - g_m sum over the row's historical
 * blocks of dlog g (the softmax backward of App. D.3); for SIGMOID
 * ds_m = dlog g_m (1 - g_m); for RAW ds_m = dlog g_m; then
 * through the scores s = qhat.kbar / (G sqrt(dh)) to the gate queries and
 * summaries and, when given, to W_gq and W_gk.  The Top-K set is piecewise
 * constant and passes no gradient; the roundings of the forward are taken
 * as identities.  Gate queries and summaries are recomputed from q and k.
 * With top_k = 0 and no dlog_gate_full every output is zero.  Score noise
 * (sas_attn_in.score_noise) is additive and needs no input here: log_gate
 * already holds the noisy gates.  ws: sas_workspace_size(cfg,
 * SAS_OP_SELECTOR_BACKWARD, batch, seq_len). */
sas_status sas_selector_backward(const sas_config* cfg, int32_t batch, int32_t seq_len,
                                 const sas_sel_bwd_in* in, sas_sel_bwd_out* out,
                                 void* ws, size_t ws_bytes, void* stream);

/* Inputs of sas_selection_stats: one layer's post-RoPE q [b,n,H,dh], k and
 * v [b,n,Hkv,dh] (activation dtype) and its selection sel_idx [b,Hkv,n,K]
 * (as sas_attention_prefill writes it; unused in DENSE mode). */
typedef struct {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* sel_idx;
  const int32_t* doc_first_block;  /* packing table (as in sas_attn_in) or NULL */
} sas_stats_in;

/* Outputs of sas_selection_stats, each optional.  W = ceil(ceil(n/B)/32).
 *  cov, cov_v [b,H,n] fp32: Eq. mass_coverage of the query's attended set
 *    (current block + selected blocks) over its causal context, with
 *    w_i = exp(z_i) and w_i = exp(z_i + log||v_i||_2), z_i = sm q.k_i
 *    (unbiased logits);
 *  sel_union [b,Hkv,n,W] uint32: bit m of word m/32 is OR-ed in for every
 *    selected block (the union over the layers it is called for);
 *  ref_union [b,Hkv,n,W] uint32: the same for the full-attention reference
 *    set: per head the top_k historical blocks by attention mass (ties to
 *    the lower block), per KV group the blocks picked by more than half of
 *    the group's heads (Sec. 6.1's majority vote).
 * The unions accumulate: clear them before the first layer. */
typedef struct {
  float* cov;
  float* cov_v;
  uint32_t* sel_union;
  uint32_t* ref_union;
} sas_stats_out;

/* Selection-analysis statistics of one layer (Sec. 6.1, Eq. mass_coverage
 * and the per-layer sets of Eq. overlap_recall).  A dense causal pass over
 * Q K^T (no values are multiplied).  ws: sas_workspace_size(cfg,
 * SAS_OP_SELECTION_STATS, batch, seq_len). */
sas_status sas_selection_stats(const sas_config* cfg, int32_t batch, int32_t seq_len,
                               const sas_stats_in* in, sas_stats_out* out,
                               void* ws, size_t ws_bytes, void* stream);

/* Eq. overlap_recall's counts over two accumulated bitmasks of `words`
 * uint32 words (DEVICE): counts[0] = |sel & ref|, counts[1] = |ref|
 * (uint64, DEVICE, overwritten); Recall = counts[0] / counts[1]. */
sas_status sas_overlap_recall(int64_t words, const uint32_t* sel_union, const uint32_t* ref_union,
                              uint64_t* counts, void* stream);

/* y = x + SwiGLU(RMSNorm(x)) for `tokens` rows of width d_model:
 * u = RMSNorm(x) * rms2; a = silu(u W_gate^T) * (u W_up^T); y = x + a W_down^T.
 * SAS defines nothing on the MLP; it is the layer's dense remainder. */
sas_status sas_mlp_forward(const sas_config* cfg, int32_t tokens, const void* x,
                           const sas_layer_weights* w, void* y,
                           void* ws, size_t ws_bytes, void* stream);

/* One pre-norm decoder layer over x [b, n, d] -> y [b, n, d]:
 * u1 = RMSNorm(x); Q,K,V = RoPE(u1 W^T); SAS attention (cfg->mode);
 * h1 = x + O W_o^T; y = h1 + SwiGLU(RMSNorm(h1)).
 * stats: optional attention outputs (o, lse, selector outputs); taps:
 * optional intermediates; cache: when non-NULL, K/V of positions 0..n-1 are
 * written to the pages of every sequence and the summaries of the complete
 * blocks to cache->k_summary (the dense-prefill half of Sec. 5.1). */
sas_status sas_layer_forward(const sas_config* cfg, int32_t batch, int32_t seq_len,
                             const void* x, const sas_layer_weights* w, void* y,
                             sas_attn_out* stats, sas_layer_taps* taps,
                             sas_paged_kv* cache, void* ws, size_t ws_bytes, void* stream);

/* One SAS decode step of one layer (Alg. 2) for `batch` sequences:
 * x [b, d] is the new token's hidden state at position pos[i] (DEVICE int32
 * array; the cache must hold positions 0..pos[i]-1 and have room for
 * pos[i]).  Appends K/V at pos[i]; when pos[i]+1 is a multiple of B the
 * block's summary is written; scores the summaries of the floor(pos/B)
 * complete blocks, keeps the Top-K per KV group and attends to them plus the
 * current block without gate bias.  y [b, d]; sel_idx [b, Hkv, K] optional.
 * taps (optional, any field NULL): the step's post-RoPE q [b, H, dh], k, v
 * [b, Hkv, dh] and h1 = x + attention [b, d].
 * Positions outside the cache are skipped by the kernels (no write). */
sas_status sas_decode_step(const sas_config* cfg, int32_t batch, const void* x,
                           const int32_t* pos, const sas_layer_weights* w,
                           sas_paged_kv* cache, void* y, int32_t* sel_idx,
                           sas_layer_taps* taps, void* ws, size_t ws_bytes, void* stream);

/* Decode weight layout (bf16 only; the memory layout of the paper's
 * decode, Alg. 2, is not specified -- this one serves the decode step's
 * weight-streaming products).  Each of the layer's four products (QKV,
 * O-projection, gate/up, down) is stored as blocks of 16 output columns x 32
 * input elements, one contiguous 1-KB block per (column group, 32-wide k
 * step), groups in order, steps ascending, so that every load instruction of
 * the decode GEMV reads 1 KB of consecutive bytes.  The column groups are
 * those of the decode step's epilogues (QKV: 8 rotary pairs; gate/up: 8 gate
 * and the matching 8 up rows; O and down: 16 rows).
 * sas_decode_packed_bytes: bytes of one layer's packed copy (0 if the
 * configuration has none: fp32, or d, H*dh or d_ff not a multiple of 128).
 * sas_pack_decode_weights: writes it from w (wq..w_down, DEVICE) into packed
 * (DEVICE, caller-owned, 256-byte aligned, at least that many bytes),
 * asynchronously on `stream`; w->decode_packed is not read. */
size_t sas_decode_packed_bytes(const sas_config* cfg);
sas_status sas_pack_decode_weights(const sas_config* cfg, const sas_layer_weights* w, void* packed,
                                   size_t packed_bytes, void* stream);

/* Scratch bytes of sas_decode_step_noalloc (one static copy per GPU). */
#define SAS_DECODE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

/* sas_decode_step for callers that cannot allocate device memory or pass a
 * workspace: code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation.  Same arguments, kernels and results as
 * sas_decode_step (without taps); the scratch is a static device array of
 * SAS_DECODE_NOALLOC_SCRATCH_BYTES per GPU, looked up on the first call on
 * each device and held until the process ends.  A call whose workspace
 * (sas_workspace_size(cfg, SAS_OP_DECODE, batch, max_blocks * B)) exceeds it
 * returns SAS_ERR_WORKSPACE before touching the GPU (32 MiB covers batch 8 of
 * the 7B shape up to 512K tokens of context).  The step needs nothing in the
 * scratch to start at zero, and nothing is allocated or freed.  Every call
 * on one GPU shares that GPU's scratch: calls that may overlap on one GPU
 * (other streams, other threads) race and must be serialised by the caller. */
sas_status sas_decode_step_noalloc(const sas_config* cfg, int32_t batch, const void* x,
                                   const int32_t* pos, const sas_layer_weights* w,
                                   sas_paged_kv* cache, void* y, int32_t* sel_idx, void* stream);

/* The selection of a decode step alone (Alg. 2's Top-K over the block
 * summaries; Sec. 5.1), for long contexts where it dominates the step:
 * q [b, H, dh] holds the post-RoPE query heads of the new tokens (activation
 * dtype, DEVICE), pos [b] their positions (DEVICE int32).  Each KV group's
 * gate query (its heads summed, then w_gq [Hkv, dh, dh] when not NULL) is
 * scored against the cache's summaries of the floor(pos/B) complete blocks
 * (exact fp64 dot products) and the Top-K (score descending, lower block
 * first on ties) is written to sel_idx [b, Hkv, K], ascending, -1 padded.
 * Only cache->k_summary and cache->max_blocks (<= 8192, i.e. 512K tokens at
 * B = 64) are read; nothing is appended.  Caches of more than 256 blocks
 * need sas_workspace_size(cfg, SAS_OP_DECODE_SELECT, batch, max context)
 * bytes of ws (b * Hkv * max_blocks doubles); sas_decode_step takes the
 * same path and needs the same room beyond its other scratch. */
sas_status sas_decode_select(const sas_config* cfg, int32_t batch, const void* q,
                             const int32_t* pos, const void* w_gq,
                             const sas_paged_kv* cache, int32_t* sel_idx,
                             void* ws, size_t ws_bytes, void* stream);

/* Token embedding for the model ends: x [b, n, d] = table[ids] for ids >= 0;
 * an id < 0 marks an image slot, filled with the next row of
 * img_embed [b, n_img, d] (n_img = number of negative ids in each row;
 * img_embed may be NULL only when there are none). ids is DEVICE memory. */
sas_status sas_embed(const sas_config* cfg, int32_t batch, int32_t seq_len, const int32_t* ids,
                     const void* table, int32_t vocab, const void* img_embed, int32_t n_img,
                     void* x, void* stream);

/* Greedy next token: logits = RMSNorm(h) W_lm^T (fp32 accumulation),
 * tokens[i] = argmax, lowest id on ties.  h [b, d]; gamma [d];
 * w_lm [vocab, d]; logits [b, vocab] fp32 optional; tokens [b] int32. */
sas_status sas_lm_head_argmax(const sas_config* cfg, int32_t batch, const void* h,
                              const void* gamma, const void* w_lm, int32_t vocab,
                              float* logits, int32_t* tokens,
                              void* ws, size_t ws_bytes, void* stream);

/* Message describing the last non-OK status on this thread ("" if none). */
const char* sas_last_error(void);

/* Library version string. */
const char* sas_version(void);

/* Kernel timing for measurement tools (not needed by the compute path).
 * sas_profiler_start(capacity): every kernel launched afterwards by this
 * library (up to `capacity` launches, on any stream) is bracketed by a pair
 * of hipEvents recorded on its stream.  sas_profiler_stop() ends recording
 * and returns the number of launches recorded.  After the caller has
 * synchronised the streams, sas_profiler_record(i, &name, &ms) returns the
 * kernel family name ("gemm_gate_up", "attention", ...) and the elapsed
 * milliseconds of launch i.  Not thread-safe; the events are reused by the
 * next sas_profiler_start (created anew only when it asks for more). */
int32_t sas_profiler_start(int32_t capacity);
/* Restrict recording to the named kernel families (comma-separated, e.g.
 * "gemm_gate_up,dec_gate_up"); NULL records every family, "" none.  Applies
 * to the launches after the call, until the next call. */
int32_t sas_profiler_select(const char* families);
int32_t sas_profiler_stop(void);
int32_t sas_profiler_record(int32_t i, const char** name, float* ms);

#ifdef __cplusplus
}
#endif
#endif /* SAS_H */
