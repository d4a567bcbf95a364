// Host-side launchers of the SAS kernels (one translation unit each).
// Every launcher enqueues on `stream` and returns hipGetLastError().
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sas {

// Kernel-exact timing for the profiler: when `start` is set, the next launch
// made through launch_ext records these events at the kernel's own start and
// end (so the interval excludes the dispatch latency that a pair of stream
// events around the launch includes) and clears them.  Launches of
// multi-kernel calls leave them unset.
struct LaunchEvents {
  hipEvent_t start, stop;
  int taken;  // set by the launch that recorded them
};
extern LaunchEvents g_launch_events;

template <typename... KArgs, typename... Args>
inline hipError_t launch_ext(void (*kern)(KArgs...), dim3 grid, dim3 block, uint32_t shm, hipStream_t s,
                             Args... args) {
  if (g_launch_events.start) {
    const LaunchEvents e = g_launch_events;
    g_launch_events = LaunchEvents{nullptr, nullptr, 1};
    hipExtLaunchKernelGGL(kern, grid, block, shm, s, e.start, e.stop, 0, args...);
  } else {
    hipLaunchKernelGGL(kern, grid, block, shm, s, args...);
  }
  return hipGetLastError();
}


inline int cdiv(int a, int b) { return (a + b - 1) / b; }
inline size_t cdiv(size_t a, int b) { return (a + (size_t)b - 1) / (size_t)b; }
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Records the thread's last-error message (returned by sas_last_error) and
// returns `status`; defined with the C ABI's entry points.
int set_error(int status, const char* fmt, ...);

// ---- elementwise.hip -------------------------------------------------------
// out[r, :] = x[r, :] / sqrt(mean(x[r, :]^2) + eps) * gamma   (fp32 math)
hipError_t launch_rmsnorm(int dtype, const void* x, const void* gamma, void* out, int rows, int d,
                          float eps, hipStream_t s);
// RMSNorm and, in the same launch, the rotary table rows [0, rope_rows) for the
// positions pos[row] (the row index when pos is NULL): rope [rope_rows, dh/2]
// float2, (cos, sin) of pos * base^(-2i/dh) evaluated in fp64; rope == NULL: norm only.
hipError_t launch_rmsnorm_rope(int dtype, const void* x, const void* gamma, void* out, int rows, int d, float eps,
                               const int32_t* pos, float2* rope, int dh, float base, int rope_rows,
                               hipStream_t s);

// ---- gemm.hip --------------------------------------------------------------
// C = A[M, K] * B[N, K]^T with one of three fused epilogues.
enum GemmEpi { EPI_QKV_ROPE = 0, EPI_SWIGLU = 1, EPI_RESID = 2, EPI_F32OUT = 3 };
struct GemmArgs {
  int epi;
  int M, K;
  const void* A;          // [M, K]
  // EPI_RESID: B0 = W [N, K]; out[M, N] = resid + A W^T
  // EPI_SWIGLU: B0 = W_gate, B1 = W_up [F, K]; out[M, F] = silu(A Wg^T) * (A Wu^T)
  // EPI_QKV_ROPE: B0 = Wq [H*dh, K], B1 = Wk, B2 = Wv [Hkv*dh, K];
  //   out = Q [M, H, dh], out1 = K, out2 = V [M, Hkv, dh]; RoPE on Q and K at
  //   position (row % seq_len) from rope table [seq_len, dh/2] float2.
  const void* B0;
  const void* B1;
  const void* B2;
  int N;                  // RESID: N; SWIGLU: F; QKV: (H + 2 Hkv) * dh
  const void* resid;      // RESID
  void* out;
  void* out1;
  void* out2;
  int n_heads, n_kv_heads, head_dim, seq_len;
  const float2* rope;
  const int32_t* row_pos; // optional per-row positions (decode), else row % seq_len
  // decode (launch_gemv, EPI_QKV_ROPE): `append` (optional, with row_pos the
  // rows' positions) also writes K/V into the paged cache and completes block
  // summaries
  const struct DecodeArgs* append;
  // decode (launch_gemv): the product's weights in the packed decode layout, or NULL
  const void* packed;
  // prefill (launch_gemm, EPI_QKV_ROPE, row_pos NULL): also write the K/V rows
  // into the paged cache, row r being position r % seq_len of sequence
  // r / seq_len (only where gemm_fills_cache holds), or NULL
  const struct DecodeArgs* prefill_cache;
};
hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t s);
// Does launch_gemm write the K/V pages of `a.prefill_cache` itself (the bf16
// staged QKV epilogue)?  Otherwise the caller fills the cache.
bool gemm_fills_cache(int dtype, const GemmArgs& a);

// ---- gemv.hip --------------------------------------------------------------
// The same products for M <= 16 rows (bf16, K % 128 == 0), streaming the
// weights: rope is a per-row table [M, dh/2]; EPI_F32OUT writes fp32 A W^T.
hipError_t launch_gemv(const GemmArgs& a, hipStream_t s);
// The packed decode layout of a product (see sas_pack_decode_weights): its
// size in elements, and the kernel that writes it from the row-major B0..B2
// of `a` (epi, N, K as launch_gemv takes them).  With a.packed set,
// launch_gemv streams the packed copy instead.
size_t gemv_packed_elems(const GemmArgs& a);
hipError_t launch_gemv_pack(const GemmArgs& a, void* out, hipStream_t s);

// Variable-length packing: doc[b, NB] holds, for each block, the first block of
// its document; a query's historical blocks are [doc_first(t), t / B).  The
// entry is clamped to [0, t / B] so that no table can send an index out of range.
__device__ __forceinline__ int doc_first(const int32_t* doc, int bi, int NB, int t, int B) {
  return doc ? min(max(doc[(size_t)bi * NB + t / B], 0), t / B) : 0;
}

// ---- selector.hip ----------------------------------------------------------
// Block summaries kbar[b, Hkv, NB, dh] of the complete blocks of K[b, n, Hkv, dh]
// (mean, fp64 ascending sum, rounded once); incomplete rows zeroed.  When
// w_gk is given the projected summary is written to `ksum` and the plain one
// to `kplain` (scratch), otherwise `ksum` holds the plain summary.
hipError_t launch_block_summaries(int dtype, const void* K, int b, int n, int Hkv, int dh, int B,
                                  const void* w_gk, void* kplain, void* ksum, hipStream_t s);
// Gate queries qhat[b, Hkv, n, dh]: the group's query heads summed (fp64,
// ascending head index) and rounded once; projected by w_gq when given (the
// unprojected query then goes to `qplain`, scratch).
hipError_t launch_gate_query(int dtype, const void* Q, int b, int n, int H, int Hkv, int dh, const void* w_gq,
                             void* qplain, void* qhat, hipStream_t s);
// Per (b, group, query) selection (Top-K, gate, tau) against kbar.
struct SelectArgs {
  int b, n, H, Hkv, dh, B, K, NB;
  const void* Q;          // [b, n, H, dh]: gate query = rounded sum of the group's heads
  const void* qhat;       // [b, Hkv, n, dh] precomputed gate queries (projection) or null
  const void* kbar;       // [b, Hkv, NB, dh]
  int32_t* sel;           // [b, Hkv, n, K] (required, scratch or user)
  float* sel_bias;        // [b, Hkv, n, K] log g of each kept block (required)
  float* log_gate;        // [b, Hkv, n, NB] optional
  float* tau;             // [b, Hkv, n] optional
  const float* noise;     // [b, Hkv, n, NB] added to the scores (optional)
  int act;                // sas_gate_act
  float* row_lse;         // [b, Hkv, n] scratch (required with log_gate)
  const int32_t* doc;     // [b, NB] first block of each block's document, or null
};
hipError_t launch_select(int dtype, const SelectArgs& a, hipStream_t s);

// ---- attention.hip ---------------------------------------------------------
struct AttnArgs {
  int b, n, H, Hkv, dh, B, K, mode;
  float sm_scale;
  const void* Q;          // [b, n, H, dh]
  const void* Kt;         // [b, n, Hkv, dh]
  const void* V;          // [b, n, Hkv, dh]
  const int32_t* sel;     // [b, Hkv, n, K] (unused in DENSE)
  const float* sel_bias;  // [b, Hkv, n, K] (GATED)
  void* O;                // [b, n, H, dh]
  float* lse;             // [b, H, n] optional
  int outer;              // GATED: the gate weights the values instead of biasing the logits
  int full;               // GATED: every historical block attended, gates from gate_table
  const float* gate_table;  // [b, Hkv, n, NB] log gates (full scope)
  const int32_t* doc;     // [b, NB] first block of each block's document, or null
  uint32_t* queue;        // [ATTN_XCDS] job counters of the bf16 kernel's work queue (reset by the launch)
  // split query tiles (bf16, fewer jobs than resident workgroups): per job slot 128 rows of
  // unnormalized sums [slot, 128, dh] and (max, sum) [slot, 128, 2]; null: no splitting
  float* part_o;
  float* part_ml;
  long long part_slots;
  int split_tiles;        // set by the launch: key tiles per part (0: no split)
  // set by the launch, work-queue order: query-tile interleave of a (batch, kv head)
  // unit, units per locality group, units of the closing longest-first group
  int unit_parts, unit_group, tail_units;
};
hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s);
// longest sequence of the bf16 attention forward (key tiles of 64 tracked in LDS)
constexpr int ATTN_MAX_SEQ = 1 << 20;
// parts of a split query tile
constexpr int ATTN_MAX_SPLIT = 4;
// accelerator dies (XCDs, each with its own L2) the work queue is split over
constexpr int ATTN_XCDS = 8;

// ---- backward.hip ----------------------------------------------------------
struct BwdArgs {
  int b, n, H, Hkv, dh, B, K, mode;
  float sm_scale;
  const void* Q;          // [b, n, H, dh]
  const void* Kt;         // [b, n, Hkv, dh]
  const void* V;          // [b, n, Hkv, dh]
  const void* O;          // [b, n, H, dh] forward output
  const void* dO;         // [b, n, H, dh]
  const float* lse;       // [b, H, n] forward LSE (natural log)
  const int32_t* sel;     // [b, Hkv, n, K]
  const float* sel_bias;  // [b, Hkv, n, K] (GATED)
  void* dQ;               // [b, n, H, dh]
  void* dK;               // [b, n, Hkv, dh]
  void* dV;
  float* dlog_gate;       // [b, Hkv, n, K] or null
  // scratch
  float* delta;           // [b, H, n]
  float* dlg_head;        // [b, H, n, K]
  const float* log_gate;  // [b, Hkv, n, ceil(n/B)] (GATED)
  uint32_t* selmask;      // [b, Hkv, n, ceil(ceil(n/B)/32)] bit m: block m selected (bf16 path)
  // rows attending each 64-key tile (bf16 path, selections): counts and offsets
  // [b, Hkv, ceil(n/64)], ascending row indices (at most 2 (K+1) per row)
  int* tile_cnt;
  int* tile_off;
  int* tile_rows;
  // gating formulation (GATED): outer gate; full scope; straight-through hard gate
  int outer, full, ste;
  float* dlog_gate_full;  // [b, Hkv, n, NB] output (full scope / straight-through)
  float* dlg_head_full;   // [b, H, n, NB] scratch (full scope / straight-through)
  const int32_t* doc;     // [b, NB] first block of each block's document, or null
  uint32_t* queue;        // [2] job counters of the bf16 pass kernels' work queues (reset by the launch)
};
// longest sequence of the bf16 attention backward (query chunks of 32 tracked in LDS)
constexpr int BWD_MAX_SEQ = 262144;
hipError_t launch_attention_backward(int dtype, const BwdArgs& a, hipStream_t s);
// p[0..n) = v with a kernel (capturable in a graph, unlike a memset node)
hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t s);
// table[r, m] = sum over the slots k of row r with sel[r, k] == m of slots[r, k]
hipError_t launch_scatter_slots(const int32_t* sel, const float* slots, int b, int n, int Hkv, int K, int NB,
                                float* table, hipStream_t s);
// bias[b, g, t, k] = log_gate[b, g, t, sel[b, g, t, k]] (0 for empty slots)
hipError_t launch_gather_gate(const int32_t* sel, const float* log_gate, int b, int n, int Hkv, int K, int NB,
                              float* bias, hipStream_t s);
// Selector backward.  ds[r, m] for rows r = (b, g, t), m < NB, from the log-gate
// gradient dl (per slot: dlog_gate at the slots of sel; or the full table):
// SOFTMAX dl_m - exp(log_gate[r, m]) sum_m' dl_m'; SIGMOID dl_m (1 - exp(log_gate));
// RAW dl_m; for m < t / B (the row's historical blocks), 0 otherwise.
hipError_t launch_selector_ds(const int32_t* sel, const float* log_gate, const float* dlog_gate,
                              const float* dlog_gate_full, int act, int b, int n, int Hkv, int K, int B, float* ds,
                              const int32_t* doc, hipStream_t s);
// C(z, split)[i, j] = alpha sum_{k in split} A(z)[i, k] B(z)[k, j] for z < Z: fp32
// A, B in the activation dtype, fp32 C; strides in elements.  With splits > 1
// each split writes its own partial at C + split * sCs.
struct SmallGemm {
  int M, N, K, Z, splits;
  float alpha;
  const float* A;
  long long sAz, sAi, sAk;
  const void* Bm;
  long long sBz, sBk, sBj;
  float* C;
  long long sCz, sCs, sCi;
};
hipError_t launch_small_gemm(int dtype, const SmallGemm& g, hipStream_t s);
// out[zo, e] = sum_{u < U} sum_{q < S} part[((u ZO + zo) S + q) E + e]
hipError_t launch_partial_sum(const float* part, int U, int ZO, int S, size_t E, float* out, hipStream_t s);

// ---- stats.hip -------------------------------------------------------------
// lvn[r] = log2 ||v_r|| over rows of dh values
hipError_t launch_vnorm(int dtype, const void* V, size_t rows, int dh, float* lvn, hipStream_t s);
struct StatsArgs {
  int b, n, H, Hkv, dh, B, K, mode;
  float sm_scale;
  const void* Q;          // [b, n, H, dh]
  const void* Kt;         // [b, n, Hkv, dh]
  const int32_t* sel;     // [b, Hkv, n, K] (unused in DENSE)
  const float* lvn;       // [b, n, Hkv] log2 of the value norms
  float* cov;             // [b, H, n] or null
  float* cov_v;           // [b, H, n] or null
  float* blk_lse;         // [b, H, n, NB] log2 mass of each historical block, or null
  const int32_t* doc;     // [b, NB] first block of each block's document, or null
  uint32_t* queue;        // job counter of the bf16 kernel's work queue (reset by the launch)
};
hipError_t launch_stats(int dtype, const StatsArgs& a, hipStream_t s);
// per-head Top-K by block mass -> head_mask [b, H, n, W]; majority per group OR-ed into uni [b, Hkv, n, W]
hipError_t launch_ref_sets(const float* blk_lse, int b, int n, int H, int Hkv, int B, int K, uint32_t* head_mask,
                           uint32_t* uni, const int32_t* doc, hipStream_t s);
// OR the selection rows into uni [rows, W]
hipError_t launch_sel_union(const int32_t* sel, size_t rows, int K, int NB, uint32_t* uni, hipStream_t s);
// counts[0] = |a & b|, counts[1] = |b| over `words` words
hipError_t launch_overlap_count(const uint32_t* a, const uint32_t* b, size_t words, unsigned long long* counts,
                                hipStream_t s);

// ---- decode.hip ------------------------------------------------------------
struct DecodeArgs {
  int b, H, Hkv, dh, B, K, d, F;
  float sm_scale, eps, rope_base;
  const int32_t* pos;
  // paged cache
  void* k_pages;
  void* v_pages;
  const int32_t* block_table;
  void* k_summary;
  int num_pages, page_size, max_pages, max_blocks;
  const void* w_gq;
  const void* w_gk;
};

// Page geometry of the cache: element offset of (sequence i, group g,
// position p) in the page pool, or -1 when the position has no page.
struct PageGeom {
  const int32_t* table;
  int num_pages, ps, max_pages;
  __device__ __forceinline__ long long offset(int i, int g, int p, int Hkv, int dh) const {
    if (p < 0) return -1;
    const int pi = p / ps;
    if (pi >= max_pages) return -1;
    const int page = table[(size_t)i * max_pages + pi];
    if (page < 0 || page >= num_pages) return -1;
    return (((long long)page * Hkv + g) * ps + (p % ps)) * dh;
  }
};
// Writes K/V of positions 0..n-1 of every sequence into the pages (unless
// `kv` is false: the QKV product wrote them) and copies the complete-block
// summaries into the summary cache.
hipError_t launch_cache_fill(int dtype, const void* K, const void* V, const void* ksum, int b, int n,
                             int Hkv, int dh, int B, int NB, const DecodeArgs& c, hipStream_t s,
                             bool kv = true);
// q [b, H, dh], k/v [b, Hkv, dh] of the new tokens -> append + summary.
hipError_t launch_kv_append(int dtype, const void* k, const void* v, const DecodeArgs& c,
                            void* kplain_scratch, hipStream_t s);
// Top-K per (seq, group) against the cached summaries -> sel [b, Hkv, K].
// Caches of more than DSEL_WAVE_MAX_BLOCKS blocks (up to DSEL_MAX_BLOCKS)
// need `scores`, b * Hkv * max_blocks doubles of scratch.
constexpr int DSEL_WAVE_MAX_BLOCKS = 256;
constexpr int DSEL_MAX_BLOCKS = 8192;
hipError_t launch_decode_select(int dtype, const void* q, const DecodeArgs& c, int32_t* sel, double* scores,
                                hipStream_t s);
// Sparse attention of the new tokens over current block + selected blocks.
hipError_t launch_decode_attention(int dtype, const void* q, const DecodeArgs& c, const int32_t* sel,
                                   float* part_ml, float* part_o, void* O, hipStream_t s);

// ---- model_ends.hip --------------------------------------------------------
hipError_t launch_embed(int dtype, int b, int n, const int32_t* ids, const void* table, int vocab,
                        const void* img, int n_img, void* x, int d, hipStream_t s);
// tokens[r] = argmax of logits[r, :V] (lowest index on ties); scratch pv/pi
// hold `slices` partial results per row.
hipError_t launch_argmax(const float* logits, int b, int V, float* pv, int32_t* pi, int slices, int32_t* tokens,
                         hipStream_t s);

}  // namespace sas
