// Backward of SAS attention (Sec. 4.3, Eq. ours_train; the recomputation
// backward of App. E) and of the selector's normalized log gate
// (Eq. normalized_log_gate), for the selector update of Alg. 1.
//
// Per (head h of group g, query t) over the forward's attended set S with
// z_i = sm q.k_i + bias_i and p = exp(z - LSE):
//   Delta = dO . O,  dp_i = dO . v_i,  ds_i = p_i (dp_i - Delta)
//   dq = sm sum_i ds_i k_i,  dk_i += sm ds_i q,  dv_i += p_i dO
//   dlog g[g, t, slot of m] = sum_{h in g} sum_{i in B_m} ds_i   (GATED)
// Pass 1 walks queries (dQ and the per-head block sums of ds); pass 2 walks
// keys (dK, dV) and visits only the query chunks that attend them.
//
// Selector (the end of this file): the gate's softmax backward gives the
// score gradient ds of each row's historical blocks; the scores are inner
// products of gate queries and block summaries, so their gradients (and
// those of the optional projections) are small batched GEMMs over ds.
#include <float.h>
#include <stdint.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace sas {

// Delta[b, h, t] = sum_d O[b, t, h, d] dO[b, t, h, d] (fp32): dh / 8 threads per
// row (rows (b, t, h) are contiguous in [b, n, H, dh]), 16-byte loads of 8
// values each, the partial sums added across the row's lanes.
template <typename T>
__global__ void __launch_bounds__(256) bwd_delta_kernel(const T* __restrict__ O, const T* __restrict__ dO, int b,
                                                        int n, int H, int dh, float* __restrict__ delta) {
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int tpr = dh / 8;  // threads per row: 16 or 8, aligned groups of lanes
  const size_t rows = (size_t)b * n * H, row = gid / tpr;
  const int c8 = (int)(gid % tpr);
  const bool valid = row < rows;
  float acc = 0.f;
  if (valid) {
    Vec8<T> o, d;
    o.load(O + row * dh + c8 * 8);
    d.load(dO + row * dh + c8 * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fmaf(o.get(e), d.get(e), acc);
  }
  for (int sh = tpr >> 1; sh > 0; sh >>= 1) acc += __shfl_xor(acc, sh, 64);
  if (valid && c8 == 0) {
    const int h = (int)(row % H), t = (int)((row / H) % n), bi = (int)(row / ((size_t)H * n));
    delta[((size_t)bi * H + h) * n + t] = acc;
  }
}

// How block m enters the attention of query t and its gradient (natural-log
// domain): att = attended (dQ, dK, dV terms); grad = receives a log-gate
// gradient; bias = logit bias; w = value weight; lg = the block's log gate;
// slot = its selection slot (-1 if none).
struct BlockGate {
  bool att, grad;
  float bias, w, lg;
  int slot;
};

__device__ BlockGate block_gate(const BwdArgs& P, int bi, int g, int t, int m) {
  BlockGate r = {false, false, 0.f, 1.f, 0.f, -1};
  const int beta = t / P.B;
  const int NBr = (P.n + P.B - 1) / P.B;
  if (m > beta || (m < beta && m < doc_first(P.doc, bi, NBr, t, P.B))) return r;  // outside the document
  if (m == beta || P.mode == SAS_MODE_DENSE) {
    r.att = true;
    return r;
  }
  const bool gated = P.mode == SAS_MODE_GATED;
  const size_t row = ((size_t)bi * P.Hkv + g) * P.n + t;
  const int NB = (P.n + P.B - 1) / P.B;
  if (gated && P.full && !P.ste) {  // every historical block, gate from the table
    r.att = r.grad = true;
    r.lg = P.log_gate[row * NB + m];
  } else {
    for (int k = 0; k < P.K; ++k) {
      const int s = P.sel[row * P.K + k];
      if (s < 0 || s > m) break;
      if (s == m) {
        r.att = true;
        r.grad = gated;
        r.slot = k;
        r.lg = gated ? P.sel_bias[row * P.K + k] : 0.f;
        break;
      }
    }
    if (!r.att && gated && P.ste && P.full) {  // straight-through gradient of a dropped block
      r.grad = true;
      r.lg = P.log_gate[row * NB + m];
    }
  }
  if (gated && !P.ste) {
    if (P.outer) r.w = expf(r.lg);
    else r.bias = r.lg;
  }
  return r;
}

// ---- fp32 path ------------------------------------------------------------------
// pass 1: one thread per (batch, head, query)
template <int DH>
__global__ void __launch_bounds__(64) bwd_dq_f32_kernel(BwdArgs P) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = P.n;
  if (idx >= (size_t)P.b * P.H * n) return;
  const int t = (int)(idx % n), h = (int)((idx / n) % P.H), bi = (int)(idx / ((size_t)n * P.H));
  const int G = P.H / P.Hkv, g = h / G, B = P.B;
  const int NB = (n + B - 1) / B;
  const float* q = (const float*)P.Q + (((size_t)bi * n + t) * P.H + h) * DH;
  const float* dO = (const float*)P.dO + (((size_t)bi * n + t) * P.H + h) * DH;
  const size_t hrow = ((size_t)bi * P.H + h) * n + t;
  const float lse = P.lse[hrow];
  const float delta = P.delta[hrow];
  float qv[DH], dov[DH], dq[DH];
#pragma unroll
  for (int j = 0; j < DH; ++j) {
    qv[j] = q[j];
    dov[j] = dO[j];
    dq[j] = 0.f;
  }
  float* dlg = P.dlg_head ? P.dlg_head + hrow * P.K : nullptr;
  const int beta = t / B;
  for (int m = 0; m <= beta; ++m) {
    const BlockGate bg = block_gate(P, bi, g, t, m);
    if (!bg.att && !bg.grad) continue;
    const int i1 = m == beta ? t : (m + 1) * B - 1;
    float dsum = 0.f;
    for (int i = m * B; i <= i1; ++i) {
      const float* k = (const float*)P.Kt + (((size_t)bi * n + i) * P.Hkv + g) * DH;
      const float* v = (const float*)P.V + (((size_t)bi * n + i) * P.Hkv + g) * DH;
      float z = 0.f, dp = 0.f;
#pragma unroll
      for (int j = 0; j < DH; ++j) {
        z = fmaf(qv[j], k[j], z);
        dp = fmaf(dov[j], v[j], dp);
      }
      const float p = expf(z * P.sm_scale + bg.bias - lse);
      const float dpw = bg.w * dp;
      const float ds = p * (dpw - delta);
      dsum += P.outer ? p * dpw : ds;
      if (bg.att) {
#pragma unroll
        for (int j = 0; j < DH; ++j) dq[j] = fmaf(ds * P.sm_scale, k[j], dq[j]);
      }
    }
    if (bg.grad && m < beta) {
      if (P.full) P.dlg_head_full[hrow * NB + m] = dsum;
      else if (dlg && bg.slot >= 0) dlg[bg.slot] = dsum;
    }
  }
  float* dqp = (float*)P.dQ + (((size_t)bi * n + t) * P.H + h) * DH;
#pragma unroll
  for (int j = 0; j < DH; ++j) dqp[j] = dq[j];
}

// pass 2: one thread per (batch, group, key)
template <int DH>
__global__ void __launch_bounds__(64) bwd_dkv_f32_kernel(BwdArgs P) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = P.n;
  if (idx >= (size_t)P.b * P.Hkv * n) return;
  const int i = (int)(idx % n), g = (int)((idx / n) % P.Hkv), bi = (int)(idx / ((size_t)n * P.Hkv));
  const int G = P.H / P.Hkv, B = P.B, m = i / B;
  const float* k = (const float*)P.Kt + (((size_t)bi * n + i) * P.Hkv + g) * DH;
  const float* v = (const float*)P.V + (((size_t)bi * n + i) * P.Hkv + g) * DH;
  float kv[DH], vv[DH], dk[DH], dv[DH];
#pragma unroll
  for (int j = 0; j < DH; ++j) {
    kv[j] = k[j];
    vv[j] = v[j];
    dk[j] = 0.f;
    dv[j] = 0.f;
  }
  for (int t = i; t < n; ++t) {
    const BlockGate bg = block_gate(P, bi, g, t, m);
    if (!bg.att) continue;
    for (int h = g * G; h < (g + 1) * G; ++h) {
      const float* q = (const float*)P.Q + (((size_t)bi * n + t) * P.H + h) * DH;
      const float* dO = (const float*)P.dO + (((size_t)bi * n + t) * P.H + h) * DH;
      float z = 0.f, dp = 0.f;
#pragma unroll
      for (int j = 0; j < DH; ++j) {
        z = fmaf(q[j], kv[j], z);
        dp = fmaf(dO[j], vv[j], dp);
      }
      const size_t hr = ((size_t)bi * P.H + h) * n + t;
      const float p = expf(z * P.sm_scale + bg.bias - P.lse[hr]);
      const float ds = p * (bg.w * dp - P.delta[hr]);
      const float pw = p * bg.w;
#pragma unroll
      for (int j = 0; j < DH; ++j) {
        dk[j] = fmaf(ds * P.sm_scale, q[j], dk[j]);
        dv[j] = fmaf(pw, dO[j], dv[j]);
      }
    }
  }
  float* dkp = (float*)P.dK + (((size_t)bi * n + i) * P.Hkv + g) * DH;
  float* dvp = (float*)P.dV + (((size_t)bi * n + i) * P.Hkv + g) * DH;
#pragma unroll
  for (int j = 0; j < DH; ++j) {
    dkp[j] = dk[j];
    dvp[j] = dv[j];
  }
}

// dLogG[b, g, t, slot] = sum over the group's heads of the per-head block sums
// (times the block's gate for the straight-through gate: the gradient of log g)
__global__ void bwd_dlog_gate_sum_kernel(const float* __restrict__ dlg_head, const float* __restrict__ sel_bias,
                                         int ste, int b, int n, int H, int Hkv, int K,
                                         float* __restrict__ dlog_gate) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)b * Hkv * n * K) return;
  const int k = (int)(idx % K), t = (int)((idx / K) % n), g = (int)((idx / ((size_t)K * n)) % Hkv);
  const int bi = (int)(idx / ((size_t)K * n * Hkv));
  const int G = H / Hkv;
  float s = 0.f;
  for (int h = g * G; h < (g + 1) * G; ++h) s += dlg_head[(((size_t)bi * H + h) * n + t) * K + k];
  dlog_gate[idx] = ste ? s * expf(sel_bias[idx]) : s;
}

// the same for every block (full scope): 0 for blocks that are not historical
__global__ void bwd_dlog_gate_full_sum_kernel(const float* __restrict__ dlg_head_full,
                                              const float* __restrict__ log_gate, int ste, int b, int n, int H,
                                              int Hkv, int B, int NB, float* __restrict__ out,
                                              const int32_t* __restrict__ doc) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)b * Hkv * n * NB) return;
  const int m = (int)(idx % NB), t = (int)((idx / NB) % n), g = (int)((idx / ((size_t)NB * n)) % Hkv);
  const int bi = (int)(idx / ((size_t)NB * n * Hkv));
  float s = 0.f;
  if (m < t / B && m >= doc_first(doc, bi, NB, t, B)) {
    const int G = H / Hkv;
    for (int h = g * G; h < (g + 1) * G; ++h) s += dlg_head_full[(((size_t)bi * H + h) * n + t) * NB + m];
    if (ste) s *= expf(log_gate[idx]);
  }
  out[idx] = s;
}

__global__ void bwd_scatter_slots_kernel(const int32_t* __restrict__ sel, const float* __restrict__ slots,
                                         size_t rows, int K, int NB, float* __restrict__ table) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * NB) return;
  const size_t row = idx / NB;
  const int m = (int)(idx % NB);
  float v = 0.f;
  for (int k = 0; k < K; ++k)
    if (sel[row * K + k] == m) v += slots[row * K + k];
  table[idx] = v;
}

hipError_t launch_scatter_slots(const int32_t* sel, const float* slots, int b, int n, int Hkv, int K, int NB,
                                float* table, hipStream_t s) {
  const size_t rows = (size_t)b * Hkv * n;
  if (rows * NB == 0) return hipSuccess;
  bwd_scatter_slots_kernel<<<(unsigned)cdiv(rows * NB, 256), 256, 0, s>>>(sel, slots, rows, K, NB, table);
  return hipGetLastError();
}

// log gate of each selected slot: bias[b, g, t, k] = log_gate[b, g, t, sel[b, g, t, k]]
__global__ void bwd_gather_gate_kernel(const int32_t* __restrict__ sel, const float* __restrict__ log_gate, int b,
                                       int n, int Hkv, int K, int NB, float* __restrict__ bias) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)b * Hkv * n * K) return;
  const int m = sel[idx];
  bias[idx] = (m >= 0 && m < NB) ? log_gate[(idx / K) * NB + m] : 0.f;
}

__global__ void fill_f32_kernel(float* p, size_t n, float v) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// ---- bf16 path ------------------------------------------------------------------
constexpr float BLOG2E = 1.4426950408889634f;

// Pass 1 (dQ and the per-head block sums of ds): one workgroup = 4 waves =
// 128 queries of one (batch, head), each lane owning one query of S^T = K Q^T
// (v_mfma_f32_32x32x16_bf16), with dP^T = V dO^T computed the same way;
// dS^T = P^T (dP^T - Delta) is formed in registers and fed back as the B
// operand of dQ^T += K^T dS^T (K staged transposed in LDS, read in the
// accumulator's key permutation).  The key tiles any query of the workgroup
// attends are flagged in LDS first; each tile's K and V are loaded into
// registers while the previous tile is multiplied.  Sub-blocks of
// 2^LSB = min(B, 64) keys carry one bias per query; a sub-block of an
// accumulator element is known at compile time (the lane-dependent part of
// its key index is below 8).  Each lane walks its query's ascending
// selection row from global memory (the next slot read one slot ahead) and
// writes a slot's block sum once the slot's last sub-block is done; a tile is
// processed as two halves of 32 keys to keep the live registers low enough
// for two workgroups per compute unit.
template <int DH, int LSB, bool PLAIN>
__device__ __forceinline__ void bwd_dq_bf16_job(const BwdArgs& P, const int qtile, const int h, const int bi) {
  constexpr int KP = DH + 8;
  constexpr int TP = 64 + 4;
  constexpr int KPG = DH / 32;   // keys per thread in the tile staging
  constexpr int C8 = DH / 8;
  constexpr int NSUB = 64 >> LSB;
  __shared__ __align__(16) bf16_t Ks[64 * KP];
  __shared__ __align__(16) bf16_t Vs[64 * KP];
  __shared__ __align__(16) bf16_t Kt[DH * TP];
  __shared__ uint32_t need[BWD_MAX_SEQ / 64 / 32];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int G = P.H / P.Hkv, g = h / G;
  const int n = P.n, B = P.B;
  const int qrow = wave * 32 + lr;  // query row of this lane in the workgroup
  const int t = qtile * 128 + qrow;
  const bool qvalid = t < n;
  const int beta = qvalid ? t / B : -1;
  const bool gated = P.mode == SAS_MODE_GATED;
  const bool dense = P.mode == SAS_MODE_DENSE;
  const bool full = gated && P.full;           // a gradient for every historical block
  const bool fullatt = full && !P.ste;         // ... which are all attended
  const bool ste = gated && P.ste, outer = gated && P.outer;
  const bool every = dense || full;            // every tile up to the query
  const int Kn = (dense || fullatt) ? 0 : P.K;
  const int ntiles = (n + 63) / 64;
  const int NB = (n + B - 1) / B;
  const size_t grow = ((size_t)bi * P.Hkv + g) * n;
  const int t_hi = min(n, qtile * 128 + 128) - 1;
  const int last_tile = t_hi / 64;
  const int fb = qvalid ? doc_first(P.doc, bi, NB, t, B) : 0;  // first block of the query's document
  const int first_tile = doc_first(P.doc, bi, NB, qtile * 128, B) * B / 64;

  bf16x8_t qb[DH / 16], dob[DH / 16];
  {
    const size_t off = (((size_t)bi * n + (qvalid ? t : 0)) * P.H + h) * DH;
    const bf16_t* qp = (const bf16_t*)P.Q + off;
    const bf16_t* dp = (const bf16_t*)P.dO + off;
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) {
      uint4 u = qvalid ? *(const uint4*)(qp + ks * 16 + lk * 8) : make_uint4(0, 0, 0, 0);
      qb[ks] = *(bf16x8_t*)&u;
      uint4 w = qvalid ? *(const uint4*)(dp + ks * 16 + lk * 8) : make_uint4(0, 0, 0, 0);
      dob[ks] = *(bf16x8_t*)&w;
    }
  }
  const size_t hrow = ((size_t)bi * P.H + h) * n + (qvalid ? t : 0);
  const float lse2 = qvalid ? P.lse[hrow] * BLOG2E : 0.f;
  const float delta = qvalid ? P.delta[hrow] : 0.f;

  // key tiles of every earlier block (DENSE, full scope), from the workgroup's earliest document start
  for (int w = tid; w < (ntiles + 31) / 32; w += 256) {
    const int lo = w * 32;
    uint32_t bits = 0;
    if (every && lo <= last_tile) bits = last_tile - lo >= 31 ? 0xffffffffu : ((1u << (last_tile - lo + 1)) - 1u);
    if (every && lo + 31 >= first_tile && lo < first_tile) bits &= ~((1u << (first_tile - lo)) - 1u);
    if (lo + 31 < first_tile) bits = 0;
    need[w] = bits;
  }
  __syncthreads();
  // this query's selection row: slots are ascending historical blocks, -1 padded
  const size_t srow = (grow + (qvalid ? t : 0)) * (size_t)Kn;
  // key tiles this workgroup attends: every query's current block, its selected blocks
  if (!every && qvalid && lk == 0) {
    for (int tl = (beta * B) / 64; tl <= t / 64; ++tl) atomicOr(&need[tl >> 5], 1u << (tl & 31));
    for (int k = 0; k < Kn; ++k) {
      const int m = P.sel[srow + k];
      if (m < 0 || m >= beta) break;  // slots are ascending historical blocks, -1 padded
      for (int tl = (m * B) / 64; tl <= ((m + 1) * B - 1) / 64; ++tl) atomicOr(&need[tl >> 5], 1u << (tl & 31));
    }
  }
  __syncthreads();

  floatx16_t dq[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) dq[dt][v] = 0.f;
  const float qk_scale = P.sm_scale * BLOG2E;
  const bf16_t* Kg = (const bf16_t*)P.Kt + (size_t)g * DH;
  const bf16_t* Vg = (const bf16_t*)P.V + (size_t)g * DH;
  const size_t kstride = (size_t)P.Hkv * DH;
  const size_t kbase = (size_t)bi * n;
  const int c8 = tid % C8, kg = tid / C8;
  uint4 rk[KPG], rv[KPG];
  float r_lg[NSUB];  // full scope: this query's log gates of the tile's blocks
  auto prefetch = [&](int kt) {
#pragma unroll
    for (int q = 0; q < KPG; ++q) {
      const int key = kt * 64 + kg * KPG + q;
      const size_t go = (kbase + key) * kstride + c8 * 8;
      rk[q] = key < n ? *(const uint4*)(Kg + go) : make_uint4(0, 0, 0, 0);
      rv[q] = key < n ? *(const uint4*)(Vg + go) : make_uint4(0, 0, 0, 0);
    }
    if (full) {
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb) {
        const int m = (kt * 64 + (sb << LSB)) / B;
        r_lg[sb] = (qvalid && m < beta && m >= fb) ? P.log_gate[(grow + t) * NB + m] : 0.f;
      }
    }
  };
  auto commit = [&]() {
#pragma unroll
    for (int q = 0; q < KPG; ++q) {
      *(uint4*)(Ks + (kg * KPG + q) * KP + c8 * 8) = rk[q];
      *(uint4*)(Vs + (kg * KPG + q) * KP + c8 * 8) = rv[q];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int sh = (e & 1) * 16, wd = e >> 1;
      bf16_t* dst = Kt + (c8 * 8 + e) * TP + kg * KPG;
      uint32_t x[KPG];
#pragma unroll
      for (int q = 0; q < KPG; ++q) x[q] = (((const uint32_t*)&rk[q])[wd] >> sh) & 0xffffu;
      if constexpr (KPG == 4) {
        *(uint2*)dst = make_uint2(x[0] | (x[1] << 16), x[2] | (x[3] << 16));
      } else {
        *(uint32_t*)dst = x[0] | (x[1] << 16);
      }
    }
  };

  // the walk over this query's slots: slot `cur` (block next_sel, bias b_cur) and the
  // one after it (read one slot ahead, so the read is done by the time it is needed)
  auto sel_at = [&](int k) -> int { return qvalid && k < Kn ? P.sel[srow + k] : -1; };
  auto bias_at = [&](int k) -> float { return gated && qvalid && k < Kn ? P.sel_bias[srow + k] : 0.f; };
  int cur = 0;
  int next_sel = sel_at(0);
  float b_cur = bias_at(0);
  int s_nx = sel_at(1);
  float b_nx = bias_at(1);
  if (next_sel < 0) next_sel = 0x7fffffff;
  float blk_acc = 0.f;   // full scope: running sum of a block wider than a tile
  float slot_acc = 0.f;  // the current slot's running sum (a block may span two tiles)
  int kt = next_set(need, 0, ntiles);
  if (kt < ntiles) prefetch(kt);
  while (kt < ntiles) {
    commit();
    lds_barrier();
    const int k0 = kt * 64;

    // per sub-block: offset (log2-domain bias - LSE; -inf: neither attended nor
    // receiving a gradient), value weight, attended, selection slot
    float offs[NSUB], wts[NSUB];
    bool attb[NSUB], gradb[NSUB];
    int slot[NSUB];
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) {
      offs[sb] = -INFINITY;
      wts[sb] = 1.f;
      attb[sb] = gradb[sb] = false;
      slot[sb] = -1;
      const int kstart = k0 + (sb << LSB);
      if (!qvalid || kstart > t) continue;
      const int m = kstart / B;
      float lg = 0.f;
      if (m == beta || (dense && m >= fb)) {
        attb[sb] = true;
      } else if (m < fb) {
        // outside the query's document
      } else if (fullatt) {
        attb[sb] = gradb[sb] = true;
        lg = r_lg[sb];
      } else {
        if (m == next_sel) {
          attb[sb] = true;
          gradb[sb] = gated;
          lg = b_cur;
          slot[sb] = cur;
          if (kstart + (1 << LSB) >= (m + 1) * B) {
            ++cur;
            next_sel = s_nx >= 0 ? s_nx : 0x7fffffff;
            b_cur = b_nx;
            s_nx = sel_at(cur + 1);
            b_nx = bias_at(cur + 1);
          }
        } else if (ste && full) {
          gradb[sb] = true;  // straight-through gradient of a dropped block
          lg = r_lg[sb];
        }
      }
      if (attb[sb] || gradb[sb]) {
        const bool biased = gated && !ste && !outer && m != beta;
        offs[sb] = (biased ? lg * BLOG2E : 0.f) - lse2;
        if (outer && m != beta) wts[sb] = __builtin_amdgcn_exp2f(lg * BLOG2E);
      }
    }
    const int nkt = next_set(need, kt + 1, ntiles);
    if (nkt < ntiles) prefetch(nkt);

    const bool diag = k0 + 63 > qtile * 128;  // keys past some query of the workgroup: mask key > t
    float dsum[NSUB];
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) dsum[sb] = 0.f;
    // the tile's two halves of 32 keys one after the other (fewer live registers):
    // S^T, dP^T of the half, dS^T in registers, then its two 16-key steps of dQ^T += K^T dS^T
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      floatx16_t sc, dp;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        sc[v] = 0.f;
        dp[v] = 0.f;
      }
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) {
        const bf16x8_t a = *(const bf16x8_t*)(Ks + (st * 32 + lr) * KP + ks * 16 + lk * 8);
        sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qb[ks], sc, 0, 0, 0);
        const bf16x8_t av = *(const bf16x8_t*)(Vs + (st * 32 + lr) * KP + ks * 16 + lk * 8);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, dob[ks], dp, 0, 0, 0);
      }
      // P, dS^T and the block sums.  PLAIN (no value weights, no straight-through gradient): a
      // sub-block that is not attended has an offset of -inf, so its dS is already zero
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int klc = st * 32 + 8 * (v >> 2);  // key offset without the lane part (4 lk + v % 4 < 8)
        const int sb = klc >> LSB;
        float p = __builtin_amdgcn_exp2f(fmaf(sc[v], qk_scale, offs[sb]));
        if (diag && k0 + klc + 4 * lk + (v & 3) > t) p = 0.f;
        if constexpr (PLAIN) {
          const float ds = p * (dp[v] - delta);
          sc[v] = ds;
          dsum[sb] += ds;
        } else {
          const float dpw = outer ? wts[sb] * dp[v] : dp[v];
          const float ds = p * (dpw - delta);
          sc[v] = attb[sb] ? ds : 0.f;
          dsum[sb] += outer ? p * dpw : ds;
        }
      }
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int ks = 2 * st + kk, v0 = 8 * kk;
        uint4 su;
        su.x = pack_bf16x2(sc[v0 + 0], sc[v0 + 1]);
        su.y = pack_bf16x2(sc[v0 + 2], sc[v0 + 3]);
        su.z = pack_bf16x2(sc[v0 + 4], sc[v0 + 5]);
        su.w = pack_bf16x2(sc[v0 + 6], sc[v0 + 7]);
        const bf16x8_t pb = *(const bf16x8_t*)&su;
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt) {
          const bf16_t* kr = Kt + (dt * 32 + lr) * TP + 16 * ks + 4 * lk;
          const uint2 lo = *(const uint2*)kr;
          const uint2 hi = *(const uint2*)(kr + 8);
          uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
          dq[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(bf16x8_t*)&u, pb, dq[dt], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) {
      const float tot = dsum[sb] + __shfl_xor(dsum[sb], 32, 64);
      const int kstart = k0 + (sb << LSB), m = kstart / B;
      const bool last = kstart + (1 << LSB) >= (m + 1) * B;  // the block's last sub-block
      if (lk == 0 && full && gradb[sb]) {
        blk_acc += tot;
        if (last) {
          P.dlg_head_full[hrow * NB + m] = blk_acc;
          blk_acc = 0.f;
        }
      } else if (lk == 0 && !full && slot[sb] >= 0) {
        if (gradb[sb]) slot_acc += tot;
        if (last) {  // the slot is complete
          if (P.dlg_head) P.dlg_head[hrow * P.K + slot[sb]] = slot_acc;
          slot_acc = 0.f;
        }
      }
    }
    lds_barrier();
    kt = nkt;
  }

  if (!qvalid) return;
  if (P.dlg_head && !full && lk == 0) {  // slots never reached (padding) get zero
    float* dlg = P.dlg_head + hrow * P.K;
    for (int k = cur; k < Kn; ++k) dlg[k] = 0.f;
  }
  bf16_t* op = (bf16_t*)P.dQ + (((size_t)bi * n + t) * P.H + h) * DH;
  const float sm = P.sm_scale;
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int d0 = dt * 32 + 8 * v4 + 4 * lk;
      const uint32_t w0 = pack_bf16x2(dq[dt][4 * v4 + 0] * sm, dq[dt][4 * v4 + 1] * sm);
      const uint32_t w1 = pack_bf16x2(dq[dt][4 * v4 + 2] * sm, dq[dt][4 * v4 + 3] * sm);
      *(uint2*)(op + d0) = make_uint2(w0, w1);
    }
}

// One job per workgroup (grid = job count, no queue) or the work queue.
// two workgroups per compute unit where the registers allow it without spills
// (one sub-block per tile, or dh = 64)
template <int DH, int LSB, bool PLAIN>
__global__ void __launch_bounds__(256, LSB == 6 || DH == 64 ? 2 : 1) bwd_dq_bf16_kernel(BwdArgs P) {
  const int nqt = (P.n + 127) / 128, per = P.H * P.b;
  const int njobs = nqt * per;
  for (int it = 0;; ++it) {
    const int job = P.queue ? queue_next_job(P.queue) : (it == 0 ? (int)blockIdx.x : njobs);
    if (job >= njobs) break;
    const int r = job % per;  // the longest (last) query tiles first, heads and batch inside
    bwd_dq_bf16_job<DH, LSB, PLAIN>(P, nqt - 1 - job / per, r % P.H, r / P.H);
  }
}

// selection bitmask of each row: bit m of word m / 32 is set when block m is selected
__global__ void bwd_selmask_kernel(const int32_t* __restrict__ sel, size_t rows, int K, int NW,
                                   uint32_t* __restrict__ mask) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * NW) return;
  const size_t row = idx / NW;
  const int w = (int)(idx % NW);
  uint32_t bits = 0;
  for (int k = 0; k < K; ++k) {
    const int m = sel[row * K + k];
    if (m >= 0 && (m >> 5) == w) bits |= 1u << (m & 31);
  }
  mask[idx] = bits;
}

// The rows of (b, g) that attend key tile j (keys 64 j .. 64 j + 63), in
// ascending order: the rows t >= 64 j whose own block lies in the tile (the
// causal part of the current block) and every later row that selected one of
// the tile's blocks (at most four; they share one mask word since a tile
// starts at a multiple of 64 / B blocks).  Without `rows` the kernel writes
// the count of tile j; with it, the rows at off[tile].  One workgroup of 256
// threads per (tile, group, batch entry); the ballot prefix sums keep the
// order, so the lists are an exact function of the selection.
__global__ void __launch_bounds__(256) bwd_tile_rows_kernel(const uint32_t* __restrict__ selmask, int n, int Hkv,
                                                            int B, int NW, int ntiles, int* __restrict__ cnt,
                                                            const int* __restrict__ off, int* __restrict__ rows) {
  __shared__ int wsum[4];
  const int j = blockIdx.x, g = blockIdx.y, bi = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t tile = ((size_t)bi * Hkv + g) * ntiles + j;
  const int k0 = j * 64, m_lo = k0 / B, m_hi = min(n - 1, k0 + 63) / B;
  const int own_end = min(n, (m_hi + 1) * B);
  const uint32_t bits = ((2u << (m_hi - m_lo)) - 1u) << (m_lo & 31);
  const uint32_t* sm = selmask + ((size_t)bi * Hkv + g) * (size_t)n * NW + (m_lo >> 5);
  const int base = rows ? off[tile] : 0;
  int total = 0;
  for (int t0 = k0; t0 < n; t0 += 256) {
    const int t = t0 + tid;
    bool f = false;
    if (t < n) f = t < own_end || (sm[(size_t)t * NW] & bits) != 0;
    const uint64_t bal = __ballot(f);
    if (lane == 0) wsum[wave] = __popcll(bal);
    __syncthreads();
    int before = __popcll(bal & ((1ull << lane) - 1ull)), all = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      before += w < wave ? wsum[w] : 0;
      all += wsum[w];
    }
    if (rows && f) rows[base + total + before] = t;
    total += all;
    __syncthreads();  // wsum is rewritten by the next step
  }
  if (!rows && tid == 0) cnt[tile] = total;
}

// exclusive prefix sum of the tile counts (one workgroup of 1024 threads; each
// thread sums a contiguous range, then the ranges are offset in order)
__global__ void __launch_bounds__(1024) bwd_rows_scan_kernel(const int* __restrict__ cnt, int T, int* __restrict__ off) {
  __shared__ int part[1024];
  const int tid = threadIdx.x;
  const int per = (T + 1023) / 1024, lo = min(T, tid * per), hi = min(T, lo + per);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += cnt[i];
  part[tid] = s;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int i = 0; i < 1024; ++i) {
      const int v = part[i];
      part[i] = run;
      run += v;
    }
  }
  __syncthreads();
  int run = part[tid];
  for (int i = lo; i < hi; ++i) {
    off[i] = run;
    run += cnt[i];
  }
}

// Pass 2 (dK, dV): one workgroup of 4 waves per 64 keys of one (batch, KV
// group); a pair of waves owns 32 keys and splits the head dimension: each
// wave holds its half of the keys' K and V as the B operands of the partial
// products S = Q K^T and dP = dO V^T over its dimensions (lane = key, 16 rows
// per lane) and accumulates dK and dV for its dimensions only; the two
// partial products are exchanged through LDS and added (the same sum in both
// waves), which keeps a wave within 256 registers (two waves per SIMD).  The rows are those of the tile's list (selections), or, when
// every earlier block is attended (DENSE, full scope), the consecutive rows
// from the tile on, in chunks of 32 that reach the tile.  Work items are
// (chunk, head of the group); the row indices of the next chunk are read one
// chunk ahead, and the Q and dO rows of the next item are loaded into
// registers while the current one is multiplied, then written to LDS both
// row-major (A of S and dP) and transposed (A of dK^T += Q^T dS and
// dV^T += dO^T P, read in the accumulator's row permutation).  P and dS stay
// in registers; the causal mask compares each key with its row's index.
template <int DH, bool PLAIN>
__device__ __forceinline__ void bwd_dkv_bf16_job(const BwdArgs& P, const int ktile, const int g, const int bi) {
  constexpr int NTH = 256, KT = 64;
  constexpr int KP = DH + 8;
  constexpr int QP = 32 + 4;
  constexpr int C8 = DH / 8;            // 16-byte pieces of a row
  constexpr int QPT = 32 * C8 / NTH;    // chunk rows staged per thread (2 or 1)
  constexpr int DHH = DH / 2;           // dimensions of a wave
  __shared__ __align__(16) bf16_t Qs[32 * KP];
  __shared__ __align__(16) bf16_t Ds[32 * KP];
  __shared__ __align__(16) bf16_t Qt[DH * QP];
  __shared__ __align__(16) bf16_t Dt[DH * QP];
  __shared__ __align__(16) float delta_s[32];
  __shared__ __align__(16) int trow_s[32];      // row index of each staged row (n: none)
  __shared__ __align__(16) float off_s[4][32];  // log2-domain bias - LSE per (sub-block, row); -inf: not attended
  __shared__ __align__(16) float wt_s[4][32];   // value weight per (sub-block, row) (outer gate)
  __shared__ uint32_t flags[BWD_MAX_SEQ / 32 / 32];
  __shared__ __align__(16) float xs[4][2][16][64];  // each wave's partial S and dP

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int kh = wave >> 1, dhf = wave & 1;  // key half, dimension half
  const int k0 = ktile * KT;
  const int n = P.n, B = P.B, H = P.H, G = H / P.Hkv;
  const int key = k0 + kh * 32 + lr;
  const bool kvalid = key < n;
  const int bshift = 31 - __clz(B < 64 ? B : 64);
  const int nsb = KT >> bshift;  // sub-blocks of min(B, 64) keys in the tile: 1, 2 or 4
  const int m_hi = min(n - 1, k0 + KT - 1) / B;
  const int NB = (n + B - 1) / B;
  const int NW = (NB + 31) / 32;
  const int nqc = (n + 31) / 32;
  const bool dense = P.mode == SAS_MODE_DENSE, gated = P.mode == SAS_MODE_GATED;
  const bool ste = gated && P.ste, outer = gated && P.outer;
  const bool fullatt = gated && P.full && !P.ste;  // every historical block attended, gates from the table
  const bool use_list = P.tile_rows != nullptr;    // selections: the tile's row list
  const size_t grow = ((size_t)bi * P.Hkv + g) * n;  // first row of (b, g) in [b, Hkv, n, ...]
  const int ntk = (n + KT - 1) / KT;
  int lbase = 0, lcnt = 0;
  if (use_list) {
    const size_t tile = ((size_t)bi * P.Hkv + g) * ntk + ktile;
    lbase = P.tile_off[tile];
    lcnt = P.tile_cnt[tile];
  }
  const int nchunk = use_list ? (lcnt + 31) / 32 : nqc;

  // without a list: the chunks that reach the tile (their rows lie in its blocks, or,
  // every earlier block being attended, their earliest row's document starts in time)
  const int qc0 = use_list ? 0 : k0 / 32;
  if (!use_list) {
    for (int w = tid; w < (nqc + 31) / 32; w += NTH) flags[w] = 0;
    __syncthreads();
    for (int qc = qc0 + tid; qc < nqc; qc += NTH) {
      const bool any = ((dense || fullatt) && doc_first(P.doc, bi, NB, qc * 32, B) <= m_hi) || (qc * 32) / B <= m_hi;
      if (any) atomicOr(&flags[qc >> 5], 1u << (qc & 31));
    }
    __syncthreads();
  }
  auto next_chunk = [&](int c) { return use_list ? c : next_set(flags, c, nqc); };

  bf16x8_t kb[DHH / 16], vb[DHH / 16];
  {
    const size_t off = (((size_t)bi * n + (kvalid ? key : 0)) * P.Hkv + g) * DH + dhf * DHH;
#pragma unroll
    for (int ks = 0; ks < DHH / 16; ++ks) {
      uint4 u = kvalid ? *(const uint4*)((const bf16_t*)P.Kt + off + ks * 16 + lk * 8) : make_uint4(0, 0, 0, 0);
      kb[ks] = *(bf16x8_t*)&u;
      uint4 w = kvalid ? *(const uint4*)((const bf16_t*)P.V + off + ks * 16 + lk * 8) : make_uint4(0, 0, 0, 0);
      vb[ks] = *(bf16x8_t*)&w;
    }
  }
  floatx16_t dk[DHH / 32], dv[DHH / 32];
#pragma unroll
  for (int dt = 0; dt < DHH / 32; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      dk[dt][v] = 0.f;
      dv[dt][v] = 0.f;
    }
  const float qk_scale = P.sm_scale * BLOG2E;

  // staging roles: rows qg * QPT + i, 16-byte piece c8; row index / delta row bq (tid < 32);
  // bias (row bq, sub-block bsb)
  const int c8 = tid % C8, qg = tid / C8;
  const int bq = tid & 31, bsb = tid >> 5;
  // row index of staged row r of chunk c (n: none)
  auto row_of = [&](int c, int r) -> int {
    if (use_list) {
      const int i = c * 32 + r;
      return i < lcnt ? P.tile_rows[lbase + i] : n;
    }
    const int t = c * 32 + r;
    return t < n ? t : n;
  };
  // row indices of the chunk being loaded (rt, bt) and of the chunk after it (rt_n, bt_n)
  int rt[QPT], rt_n[QPT], bt = n, bt_n = n;
  uint4 rq[QPT], rd[QPT];
  float r_lse = 0.f, r_delta = 0.f, r_lg = 0.f;
  uint32_t r_mw = 0;
  int r_fb = 0;  // first block of the row's document
  int pc = -1;   // chunk whose row indices are in rt

  auto load_rows = [&](int c, int* dst, int& b) {
#pragma unroll
    for (int i = 0; i < QPT; ++i) dst[i] = c < nchunk ? row_of(c, qg * QPT + i) : n;
    b = c < nchunk ? row_of(c, bq) : n;
  };
  auto prefetch = [&](int qc, int hg) {
    if (qc != pc) {  // a new chunk: its rows were read one chunk ahead
#pragma unroll
      for (int i = 0; i < QPT; ++i) rt[i] = rt_n[i];
      bt = bt_n;
      pc = qc;
      load_rows(next_chunk(qc + 1), rt_n, bt_n);
    }
    const int h = g * G + hg;
#pragma unroll
    for (int i = 0; i < QPT; ++i) {
      const int t = rt[i];
      const size_t off = (((size_t)bi * n + t) * H + h) * DH + c8 * 8;
      rq[i] = t < n ? *(const uint4*)((const bf16_t*)P.Q + off) : make_uint4(0, 0, 0, 0);
      rd[i] = t < n ? *(const uint4*)((const bf16_t*)P.dO + off) : make_uint4(0, 0, 0, 0);
    }
    const int t = bt;
    if (tid < 32) r_delta = t < n ? P.delta[((size_t)bi * H + h) * n + t] : 0.f;
    if (bsb < nsb) {
      const int kstart = k0 + (bsb << bshift), m = kstart / B;
      r_lse = t < n ? P.lse[((size_t)bi * H + h) * n + t] : 0.f;
      r_fb = t < n ? doc_first(P.doc, bi, NB, t, B) : 0;
      r_mw = 0u;
      r_lg = 0.f;
      if (t < n && kstart <= t && m != t / B) {
        r_mw = use_list ? P.selmask[(grow + t) * NW + (m >> 5)] : 0u;
        r_lg = gated && (use_list || fullatt) ? P.log_gate[(grow + t) * NB + m] : 0.f;
      }
    }
  };
  auto commit = [&]() {
#pragma unroll
    for (int i = 0; i < QPT; ++i) {
      *(uint4*)(Qs + (qg * QPT + i) * KP + c8 * 8) = rq[i];
      *(uint4*)(Ds + (qg * QPT + i) * KP + c8 * 8) = rd[i];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int sh = (e & 1) * 16;
      const int wd = e >> 1;
      uint32_t x[QPT], y[QPT];
#pragma unroll
      for (int i = 0; i < QPT; ++i) {
        x[i] = (((const uint32_t*)&rq[i])[wd] >> sh) & 0xffffu;
        y[i] = (((const uint32_t*)&rd[i])[wd] >> sh) & 0xffffu;
      }
      bf16_t* qd = Qt + (c8 * 8 + e) * QP + qg * QPT;
      bf16_t* dd = Dt + (c8 * 8 + e) * QP + qg * QPT;
      if constexpr (QPT == 2) {
        *(uint32_t*)qd = x[0] | (x[1] << 16);
        *(uint32_t*)dd = y[0] | (y[1] << 16);
      } else {
        *(uint16_t*)qd = (uint16_t)x[0];
        *(uint16_t*)dd = (uint16_t)y[0];
      }
    }
    if (tid < 32) {
      delta_s[tid] = r_delta;
      trow_s[tid] = bt;
    }
    if (bsb < nsb) {
      const int t = bt, kstart = k0 + (bsb << bshift), m = kstart / B;
      float bb = -INFINITY, w = 1.f;
      if (t < n && kstart <= t) {
        if (m == t / B || (dense && m >= r_fb)) {
          bb = 0.f;
        } else if ((fullatt && m >= r_fb) || ((r_mw >> (m & 31)) & 1u)) {
          const bool gate = gated && !ste;
          bb = gate && !outer ? r_lg * BLOG2E : 0.f;
          if (gate && outer) w = __builtin_amdgcn_exp2f(r_lg * BLOG2E);
        }
      }
      off_s[bsb][bq] = bb - r_lse * BLOG2E;
      wt_s[bsb][bq] = w;
    }
  };

  int qc = next_chunk(qc0), hg = 0;
  load_rows(qc, rt_n, bt_n);
  if (qc < nchunk) prefetch(qc, 0);
  while (qc < nchunk) {
    commit();
    lds_barrier();
    int nq = qc, nh = hg + 1;
    if (nh == G) {
      nh = 0;
      nq = next_chunk(qc + 1);
    }
    if (nq < nchunk) prefetch(nq, nh);

    floatx16_t sc, dp;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      sc[v] = 0.f;
      dp[v] = 0.f;
    }
#pragma unroll
    for (int ks = 0; ks < DHH / 16; ++ks) {
      const bf16x8_t aq = *(const bf16x8_t*)(Qs + lr * KP + dhf * DHH + ks * 16 + lk * 8);
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq, kb[ks], sc, 0, 0, 0);
      const bf16x8_t ad = *(const bf16x8_t*)(Ds + lr * KP + dhf * DHH + ks * 16 + lk * 8);
      dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ad, vb[ks], dp, 0, 0, 0);
    }
    // the pair's partial products: written, exchanged, added (commutative, the same in both)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      xs[wave][0][v][lane] = sc[v];
      xs[wave][1][v][lane] = dp[v];
    }
    lds_barrier();
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      sc[v] += xs[wave ^ 1][0][v][lane];
      dp[v] += xs[wave ^ 1][1][v][lane];
    }
    // lane: key column `key`; staged rows 8 j + 4 lk + i (v = 4 j + i)
    const int sbk = (kh * 32 + lr) >> bshift;
    const bool diag = trow_s[0] < k0 + KT - 1;  // some row precedes a key of the tile: mask key > row
    // dV^T += dO^T P and dK^T += Q^T dS, 16 rows per step in the accumulator's row permutation;
    // each step's P and dS are formed and packed just before its MFMAs
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      float pv[8], sv[8];
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int j = 2 * ks + jj;
        const float4 of = *(const float4*)&off_s[sbk][8 * j + 4 * lk];
        const float4 de = *(const float4*)&delta_s[8 * j + 4 * lk];
        const int4 tr = *(const int4*)&trow_s[8 * j + 4 * lk];
        float4 wt = make_float4(1.f, 1.f, 1.f, 1.f);
        if (!PLAIN && outer) wt = *(const float4*)&wt_s[sbk][8 * j + 4 * lk];
        const float ofv[4] = {of.x, of.y, of.z, of.w}, dev[4] = {de.x, de.y, de.z, de.w};
        const float wv[4] = {wt.x, wt.y, wt.z, wt.w};
        const int trv[4] = {tr.x, tr.y, tr.z, tr.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int v = 4 * j + i;
          float p = __builtin_amdgcn_exp2f(fmaf(sc[v], qk_scale, ofv[i]));
          if (diag && key > trv[i]) p = 0.f;
          if constexpr (PLAIN) {  // unit value weights
            pv[4 * jj + i] = p;
            sv[4 * jj + i] = p * (dp[v] - dev[i]);
          } else {
            pv[4 * jj + i] = p * wv[i];
            sv[4 * jj + i] = p * (wv[i] * dp[v] - dev[i]);
          }
        }
      }
      uint4 pu, su;
      pu.x = pack_bf16x2(pv[0], pv[1]);
      pu.y = pack_bf16x2(pv[2], pv[3]);
      pu.z = pack_bf16x2(pv[4], pv[5]);
      pu.w = pack_bf16x2(pv[6], pv[7]);
      su.x = pack_bf16x2(sv[0], sv[1]);
      su.y = pack_bf16x2(sv[2], sv[3]);
      su.z = pack_bf16x2(sv[4], sv[5]);
      su.w = pack_bf16x2(sv[6], sv[7]);
      const bf16x8_t pb = *(const bf16x8_t*)&pu, sb8 = *(const bf16x8_t*)&su;
#pragma unroll
      for (int dt = 0; dt < DHH / 32; ++dt) {
        const bf16_t* dr = Dt + (dhf * DHH + dt * 32 + lr) * QP + 16 * ks + 4 * lk;
        const uint2 dlo = *(const uint2*)dr;
        const uint2 dhi = *(const uint2*)(dr + 8);
        uint4 du = make_uint4(dlo.x, dlo.y, dhi.x, dhi.y);
        dv[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(bf16x8_t*)&du, pb, dv[dt], 0, 0, 0);
        const bf16_t* qrp = Qt + (dhf * DHH + dt * 32 + lr) * QP + 16 * ks + 4 * lk;
        const uint2 qlo = *(const uint2*)qrp;
        const uint2 qhi = *(const uint2*)(qrp + 8);
        uint4 qu = make_uint4(qlo.x, qlo.y, qhi.x, qhi.y);
        dk[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(bf16x8_t*)&qu, sb8, dk[dt], 0, 0, 0);
      }
    }
    lds_barrier();
    qc = nq;
    hg = nh;
  }
  if (!kvalid) return;
  const size_t off = (((size_t)bi * n + key) * P.Hkv + g) * DH + dhf * DHH;
  bf16_t* dkp = (bf16_t*)P.dK + off;
  bf16_t* dvp = (bf16_t*)P.dV + off;
  const float sm = P.sm_scale;
#pragma unroll
  for (int dt = 0; dt < DHH / 32; ++dt)
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int d0 = dt * 32 + 8 * v4 + 4 * lk;
      uint32_t w0 = pack_bf16x2(dk[dt][4 * v4 + 0] * sm, dk[dt][4 * v4 + 1] * sm);
      uint32_t w1 = pack_bf16x2(dk[dt][4 * v4 + 2] * sm, dk[dt][4 * v4 + 3] * sm);
      *(uint2*)(dkp + d0) = make_uint2(w0, w1);
      w0 = pack_bf16x2(dv[dt][4 * v4 + 0], dv[dt][4 * v4 + 1]);
      w1 = pack_bf16x2(dv[dt][4 * v4 + 2], dv[dt][4 * v4 + 3]);
      *(uint2*)(dvp + d0) = make_uint2(w0, w1);
    }
}

template <int DH, bool PLAIN>
__global__ void __launch_bounds__(256, 2) bwd_dkv_bf16_kernel(BwdArgs P) {
  const int nkt = (P.n + 63) / 64, per = P.Hkv * P.b;
  const int njobs = nkt * per;
  for (int it = 0;; ++it) {
    const int job = P.queue ? queue_next_job(P.queue) : (it == 0 ? (int)blockIdx.x : njobs);
    if (job >= njobs) break;
    const int r = job % per;  // the first (longest) key tiles first
    bwd_dkv_bf16_job<DH, PLAIN>(P, job / per, r % P.Hkv, r / P.Hkv);
  }
}

static hipError_t launch_attention_backward_bf16(const BwdArgs& P, hipStream_t s) {
  if (P.n > BWD_MAX_SEQ) return hipErrorInvalidValue;
  if (P.K > 32) return hipErrorInvalidValue;
  if (!P.queue) return hipErrorInvalidValue;
  const int NB = cdiv(P.n, P.B), NW = cdiv(NB, 32), ntk = cdiv(P.n, 64);
  BwdArgs Q = P;
  const bool marks = P.mode != SAS_MODE_DENSE && P.K > 0;  // selected blocks to mark
  const bool fullatt = P.mode == SAS_MODE_GATED && P.full && !P.ste;
  Q.tile_rows = nullptr;
  Q.tile_cnt = nullptr;
  Q.tile_off = nullptr;
  if (!marks) {
    Q.selmask = nullptr;
  } else {
    const size_t rows = (size_t)P.b * P.Hkv * P.n;
    bwd_selmask_kernel<<<(unsigned)cdiv(rows * NW, 256), 256, 0, s>>>(P.sel, rows, P.K, NW, P.selmask);
    if (!fullatt) {
      // each tile's list of attending rows: counts, offsets, rows
      if (!P.tile_rows || !P.tile_cnt || !P.tile_off) return hipErrorInvalidValue;
      const long long T = (long long)P.b * P.Hkv * ntk;
      if (T > INT32_MAX || rows * 2 * (P.K + 1) > (size_t)INT32_MAX) return hipErrorInvalidValue;
      const dim3 grid(ntk, P.Hkv, P.b);
      bwd_tile_rows_kernel<<<grid, 256, 0, s>>>(P.selmask, P.n, P.Hkv, P.B, NW, ntk, P.tile_cnt, nullptr, nullptr);
      bwd_rows_scan_kernel<<<1, 1024, 0, s>>>(P.tile_cnt, (int)T, P.tile_off);
      bwd_tile_rows_kernel<<<grid, 256, 0, s>>>(P.selmask, P.n, P.Hkv, P.B, NW, ntk, P.tile_cnt, P.tile_off,
                                                P.tile_rows);
      Q.tile_rows = P.tile_rows;
      Q.tile_cnt = P.tile_cnt;
      Q.tile_off = P.tile_off;
    }
  }
  const int lsb = P.B >= 64 ? 6 : (P.B == 32 ? 5 : 4);
  // no value weights and no straight-through gradient: the plain elementwise step
  const bool plain = !(P.mode == SAS_MODE_GATED && (P.outer || P.ste));
  void (*dq)(BwdArgs);
  if (plain)
    dq = P.dh == 128 ? (lsb == 6 ? bwd_dq_bf16_kernel<128, 6, true> : lsb == 5 ? bwd_dq_bf16_kernel<128, 5, true>
                                                                             : bwd_dq_bf16_kernel<128, 4, true>)
                     : (lsb == 6 ? bwd_dq_bf16_kernel<64, 6, true> : lsb == 5 ? bwd_dq_bf16_kernel<64, 5, true>
                                                                            : bwd_dq_bf16_kernel<64, 4, true>);
  else
    dq = P.dh == 128 ? (lsb == 6 ? bwd_dq_bf16_kernel<128, 6, false> : lsb == 5 ? bwd_dq_bf16_kernel<128, 5, false>
                                                                              : bwd_dq_bf16_kernel<128, 4, false>)
                     : (lsb == 6 ? bwd_dq_bf16_kernel<64, 6, false> : lsb == 5 ? bwd_dq_bf16_kernel<64, 5, false>
                                                                             : bwd_dq_bf16_kernel<64, 4, false>);
  auto dkv = P.dh == 128 ? (plain ? bwd_dkv_bf16_kernel<128, true> : bwd_dkv_bf16_kernel<128, false>)
                         : (plain ? bwd_dkv_bf16_kernel<64, true> : bwd_dkv_bf16_kernel<64, false>);
  const long long jq = (long long)cdiv(P.n, 128) * P.H * P.b, jk = (long long)ntk * P.Hkv * P.b;
  const int rq = resident_workgroups(dq, 256), rk = resident_workgroups(dkv, 256);
  if (rq <= 0 || rk <= 0 || jq > INT32_MAX || jk > INT32_MAX) return hipErrorInvalidValue;
  if (jq > rq || jk > rk) fill_f32_kernel<<<1, 64, 0, s>>>((float*)P.queue, 2, 0.f);  // job counters to zero
  BwdArgs A = Q;
  A.queue = jq > rq ? P.queue : nullptr;
  if (jq > 0) dq<<<(unsigned)std::min<long long>(jq, rq), 256, 0, s>>>(A);
  A.queue = jk > rk ? P.queue + 1 : nullptr;
  if (jk > 0) dkv<<<(unsigned)std::min<long long>(jk, rk), 256, 0, s>>>(A);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t s) {
  if (n == 0) return hipSuccess;
  fill_f32_kernel<<<(unsigned)cdiv(n, 256), 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

hipError_t launch_gather_gate(const int32_t* sel, const float* log_gate, int b, int n, int Hkv, int K, int NB,
                              float* bias, hipStream_t s) {
  const size_t tot = (size_t)b * Hkv * n * K;
  if (tot == 0) return hipSuccess;
  bwd_gather_gate_kernel<<<(unsigned)cdiv(tot, 256), 256, 0, s>>>(sel, log_gate, b, n, Hkv, K, NB, bias);
  return hipGetLastError();
}

// ---- selector ------------------------------------------------------------------
// one wave per row (b, g, t); lane k < K holds slot k (per-slot input)
__global__ void __launch_bounds__(256) selector_ds_kernel(const int32_t* __restrict__ sel,
                                                          const float* __restrict__ log_gate,
                                                          const float* __restrict__ dlog_gate,
                                                          const float* __restrict__ dfull, int act, int rows,
                                                          int n, int Hkv, int K, int B, int NB,
                                                          float* __restrict__ ds, const int32_t* __restrict__ doc) {
  const int row = (int)(((size_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int C = (row % n) / B;
  const int F = doc_first(doc, row / (n * Hkv), NB, row % n, B);  // historical blocks are [F, C)
  const float* lg = log_gate + (size_t)row * NB;
  const float* dfr = dfull ? dfull + (size_t)row * NB : nullptr;
  // every load of the row issued together (slot and its gradient, the first 64 log gates),
  // masked afterwards, so the row costs one memory round trip
  int sk = -1;
  float dk = 0.f;
  const bool has_slot = !dfr && lane < K;
  {
    const size_t so = (size_t)row * K + (has_slot ? lane : 0);
    const int s0 = K > 0 && sel ? sel[so] : -1;
    const float d0 = K > 0 && !dfr && dlog_gate ? dlog_gate[so] : 0.f;
    if (has_slot && s0 >= 0) {
      sk = s0;
      dk = d0;
    }
  }
  const float lg0 = lg[min(lane, NB - 1)];
  float D = 0.f;  // sum of the row's log-gate gradient (softmax)
  if (act == SAS_ACT_SOFTMAX) {
    if (dfr) {
      for (int m = F + lane; m < C; m += 64) D += dfr[m];
      D = wave_sum(D);
    } else {
      D = wave_sum(dk);
    }
  }
  float* out = ds + (size_t)row * NB;
  for (int m0 = 0; m0 < NB; m0 += 64) {
    const int m = m0 + lane;
    float dl = 0.f;
    if (dfr) {
      if (m < C && m >= F) dl = dfr[m];
    } else {
      for (int k = 0; k < K; ++k) {  // every lane shuffles (the sources must be active)
        const int s = __shfl(sk, k, 64);
        const float d = __shfl(dk, k, 64);
        if (s == m) dl += d;
      }
    }
    float v = 0.f;
    if (m < C && m >= F) {
      const float lgm = m0 == 0 ? lg0 : lg[m];
      if (act == SAS_ACT_SOFTMAX) v = dl - expf(lgm) * D;
      else if (act == SAS_ACT_SIGMOID) v = dl * (1.f - expf(lgm));
      else v = dl;
    }
    if (m < NB) out[m] = v;
  }
}

hipError_t launch_selector_ds(const int32_t* sel, const float* log_gate, const float* dlog_gate,
                              const float* dlog_gate_full, int act, int b, int n, int Hkv, int K, int B, float* ds,
                              const int32_t* doc, hipStream_t s) {
  const int rows = b * Hkv * n;
  if (rows <= 0) return hipSuccess;
  if (K > 64) return hipErrorInvalidValue;
  selector_ds_kernel<<<cdiv(rows, 4), 256, 0, s>>>(sel, log_gate, dlog_gate, dlog_gate_full, act, rows, n, Hkv, K, B,
                                                   cdiv(n, B), ds, doc);
  return hipGetLastError();
}

// 64 x 64 output tile per workgroup, 16-deep k steps staged in LDS as fp32
// (the next step's values loaded into registers during this step's FMAs);
// thread (tx, ty) owns rows ty + 16 r and columns tx + 16 c.  Tile loads run
// along whichever of the operand's two indices is contiguous.
template <typename T>
__global__ void __launch_bounds__(256) small_gemm_kernel(SmallGemm P) {
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int j0 = blockIdx.x * 64, i0 = blockIdx.y * 64;
  const int z = blockIdx.z / P.splits, sp = blockIdx.z % P.splits;
  const int kc = (P.K + P.splits - 1) / P.splits;
  const int kb = sp * kc, ke = min(P.K, kb + kc);
  const float* A = P.A + z * P.sAz;
  const T* Bm = (const T*)P.Bm + z * P.sBz;
  float acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.f;
  // the next k step's tile values are loaded into registers while this one is multiplied
  float ra[4], rb[4];
  auto load = [&](int k0) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int idx = tid + e * 256;
      int ii, kk;
      if (P.sAi == 1) {
        ii = idx & 63;
        kk = idx >> 6;
      } else {
        kk = idx & 15;
        ii = idx >> 4;
      }
      const int i = i0 + ii, k = k0 + kk;
      ra[e] = (i < P.M && k < ke) ? A[i * P.sAi + k * P.sAk] : 0.f;
      int jj;
      if (P.sBj == 1) {
        jj = idx & 63;
        kk = idx >> 6;
      } else {
        kk = idx & 15;
        jj = idx >> 4;
      }
      const int j = j0 + jj, k2 = k0 + kk;
      rb[e] = (j < P.N && k2 < ke) ? Act<T>::to_f32(Bm[j * P.sBj + k2 * P.sBk]) : 0.f;
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int idx = tid + e * 256;
      if (P.sAi == 1) As[idx >> 6][idx & 63] = ra[e];
      else As[idx & 15][idx >> 4] = ra[e];
      if (P.sBj == 1) Bs[idx >> 6][idx & 63] = rb[e];
      else Bs[idx & 15][idx >> 4] = rb[e];
    }
  };
  if (kb < ke) load(kb);
  for (int k0 = kb; k0 < ke; k0 += 16) {
    store();
    __syncthreads();
    if (k0 + 16 < ke) load(k0 + 16);
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], bv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) a[r] = As[kk][ty + 16 * r];
#pragma unroll
      for (int c = 0; c < 4; ++c) bv[c] = Bs[kk][tx + 16 * c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(a[r], bv[c], acc[r][c]);
    }
    __syncthreads();
  }
  float* C = P.C + z * P.sCz + sp * P.sCs;
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int i = i0 + ty + 16 * r, j = j0 + tx + 16 * c;
      if (i < P.M && j < P.N) C[i * P.sCi + j] = P.alpha * acc[r][c];
    }
}

hipError_t launch_small_gemm(int dtype, const SmallGemm& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0 || g.Z <= 0) return hipSuccess;
  if (g.splits < 1 || (size_t)g.Z * g.splits > 65535) return hipErrorInvalidValue;
  dim3 grid(cdiv(g.N, 64), cdiv(g.M, 64), g.Z * g.splits);
  if (dtype == SAS_BF16) small_gemm_kernel<bf16_t><<<grid, 256, 0, s>>>(g);
  else small_gemm_kernel<float><<<grid, 256, 0, s>>>(g);
  return hipGetLastError();
}

__global__ void partial_sum_kernel(const float* __restrict__ part, int U, int ZO, int S, size_t E,
                                   float* __restrict__ out) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)ZO * E) return;
  const size_t zo = idx / E, e = idx % E;
  float acc = 0.f;
  for (int u = 0; u < U; ++u)
    for (int q = 0; q < S; ++q) acc += part[(((size_t)u * ZO + zo) * S + q) * E + e];
  out[idx] = acc;
}

hipError_t launch_partial_sum(const float* part, int U, int ZO, int S, size_t E, float* out, hipStream_t s) {
  const size_t tot = (size_t)ZO * E;
  if (tot == 0) return hipSuccess;
  partial_sum_kernel<<<(unsigned)cdiv(tot, 256), 256, 0, s>>>(part, U, ZO, S, E, out);
  return hipGetLastError();
}

hipError_t launch_attention_backward(int dtype, const BwdArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.b <= 0) return hipSuccess;
  if (a.dh != 64 && a.dh != 128) return hipErrorInvalidValue;
  const size_t dthreads = (size_t)a.b * a.n * a.H * (a.dh / 8);
  if (dtype == SAS_BF16)
    bwd_delta_kernel<bf16_t><<<(unsigned)cdiv(dthreads, 256), 256, 0, s>>>((const bf16_t*)a.O, (const bf16_t*)a.dO,
                                                                            a.b, a.n, a.H, a.dh, a.delta);
  else
    bwd_delta_kernel<float><<<(unsigned)cdiv(dthreads, 256), 256, 0, s>>>((const float*)a.O, (const float*)a.dO,
                                                                           a.b, a.n, a.H, a.dh, a.delta);
  const bool need_dlg = a.dlog_gate && a.mode == SAS_MODE_GATED && a.K > 0 && !a.full;
  BwdArgs P = a;
  if (!need_dlg) P.dlg_head = nullptr;
  if (!(a.mode == SAS_MODE_GATED && a.full)) P.dlg_head_full = nullptr;
  if (P.dlg_head) {
    const size_t tot = (size_t)a.b * a.H * a.n * a.K;
    fill_f32_kernel<<<(unsigned)cdiv(tot, 256), 256, 0, s>>>(P.dlg_head, tot, 0.f);
  }
  if (dtype == SAS_BF16) {
    const hipError_t e = launch_attention_backward_bf16(P, s);
    if (e != hipSuccess) return e;
  } else {
    const size_t tq = (size_t)a.b * a.H * a.n, tk = (size_t)a.b * a.Hkv * a.n;
    if (a.dh == 128) {
      bwd_dq_f32_kernel<128><<<(unsigned)cdiv(tq, 64), 64, 0, s>>>(P);
      bwd_dkv_f32_kernel<128><<<(unsigned)cdiv(tk, 64), 64, 0, s>>>(P);
    } else {
      bwd_dq_f32_kernel<64><<<(unsigned)cdiv(tq, 64), 64, 0, s>>>(P);
      bwd_dkv_f32_kernel<64><<<(unsigned)cdiv(tk, 64), 64, 0, s>>>(P);
    }
  }
  if (need_dlg) {
    const size_t tot = (size_t)a.b * a.Hkv * a.n * a.K;
    bwd_dlog_gate_sum_kernel<<<(unsigned)cdiv(tot, 256), 256, 0, s>>>(P.dlg_head, a.sel_bias, a.ste, a.b, a.n,
                                                                        a.H, a.Hkv, a.K, a.dlog_gate);
  }
  if (P.dlg_head_full) {
    const int NB = cdiv(a.n, a.B);
    const size_t tot = (size_t)a.b * a.Hkv * a.n * NB;
    bwd_dlog_gate_full_sum_kernel<<<(unsigned)cdiv(tot, 256), 256, 0, s>>>(
        P.dlg_head_full, a.log_gate, a.ste, a.b, a.n, a.H, a.Hkv, a.B, NB, a.dlog_gate_full, a.doc);
  }
  return hipGetLastError();
}

}  // namespace sas
