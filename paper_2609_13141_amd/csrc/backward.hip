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

#include "common.h"
#include "kernels.h"

namespace sas {

// Delta[b, h, t] = sum_d O[b, t, h, d] dO[b, t, h, d] (fp32)
template <typename T>
__global__ void bwd_delta_kernel(const T* __restrict__ O, const T* __restrict__ dO, int b, int n, int H, int dh,
                                 float* __restrict__ delta) {
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6, lane = threadIdx.x & 63;
  if (wave >= b * n * H) return;
  const int h = wave % H, t = (wave / H) % n, bi = wave / (H * n);
  const size_t off = (((size_t)bi * n + t) * H + h) * dh;
  float acc = 0.f;
  for (int d = lane; d < dh; d += 64) acc = fmaf(Act<T>::to_f32(O[off + d]), Act<T>::to_f32(dO[off + d]), acc);
  acc = wave_sum(acc);
  if (lane == 0) delta[((size_t)bi * H + h) * n + t] = acc;
}

// key range / bias of the sets: returns the bias of block m for query t (natural
// log domain), -inf when m is not attended; `slot` = its selection slot or -1
__device__ __forceinline__ float block_bias(const BwdArgs& P, int bi, int g, int t, int m, int& slot) {
  slot = -1;
  const int beta = t / P.B;
  if (m > beta) return -INFINITY;
  if (m == beta || P.mode == SAS_MODE_DENSE) return 0.f;
  if (P.K <= 0) return -INFINITY;
  const size_t row = (((size_t)bi * P.Hkv + g) * P.n + t) * P.K;
  for (int k = 0; k < P.K; ++k) {
    const int s = P.sel[row + k];
    if (s < 0 || s > m) break;
    if (s == m) {
      slot = k;
      return P.mode == SAS_MODE_GATED ? P.sel_bias[row + k] : 0.f;
    }
  }
  return -INFINITY;
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
  const float* q = (const float*)P.Q + (((size_t)bi * n + t) * P.H + h) * DH;
  const float* dO = (const float*)P.dO + (((size_t)bi * n + t) * P.H + h) * DH;
  const float lse = P.lse[((size_t)bi * P.H + h) * n + t];
  const float delta = P.delta[((size_t)bi * P.H + h) * n + t];
  float qv[DH], dov[DH], dq[DH];
#pragma unroll
  for (int j = 0; j < DH; ++j) {
    qv[j] = q[j];
    dov[j] = dO[j];
    dq[j] = 0.f;
  }
  float* dlg = P.dlg_head ? P.dlg_head + (((size_t)bi * P.H + h) * n + t) * P.K : nullptr;
  const int beta = t / B;
  for (int m = 0; m <= beta; ++m) {
    int slot;
    const float bias = block_bias(P, bi, g, t, m, slot);
    if (bias == -INFINITY) continue;
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
      const float p = expf(z * P.sm_scale + bias - lse);
      const float ds = p * (dp - delta);
      dsum += ds;
#pragma unroll
      for (int j = 0; j < DH; ++j) dq[j] = fmaf(ds * P.sm_scale, k[j], dq[j]);
    }
    if (dlg && slot >= 0) dlg[slot] = dsum;
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
    int slot;
    const float bias = block_bias(P, bi, g, t, m, slot);
    if (bias == -INFINITY) continue;
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
      const float p = expf(z * P.sm_scale + bias - P.lse[hr]);
      const float ds = p * (dp - P.delta[hr]);
#pragma unroll
      for (int j = 0; j < DH; ++j) {
        dk[j] = fmaf(ds * P.sm_scale, q[j], dk[j]);
        dv[j] = fmaf(p, dO[j], dv[j]);
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
__global__ void bwd_dlog_gate_sum_kernel(const float* __restrict__ dlg_head, int b, int n, int H, int Hkv, int K,
                                         float* __restrict__ dlog_gate) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)b * Hkv * n * K) return;
  const int k = (int)(idx % K), t = (int)((idx / K) % n), g = (int)((idx / ((size_t)K * n)) % Hkv);
  const int bi = (int)(idx / ((size_t)K * n * Hkv));
  const int G = H / Hkv;
  float s = 0.f;
  for (int h = g * G; h < (g + 1) * G; ++h) s += dlg_head[(((size_t)bi * H + h) * n + t) * K + k];
  dlog_gate[idx] = s;
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

// Pass 1 (dQ and the per-head block sums of ds): the forward kernel's
// layout -- one workgroup = 4 waves = 128 queries of one (batch, head), each
// lane owning one query of S^T = K Q^T (v_mfma_f32_32x32x16_bf16) -- with
// dP^T = V dO^T computed the same way, dS^T = P^T (dP^T - Delta) formed in
// registers and fed back as the B operand of dQ^T += K^T dS^T (K staged
// transposed in LDS, read in the accumulator's key permutation).  Tiles no
// query of the workgroup attends are skipped.
template <int DH, bool SINGLE>
__global__ void __launch_bounds__(256) bwd_dq_bf16_kernel(BwdArgs P) {
  constexpr int KP = DH + 8;
  constexpr int TP = 64 + 4;
  constexpr int KPG = DH / 32;
  __shared__ __align__(16) bf16_t Ks[64 * KP];
  __shared__ __align__(16) bf16_t Vs[64 * KP];
  __shared__ __align__(16) bf16_t Kt[DH * TP];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int qtile = gridDim.x - 1 - blockIdx.x;
  const int h = blockIdx.y, bi = blockIdx.z;
  const int G = P.H / P.Hkv, g = h / G;
  const int n = P.n, B = P.B, Kn = P.K;
  const int t = qtile * 128 + wave * 32 + lr;
  const bool qvalid = t < n;
  const int beta = qvalid ? t / B : -1;
  const int bshift = 31 - __clz(B < 64 ? B : 64);

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
  float* dlg = (P.dlg_head && qvalid) ? P.dlg_head + hrow * Kn : nullptr;

  const int32_t* selp = nullptr;
  const float* biasp = nullptr;
  int cur = 0, next_sel = 0x7fffffff;
  if (P.mode != SAS_MODE_DENSE && qvalid && Kn > 0) {
    const size_t row = (((size_t)bi * P.Hkv + g) * n + t) * Kn;
    selp = P.sel + row;
    biasp = P.sel_bias + row;
    const int s0 = selp[0];
    next_sel = s0 >= 0 ? s0 : 0x7fffffff;
  }
  const bool gated = P.mode == SAS_MODE_GATED;
  const bool dense = P.mode == SAS_MODE_DENSE;

  floatx16_t dq[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) dq[dt][v] = 0.f;
  const float qk_scale = P.sm_scale * BLOG2E;

  const int t_hi = min(n, qtile * 128 + 128) - 1;
  const int last_tile = t_hi / 64;
  const bf16_t* Kg = (const bf16_t*)P.Kt + (size_t)g * DH;
  const bf16_t* Vg = (const bf16_t*)P.V + (size_t)g * DH;
  const size_t kstride = (size_t)P.Hkv * DH;
  const size_t kbase = (size_t)bi * n;

  for (int kt = 0; kt <= last_tile; ++kt) {
    const int k0 = kt * 64;
    constexpr int NSUB = SINGLE ? 1 : 4;
    float bsub[NSUB];
    int slot[NSUB];
    bool need = false;
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) {
      bsub[sb] = -INFINITY;
      slot[sb] = -1;
      const int kstart = k0 + (sb << bshift);
      if (!qvalid || kstart > t || (!SINGLE && (sb << bshift) >= 64)) continue;
      const int m = kstart / B;
      if (m == beta || dense) {
        bsub[sb] = 0.f;
      } else if (m == next_sel) {
        bsub[sb] = gated ? biasp[cur] * BLOG2E : 0.f;
        slot[sb] = cur;
        if (kstart + (1 << bshift) >= (m + 1) * B) {
          ++cur;
          const int s1 = cur < Kn ? selp[cur] : -1;
          next_sel = s1 >= 0 ? s1 : 0x7fffffff;
        }
      }
      need |= bsub[sb] != -INFINITY;
    }
    if (!__syncthreads_or(need)) continue;

    // stage K and V row-major and K transposed
    {
#pragma unroll
      for (int i = 0; i < (64 * DH / 8) / 256; ++i) {
        const int c = tid + i * 256;
        const int kr = c / (DH / 8), c8 = c % (DH / 8);
        const int key = k0 + kr;
        const size_t go = (kbase + key) * kstride + c8 * 8;
        uint4 ku = key < n ? *(const uint4*)(Kg + go) : make_uint4(0, 0, 0, 0);
        uint4 vu = key < n ? *(const uint4*)(Vg + go) : make_uint4(0, 0, 0, 0);
        *(uint4*)(Ks + kr * KP + c8 * 8) = ku;
        *(uint4*)(Vs + kr * KP + c8 * 8) = vu;
      }
      const int c8 = tid % (DH / 8), kg = tid / (DH / 8);
      uint32_t w[KPG][4];
#pragma unroll
      for (int q = 0; q < KPG; ++q) {
        const int key = k0 + kg * KPG + q;
        uint4 ku = key < n ? *(const uint4*)(Kg + (kbase + key) * kstride + c8 * 8) : make_uint4(0, 0, 0, 0);
        w[q][0] = ku.x; w[q][1] = ku.y; w[q][2] = ku.z; w[q][3] = ku.w;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int sh = (e & 1) * 16;
        bf16_t* dst = Kt + (c8 * 8 + e) * TP + kg * KPG;
        if constexpr (KPG == 4) {
          uint2 pk;
          pk.x = ((w[0][e >> 1] >> sh) & 0xffffu) | (((w[1][e >> 1] >> sh) & 0xffffu) << 16);
          pk.y = ((w[2][e >> 1] >> sh) & 0xffffu) | (((w[3][e >> 1] >> sh) & 0xffffu) << 16);
          *(uint2*)dst = pk;
        } else {
          *(uint32_t*)dst = ((w[0][e >> 1] >> sh) & 0xffffu) | (((w[1][e >> 1] >> sh) & 0xffffu) << 16);
        }
      }
    }
    __syncthreads();

    floatx16_t sc[2], dp[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        sc[st][v] = 0.f;
        dp[st][v] = 0.f;
      }
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) {
        const bf16x8_t a = *(const bf16x8_t*)(Ks + (st * 32 + lr) * KP + ks * 16 + lk * 8);
        sc[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qb[ks], sc[st], 0, 0, 0);
        const bf16x8_t av = *(const bf16x8_t*)(Vs + (st * 32 + lr) * KP + ks * 16 + lk * 8);
        dp[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, dob[ks], dp[st], 0, 0, 0);
      }
    }
    const int lim = t - k0;
    float dsum[NSUB];
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) dsum[sb] = 0.f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kl = st * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
        int sb = 0;
        float bb;
        if constexpr (SINGLE) {
          bb = bsub[0];
        } else {
          sb = kl >> bshift;
          bb = sb == 0 ? bsub[0] : sb == 1 ? bsub[1] : sb == 2 ? bsub[2] : bsub[3];
        }
        float ds = 0.f;
        if (kl <= lim && bb != -INFINITY) {
          const float p = __builtin_amdgcn_exp2f(sc[st][v] * qk_scale + bb - lse2);
          ds = p * (dp[st][v] - delta);
        }
        sc[st][v] = ds;
        if constexpr (SINGLE) dsum[0] += ds;
        else {
          if (sb == 0) dsum[0] += ds;
          else if (sb == 1) dsum[1] += ds;
          else if (sb == 2) dsum[2] += ds;
          else dsum[3] += ds;
        }
      }
    if (dlg) {
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb) {
        const float tot = dsum[sb] + __shfl_xor(dsum[sb], 32, 64);
        if (slot[sb] >= 0 && lk == 0) dlg[slot[sb]] += tot;
      }
    }
    // dQ^T += K^T dS^T, 16 keys per step in the accumulator's key permutation
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      bf16x8_t pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf16_t hb = f32_to_bf16(sc[ks >> 1][8 * (ks & 1) + e]);
        pb[e] = *(__bf16*)&hb;
      }
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

  if (!qvalid) return;
  bf16_t* op = (bf16_t*)P.dQ + (((size_t)bi * n + t) * P.H + h) * DH;
  const float sm = P.sm_scale;
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int d0 = dt * 32 + 8 * v4 + 4 * lk;
      const uint32_t w0 = (uint32_t)f32_to_bf16(dq[dt][4 * v4 + 0] * sm) |
                          ((uint32_t)f32_to_bf16(dq[dt][4 * v4 + 1] * sm) << 16);
      const uint32_t w1 = (uint32_t)f32_to_bf16(dq[dt][4 * v4 + 2] * sm) |
                          ((uint32_t)f32_to_bf16(dq[dt][4 * v4 + 3] * sm) << 16);
      *(uint2*)(op + d0) = make_uint2(w0, w1);
    }
}

// which 32-query chunks select which blocks: mask[b, g, t / 32, m] = 1
__global__ void bwd_chunk_mask_kernel(const int32_t* __restrict__ sel, int b, int n, int Hkv, int K, int NB,
                                      uint8_t* __restrict__ mask) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)b * Hkv * n * K) return;
  const int m = sel[idx];
  if (m < 0 || m >= NB) return;
  const size_t bgt = idx / K;  // (b, g, t)
  const int t = (int)(bgt % n);
  const size_t bg = bgt / n;
  const int nqc = (n + 31) / 32;
  mask[(bg * nqc + t / 32) * NB + m] = 1;
}

// Pass 2 (dK, dV): one workgroup of 2 waves per 64 keys of one (batch, KV
// group); each wave owns 32 keys, held in registers as the B operands of
// S = Q K^T and dP = dO V^T over 32-query chunks (lane = key, 16 query rows).
// For every chunk that attends the tile and every head of the group, the
// chunk's Q and dO are staged in LDS both row-major (A of S and dP) and
// transposed (A of dK^T += Q^T dS and dV^T += dO^T P, read in the
// accumulator's query permutation); P and dS stay in registers.
template <int DH>
__global__ void __launch_bounds__(128) bwd_dkv_bf16_kernel(BwdArgs P) {
  constexpr int KP = DH + 8;
  constexpr int QP = 32 + 4;
  constexpr int NTH = 128;
  __shared__ __align__(16) bf16_t Qs[32 * KP];
  __shared__ __align__(16) bf16_t Ds[32 * KP];
  __shared__ __align__(16) bf16_t Qt[DH * QP];
  __shared__ __align__(16) bf16_t Dt[DH * QP];
  __shared__ float lse_s[32], delta_s[32];
  __shared__ float bias_s[32][4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int ktile = blockIdx.x, g = blockIdx.y, bi = blockIdx.z;
  const int n = P.n, B = P.B, H = P.H, G = H / P.Hkv;
  const int k0 = ktile * 64;
  const int key = k0 + wave * 32 + lr;
  const bool kvalid = key < n;
  const int bshift = 31 - __clz(B < 64 ? B : 64);
  const int nsb = 64 >> bshift;  // SAS blocks (or parts of one) in the tile
  const int m_lo = k0 / B, m_hi = min(n - 1, k0 + 63) / B;
  const int NB = (n + B - 1) / B;
  const int nqc = (n + 31) / 32;
  const uint8_t* cmask = P.chunk_mask ? P.chunk_mask + ((size_t)bi * P.Hkv + g) * nqc * NB : nullptr;

  bf16x8_t kb[DH / 16], vb[DH / 16];
  {
    const size_t off = (((size_t)bi * n + (kvalid ? key : 0)) * P.Hkv + g) * DH;
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) {
      uint4 u = kvalid ? *(const uint4*)((const bf16_t*)P.Kt + off + ks * 16 + lk * 8) : make_uint4(0, 0, 0, 0);
      kb[ks] = *(bf16x8_t*)&u;
      uint4 w = kvalid ? *(const uint4*)((const bf16_t*)P.V + off + ks * 16 + lk * 8) : make_uint4(0, 0, 0, 0);
      vb[ks] = *(bf16x8_t*)&w;
    }
  }
  floatx16_t dk[DH / 32], dv[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      dk[dt][v] = 0.f;
      dv[dt][v] = 0.f;
    }
  const float qk_scale = P.sm_scale * BLOG2E;
  const bool dense = P.mode == SAS_MODE_DENSE;

  for (int qc = k0 / 32; qc < nqc; ++qc) {
    const int q0 = qc * 32;
    // does any query of the chunk attend a key of the tile?  (the chunk reaches
    // into the tile's current blocks, or selects one of them; thread j checks
    // block m_lo + j, at most 64 / B + 1 of them)
    bool any = dense || (q0 / B <= m_hi);
    if (!any && cmask && tid <= m_hi - m_lo) any = cmask[(size_t)qc * NB + m_lo + tid] != 0;
    if (!__syncthreads_or(any)) continue;
    for (int hg = 0; hg < G; ++hg) {
      const int h = g * G + hg;
      // stage the chunk: Q, dO row-major and transposed; LSE, Delta; block biases
      for (int c = tid; c < 32 * (DH / 8); c += NTH) {
        const int qr = c / (DH / 8), c8 = c % (DH / 8);
        const int t = q0 + qr;
        const size_t off = (((size_t)bi * n + t) * H + h) * DH + c8 * 8;
        uint4 qu = t < n ? *(const uint4*)((const bf16_t*)P.Q + off) : make_uint4(0, 0, 0, 0);
        uint4 du = t < n ? *(const uint4*)((const bf16_t*)P.dO + off) : make_uint4(0, 0, 0, 0);
        *(uint4*)(Qs + qr * KP + c8 * 8) = qu;
        *(uint4*)(Ds + qr * KP + c8 * 8) = du;
      }
      if (tid < (DH / 8) * 8) {
        const int c8 = tid % (DH / 8), qg = tid / (DH / 8);  // 8 query groups of 4
        uint32_t wq[4][4], wd[4][4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int t = q0 + qg * 4 + q;
          const size_t off = (((size_t)bi * n + t) * H + h) * DH + c8 * 8;
          uint4 qu = t < n ? *(const uint4*)((const bf16_t*)P.Q + off) : make_uint4(0, 0, 0, 0);
          uint4 du = t < n ? *(const uint4*)((const bf16_t*)P.dO + off) : make_uint4(0, 0, 0, 0);
          wq[q][0] = qu.x; wq[q][1] = qu.y; wq[q][2] = qu.z; wq[q][3] = qu.w;
          wd[q][0] = du.x; wd[q][1] = du.y; wd[q][2] = du.z; wd[q][3] = du.w;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int sh = (e & 1) * 16;
          uint2 pq, pd;
          pq.x = ((wq[0][e >> 1] >> sh) & 0xffffu) | (((wq[1][e >> 1] >> sh) & 0xffffu) << 16);
          pq.y = ((wq[2][e >> 1] >> sh) & 0xffffu) | (((wq[3][e >> 1] >> sh) & 0xffffu) << 16);
          pd.x = ((wd[0][e >> 1] >> sh) & 0xffffu) | (((wd[1][e >> 1] >> sh) & 0xffffu) << 16);
          pd.y = ((wd[2][e >> 1] >> sh) & 0xffffu) | (((wd[3][e >> 1] >> sh) & 0xffffu) << 16);
          *(uint2*)(Qt + (c8 * 8 + e) * QP + qg * 4) = pq;
          *(uint2*)(Dt + (c8 * 8 + e) * QP + qg * 4) = pd;
        }
      }
      if (tid < 32) {
        const int t = q0 + tid;
        const size_t hr = ((size_t)bi * H + h) * n + (t < n ? t : 0);
        lse_s[tid] = t < n ? P.lse[hr] * BLOG2E : 0.f;
        delta_s[tid] = t < n ? P.delta[hr] : 0.f;
      }
      for (int j = tid; j < 32 * 4; j += NTH) {
        const int qr = j & 31, sb = j >> 5;
        const int t = q0 + qr;
        float bb = -INFINITY;
        if (t < n && sb < nsb) {
          const int kstart = k0 + (sb << bshift);
          int slot;
          if (kstart <= t) bb = block_bias(P, bi, g, t, kstart / B, slot);
          if (bb != -INFINITY) bb *= BLOG2E;
        }
        bias_s[qr][sb] = bb;
      }
      __syncthreads();

      floatx16_t sc, dp;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        sc[v] = 0.f;
        dp[v] = 0.f;
      }
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) {
        const bf16x8_t aq = *(const bf16x8_t*)(Qs + lr * KP + ks * 16 + lk * 8);
        sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq, kb[ks], sc, 0, 0, 0);
        const bf16x8_t ad = *(const bf16x8_t*)(Ds + lr * KP + ks * 16 + lk * 8);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ad, vb[ks], dp, 0, 0, 0);
      }
      // lane: key column `key`; rows = queries q0 + 8 (v / 4) + 4 lk + v % 4
      const int sbk = (wave * 32 + lr) >> bshift;
      floatx16_t pp;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int qr = 8 * (v >> 2) + 4 * lk + (v & 3);
        const int t = q0 + qr;
        const float bb = bias_s[qr][sbk];
        float p = 0.f, ds = 0.f;
        if (kvalid && key <= t && bb != -INFINITY) {
          p = __builtin_amdgcn_exp2f(sc[v] * qk_scale + bb - lse_s[qr]);
          ds = p * (dp[v] - delta_s[qr]);
        }
        pp[v] = p;
        sc[v] = ds;
      }
      // dV^T += dO^T P and dK^T += Q^T dS, 16 queries per step in the accumulator's query permutation
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        bf16x8_t pb, sb8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          bf16_t hp = f32_to_bf16(pp[8 * ks + e]);
          bf16_t hs = f32_to_bf16(sc[8 * ks + e]);
          pb[e] = *(__bf16*)&hp;
          sb8[e] = *(__bf16*)&hs;
        }
#pragma unroll
        for (int dt = 0; dt < DH / 32; ++dt) {
          const bf16_t* dr = Dt + (dt * 32 + lr) * QP + 16 * ks + 4 * lk;
          const uint2 dlo = *(const uint2*)dr;
          const uint2 dhi = *(const uint2*)(dr + 8);
          uint4 du = make_uint4(dlo.x, dlo.y, dhi.x, dhi.y);
          dv[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(bf16x8_t*)&du, pb, dv[dt], 0, 0, 0);
          const bf16_t* qrp = Qt + (dt * 32 + lr) * QP + 16 * ks + 4 * lk;
          const uint2 qlo = *(const uint2*)qrp;
          const uint2 qhi = *(const uint2*)(qrp + 8);
          uint4 qu = make_uint4(qlo.x, qlo.y, qhi.x, qhi.y);
          dk[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(bf16x8_t*)&qu, sb8, dk[dt], 0, 0, 0);
        }
      }
      __syncthreads();
    }
  }
  if (!kvalid) return;
  const size_t off = (((size_t)bi * n + key) * P.Hkv + g) * DH;
  bf16_t* dkp = (bf16_t*)P.dK + off;
  bf16_t* dvp = (bf16_t*)P.dV + off;
  const float sm = P.sm_scale;
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int d0 = dt * 32 + 8 * v4 + 4 * lk;
      uint32_t w0 = (uint32_t)f32_to_bf16(dk[dt][4 * v4 + 0] * sm) | ((uint32_t)f32_to_bf16(dk[dt][4 * v4 + 1] * sm) << 16);
      uint32_t w1 = (uint32_t)f32_to_bf16(dk[dt][4 * v4 + 2] * sm) | ((uint32_t)f32_to_bf16(dk[dt][4 * v4 + 3] * sm) << 16);
      *(uint2*)(dkp + d0) = make_uint2(w0, w1);
      w0 = (uint32_t)f32_to_bf16(dv[dt][4 * v4 + 0]) | ((uint32_t)f32_to_bf16(dv[dt][4 * v4 + 1]) << 16);
      w1 = (uint32_t)f32_to_bf16(dv[dt][4 * v4 + 2]) | ((uint32_t)f32_to_bf16(dv[dt][4 * v4 + 3]) << 16);
      *(uint2*)(dvp + d0) = make_uint2(w0, w1);
    }
}

static hipError_t launch_attention_backward_bf16(const BwdArgs& P, hipStream_t s) {
  const int NB = cdiv(P.n, P.B), nqc = cdiv(P.n, 32);
  BwdArgs Q = P;
  if (P.mode == SAS_MODE_DENSE || P.K <= 0) Q.chunk_mask = nullptr;  // no selected blocks to mark
  if (Q.chunk_mask) {
    const size_t bytes = (size_t)P.b * P.Hkv * nqc * NB;
    fill_f32_kernel<<<(unsigned)cdiv(cdiv(bytes, 4), 256), 256, 0, s>>>((float*)P.chunk_mask, cdiv(bytes, 4), 0.f);
    const size_t tot = (size_t)P.b * P.Hkv * P.n * P.K;
    bwd_chunk_mask_kernel<<<(unsigned)cdiv(tot, 256), 256, 0, s>>>(P.sel, P.b, P.n, P.Hkv, P.K, NB, P.chunk_mask);
  }
  dim3 g1(cdiv(P.n, 128), P.H, P.b);
  const bool single = P.B >= 64;
  if (P.dh == 128) {
    if (single) bwd_dq_bf16_kernel<128, true><<<g1, 256, 0, s>>>(P);
    else bwd_dq_bf16_kernel<128, false><<<g1, 256, 0, s>>>(P);
  } else {
    if (single) bwd_dq_bf16_kernel<64, true><<<g1, 256, 0, s>>>(P);
    else bwd_dq_bf16_kernel<64, false><<<g1, 256, 0, s>>>(P);
  }
  dim3 g2(cdiv(P.n, 64), P.Hkv, P.b);
  if (P.dh == 128) bwd_dkv_bf16_kernel<128><<<g2, 128, 0, s>>>(Q);
  else bwd_dkv_bf16_kernel<64><<<g2, 128, 0, s>>>(Q);
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
// one wave per row (b, g, t); lane k < K holds slot k
__global__ void __launch_bounds__(256) selector_ds_kernel(const int32_t* __restrict__ sel,
                                                          const float* __restrict__ log_gate,
                                                          const float* __restrict__ dlog_gate, int rows, int n,
                                                          int K, int B, int NB, float* __restrict__ ds) {
  const int row = (int)(((size_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int C = (row % n) / B;
  const int sk = lane < K ? sel[(size_t)row * K + lane] : -1;
  const float dk = sk >= 0 ? dlog_gate[(size_t)row * K + lane] : 0.f;
  const float D = wave_sum(dk);
  const float* lg = log_gate + (size_t)row * NB;
  float* out = ds + (size_t)row * NB;
  for (int m0 = 0; m0 < NB; m0 += 64) {
    const int m = m0 + lane;
    float v = 0.f;
    if (m < C) v = -expf(lg[m]) * D;
    for (int k = 0; k < K; ++k) {
      const int s = __shfl(sk, k, 64);
      const float d = __shfl(dk, k, 64);
      if (s == m && m < C) v += d;
    }
    if (m < NB) out[m] = v;
  }
}

hipError_t launch_selector_ds(const int32_t* sel, const float* log_gate, const float* dlog_gate, int b, int n,
                              int Hkv, int K, int B, float* ds, hipStream_t s) {
  const int rows = b * Hkv * n;
  if (rows <= 0) return hipSuccess;
  if (K > 64) return hipErrorInvalidValue;
  selector_ds_kernel<<<cdiv(rows, 4), 256, 0, s>>>(sel, log_gate, dlog_gate, rows, n, K, B, cdiv(n, B), ds);
  return hipGetLastError();
}

// 64 x 64 output tile per workgroup, 16-deep k steps staged in LDS as fp32;
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
  for (int k0 = kb; k0 < ke; k0 += 16) {
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
      As[kk][ii] = (i < P.M && k < ke) ? A[i * P.sAi + k * P.sAk] : 0.f;
      int jj;
      if (P.sBj == 1) {
        jj = idx & 63;
        kk = idx >> 6;
      } else {
        kk = idx & 15;
        jj = idx >> 4;
      }
      const int j = j0 + jj, k2 = k0 + kk;
      Bs[kk][jj] = (j < P.N && k2 < ke) ? Act<T>::to_f32(Bm[j * P.sBj + k2 * P.sBk]) : 0.f;
    }
    __syncthreads();
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
  const int waves = a.b * a.n * a.H;
  if (dtype == SAS_BF16)
    bwd_delta_kernel<bf16_t><<<cdiv(waves, 4), 256, 0, s>>>((const bf16_t*)a.O, (const bf16_t*)a.dO, a.b, a.n, a.H,
                                                              a.dh, a.delta);
  else
    bwd_delta_kernel<float><<<cdiv(waves, 4), 256, 0, s>>>((const float*)a.O, (const float*)a.dO, a.b, a.n, a.H,
                                                             a.dh, a.delta);
  const bool need_dlg = a.dlog_gate && a.mode == SAS_MODE_GATED && a.K > 0;
  BwdArgs P = a;
  if (!need_dlg) P.dlg_head = nullptr;
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
    bwd_dlog_gate_sum_kernel<<<(unsigned)cdiv(tot, 256), 256, 0, s>>>(P.dlg_head, a.b, a.n, a.H, a.Hkv, a.K,
                                                                        a.dlog_gate);
  }
  return hipGetLastError();
}

}  // namespace sas
