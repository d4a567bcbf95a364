// Selection-analysis statistics (Sec. 6.1): attention mass coverage of the
// attended set (Eq. mass_coverage, raw and value-norm weights), the
// full-attention reference sets (per-head Top-K blocks by attention mass,
// merged per KV group by majority vote) and the cross-layer overlap recall
// (Eq. overlap_recall) on OR-accumulated block bitmasks.
//
// The coverage pass is a dense causal pass in the forward attention's layout
// (S^T = K Q^T on v_mfma_f32_32x32x16_bf16, lane = query, partner lane l^32)
// without the PV product: per query it keeps two running maxima (raw and
// value-aware logits, log2 domain) and four sums (all keys / attended keys,
// each weighting), and the log-sum-exp of every historical block's raw
// logits for the reference Top-K.
#include <float.h>

#include <stdint.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace sas {

constexpr float SLOG2E = 1.4426950408889634f;

// lvn[b, t, g] = log2 ||v[b, t, g, :]||_2 (fp32 sum of squares; -inf for a zero row)
template <typename T, int DH>
__global__ void vnorm_kernel(const T* __restrict__ V, size_t rows, float* __restrict__ lvn) {
  const size_t r = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows) return;
  const T* v = V + r * DH;
  float ss = 0.f;
  for (int j = 0; j < DH; j += 8) {
    Vec8<T> x;
    x.load(v + j);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(x.get(e), x.get(e), ss);
  }
  lvn[r] = 0.5f * log2f(ss);
}

// log2(2^a + 2^b), either may be -inf
__device__ __forceinline__ float lse2(float a, float b) {
  const float m = fmaxf(a, b);
  if (m == -INFINITY) return -INFINITY;
  return m + log2f(exp2f(a - m) + exp2f(b - m));
}

template <int DH, int LSB>
__device__ __forceinline__ void stats_bf16_job(const StatsArgs& P, const int qtile, const int h, const int bi) {
  constexpr int KP = DH + 8;
  constexpr int KPG = DH / 32;
  constexpr int C8 = DH / 8;
  constexpr int NSUB = 64 >> LSB;
  constexpr int KMAX = 32;
  __shared__ __align__(16) bf16_t Ks[64 * KP];
  __shared__ float lv_s[64];
  __shared__ int sel_s[128 * KMAX];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int G = P.H / P.Hkv, g = h / G;
  const int n = P.n, B = P.B;
  const int qrow = wave * 32 + lr;
  const int t = qtile * 128 + qrow;
  const bool qvalid = t < n;
  const int beta = qvalid ? t / B : -1;
  const bool dense = P.mode == SAS_MODE_DENSE;
  const int Kn = dense ? 0 : P.K;
  const int NB = (n + B - 1) / B;
  const int t_hi = min(n, qtile * 128 + 128) - 1;
  const int last_tile = t_hi / 64;
  const size_t grow = ((size_t)bi * P.Hkv + g) * n;
  const size_t hrow = ((size_t)bi * P.H + h) * n + (qvalid ? t : 0);
  const int fb = qvalid ? doc_first(P.doc, bi, NB, t, B) : 0;  // the query's document starts at block fb
  const int first_tile = doc_first(P.doc, bi, NB, qtile * 128, B) * B / 64;

  bf16x8_t qb[DH / 16];
  {
    const bf16_t* qp = (const bf16_t*)P.Q + (((size_t)bi * n + (qvalid ? t : 0)) * P.H + h) * DH;
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) {
      uint4 u = qvalid ? *(const uint4*)(qp + ks * 16 + lk * 8) : make_uint4(0, 0, 0, 0);
      qb[ks] = *(bf16x8_t*)&u;
    }
  }
  if (Kn > 0 && qvalid)
    for (int k = lk; k < Kn; k += 2) sel_s[qrow * KMAX + k] = P.sel[(grow + t) * Kn + k];
  __syncthreads();

  const float qk_scale = P.sm_scale * SLOG2E;
  const bf16_t* Kg = (const bf16_t*)P.Kt + (size_t)g * DH;
  const size_t kstride = (size_t)P.Hkv * DH;
  const size_t kbase = (size_t)bi * n;
  const int c8 = tid % C8, kg = tid / C8;
  uint4 rk[KPG];
  float rl = 0.f;
  auto prefetch = [&](int kt) {
#pragma unroll
    for (int q = 0; q < KPG; ++q) {
      const int key = kt * 64 + kg * KPG + q;
      rk[q] = key < n ? *(const uint4*)(Kg + (kbase + key) * kstride + c8 * 8) : make_uint4(0, 0, 0, 0);
    }
    if (tid < 64) {
      const int key = kt * 64 + tid;
      rl = key < n ? P.lvn[(kbase + key) * P.Hkv + g] : -INFINITY;
    }
  };

  float m_raw = -INFINITY, m_val = -INFINITY;         // running maxima (log2 domain)
  float l_all = 0.f, l_S = 0.f, l_vall = 0.f, l_vS = 0.f;
  float blk_acc = -INFINITY;                           // log2 mass of a block wider than a tile so far
  int cur = 0, next_sel = 0x7fffffff;
  if (Kn > 0 && qvalid) {
    const int s0 = sel_s[qrow * KMAX];
    next_sel = s0 >= 0 ? s0 : 0x7fffffff;
  }
  prefetch(first_tile);
  for (int kt = first_tile; kt <= last_tile; ++kt) {
#pragma unroll
    for (int q = 0; q < KPG; ++q) *(uint4*)(Ks + (kg * KPG + q) * KP + c8 * 8) = rk[q];
    if (tid < 64) lv_s[tid] = rl;
    lds_barrier();
    const int k0 = kt * 64;
    // membership of the attended set per sub-block (causal context only)
    bool inS[NSUB], ctx[NSUB];
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) {
      const int kstart = k0 + (sb << LSB);
      ctx[sb] = qvalid && kstart <= t && kstart / B >= fb;
      inS[sb] = false;
      if (!ctx[sb]) continue;
      const int m = kstart / B;
      if (m == beta || dense) {
        inS[sb] = true;
      } else if (m == next_sel) {
        inS[sb] = true;
        if (kstart + (1 << LSB) >= (m + 1) * B) {
          ++cur;
          const int s1 = cur < Kn ? sel_s[qrow * KMAX + cur] : -1;
          next_sel = s1 >= 0 ? s1 : 0x7fffffff;
        }
      }
    }
    if (kt + 1 <= last_tile) prefetch(kt + 1);

    floatx16_t s[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int v = 0; v < 16; ++v) s[st][v] = 0.f;
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) {
        const bf16x8_t a = *(const bf16x8_t*)(Ks + (st * 32 + lr) * KP + ks * 16 + lk * 8);
        s[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qb[ks], s[st], 0, 0, 0);
      }
    }
    const bool diag = k0 + 63 > qtile * 128;
    float xv[2][16];
    float mx = -INFINITY, mxv = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int klc = st * 32 + 8 * (v >> 2);
        const int kl = klc + 4 * lk + (v & 3);
        float x = s[st][v] * qk_scale;
        if (!ctx[klc >> LSB] || (diag && k0 + kl > t)) x = -INFINITY;
        const float y = x + lv_s[kl];
        s[st][v] = x;
        xv[st][v] = y;
        mx = fmaxf(mx, x);
        mxv = fmaxf(mxv, y);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    mxv = fmaxf(mxv, __shfl_xor(mxv, 32, 64));
    const float mn = fmaxf(m_raw, mx), mnv = fmaxf(m_val, mxv);
    const float mu = mn == -INFINITY ? 0.f : mn, muv = mnv == -INFINITY ? 0.f : mnv;
    const float a = exp2f(m_raw - mu), av = exp2f(m_val - muv);
    float sa = 0.f, sS = 0.f, sva = 0.f, svS = 0.f, bsum[NSUB];
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) bsum[sb] = 0.f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int sb = (st * 32 + 8 * (v >> 2)) >> LSB;
        const float p = exp2f(s[st][v] - mu);
        const float pv = exp2f(xv[st][v] - muv);
        sa += p;
        sva += pv;
        bsum[sb] += p;
        if (inS[sb]) {
          sS += p;
          svS += pv;
        }
      }
    sa += __shfl_xor(sa, 32, 64);
    sS += __shfl_xor(sS, 32, 64);
    sva += __shfl_xor(sva, 32, 64);
    svS += __shfl_xor(svS, 32, 64);
    l_all = l_all * a + sa;
    l_S = l_S * a + sS;
    l_vall = l_vall * av + sva;
    l_vS = l_vS * av + svS;
    m_raw = mn;
    m_val = mnv;
    // block masses of the historical blocks (reference Top-K)
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) {
      const float tot = bsum[sb] + __shfl_xor(bsum[sb], 32, 64);
      const int kstart = k0 + (sb << LSB), m = kstart / B;
      if (P.blk_lse && lk == 0 && ctx[sb] && m < beta) {
        blk_acc = lse2(blk_acc, tot > 0.f ? mu + log2f(tot) : -INFINITY);
        if (kstart + (1 << LSB) >= (m + 1) * B) {
          P.blk_lse[hrow * NB + m] = blk_acc;
          blk_acc = -INFINITY;
        }
      }
    }
    lds_barrier();
  }
  if (!qvalid || lk != 0) return;
  if (P.cov) P.cov[hrow] = l_S / l_all;
  if (P.cov_v) P.cov_v[hrow] = l_vS / l_vall;
}

// One job (query tile, head, batch entry) per workgroup (grid = job count, no
// queue) or the work queue; the heavy (late) query tiles first.
template <int DH, int LSB>
__global__ void __launch_bounds__(256, 2) stats_bf16_kernel(StatsArgs P) {
  const int nqt = (P.n + 127) / 128, per = P.H * P.b;
  const int njobs = nqt * per;
  for (int it = 0;; ++it) {
    const int job = P.queue ? queue_next_job(P.queue) : (it == 0 ? (int)blockIdx.x : njobs);
    if (job >= njobs) break;
    const int r = job % per;
    stats_bf16_job<DH, LSB>(P, nqt - 1 - job / per, r % P.H, r / P.H);
  }
}

// fp32: one thread per (batch, head, query), sums in fp32 against running maxima
template <int DH>
__global__ void stats_f32_kernel(StatsArgs P) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = P.n;
  if (idx >= (size_t)P.b * P.H * n) return;
  const int t = (int)(idx % n), h = (int)((idx / n) % P.H), bi = (int)(idx / ((size_t)n * P.H));
  const int G = P.H / P.Hkv, g = h / G, B = P.B, beta = t / B;
  const int NB = (n + B - 1) / B;
  const float* q = (const float*)P.Q + (((size_t)bi * n + t) * P.H + h) * DH;
  const size_t row = ((size_t)bi * P.Hkv + g) * n + t;
  const size_t hrow = ((size_t)bi * P.H + h) * n + t;
  float qv[DH];
#pragma unroll
  for (int j = 0; j < DH; ++j) qv[j] = q[j];
  float m_raw = -INFINITY, m_val = -INFINITY, l_all = 0.f, l_S = 0.f, l_vall = 0.f, l_vS = 0.f;
  int cur = 0;
  for (int m = doc_first(P.doc, bi, NB, t, B); m <= beta; ++m) {
    bool in = m == beta || P.mode == SAS_MODE_DENSE;
    if (!in && P.K > 0) {
      while (cur < P.K && P.sel[row * P.K + cur] >= 0 && P.sel[row * P.K + cur] < m) ++cur;
      in = cur < P.K && P.sel[row * P.K + cur] == m;
    }
    float bm = -INFINITY, bl = 0.f;  // the block's own log2 mass
    const int i1 = m == beta ? t : (m + 1) * B - 1;
    for (int i = m * B; i <= i1; ++i) {
      const float* k = (const float*)P.Kt + (((size_t)bi * n + i) * P.Hkv + g) * DH;
      float z = 0.f;
#pragma unroll
      for (int j = 0; j < DH; ++j) z = fmaf(qv[j], k[j], z);
      const float x = z * P.sm_scale * SLOG2E;
      const float y = x + P.lvn[((size_t)bi * n + i) * P.Hkv + g];
      if (x > m_raw) {
        const float a = exp2f(m_raw - x);
        l_all *= a;
        l_S *= a;
        m_raw = x;
      }
      if (y > m_val) {
        const float a = exp2f(m_val - y);
        l_vall *= a;
        l_vS *= a;
        m_val = y;
      }
      const float p = exp2f(x - m_raw), pv = exp2f(y - m_val);
      l_all += p;
      l_vall += pv;
      if (in) {
        l_S += p;
        l_vS += pv;
      }
      if (x > bm) {
        bl = bl * exp2f(bm - x) + 1.f;
        bm = x;
      } else {
        bl += exp2f(x - bm);
      }
    }
    if (P.blk_lse && m < beta) P.blk_lse[hrow * NB + m] = bm + log2f(bl);
  }
  if (P.cov) P.cov[hrow] = l_S / l_all;
  if (P.cov_v) P.cov_v[hrow] = l_vS / l_vall;
}

// Per-head Top-K historical blocks by block mass (descending, lower block
// first on ties), as a bitmask row [W words]; one thread per (b, h, t).
template <int KMAX>
__global__ void ref_topk_kernel(const float* __restrict__ blk_lse, size_t rows, int n, int H, int B, int K, int NB,
                                int W, uint32_t* __restrict__ head_mask, const int32_t* __restrict__ doc) {
  const size_t r = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows) return;
  const int t = (int)(r % n);
  const int C = t / B;
  const int F = doc_first(doc, (int)(r / ((size_t)n * H)), NB, t, B);  // historical blocks [F, C)
  float tv[KMAX];
  int tm[KMAX];
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    tv[i] = -INFINITY;
    tm[i] = 0x7fffffff;
  }
  const float* row = blk_lse + r * NB;
  for (int m = F; m < C; ++m) {
    float cv = row[m];
    int cm = m;
    if (!(cv > tv[KMAX - 1] || (cv == tv[KMAX - 1] && cm < tm[KMAX - 1]))) continue;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      // (value desc, block asc): an equal value keeps the lower block ahead; empty slots hold (-inf, max)
      const bool better = cv > tv[i] || (cv == tv[i] && cm < tm[i]);
      const float ov = tv[i];
      const int om = tm[i];
      tv[i] = better ? cv : ov;
      tm[i] = better ? cm : om;
      cv = better ? ov : cv;
      cm = better ? om : cm;
    }
  }
  const int kk = min(K, C - F);
  uint32_t* out = head_mask + r * W;
  for (int w = 0; w < W; ++w) {
    uint32_t bits = 0;
#pragma unroll
    for (int i = 0; i < KMAX; ++i)
      if (i < kk && (tm[i] >> 5) == w) bits |= 1u << (tm[i] & 31);
    out[w] = bits;
  }
}

// group set = blocks chosen by more than half of the group's heads; OR into the union
__global__ void vote_union_kernel(const uint32_t* __restrict__ head_mask, int b, int n, int H, int Hkv, int W,
                                  uint32_t* __restrict__ uni) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)b * Hkv * n * W) return;
  const int w = (int)(idx % W), t = (int)((idx / W) % n), g = (int)((idx / ((size_t)W * n)) % Hkv);
  const int bi = (int)(idx / ((size_t)W * n * Hkv));
  const int G = H / Hkv;
  uint32_t bits = 0;
  for (int j = 0; j < 32; ++j) {
    int cnt = 0;
    for (int hh = g * G; hh < (g + 1) * G; ++hh)
      cnt += (head_mask[(((size_t)bi * H + hh) * n + t) * W + w] >> j) & 1u;
    if (2 * cnt > G) bits |= 1u << j;
  }
  uni[idx] |= bits;
}

// OR the selection rows [b, Hkv, n, K] into the union bitmask
__global__ void sel_union_kernel(const int32_t* __restrict__ sel, size_t rows, int K, int NB, int W,
                                 uint32_t* __restrict__ uni) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * W) return;
  const size_t row = idx / W;
  const int w = (int)(idx % W);
  uint32_t bits = 0;
  for (int k = 0; k < K; ++k) {
    const int m = sel[row * K + k];
    if (m >= 0 && m < NB && (m >> 5) == w) bits |= 1u << (m & 31);
  }
  uni[idx] |= bits;
}

__global__ void zero_u64_kernel(unsigned long long* p, int n) {
  if ((int)threadIdx.x < n) p[threadIdx.x] = 0ull;
}

// counts[0] += |a & b|, counts[1] += |b| over every word
__global__ void overlap_count_kernel(const uint32_t* __restrict__ a, const uint32_t* __restrict__ b, size_t words,
                                     unsigned long long* __restrict__ counts) {
  __shared__ unsigned long long part[2][4];
  unsigned long long ci = 0, cb = 0;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += (size_t)gridDim.x * blockDim.x) {
    const uint32_t bw = b[i];
    ci += __popc(a[i] & bw);
    cb += __popc(bw);
  }
  for (int off = 32; off > 0; off >>= 1) {
    ci += __shfl_xor(ci, off, 64);
    cb += __shfl_xor(cb, off, 64);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    part[0][wave] = ci;
    part[1][wave] = cb;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long si = 0, sb = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
      si += part[0][w];
      sb += part[1][w];
    }
    atomicAdd(&counts[0], si);
    atomicAdd(&counts[1], sb);
  }
}

hipError_t launch_vnorm(int dtype, const void* V, size_t rows, int dh, float* lvn, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const unsigned grid = (unsigned)cdiv(rows, 256);
  if (dtype == SAS_BF16) {
    if (dh == 128) vnorm_kernel<bf16_t, 128><<<grid, 256, 0, s>>>((const bf16_t*)V, rows, lvn);
    else vnorm_kernel<bf16_t, 64><<<grid, 256, 0, s>>>((const bf16_t*)V, rows, lvn);
  } else {
    if (dh == 128) vnorm_kernel<float, 128><<<grid, 256, 0, s>>>((const float*)V, rows, lvn);
    else vnorm_kernel<float, 64><<<grid, 256, 0, s>>>((const float*)V, rows, lvn);
  }
  return hipGetLastError();
}

hipError_t launch_stats(int dtype, const StatsArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.b <= 0) return hipSuccess;
  if (a.K > 32) return hipErrorInvalidValue;
  if (dtype != SAS_BF16) {
    const size_t tot = (size_t)a.b * a.H * a.n;
    if (a.dh == 128) stats_f32_kernel<128><<<(unsigned)cdiv(tot, 64), 64, 0, s>>>(a);
    else stats_f32_kernel<64><<<(unsigned)cdiv(tot, 64), 64, 0, s>>>(a);
    return hipGetLastError();
  }
  const int lsb = a.B >= 64 ? 6 : (a.B == 32 ? 5 : 4);
  auto kern = a.dh == 128 ? (lsb == 6 ? stats_bf16_kernel<128, 6> : lsb == 5 ? stats_bf16_kernel<128, 5>
                                                                              : stats_bf16_kernel<128, 4>)
                          : (lsb == 6 ? stats_bf16_kernel<64, 6> : lsb == 5 ? stats_bf16_kernel<64, 5>
                                                                             : stats_bf16_kernel<64, 4>);
  const long long jobs = (long long)cdiv(a.n, 128) * a.H * a.b;
  const int res = resident_workgroups(kern, 256);
  if (res <= 0 || jobs > INT32_MAX) return hipErrorInvalidValue;
  StatsArgs A = a;
  A.queue = nullptr;
  if (jobs > res) {
    if (!a.queue) return hipErrorInvalidValue;
    const hipError_t e = launch_fill_f32((float*)a.queue, 1, 0.f, s);  // the job counter to zero
    if (e != hipSuccess) return e;
    A.queue = a.queue;
  }
  kern<<<(unsigned)std::min<long long>(jobs, res), 256, 0, s>>>(A);
  return hipGetLastError();
}

hipError_t launch_ref_sets(const float* blk_lse, int b, int n, int H, int Hkv, int B, int K, uint32_t* head_mask,
                           uint32_t* uni, const int32_t* doc, hipStream_t s) {
  const int NB = cdiv(n, B), W = cdiv(NB, 32);
  const size_t rows = (size_t)b * H * n;
  if (rows == 0) return hipSuccess;
  const unsigned grid = (unsigned)cdiv(rows, 128);
  if (K <= 8) ref_topk_kernel<8><<<grid, 128, 0, s>>>(blk_lse, rows, n, H, B, K, NB, W, head_mask, doc);
  else if (K <= 16) ref_topk_kernel<16><<<grid, 128, 0, s>>>(blk_lse, rows, n, H, B, K, NB, W, head_mask, doc);
  else ref_topk_kernel<32><<<grid, 128, 0, s>>>(blk_lse, rows, n, H, B, K, NB, W, head_mask, doc);
  const size_t tot = (size_t)b * Hkv * n * W;
  vote_union_kernel<<<(unsigned)cdiv(tot, 256), 256, 0, s>>>(head_mask, b, n, H, Hkv, W, uni);
  return hipGetLastError();
}

hipError_t launch_sel_union(const int32_t* sel, size_t rows, int K, int NB, uint32_t* uni, hipStream_t s) {
  const int W = cdiv(NB, 32);
  if (rows * W == 0) return hipSuccess;
  sel_union_kernel<<<(unsigned)cdiv(rows * W, 256), 256, 0, s>>>(sel, rows, K, NB, W, uni);
  return hipGetLastError();
}

hipError_t launch_overlap_count(const uint32_t* a, const uint32_t* b, size_t words, unsigned long long* counts,
                                hipStream_t s) {
  zero_u64_kernel<<<1, 64, 0, s>>>(counts, 2);
  if (words == 0) return hipGetLastError();
  const size_t blocks = cdiv(words, 256);
  const unsigned grid = (unsigned)(blocks < 1024 ? blocks : 1024);
  overlap_count_kernel<<<grid, 256, 0, s>>>(a, b, words, counts);
  return hipGetLastError();
}

}  // namespace sas
