// SAS inference step over a paged KV cache (Alg. 2; Sec. 5.1: the prefill is
// dense and fills the cache, every decode step scores the cached block
// summaries, keeps the Top-K blocks per KV group and attends to them plus the
// current block, without gate bias).
//
// Cache layout: pages [num_pages, Hkv, page_size, dh]; position p of sequence
// i lives in page block_table[i][p / page_size], slot p % page_size, so one
// page of one KV head is page_size * dh contiguous values.  Block summaries
// [b, Hkv, max_blocks, dh] hold the selector's pooled key of every complete
// SAS block.  Every kernel checks positions and page ids against the cache
// geometry and skips what falls outside.
#include <float.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace sas {

__device__ __forceinline__ PageGeom geom_of(const DecodeArgs& c) {
  PageGeom G;
  G.table = c.block_table;
  G.num_pages = c.num_pages;
  G.ps = c.page_size;
  G.max_pages = c.max_pages;
  return G;
}

// ---- prefill -> cache ---------------------------------------------------------
// thread per (b, t, g, 8-value chunk): K and V into their pages; thread per
// (b, g, m, chunk) copies the complete-block summaries.
template <typename T>
__global__ void cache_fill_kernel(const T* __restrict__ K, const T* __restrict__ V, int b, int n, int Hkv, int dh,
                                  DecodeArgs c, size_t total) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int nc = dh / 8;
  const int c8 = (int)(idx % nc);
  size_t r = idx / nc;
  const int g = (int)(r % Hkv);
  r /= Hkv;
  const int t = (int)(r % n);
  const int i = (int)(r / n);
  const long long off = geom_of(c).offset(i, g, t, Hkv, dh);
  if (off < 0) return;
  const size_t src = (((size_t)i * n + t) * Hkv + g) * dh + c8 * 8;
  *(uint4*)((T*)c.k_pages + off + c8 * 8) = *(const uint4*)(K + src);
  *(uint4*)((T*)c.v_pages + off + c8 * 8) = *(const uint4*)(V + src);
  if (sizeof(T) == 4) {
    *(uint4*)((T*)c.k_pages + off + c8 * 8 + 4) = *(const uint4*)(K + src + 4);
    *(uint4*)((T*)c.v_pages + off + c8 * 8 + 4) = *(const uint4*)(V + src + 4);
  }
}

template <typename T>
__global__ void summary_copy_kernel(const T* __restrict__ ksum, int b, int Hkv, int NB, int nfull, int dh,
                                    T* __restrict__ cache_sum, int max_blocks, size_t total) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int j = (int)(idx % dh);
  size_t r = idx / dh;
  const int m = (int)(r % nfull);
  r /= nfull;
  const int g = (int)(r % Hkv);
  const int i = (int)(r / Hkv);
  if (m >= max_blocks) return;
  cache_sum[(((size_t)i * Hkv + g) * max_blocks + m) * dh + j] = ksum[(((size_t)i * Hkv + g) * NB + m) * dh + j];
}

hipError_t launch_cache_fill(int dtype, const void* K, const void* V, const void* ksum, int b, int n, int Hkv,
                             int dh, int B, int NB, const DecodeArgs& c, hipStream_t s, bool kv) {
  const size_t total = kv ? (size_t)b * n * Hkv * (dh / 8) : 0;
  const int nfull = n / B;
  const size_t stot = (size_t)b * Hkv * nfull * dh;
  if (dtype == SAS_BF16) {
    if (total) cache_fill_kernel<bf16_t><<<(unsigned)((total + 255) / 256), 256, 0, s>>>(
        (const bf16_t*)K, (const bf16_t*)V, b, n, Hkv, dh, c, total);
    if (stot) summary_copy_kernel<bf16_t><<<(unsigned)((stot + 255) / 256), 256, 0, s>>>(
        (const bf16_t*)ksum, b, Hkv, NB, nfull, dh, (bf16_t*)c.k_summary, c.max_blocks, stot);
  } else {
    if (total) cache_fill_kernel<float><<<(unsigned)((total + 255) / 256), 256, 0, s>>>(
        (const float*)K, (const float*)V, b, n, Hkv, dh, c, total);
    if (stot) summary_copy_kernel<float><<<(unsigned)((stot + 255) / 256), 256, 0, s>>>(
        (const float*)ksum, b, Hkv, NB, nfull, dh, (float*)c.k_summary, c.max_blocks, stot);
  }
  return hipGetLastError();
}

// ---- append the new token, complete the block summary -----------------------
// thread per (i, g, j): writes k/v at pos[i]; when pos+1 closes a SAS block it
// sums the block's keys (its own dimension j, ascending positions, fp64) and
// writes the summary (plain, or to `kplain` when a projection follows).
template <typename T>
__global__ void kv_append_kernel(const T* __restrict__ k, const T* __restrict__ v, DecodeArgs c, T* kplain) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= c.b * c.Hkv * c.dh) return;
  const int j = idx % c.dh;
  const int g = (idx / c.dh) % c.Hkv;
  const int i = idx / (c.dh * c.Hkv);
  const int p = c.pos[i];
  const PageGeom G = geom_of(c);
  const long long off = G.offset(i, g, p, c.Hkv, c.dh);
  if (off < 0) return;
  const T kv = k[((size_t)i * c.Hkv + g) * c.dh + j];
  ((T*)c.k_pages)[off + j] = kv;
  ((T*)c.v_pages)[off + j] = v[((size_t)i * c.Hkv + g) * c.dh + j];
  if ((p + 1) % c.B != 0) return;
  const int m = p / c.B;
  if (m >= c.max_blocks) return;
  // positions in chunks of SUMC: the chunk's page ids, then its keys, loaded
  // unconditionally from clamped addresses and masked afterwards (two memory
  // round trips per chunk instead of two per position); the fp64 sum keeps
  // the ascending order
  constexpr int SUMC = 16;
  const T* kp = (const T*)c.k_pages;
  const int32_t* trow = c.block_table + (size_t)i * c.max_pages;
  double acc = 0.0;
  for (int q0 = m * c.B; q0 < p; q0 += SUMC) {
    long long o[SUMC];
#pragma unroll
    for (int u = 0; u < SUMC; ++u) {
      const int q = q0 + u, pi = q / c.page_size;
      const int page = trow[min(pi, c.max_pages - 1)];
      const bool ok = q < p && pi < c.max_pages && page >= 0 && page < c.num_pages;
      o[u] = ok ? (((long long)page * c.Hkv + g) * c.page_size + (q % c.page_size)) * c.dh : -1;
    }
    float kq[SUMC];
#pragma unroll
    for (int u = 0; u < SUMC; ++u) {
      const float x = Act<T>::to_f32(kp[(o[u] >= 0 ? o[u] : 0) + j]);
      kq[u] = o[u] >= 0 ? x : 0.f;  // a position without a page adds zero
    }
#pragma unroll
    for (int u = 0; u < SUMC; ++u)
      if (q0 + u < p) acc += (double)kq[u];
  }
  acc += (double)Act<T>::to_f32(kv);
  T* dst = kplain ? kplain + ((size_t)i * c.Hkv + g) * c.dh
                  : (T*)c.k_summary + (((size_t)i * c.Hkv + g) * c.max_blocks + m) * c.dh;
  dst[j] = Act<T>::from_f64(acc / (double)c.B);
}

// projected summary of a block completed at this step: thread per (i, g, k)
template <typename T>
__global__ void kv_summary_project_kernel(const T* __restrict__ kplain, const T* __restrict__ W, DecodeArgs c) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= c.b * c.Hkv * c.dh) return;
  const int kk = idx % c.dh;
  const int g = (idx / c.dh) % c.Hkv;
  const int i = idx / (c.dh * c.Hkv);
  const int p = c.pos[i];
  if (p < 0 || (p + 1) % c.B != 0 || p / c.B >= c.max_blocks) return;
  if (geom_of(c).offset(i, g, p, c.Hkv, c.dh) < 0) return;
  const T* x = kplain + ((size_t)i * c.Hkv + g) * c.dh;
  const T* w = W + ((size_t)g * c.dh + kk) * c.dh;
  double acc = 0.0;
  for (int j = 0; j < c.dh; ++j) acc = fma((double)Act<T>::to_f32(w[j]), (double)Act<T>::to_f32(x[j]), acc);
  ((T*)c.k_summary)[(((size_t)i * c.Hkv + g) * c.max_blocks + p / c.B) * c.dh + kk] = Act<T>::from_f64(acc);
}

hipError_t launch_kv_append(int dtype, const void* k, const void* v, const DecodeArgs& c, void* kplain_scratch,
                            hipStream_t s) {
  const int tot = c.b * c.Hkv * c.dh;
  void* kp = c.w_gk ? kplain_scratch : nullptr;
  if (dtype == SAS_BF16) {
    kv_append_kernel<bf16_t><<<cdiv(tot, 256), 256, 0, s>>>((const bf16_t*)k, (const bf16_t*)v, c, (bf16_t*)kp);
    if (c.w_gk)
      kv_summary_project_kernel<bf16_t><<<cdiv(tot, 256), 256, 0, s>>>((const bf16_t*)kp, (const bf16_t*)c.w_gk, c);
  } else {
    kv_append_kernel<float><<<cdiv(tot, 256), 256, 0, s>>>((const float*)k, (const float*)v, c, (float*)kp);
    if (c.w_gk)
      kv_summary_project_kernel<float><<<cdiv(tot, 256), 256, 0, s>>>((const float*)kp, (const float*)c.w_gk, c);
  }
  return hipGetLastError();
}

// ---- Top-K blocks per (sequence, group) ------------------------------------------
// One wave per (i, g).  Gate query: rho(sum of the group's heads), optionally
// projected; scores: sequential fp64 sums over ascending j; rank of a block =
// number of blocks strictly ahead of it under (r desc, m asc); kept if rank < K,
// written in ascending block order.  A lane reads its summary row with 16-byte
// loads issued together.

template <typename T, int DH>
__global__ void __launch_bounds__(64) decode_select_kernel(const T* __restrict__ q, DecodeArgs c,
                                                           int32_t* __restrict__ sel) {
  __shared__ double qh[128];
  __shared__ double qp[128];
  __shared__ double rs[DSEL_WAVE_MAX_BLOCKS];
  const int lane = threadIdx.x;
  const int g = blockIdx.x, i = blockIdx.y;
  const int G = c.H / c.Hkv, dh = DH, K = c.K;
  // this lane's first summary row, loaded before the position is known so
  // that its latency overlaps the position's and the queries' (a row past the
  // cache's blocks is clamped and its score is never used)
  const T* ks = (const T*)c.k_summary + ((size_t)i * c.Hkv + g) * c.max_blocks * dh;
  Vec8<T> kv0[DH / 8];
  if (c.max_blocks > 0) {
    const T* kr = ks + (size_t)min(lane, c.max_blocks - 1) * DH;
#pragma unroll
    for (int c8 = 0; c8 < DH / 8; ++c8) kv0[c8].load(kr + c8 * 8);
  }
  const int p = c.pos[i];
  const int ct = max(0, min(p / c.B, min(c.max_blocks, DSEL_WAVE_MAX_BLOCKS)));
  for (int j = lane; j < dh; j += 64) {
    double acc = 0.0;
    for (int h = 0; h < G; ++h) acc += (double)Act<T>::to_f32(q[((size_t)i * c.H + g * G + h) * dh + j]);
    qh[j] = (double)Act<T>::to_f32(Act<T>::from_f64(acc));
  }
  __syncthreads();
  if (c.w_gq) {
    const T* W = (const T*)c.w_gq + (size_t)g * dh * dh;
    for (int kk = lane; kk < dh; kk += 64) {
      double acc = 0.0;
      for (int j = 0; j < dh; ++j) acc = fma((double)Act<T>::to_f32(W[(size_t)kk * dh + j]), qh[j], acc);
      qp[kk] = (double)Act<T>::to_f32(Act<T>::from_f64(acc));
    }
    __syncthreads();
    for (int j = lane; j < dh; j += 64) qh[j] = qp[j];
    __syncthreads();
  }
  auto score = [&](const Vec8<T>(&kv)[DH / 8]) {
    double acc = 0.0;
#pragma unroll
    for (int c8 = 0; c8 < DH / 8; ++c8)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc = fma(qh[c8 * 8 + e], (double)kv[c8].get(e), acc);
    return acc;
  };
  if (lane < ct) rs[lane] = score(kv0);
  for (int m = lane + 64; m < ct; m += 64) {
    const T* kr = ks + (size_t)m * DH;
    Vec8<T> kv[DH / 8];
#pragma unroll
    for (int c8 = 0; c8 < DH / 8; ++c8) kv[c8].load(kr + c8 * 8);
    rs[m] = score(kv);
  }
  __syncthreads();
  int32_t* out = sel + ((size_t)i * c.Hkv + g) * K;
  int base = 0;
  for (int m0 = 0; m0 < ct; m0 += 64) {
    const int m = m0 + lane;
    bool keep = false;
    if (m < ct) {
      const double r = rs[m];
      // rank = the blocks ahead of m (a full pass without an early exit, so
      // that the unrolled LDS reads are issued together)
      int rank = 0;
#pragma unroll 8
      for (int o = 0; o < ct; ++o) {
        const double ro = rs[o];
        rank += (ro > r || (ro == r && o < m)) ? 1 : 0;
      }
      keep = rank < K;
    }
    const unsigned long long mask = __ballot(keep);
    if (keep) {
      const int slot = base + __popcll(mask & ((1ull << lane) - 1ull));
      if (slot < K) out[slot] = m;
    }
    base += __popcll(mask);
  }
  for (int s2 = base + lane; s2 < K; s2 += 64) out[s2] = -1;
}

// ---- selection over long contexts ----------------------------------------------
// Caches of more than DSEL_WAVE_MAX_BLOCKS blocks take two phases.  decode_score_kernel:
// a workgroup per ROWS blocks of one (group, sequence) stages their summary
// rows in LDS with coalesced 16-byte loads (rows padded by 16 bytes so the
// lanes of one 128-bit read pass hit distinct banks) and gives each thread one
// block, whose score r is the same sequential fp64 sum over ascending j as in
// the single-wave kernel; scores go to a scratch row per (sequence, group).
// decode_topk_kernel: a workgroup of 1024 threads per (group, sequence) holds
// the scores as order-preserving 64-bit keys (-0 folded into +0, so equal
// scores tie) in registers, KPT consecutive blocks per thread, and finds the
// key of the K-th largest by eight passes of 8-bit radix histograms in LDS.
// Every key above it is kept, and of the keys equal to it the lowest block
// indices; block-wide scans in block order write them ascending.
constexpr int DSEL_TOPK_KPT = 8;      // blocks per thread of the radix Top-K
constexpr int DSEL_TOPK_NT = 1024;
constexpr int DSEL_LONG_MAXB = DSEL_TOPK_KPT * DSEL_TOPK_NT;  // 8192 blocks: 512K tokens at B = 64
static_assert(DSEL_LONG_MAXB == DSEL_MAX_BLOCKS, "selection limit");

template <typename T, int DH, int ROWS>
__global__ void __launch_bounds__(ROWS) decode_score_kernel(const T* __restrict__ q, DecodeArgs c,
                                                            double* __restrict__ scores) {
  constexpr int RS = DH * (int)sizeof(T) + 16;  // bytes per staged row
  constexpr int CH = DH * (int)sizeof(T) / 16;  // 16-byte chunks per row
  __shared__ double qh[DH], qp[DH];
  __shared__ __align__(16) unsigned char rows[ROWS * RS];
  const int tid = threadIdx.x;
  const int g = blockIdx.y, i = blockIdx.z;
  const int m0 = blockIdx.x * ROWS;
  const int p = c.pos[i];
  const int ct = p < 0 ? 0 : min(p / c.B, c.max_blocks);
  if (m0 >= ct) return;
  const int G = c.H / c.Hkv;
  for (int j = tid; j < DH; j += ROWS) {
    double acc = 0.0;
    for (int h = 0; h < G; ++h) acc += (double)Act<T>::to_f32(q[((size_t)i * c.H + g * G + h) * DH + j]);
    qh[j] = (double)Act<T>::to_f32(Act<T>::from_f64(acc));
  }
  __syncthreads();
  if (c.w_gq) {
    const T* W = (const T*)c.w_gq + (size_t)g * DH * DH;
    for (int kk = tid; kk < DH; kk += ROWS) {
      double acc = 0.0;
      for (int j = 0; j < DH; ++j) acc = fma((double)Act<T>::to_f32(W[(size_t)kk * DH + j]), qh[j], acc);
      qp[kk] = (double)Act<T>::to_f32(Act<T>::from_f64(acc));
    }
    __syncthreads();
    for (int j = tid; j < DH; j += ROWS) qh[j] = qp[j];
  }
  const T* ks = (const T*)c.k_summary + ((size_t)i * c.Hkv + g) * c.max_blocks * DH;
  const int nrow = min(ROWS, ct - m0);
  for (int x = tid; x < nrow * CH; x += ROWS) {
    const int r = x / CH, cc = x % CH;
    *(uint4*)(rows + r * RS + cc * 16) = *(const uint4*)((const unsigned char*)(ks + (size_t)(m0 + r) * DH) + cc * 16);
  }
  __syncthreads();
  if (tid < nrow) {
    const T* row = (const T*)(rows + tid * RS);
    double acc = 0.0;
    for (int j0 = 0; j0 < DH; j0 += 8) {
      Vec8<T> v;
      v.load(row + j0);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc = fma(qh[j0 + e], (double)v.get(e), acc);
    }
    scores[((size_t)i * c.Hkv + g) * c.max_blocks + m0 + tid] = acc;
  }
}

// exclusive prefix sum of v over the workgroup in thread order; total in *tot
__device__ __forceinline__ int block_exclusive_scan(int v, int* wsum, int* tot) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wv] = x;
  __syncthreads();
  int before = 0, all = 0;
  for (int w = 0; w < nw; ++w) {
    const int sw = wsum[w];
    before += w < wv ? sw : 0;
    all += sw;
  }
  __syncthreads();
  *tot = all;
  return before + x - v;
}

__global__ void __launch_bounds__(DSEL_TOPK_NT) decode_topk_kernel(const double* __restrict__ scores, DecodeArgs c,
                                                                   int32_t* __restrict__ sel) {
  constexpr int KPT = DSEL_TOPK_KPT;
  __shared__ int hist[256];
  __shared__ int sh_digit, sh_above;
  __shared__ int wsum[DSEL_TOPK_NT / 64];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g = blockIdx.x, i = blockIdx.y;
  const int K = c.K;
  int32_t* out = sel + ((size_t)i * c.Hkv + g) * K;
  const int p = c.pos[i];
  const int ct = p < 0 ? 0 : min(p / c.B, c.max_blocks);
  const int kk = min(K, ct);
  const double* rs = scores + ((size_t)i * c.Hkv + g) * c.max_blocks;
  unsigned long long key[KPT];
#pragma unroll
  for (int e = 0; e < KPT; ++e) {
    const int m = tid * KPT + e;
    key[e] = 0;
    if (m < ct) {
      const unsigned long long u = (unsigned long long)__double_as_longlong(rs[m] + 0.0);  // -0 -> +0
      key[e] = (u >> 63) ? ~u : (u | (1ull << 63));
    }
  }
  unsigned long long prefix = 0, pmask = 0;
  int need = kk;
  const bool all = ct <= K;  // every historical block is kept
  if (!all) {
    for (int pass = 7; pass >= 0; --pass) {
      const int sh = 8 * pass;
      for (int x = tid; x < 256; x += DSEL_TOPK_NT) hist[x] = 0;
      __syncthreads();
#pragma unroll
      for (int e = 0; e < KPT; ++e)
        if (tid * KPT + e < ct && (key[e] & pmask) == prefix) atomicAdd(&hist[(int)((key[e] >> sh) & 255)], 1);
      __syncthreads();
      if (wv == 0) {
        // lane l holds digits 255-4l .. 252-4l (descending); find the digit whose
        // bin holds the need-th largest remaining key
        int cnt[4], cum = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          cnt[e] = hist[255 - 4 * lane - e];
          cum += cnt[e];
        }
        int x = cum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(x, o, 64);
          if (lane >= o) x += y;
        }
        int above = x - cum;  // keys with a higher digit than this lane's first
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (above < need && above + cnt[e] >= need) {
            sh_digit = 255 - 4 * lane - e;
            sh_above = above;
          }
          above += cnt[e];
        }
      }
      __syncthreads();
      need -= sh_above;
      prefix |= (unsigned long long)sh_digit << sh;
      pmask |= 255ull << sh;
      __syncthreads();
    }
  }
  // prefix = key of the K-th largest; keep every key above it and the `need`
  // lowest-index keys equal to it
  int n_eq = 0;
#pragma unroll
  for (int e = 0; e < KPT; ++e) n_eq += (!all && tid * KPT + e < ct && key[e] == prefix) ? 1 : 0;
  int tot;
  const int eq_before = block_exclusive_scan(n_eq, wsum, &tot);
  bool keep[KPT];
  int n_keep = 0, eq_seen = 0;
#pragma unroll
  for (int e = 0; e < KPT; ++e) {
    const bool valid = tid * KPT + e < ct;
    bool k = valid && (all || key[e] > prefix);
    if (valid && !all && key[e] == prefix) {
      k = eq_before + eq_seen < need;
      ++eq_seen;
    }
    keep[e] = k;
    n_keep += k ? 1 : 0;
  }
  const int slot0 = block_exclusive_scan(n_keep, wsum, &tot);
  int slot = slot0;
#pragma unroll
  for (int e = 0; e < KPT; ++e)
    if (keep[e]) {
      if (slot < K) out[slot] = tid * KPT + e;
      ++slot;
    }
  for (int s2 = kk + tid; s2 < K; s2 += DSEL_TOPK_NT) out[s2] = -1;
}

hipError_t launch_decode_select(int dtype, const void* q, const DecodeArgs& c, int32_t* sel, double* scores,
                                hipStream_t s) {
  if (c.K <= 0) return hipSuccess;
  if (c.max_blocks <= DSEL_WAVE_MAX_BLOCKS) {
    dim3 grid(c.Hkv, c.b);
    if (c.dh != 64 && c.dh != 128) return hipErrorInvalidValue;
    if (dtype == SAS_BF16) {
      if (c.dh == 128) decode_select_kernel<bf16_t, 128><<<grid, 64, 0, s>>>((const bf16_t*)q, c, sel);
      else decode_select_kernel<bf16_t, 64><<<grid, 64, 0, s>>>((const bf16_t*)q, c, sel);
    } else {
      if (c.dh == 128) decode_select_kernel<float, 128><<<grid, 64, 0, s>>>((const float*)q, c, sel);
      else decode_select_kernel<float, 64><<<grid, 64, 0, s>>>((const float*)q, c, sel);
    }
    return hipGetLastError();
  }
  if (c.max_blocks > DSEL_LONG_MAXB || !scores) return hipErrorInvalidValue;
  if (dtype == SAS_BF16) {
    dim3 grid(cdiv(c.max_blocks, 128), c.Hkv, c.b);
    if (c.dh == 128) decode_score_kernel<bf16_t, 128, 128><<<grid, 128, 0, s>>>((const bf16_t*)q, c, scores);
    else decode_score_kernel<bf16_t, 64, 128><<<grid, 128, 0, s>>>((const bf16_t*)q, c, scores);
  } else {
    dim3 grid(cdiv(c.max_blocks, 64), c.Hkv, c.b);
    if (c.dh == 128) decode_score_kernel<float, 128, 64><<<grid, 64, 0, s>>>((const float*)q, c, scores);
    else decode_score_kernel<float, 64, 64><<<grid, 64, 0, s>>>((const float*)q, c, scores);
  }
  decode_topk_kernel<<<dim3(c.Hkv, c.b), DSEL_TOPK_NT, 0, s>>>(scores, c, sel);
  return hipGetLastError();
}

// ---- sparse attention of the new tokens ----------------------------------------
// One workgroup of NW waves per (split, head chunk, group, sequence).  The kept
// keys of a group are walked in segments of SEG keys: the K selected blocks in
// selection order (a block of B > SEG keys is B / SEG segments), then the
// current block [B*floor(p/B), p].  A split is a contiguous range of segments;
// the workgroup first resolves where each of its segments starts (one pass,
// into LDS) and the page ids of every block it touches (a block's pages are
// consecutive entries of the block table), so that a segment's key and value
// loads depend on no global load: a wait on the page ids would also wait for
// the loads of the segment in flight before it.  Segments are dealt to the
// waves round-robin.  Keys and values are not staged
// in LDS: with NC = dh/8 lanes per key, lane l holds the 8-value slice l % NC
// of keys l / NC + (64/NC) * it, loaded with coalesced 16-byte loads (a page of
// one KV head is contiguous).  A wave holds K and V of two segments in
// registers and issues the loads of the next segment before it computes the
// current one; the keys serve every head of the head chunk.  A key's score is
// the partial dot product reduced over its NC lanes; each wave keeps an online
// softmax per head (running max, sum of exp, unnormalised P V per slice).  The
// waves are merged in LDS; with one split the result is O itself, otherwise an
// fp32 partial (max, sum of exp, unnormalised output) that
// decode_combine_kernel merges.
template <typename T, int DH>
struct DecodeSeg {
  static constexpr int NC = DH / 8;                          // lanes per key
  static constexpr int KPI = 64 / NC;                        // keys per load instruction
  static constexpr int SEG = 4096 / (DH * (int)sizeof(T));   // keys per segment: K and V in 32 VGPRs
  static constexpr int IT = SEG / KPI;                       // load steps per segment
  Vec8<T> k[IT], v[IT];
  bool ok[IT];
  int count;
};

constexpr int DSEG_MAX = 33 * 16;  // segments of a split: (K + 1) blocks of at most 16 segments
constexpr int DPAGE_MAX = 33 * 64;  // page ids of a split: (K + 1) blocks of at most 64 pages

// Sum over groups of NC consecutive lanes (NC = 8 or 16) with DPP moves:
// swaps within pairs and quads, then the mirror of each 8 and of each 16.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
template <int NC>
__device__ __forceinline__ float lane_group_sum(float v) {
  static_assert(NC == 8 || NC == 16, "groups of 8 or 16 lanes");
  v += dpp_move<0xB1>(v);                       // quad_perm 1,0,3,2
  v += dpp_move<0x4E>(v);                       // quad_perm 2,3,0,1
  v += dpp_move<0x141>(v);                      // row_half_mirror
  if constexpr (NC == 16) v += dpp_move<0x140>(v);  // row_mirror
  return v;
}

template <typename T, int DH, int GMAX, int NW>
__global__ void __launch_bounds__(NW * 64) decode_attn_kernel(const T* __restrict__ q, DecodeArgs c,
                                                              const int32_t* __restrict__ sel, int nsplit,
                                                              float* __restrict__ part_ml,
                                                              float* __restrict__ part_o, T* __restrict__ O) {
  using Seg = DecodeSeg<T, DH>;
  constexpr int NC = Seg::NC, KPI = Seg::KPI, SEG = Seg::SEG, IT = Seg::IT;
  __shared__ float sm_o[NW][GMAX][DH];
  __shared__ float sm_ml[NW][GMAX][2];
  __shared__ int sm_count[DSEG_MAX];
  __shared__ int sm_pages[DPAGE_MAX];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int G = c.H / c.Hkv, nhc = (G + GMAX - 1) / GMAX;
  const int split = blockIdx.x / nhc, hc = blockIdx.x % nhc;
  const int g = blockIdx.y, i = blockIdx.z;
  const int K = c.K, B = c.B;
  const int spb = B > SEG ? B / SEG : 1;  // segments per block (a power of two)
  const int spb_shift = __builtin_ctz(spb);
  const int seg_len = B > SEG ? SEG : B;
  const int nseg = (K + 1) * spb;
  const int per = (nseg + nsplit - 1) / nsplit;
  const int s0 = split * per, s1 = min(nseg, s0 + per);
  const int p = c.pos[i];
  const int sl = lane % NC, kq = lane / NC;
  const int ps = c.page_size;  // a power of two (it divides the power-of-two block size)
  const int pshift = __builtin_ctz(ps);
  const size_t kvstride = (size_t)c.Hkv * ps * DH;  // elements per page

  // block of selection slot ch (slot K: the current block), -1 if none
  auto block_of = [&](int ch) -> int {
    if (p < 0) return -1;
    return ch < K ? sel[((size_t)i * c.Hkv + g) * K + ch] : p / B;
  };
  // page ids of the blocks the split touches, and key count of every segment
  const int ppb = B / ps;  // pages per block (B is a multiple of the page size, ppb <= 64)
  const int ch0 = s0 / spb;
  const int nbl = s1 > s0 ? (s1 - 1) / spb - ch0 + 1 : 0;
  for (int t = threadIdx.x; t < nbl * ppb; t += NW * 64) {
    const int mb = block_of(ch0 + t / ppb);
    int pid = -1;
    if (mb >= 0) {
      const int pi = mb * ppb + t % ppb;
      if (pi < c.max_pages) pid = c.block_table[(size_t)i * c.max_pages + pi];
      if (pid >= c.num_pages) pid = -1;
    }
    sm_pages[t] = pid;
  }
  for (int t = threadIdx.x; t < s1 - s0; t += NW * 64) {
    const int sg = s0 + t, ch = sg / spb, sub = sg % spb;
    const int mb = block_of(ch);
    int count = 0;
    if (mb >= 0) count = ch < K ? seg_len : max(0, min(seg_len, p - (mb * B + sub * seg_len) + 1));
    sm_count[t] = count;
  }
  __syncthreads();

  const int ns = s1 - s0;
  // segment t of the split into S.  Every load is issued unconditionally,
  // also for segments without keys (past the split's end, or past the
  // position in the current block): loads under a branch, even a uniform
  // one, make the compiler wait for all loads in flight.  Keys past the count
  // reload the segment's last key (lines the same instruction reads anyway);
  // segments without keys and keys without a page reload the workgroup's own
  // query slice (cached, and different for every workgroup: padding loads of
  // one shared address from every workgroup crowd a few L2 channels).  ok
  // masks them all.
  const T* qpad = q + ((size_t)i * c.H + g * G + min(hc * GMAX, G - 1)) * DH + sl * 8;
  auto load = [&](Seg& S, int t) {
    const bool live = t < ns;
    const int cnt = live ? sm_count[t] : 0;
    S.count = cnt;
    const int sg = s0 + (live ? t : 0), chl = (sg >> spb_shift) - ch0;
    const int base = (sg & (spb - 1)) * seg_len;  // the segment's first key within its block
    size_t off[IT];
    bool use[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int kl = kq + KPI * it;
      const int a = base + max(0, min(kl, cnt - 1));  // key within the block
      const int page = sm_pages[chl * ppb + (a >> pshift)];
      use[it] = cnt > 0 && page >= 0;
      S.ok[it] = kl < cnt && use[it];
      off[it] = (size_t)(use[it] ? page : 0) * kvstride + (uint32_t)(((g << pshift) + (a & (ps - 1))) * DH + sl * 8);
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      S.k[it].load(use[it] ? (const T*)c.k_pages + off[it] : qpad);
      S.v[it].load(use[it] ? (const T*)c.v_pages + off[it] : qpad);
    }
  };

  float m[GMAX], l[GMAX], o[GMAX][8];
#pragma unroll
  for (int hg = 0; hg < GMAX; ++hg) {
    m[hg] = -INFINITY;
    l[hg] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[hg][e] = 0.f;
  }
  // Every lane reads every K and V register of the segment, whatever the keys'
  // validity (keys without data contribute zero through selects): the
  // compiler's wait for a segment's loads then does not depend on a branch,
  // and the next loads into these registers need no wait for older loads.
  // the scaled query slices of the chunk's heads, loaded once: a query load
  // issued after a segment's loads would make its use wait for all of them
  // (bf16: the raw query pairs, for bf16 dot products; the scale is applied
  // to the reduced score)
  constexpr bool BF = sizeof(T) == 2;
  float qsl[GMAX][8];
  uint32_t qpair[GMAX][4];
#pragma unroll
  for (int hg = 0; hg < GMAX; ++hg) {
    const int hl = min(hc * GMAX + hg, G - 1);
    Vec8<T> v;
    v.load(q + ((size_t)i * c.H + g * G + hl) * DH + sl * 8);
    if constexpr (BF) {
      const uint32_t* w = (const uint32_t*)&v;
#pragma unroll
      for (int e = 0; e < 4; ++e) qpair[hg][e] = w[e];
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) qsl[hg][e] = v.get(e) * c.sm_scale;
    }
  }
  auto compute = [&](const Seg& S) {
#pragma unroll
    for (int hg = 0; hg < GMAX; ++hg) {
      const int hl = hc * GMAX + hg;
      if (hl >= G) break;
      const float* qs = qsl[hg];
      float sc[IT];
      float mx = -INFINITY;
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        float acc = 0.f;
        if constexpr (BF) {
          const uint32_t* kw = (const uint32_t*)&S.k[it];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, kw[e]),
                                                  __builtin_bit_cast(bf16x2_t, qpair[hg][e]), acc, false);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) acc = fmaf(qs[e], S.k[it].get(e), acc);
        }
        acc = S.ok[it] ? acc : 0.f;
        acc = lane_group_sum<NC>(acc);
        if constexpr (BF) acc *= c.sm_scale;
        sc[it] = S.ok[it] ? acc : -INFINITY;  // keys past the count or without a page take no part
        mx = fmaxf(mx, sc[it]);
      }
      mx = wave_max(mx);
      const float mn = fmaxf(m[hg], mx);
      const bool any = mn > -INFINITY;  // some key so far (uniform across the wave)
      const float scale = any ? __expf(m[hg] - mn) : 1.f;
      m[hg] = mn;
      l[hg] *= scale;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[hg][e] *= scale;
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const float pk = any && S.ok[it] ? __expf(sc[it] - mn) : 0.f;
        l[hg] += pk;
        // keys without data read arbitrary bytes: their values are zeroed
        // (the probability alone would give 0 x NaN)
        Vec8<T> vz = S.v[it];
        if constexpr (BF) {
          uint32_t* vw = (uint32_t*)&vz;
#pragma unroll
          for (int e = 0; e < 4; ++e) vw[e] = S.ok[it] ? vw[e] : 0u;
        } else {
          float* vf = (float*)&vz;
#pragma unroll
          for (int e = 0; e < 8; ++e) vf[e] = S.ok[it] ? vf[e] : 0.f;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) o[hg][e] = fmaf(pk, vz.get(e), o[hg][e]);
      }
    }
  };

  // two segments in registers: the next one's loads are in flight while one
  // is computed.  Loads and computes are unconditional (empty segments past
  // the end), so the compiler's waits count exactly the other buffer's loads.
  // (Measured at batch 8, 7B shape, per layer step: segments of 16 keys
  // 30.8 us, of 8 keys 31.4, of 32 keys 31.9; a third segment of 32 keys in
  // flight 37 us: more bytes in flight per wave make the stream slower.)
  Seg sa, sb;
  load(sa, wave);
  for (int t = wave; t < ns; t += 2 * NW) {
    load(sb, t + NW);
    compute(sa);
    load(sa, t + 2 * NW);
    compute(sb);
  }

  // lanes sharing a slice hold different keys: reduce over them, then merge the waves
#pragma unroll
  for (int hg = 0; hg < GMAX; ++hg) {
#pragma unroll
    for (int off = NC; off < 64; off <<= 1) {
      l[hg] += __shfl_xor(l[hg], off, 64);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[hg][e] += __shfl_xor(o[hg][e], off, 64);
    }
    if (kq == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) sm_o[wave][hg][sl * 8 + e] = o[hg][e];
    }
    if (lane == 0) {
      sm_ml[wave][hg][0] = m[hg];
      sm_ml[wave][hg][1] = l[hg];
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < GMAX * DH; idx += NW * 64) {
    const int hg = idx / DH, d = idx % DH;
    const int hl = hc * GMAX + hg;
    if (hl >= G) break;
    const int h = g * G + hl;
    float mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) mx = fmaxf(mx, sm_ml[w][hg][0]);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = sm_ml[w][hg][0];
      if (mw == -INFINITY) continue;
      const float wt = __expf(mw - mx);
      num += wt * sm_o[w][hg][d];
      den += wt * sm_ml[w][hg][1];
    }
    const size_t ih = (size_t)i * c.H + h;
    if (nsplit == 1) {
      O[ih * DH + d] = Act<T>::from_f32(den > 0.f ? num / den : 0.f);
    } else {
      const size_t pidx = ih * nsplit + split;
      part_o[pidx * DH + d] = num;
      if (d == 0) {
        part_ml[pidx * 2 + 0] = den > 0.f ? mx : -INFINITY;
        part_ml[pidx * 2 + 1] = den;
      }
    }
  }
}

// O[i, h, :] = sum_ch w_ch o_ch / sum_ch w_ch l_ch, w_ch = exp(m_ch - max m)
template <typename T>
__global__ void decode_combine_kernel(const float* __restrict__ part_ml, const float* __restrict__ part_o, int b,
                                      int H, int nch, int dh, T* __restrict__ O) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= b * H * dh) return;
  const int d = idx % dh;
  const size_t ih = idx / dh;
  const float* ml = part_ml + ih * nch * 2;
  float mx = -INFINITY;
  for (int k = 0; k < nch; ++k) mx = fmaxf(mx, ml[2 * k]);
  float num = 0.f, den = 0.f;
  for (int k = 0; k < nch; ++k) {
    const float mk = ml[2 * k];
    if (mk == -INFINITY) continue;
    const float w = expf(mk - mx);
    den += w * ml[2 * k + 1];
    num += w * part_o[(ih * nch + k) * dh + d];
  }
  O[idx] = Act<T>::from_f32(den > 0.f ? num / den : 0.f);
}

hipError_t launch_decode_attention(int dtype, const void* q, const DecodeArgs& c, const int32_t* sel,
                                   float* part_ml, float* part_o, void* O, hipStream_t s) {
  constexpr int NW = 8;
  const int G = c.H / c.Hkv;
  // heads per workgroup: up to 4, whose softmax state fits in registers beside two segments
  const int gmax = G <= 1 ? 1 : G <= 2 ? 2 : 4;
  const int nhc = cdiv(G, gmax);
  // splits of the kept keys: enough workgroups for 256 CUs; the partial
  // buffers hold K + 1 per head
  const int groups = c.b * c.Hkv * nhc;
  const int nsplit = std::max(1, std::min(c.K + 1, cdiv(256, groups)));
  dim3 grid(nsplit * nhc, c.Hkv, c.b);
#define DA_LAUNCH(T, DH, GM)                                                                                   \
  decode_attn_kernel<T, DH, GM, NW><<<grid, NW * 64, 0, s>>>((const T*)q, c, sel, nsplit, part_ml, part_o, \
                                                              (T*)O)
#define DA_GMAX(T, DH)                       \
  do {                                       \
    if (gmax == 1) DA_LAUNCH(T, DH, 1);      \
    else if (gmax == 2) DA_LAUNCH(T, DH, 2); \
    else DA_LAUNCH(T, DH, 4);                \
  } while (0)
  if (dtype == SAS_BF16) {
    if (c.dh == 128) DA_GMAX(bf16_t, 128);
    else DA_GMAX(bf16_t, 64);
  } else {
    if (c.dh == 128) DA_GMAX(float, 128);
    else DA_GMAX(float, 64);
  }
#undef DA_GMAX
#undef DA_LAUNCH
  if (nsplit == 1) return hipGetLastError();
  const int tot = c.b * c.H * c.dh;
  if (dtype == SAS_BF16)
    decode_combine_kernel<bf16_t><<<cdiv(tot, 256), 256, 0, s>>>(part_ml, part_o, c.b, c.H, nsplit, c.dh, (bf16_t*)O);
  else
    decode_combine_kernel<float><<<cdiv(tot, 256), 256, 0, s>>>(part_ml, part_o, c.b, c.H, nsplit, c.dh, (float*)O);
  return hipGetLastError();
}

}  // namespace sas
