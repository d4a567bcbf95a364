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

struct PageGeom {
  const int32_t* table;
  int num_pages, ps, max_pages;
  // element offset of (seq, group, position) in the page pool, or -1
  __device__ __forceinline__ long long offset(int i, int g, int p, int Hkv, int dh) const {
    if (p < 0) return -1;
    const int pi = p / ps;
    if (pi >= max_pages) return -1;
    const int page = table[(size_t)i * max_pages + pi];
    if (page < 0 || page >= num_pages) return -1;
    return (((long long)page * Hkv + g) * ps + (p % ps)) * dh;
  }
};

__device__ __forceinline__ PageGeom geom_of(const DecodeArgs& c) {
  PageGeom G;
  G.table = c.block_table;
  G.num_pages = c.num_pages;
  G.ps = c.page_size;
  G.max_pages = c.max_pages;
  return G;
}

// ---- rotary table for the positions of the new tokens -----------------------
__global__ void rope_rows_kernel(const int32_t* __restrict__ pos, float2* __restrict__ rope, int b, int half,
                                 int dh, double base) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= b * half) return;
  const int r = idx / half, i = idx % half;
  const double ang = (double)pos[r] * pow(base, -2.0 * (double)i / (double)dh);
  rope[idx] = make_float2((float)cos(ang), (float)sin(ang));
}

hipError_t launch_rope_rows(const int32_t* pos, float2* rope, int b, int dh, float base, hipStream_t s) {
  const int tot = b * (dh / 2);
  rope_rows_kernel<<<cdiv(tot, 256), 256, 0, s>>>(pos, rope, b, dh / 2, dh, (double)base);
  return hipGetLastError();
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
                             int dh, int B, int NB, const DecodeArgs& c, hipStream_t s) {
  const size_t total = (size_t)b * n * Hkv * (dh / 8);
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
  double acc = 0.0;
  for (int q = m * c.B; q < p; ++q) {
    const long long o = G.offset(i, g, q, c.Hkv, c.dh);
    acc += (double)Act<T>::to_f32(o >= 0 ? ((const T*)c.k_pages)[o + j] : Act<T>::from_f32(0.f));
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
// written in ascending block order.
constexpr int DSEL_MAXB = 2048;  // historical blocks per query supported by this kernel

template <typename T>
__global__ void __launch_bounds__(64) decode_select_kernel(const T* __restrict__ q, DecodeArgs c,
                                                           int32_t* __restrict__ sel) {
  __shared__ double qh[128];
  __shared__ double qp[128];
  __shared__ double rs[DSEL_MAXB];
  const int lane = threadIdx.x;
  const int g = blockIdx.x, i = blockIdx.y;
  const int G = c.H / c.Hkv, dh = c.dh, K = c.K;
  const int p = c.pos[i];
  const int ct = max(0, min(p / c.B, min(c.max_blocks, DSEL_MAXB)));
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
  const T* ks = (const T*)c.k_summary + ((size_t)i * c.Hkv + g) * c.max_blocks * dh;
  for (int m = lane; m < ct; m += 64) {
    const T* kr = ks + (size_t)m * dh;
    double acc = 0.0;
    for (int j = 0; j < dh; ++j) acc = fma(qh[j], (double)Act<T>::to_f32(kr[j]), acc);
    rs[m] = acc;
  }
  __syncthreads();
  int32_t* out = sel + ((size_t)i * c.Hkv + g) * K;
  int base = 0;
  for (int m0 = 0; m0 < ct; m0 += 64) {
    const int m = m0 + lane;
    bool keep = false;
    if (m < ct) {
      const double r = rs[m];
      int rank = 0;
      for (int o = 0; o < ct && rank < K; ++o) {
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

hipError_t launch_decode_select(int dtype, const void* q, const DecodeArgs& c, int32_t* sel, hipStream_t s) {
  if (c.K <= 0) return hipSuccess;
  dim3 grid(c.Hkv, c.b);
  if (dtype == SAS_BF16) decode_select_kernel<bf16_t><<<grid, 64, 0, s>>>((const bf16_t*)q, c, sel);
  else decode_select_kernel<float><<<grid, 64, 0, s>>>((const float*)q, c, sel);
  return hipGetLastError();
}

// ---- sparse attention of the new tokens ----------------------------------------
// One workgroup of NW waves per (split, head chunk, group, sequence).  The kept
// keys of a group are walked in segments of SEG keys: the K selected blocks in
// selection order (a block of B > SEG keys is B / SEG segments), then the
// current block [B*floor(p/B), p].  A split is a contiguous range of segments;
// the workgroup first resolves where each of its segments starts (one pass,
// into LDS), then deals them to its waves round-robin.  Nothing else is staged
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
  static constexpr int SEG = 8192 / (DH * (int)sizeof(T));   // keys per segment: K and V in 64 VGPRs
  static constexpr int IT = SEG / KPI;                       // load steps per segment
  Vec8<T> k[IT], v[IT];
  bool ok[IT];
  int count;
};

constexpr int DSEG_MAX = 33 * 8;  // segments of a split: (K + 1) blocks of at most 8 segments

template <typename T, int DH, int GMAX, int NW>
__global__ void __launch_bounds__(NW * 64) decode_attn_kernel(const T* __restrict__ q, DecodeArgs c,
                                                              const int32_t* __restrict__ sel, int nsplit,
                                                              float* __restrict__ part_ml,
                                                              float* __restrict__ part_o, T* __restrict__ O) {
  using Seg = DecodeSeg<T, DH>;
  constexpr int NC = Seg::NC, KPI = Seg::KPI, SEG = Seg::SEG, IT = Seg::IT;
  __shared__ float sm_o[NW][GMAX][DH];
  __shared__ float sm_ml[NW][GMAX][2];
  __shared__ int sm_first[DSEG_MAX], sm_count[DSEG_MAX];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int G = c.H / c.Hkv, nhc = (G + GMAX - 1) / GMAX;
  const int split = blockIdx.x / nhc, hc = blockIdx.x % nhc;
  const int g = blockIdx.y, i = blockIdx.z;
  const int K = c.K, B = c.B;
  const int spb = B > SEG ? B / SEG : 1;  // segments per block
  const int seg_len = B > SEG ? SEG : B;
  const int nseg = (K + 1) * spb;
  const int per = (nseg + nsplit - 1) / nsplit;
  const int s0 = split * per, s1 = min(nseg, s0 + per);
  const int p = c.pos[i];
  const int sl = lane % NC, kq = lane / NC;
  const int ps = c.page_size;
  const size_t kvstride = (size_t)c.Hkv * ps * DH;  // elements per page

  // key range [first, first + count) of every segment of the split
  for (int t = threadIdx.x; t < s1 - s0; t += NW * 64) {
    const int sg = s0 + t, ch = sg / spb, sub = sg % spb;
    int first = 0, count = 0;
    if (p >= 0) {
      if (ch < K) {
        const int mb = sel[((size_t)i * c.Hkv + g) * K + ch];
        if (mb >= 0) {
          first = mb * B + sub * seg_len;
          count = seg_len;
        }
      } else {
        first = (p / B) * B + sub * seg_len;
        count = max(0, min(seg_len, p - first + 1));
      }
    }
    sm_first[t] = first;
    sm_count[t] = count;
  }
  __syncthreads();

  auto load = [&](Seg& S, int t) {
    const int first = sm_first[t];
    S.count = sm_count[t];
    // page ids of the segment: lane j holds the j-th page from the one holding `first`
    // (a segment spans at most 64 pages)
    const int koff = first % ps;
    const int npg = (koff + S.count + ps - 1) / ps;
    int pid = -1;
    if (lane < npg) {
      const int pi = first / ps + lane;
      if (pi < c.max_pages) pid = c.block_table[(size_t)i * c.max_pages + pi];
      if (pid >= c.num_pages) pid = -1;
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int kl = kq + KPI * it;
      const int a = koff + kl;  // offset from the start of the first page
      const int page = __shfl(pid, min(a / ps, 63), 64);
      S.ok[it] = kl < S.count && page >= 0;
      if (S.ok[it]) {
        const size_t off = (size_t)page * kvstride + ((size_t)g * ps + a % ps) * DH + sl * 8;
        S.k[it].load((const T*)c.k_pages + off);
        S.v[it].load((const T*)c.v_pages + off);
      }
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
  auto compute = [&](const Seg& S) {
    if (S.count <= 0) return;
#pragma unroll
    for (int hg = 0; hg < GMAX; ++hg) {
      const int hl = hc * GMAX + hg;
      if (hl >= G) break;
      const int h = g * G + hl;
      float qs[8];
      {
        Vec8<T> v;
        v.load(q + ((size_t)i * c.H + h) * DH + sl * 8);
#pragma unroll
        for (int e = 0; e < 8; ++e) qs[e] = v.get(e) * c.sm_scale;
      }
      float sc[IT];
      float mx = -INFINITY;
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        float acc = 0.f;
        if (S.ok[it]) {
#pragma unroll
          for (int e = 0; e < 8; ++e) acc = fmaf(qs[e], S.k[it].get(e), acc);
        }
#pragma unroll
        for (int off = NC / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
        sc[it] = kq + KPI * it < S.count ? acc : -INFINITY;
        mx = fmaxf(mx, sc[it]);
      }
      mx = wave_max(mx);
      const float mn = fmaxf(m[hg], mx);
      const float scale = __expf(m[hg] - mn);
      m[hg] = mn;
      l[hg] *= scale;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[hg][e] *= scale;
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const float pk = kq + KPI * it < S.count ? __expf(sc[it] - mn) : 0.f;
        l[hg] += pk;
        if (S.ok[it]) {
#pragma unroll
          for (int e = 0; e < 8; ++e) o[hg][e] = fmaf(pk, S.v[it].get(e), o[hg][e]);
        }
      }
    }
  };

  // two segments in registers: the next one's loads are in flight while one is computed
  const int ns = s1 - s0;
  Seg sa, sb;
  if (wave < ns) load(sa, wave);
  for (int t = wave; t < ns; t += 2 * NW) {
    if (t + NW < ns) load(sb, t + NW);
    compute(sa);
    if (t + NW >= ns) break;
    if (t + 2 * NW < ns) load(sa, t + 2 * NW);
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
