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
// One wave per (chunk, group, sequence); chunk ch < K is the ch-th kept block,
// ch == K the current block [B*floor(p/B), p].  Nothing is staged in LDS: with
// NC = dh/8 lanes per key, lane l holds the 8-value slice l % NC of keys
// l / NC + (64/NC) * it, loaded with coalesced 16-byte loads (a page of one KV
// head is contiguous).  A key's score is the partial dot product reduced over
// its NC lanes with shuffles; P V accumulates per slice and is reduced over
// the lanes that share a slice.  The partial (max, sum of exp, unnormalised
// output) is written in fp32 and merged by decode_combine_kernel.
template <typename T, int DH, int MAXKEYS>
__global__ void __launch_bounds__(64) decode_attn_kernel(const T* __restrict__ q, DecodeArgs c,
                                                         const int32_t* __restrict__ sel,
                                                         float* __restrict__ part_ml, float* __restrict__ part_o) {
  constexpr int NC = DH / 8;          // lanes per key (one 8-value slice each)
  constexpr int KPI = 64 / NC;        // keys per load instruction
  constexpr int IT = MAXKEYS / KPI;   // load steps
  const int lane = threadIdx.x;
  const int ch = blockIdx.x, g = blockIdx.y, i = blockIdx.z;
  const int K = c.K, G = c.H / c.Hkv, B = c.B;
  const int p = c.pos[i];
  int first = 0, count = 0;  // key positions [first, first + count)
  if (p >= 0) {
    if (ch < K) {
      const int m = sel[((size_t)i * c.Hkv + g) * K + ch];
      if (m >= 0) {
        first = m * B;
        count = B;
      }
    } else {
      first = (p / B) * B;
      count = p - first + 1;
    }
  }
  const int sl = lane % NC, kq = lane / NC;
  // page ids of the chunk (blocks are page aligned): lane j holds page j
  const int ps = c.page_size;
  const int npg = (count + ps - 1) / ps;
  int pid = -1;
  if (lane < npg) {
    const int pi = first / ps + lane;
    if (pi < c.max_pages) pid = c.block_table[(size_t)i * c.max_pages + pi];
    if (pid >= c.num_pages) pid = -1;
  }
  const size_t kvstride = (size_t)c.Hkv * ps * DH;  // elements per page
  for (int hg = 0; hg < G; ++hg) {
    const int h = g * G + hg;
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
      const int kl = kq + KPI * it;
      sc[it] = -INFINITY;
      if (KPI * it >= count) continue;
      const int page = __shfl(pid, kl / ps, 64);
      const bool ok = kl < count && page >= 0;
      Vec8<T> kv;
      if (ok) kv.load((const T*)c.k_pages + (size_t)page * kvstride + ((size_t)g * ps + kl % ps) * DH + sl * 8);
      float acc = 0.f;
      if (ok) {
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = fmaf(qs[e], kv.get(e), acc);
      }
#pragma unroll
      for (int o = NC / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
      sc[it] = kl < count ? acc : -INFINITY;
      mx = fmaxf(mx, sc[it]);
    }
    mx = wave_max(mx);
    float ls = 0.f, o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = 0.f;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int kl = kq + KPI * it;
      if (KPI * it >= count) continue;
      const int page = __shfl(pid, kl / ps, 64);
      const bool ok = kl < count && page >= 0;
      Vec8<T> vv;
      if (ok) vv.load((const T*)c.v_pages + (size_t)page * kvstride + ((size_t)g * ps + kl % ps) * DH + sl * 8);
      const float pk = kl < count ? __expf(sc[it] - mx) : 0.f;
      ls += pk;
      if (ok) {
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = fmaf(pk, vv.get(e), o[e]);
      }
    }
    // lanes sharing a slice hold different keys: reduce over them
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int off = NC; off < 64; off <<= 1) o[e] += __shfl_xor(o[e], off, 64);
#pragma unroll
    for (int off = NC; off < 64; off <<= 1) ls += __shfl_xor(ls, off, 64);  // each key once per slice
    const size_t pidx = ((size_t)i * c.H + h) * (K + 1) + ch;
    if (kq == 0) {
      float4* dst = (float4*)(part_o + pidx * DH + sl * 8);
      dst[0] = make_float4(o[0], o[1], o[2], o[3]);
      dst[1] = make_float4(o[4], o[5], o[6], o[7]);
    }
    if (lane == 0) {
      part_ml[pidx * 2 + 0] = count > 0 ? mx : -INFINITY;
      part_ml[pidx * 2 + 1] = count > 0 ? ls : 0.f;
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
  const int nch = c.K + 1;
  dim3 grid(nch, c.Hkv, c.b);
#define DA_LAUNCH(T, DH, MK) \
  decode_attn_kernel<T, DH, MK><<<grid, 64, 0, s>>>((const T*)q, c, sel, part_ml, part_o)
  const bool wide = c.B > 64;
  if (dtype == SAS_BF16) {
    if (c.dh == 128) {
      if (wide) DA_LAUNCH(bf16_t, 128, 128); else DA_LAUNCH(bf16_t, 128, 64);
    } else {
      if (wide) DA_LAUNCH(bf16_t, 64, 128); else DA_LAUNCH(bf16_t, 64, 64);
    }
  } else {
    if (c.dh == 128) {
      if (wide) DA_LAUNCH(float, 128, 128); else DA_LAUNCH(float, 128, 64);
    } else {
      if (wide) DA_LAUNCH(float, 64, 128); else DA_LAUNCH(float, 64, 64);
    }
  }
#undef DA_LAUNCH
  const int tot = c.b * c.H * c.dh;
  if (dtype == SAS_BF16)
    decode_combine_kernel<bf16_t><<<cdiv(tot, 256), 256, 0, s>>>(part_ml, part_o, c.b, c.H, nch, c.dh, (bf16_t*)O);
  else
    decode_combine_kernel<float><<<cdiv(tot, 256), 256, 0, s>>>(part_ml, part_o, c.b, c.H, nch, c.dh, (float*)O);
  return hipGetLastError();
}

}  // namespace sas
