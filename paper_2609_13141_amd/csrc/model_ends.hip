// Model ends for the serving loop: token embedding (with image slots filled
// from precomputed image embeddings) and the greedy LM head (logits through
// the skinny GEMM, argmax here).
#include <float.h>

#include "common.h"
#include "kernels.h"

namespace sas {

// One workgroup per (b, t): an id >= 0 copies table row id; an id < 0 marks an
// image slot that takes the next row of img[b] (its rank among the row's
// negative ids so far).
template <typename T>
__global__ void __launch_bounds__(256) embed_kernel(const int32_t* __restrict__ ids, const T* __restrict__ table,
                                                    int vocab, const T* __restrict__ img, int n_img, T* __restrict__ x,
                                                    int n, int d) {
  const int t = blockIdx.x, bi = blockIdx.y;
  const int32_t* row = ids + (size_t)bi * n;
  const int id = row[t];
  const T* src = nullptr;
  if (id >= 0) {
    if (id < vocab) src = table + (size_t)id * d;
  } else {
    int cnt = 0;
    for (int u = threadIdx.x; u < t; u += 256) cnt += row[u] < 0 ? 1 : 0;
    __shared__ int part[4];
    cnt = (int)wave_sum((float)cnt);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = cnt;
    __syncthreads();
    const int slot = part[0] + part[1] + part[2] + part[3];
    if (img && slot < n_img) src = img + ((size_t)bi * n_img + slot) * d;
  }
  // 16-byte chunks (d is a multiple of 8, so rows are 16-byte aligned), up to
  // four per thread loaded before any is stored
  uint4* dst = (uint4*)(x + ((size_t)bi * n + t) * d);
  const uint4* s16 = (const uint4*)src;
  const int nch = d * (int)sizeof(T) / 16;
  for (int c0 = threadIdx.x; c0 < nch; c0 += 4 * 256) {
    uint4 r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) r[u] = src ? s16[min(c0 + u * 256, nch - 1)] : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (c0 + u * 256 < nch) dst[c0 + u * 256] = r[u];
  }
}

hipError_t launch_embed(int dtype, int b, int n, const int32_t* ids, const void* table, int vocab, const void* img,
                        int n_img, void* x, int d, hipStream_t s) {
  dim3 grid(n, b);
  if (dtype == SAS_BF16)
    embed_kernel<bf16_t><<<grid, 256, 0, s>>>(ids, (const bf16_t*)table, vocab, (const bf16_t*)img, n_img,
                                              (bf16_t*)x, n, d);
  else
    embed_kernel<float><<<grid, 256, 0, s>>>(ids, (const float*)table, vocab, (const float*)img, n_img, (float*)x,
                                             n, d);
  return hipGetLastError();
}

// argmax over logits[row, :] (fp32), lowest index on ties.  Stage 1: one
// workgroup per (row, slice) writes its best (value, index); stage 2 reduces
// the slices of a row.
__device__ __forceinline__ void better_of(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

__global__ void __launch_bounds__(256) argmax_stage1(const float* __restrict__ logits, int V, int slices,
                                                     float* __restrict__ pv, int32_t* __restrict__ pi) {
  const int row = blockIdx.y, sl = blockIdx.x;
  const int per = (V + slices - 1) / slices;
  const int lo = sl * per, hi = min(V, lo + per);
  float v = -INFINITY;
  int idx = 0x7fffffff;
  for (int j = lo + threadIdx.x; j < hi; j += 256) better_of(v, idx, logits[(size_t)row * V + j], j);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(v, o, 64);
    const int i2 = __shfl_xor(idx, o, 64);
    better_of(v, idx, v2, i2);
  }
  __shared__ float sv[4];
  __shared__ int si[4];
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = v;
    si[threadIdx.x >> 6] = idx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) better_of(v, idx, sv[w], si[w]);
    pv[(size_t)row * slices + sl] = v;
    pi[(size_t)row * slices + sl] = idx;
  }
}

// one wave per row: lane l takes slices l, l + 64, ... (the reduction under
// better_of does not depend on the order: larger value, then lower index)
__global__ void __launch_bounds__(64) argmax_stage2(const float* __restrict__ pv, const int32_t* __restrict__ pi,
                                                    int slices, int32_t* __restrict__ tokens) {
  const size_t row = blockIdx.x;
  float v = -INFINITY;
  int idx = 0x7fffffff;
  for (int s2 = threadIdx.x; s2 < slices; s2 += 64) better_of(v, idx, pv[row * slices + s2], pi[row * slices + s2]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(v, o, 64);
    const int i2 = __shfl_xor(idx, o, 64);
    better_of(v, idx, v2, i2);
  }
  if (threadIdx.x == 0) tokens[row] = idx;
}

hipError_t launch_argmax(const float* logits, int b, int V, float* pv, int32_t* pi, int slices, int32_t* tokens,
                         hipStream_t s) {
  if (b <= 0) return hipSuccess;
  argmax_stage1<<<dim3(slices, b), 256, 0, s>>>(logits, V, slices, pv, pi);
  argmax_stage2<<<b, 64, 0, s>>>(pv, pi, slices, tokens);
  return hipGetLastError();
}

}  // namespace sas
