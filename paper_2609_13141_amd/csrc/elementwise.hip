// RMSNorm, optionally with the rotary-embedding table of its rows.
#include "common.h"
#include "kernels.h"

namespace sas {

// One workgroup of 256 threads per row; each thread keeps its 16-byte
// chunks of the row in registers between the sum of squares (fp32) and the
// scaled write, rounded once to the activation dtype.  With ROPE a row
// below rope_rows also writes its rotary table entries for position pos[row]
// (the row index itself without pos): rope[row, i] = (cos, sin) of
// pos * base^(-2i/dh), evaluated in fp64 and rounded to fp32, computed while
// the row's loads are in flight.
template <typename T, int CPT, bool ROPE>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const T* __restrict__ x, const T* __restrict__ gamma,
                                                      T* __restrict__ out, int d, float eps,
                                                      const int32_t* __restrict__ pos, float2* __restrict__ rope,
                                                      int dh, double base, int rope_rows) {
  constexpr int EPC = 16 / sizeof(T);  // elements per 16-byte chunk
  const size_t row = blockIdx.x;
  const T* xr = x + row * (size_t)d;
  T* o = out + row * (size_t)d;
  const int nch = d / EPC;
  // the row and the gains are loaded together: one memory round trip before the reduction
  uint4 v[CPT], gv[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = threadIdx.x + i * 256;
    v[i] = c < nch ? *(const uint4*)(xr + (size_t)c * EPC) : make_uint4(0, 0, 0, 0);
    gv[i] = c < nch ? *(const uint4*)(gamma + (size_t)c * EPC) : make_uint4(0, 0, 0, 0);
  }
  if constexpr (ROPE) {
    const int half = dh >> 1;
    if (row < (size_t)rope_rows) {
      const double p = pos ? (double)pos[row] : (double)row;
      for (int i = threadIdx.x; i < half; i += 256) {
        const double ang = p * pow(base, -2.0 * (double)i / (double)dh);
        rope[row * (size_t)half + i] = make_float2((float)cos(ang), (float)sin(ang));
      }
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const T* e = (const T*)&v[i];
#pragma unroll
    for (int k = 0; k < EPC; ++k) {
      const float f = Act<T>::to_f32(e[k]);
      ss += f * f;
    }
  }
  ss = wave_sum(ss);
  __shared__ float part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = part[0] + part[1] + part[2] + part[3];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int c = threadIdx.x + i * 256;
    if (c >= nch) continue;
    const T* e = (const T*)&v[i];
    const T* ge = (const T*)&gv[i];
    uint4 r;
    T* re = (T*)&r;
#pragma unroll
    for (int k = 0; k < EPC; ++k) re[k] = Act<T>::from_f32(Act<T>::to_f32(e[k]) * inv * Act<T>::to_f32(ge[k]));
    *(uint4*)(o + (size_t)c * EPC) = r;
  }
}

hipError_t launch_rmsnorm_rope(int dtype, const void* x, const void* gamma, void* out, int rows, int d, float eps,
                               const int32_t* pos, float2* rope, int dh, float base, int rope_rows,
                               hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  // d is a multiple of 8 (validated); up to 16 chunks of 16 bytes per thread
  const int epc = dtype == SAS_BF16 ? 8 : 4;
  const int cpt = (d / epc + 255) / 256;
  if (cpt > 16) return hipErrorInvalidValue;
  if (rope && rope_rows > rows) return hipErrorInvalidValue;
#define RMS_LAUNCH(T, C)                                                                                      \
  (rope ? rmsnorm_kernel<T, C, true><<<rows, 256, 0, s>>>((const T*)x, (const T*)gamma, (T*)out, d, eps, pos, \
                                                          rope, dh, (double)base, rope_rows)                  \
        : rmsnorm_kernel<T, C, false><<<rows, 256, 0, s>>>((const T*)x, (const T*)gamma, (T*)out, d, eps,     \
                                                           nullptr, nullptr, dh, 0.0, 0))
  if (dtype == SAS_BF16) {
    if (cpt <= 2) RMS_LAUNCH(bf16_t, 2);
    else if (cpt <= 4) RMS_LAUNCH(bf16_t, 4);
    else RMS_LAUNCH(bf16_t, 16);
  } else {
    if (cpt <= 2) RMS_LAUNCH(float, 2);
    else if (cpt <= 4) RMS_LAUNCH(float, 4);
    else RMS_LAUNCH(float, 16);
  }
#undef RMS_LAUNCH
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int dtype, const void* x, const void* gamma, void* out, int rows, int d,
                          float eps, hipStream_t s) {
  return launch_rmsnorm_rope(dtype, x, gamma, out, rows, d, eps, nullptr, nullptr, 0, 0.f, 0, s);
}

}  // namespace sas
