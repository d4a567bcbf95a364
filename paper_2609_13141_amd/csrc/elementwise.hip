// RMSNorm and the rotary-embedding table.
#include "common.h"
#include "kernels.h"

namespace sas {

// One workgroup of 256 threads per row; the row is read twice (L2-resident),
// sum of squares in fp32, output rounded once to the activation dtype.
template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const T* __restrict__ x, const T* __restrict__ gamma,
                                                      T* __restrict__ out, int d, float eps) {
  const size_t row = blockIdx.x;
  const T* xr = x + row * (size_t)d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    float v = Act<T>::to_f32(xr[i]);
    ss += v * v;
  }
  ss = wave_sum(ss);
  __shared__ float part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = part[0] + part[1] + part[2] + part[3];
  float inv = 1.0f / sqrtf(tot / (float)d + eps);
  T* o = out + row * (size_t)d;
  for (int i = threadIdx.x; i < d; i += 256) {
    float v = Act<T>::to_f32(xr[i]) * inv * Act<T>::to_f32(gamma[i]);
    o[i] = Act<T>::from_f32(v);
  }
}

hipError_t launch_rmsnorm(int dtype, const void* x, const void* gamma, void* out, int rows, int d,
                          float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (dtype == SAS_BF16)
    rmsnorm_kernel<bf16_t><<<rows, 256, 0, s>>>((const bf16_t*)x, (const bf16_t*)gamma, (bf16_t*)out, d, eps);
  else
    rmsnorm_kernel<float><<<rows, 256, 0, s>>>((const float*)x, (const float*)gamma, (float*)out, d, eps);
  return hipGetLastError();
}

__global__ void rope_table_kernel(float2* __restrict__ rope, int n, int half, int dh, double base) {
  int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n * half) return;
  int p = idx / half, i = idx % half;
  double theta = pow(base, -2.0 * (double)i / (double)dh);
  double ang = (double)p * theta;
  rope[idx] = make_float2((float)cos(ang), (float)sin(ang));
}

hipError_t launch_rope_table(float2* rope, int n, int dh, float base, hipStream_t s) {
  int half = dh / 2;
  int tot = n * half;
  if (tot <= 0) return hipSuccess;
  rope_table_kernel<<<cdiv(tot, 256), 256, 0, s>>>(rope, n, half, dh, (double)base);
  return hipGetLastError();
}

}  // namespace sas
