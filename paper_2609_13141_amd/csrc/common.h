// Device helpers shared by the SAS kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sas.h"

namespace sas {

typedef uint16_t bf16_t;  // bfloat16 storage

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16_t;

constexpr int WAVE = 64;

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// float -> bfloat16 with the hardware conversion (v_cvt_pk_bf16_f32): round
// to nearest even, NaN stays NaN; pack_bf16x2 converts two values at once.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));  // 16 bytes as a native vector
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t f = {lo, hi};
  const bf16x2_t h = __builtin_convertvector(f, bf16x2_t);
  return __builtin_bit_cast(uint32_t, h);
}
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, (__bf16)f);
}

// Workgroup barrier after this wave's LDS accesses complete (s_waitcnt
// lgkmcnt(0); s_barrier).  Unlike __syncthreads() it does not wait for
// outstanding global loads, so loads issued for the next step stay in flight.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// next set bit at or after p in an LDS bitmask of `count` bits (count if none)
__device__ __forceinline__ int next_set(const uint32_t* bits, int p, int count) {
  while (p < count) {
    const uint32_t w = bits[p >> 5] >> (p & 31);
    if (w) return p + __builtin_ctz(w);
    p = (p | 31) + 1;
  }
  return count;
}

// double -> bfloat16 directly (one rounding, ties to even), including
// subnormal results and overflow to infinity.
__device__ __forceinline__ bf16_t f64_to_bf16(double d) {
  uint64_t u = (uint64_t)__double_as_longlong(d);
  uint32_t sign = (uint32_t)(u >> 48) & 0x8000u;
  uint64_t a = u & 0x7fffffffffffffffull;
  if (a >= 0x7ff0000000000000ull) {  // inf / nan
    return (bf16_t)(sign | 0x7f80u | (a > 0x7ff0000000000000ull ? 0x40u : 0u));
  }
  double ad = __longlong_as_double((long long)a);
  if (ad < 0x1p-126) {  // bfloat16 subnormal range: spacing 2^-133
    double r = rint(ad * 0x1p133);  // <= 128, exact; 128 is the smallest normal
    return (bf16_t)(sign | (uint32_t)r);
  }
  // keep 7 mantissa bits of the double: round at bit 45 (ties to even); a
  // carry propagates into the exponent naturally
  uint64_t r = (a + 0x00000fffffffffffull + ((a >> 45) & 1ull)) >> 45;
  // r = (biased_exp_d << 7) | mant7 ; rebias 1023 -> 127
  int64_t e = (int64_t)(r >> 7) - 1023 + 127;
  if (e >= 255) return (bf16_t)(sign | 0x7f80u);
  return (bf16_t)(sign | ((uint32_t)e << 7) | (uint32_t)(r & 0x7f));
}

template <typename T> struct Act;
template <> struct Act<float> {
  static __device__ __forceinline__ float load(const float* p, size_t i) { return p[i]; }
  static __device__ __forceinline__ float to_f32(float v) { return v; }
  static __device__ __forceinline__ float from_f32(float v) { return v; }
  static __device__ __forceinline__ float from_f64(double v) { return (float)v; }
};
template <> struct Act<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p, size_t i) { return bf16_to_f32(p[i]); }
  static __device__ __forceinline__ float to_f32(bf16_t v) { return bf16_to_f32(v); }
  static __device__ __forceinline__ bf16_t from_f32(float v) { return f32_to_bf16(v); }
  static __device__ __forceinline__ bf16_t from_f64(double v) { return f64_to_bf16(v); }
};

// 8 consecutive activation values as floats (one 16-byte load for bf16).
template <typename T> struct Vec8;
template <> struct Vec8<bf16_t> {
  uint4 u;
  __device__ __forceinline__ void load(const bf16_t* p) { u = *(const uint4*)p; }
  __device__ __forceinline__ float get(int e) const {
    const uint32_t w = e < 2 ? u.x : e < 4 ? u.y : e < 6 ? u.z : u.w;
    return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
  }
};
template <> struct Vec8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = *(const float4*)p;
    b = *(const float4*)(p + 4);
  }
  __device__ __forceinline__ float get(int e) const {
    const float4& v = e < 4 ? a : b;
    const int k = e & 3;
    return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
  }
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Work queue of the attention kernels: the grid holds only as many
// workgroups as the chip runs at once, and each takes the next job from a
// counter in global memory until none is left.  Their jobs (query or key
// tiles) vary in length by the causal prefix they walk, and a launch of one
// workgroup per job leaves a large share of the compute units idle while the
// dispatcher waits to place the next workgroup; jobs are numbered longest
// first.  The counter is reset by the launch before the kernel runs, and
// every workgroup leaves once the counter has passed the job count.
__device__ __forceinline__ int queue_next_job(uint32_t* counter) {
  __shared__ int job_s;
  __syncthreads();  // every thread has finished the previous job and read job_s
  if (threadIdx.x == 0) job_s = (int)atomicAdd(counter, 1u);
  __syncthreads();
  return job_s;
}

// workgroups of `kernel` with `threads` threads resident on the current device
// at once (0 when the runtime cannot tell)
template <typename F>
inline int resident_workgroups(F kernel, int threads) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) return 0;
  return cus * (per_cu > 0 ? per_cu : 1);
}

}  // namespace sas
