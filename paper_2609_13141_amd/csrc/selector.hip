// SAS selector on the GPU: block summaries, gate query, exact scores,
// normalized log gate (Eq. normalized_log_gate) and Top-K selection
// (Eq. selected_context), one lane per query row.
//
// Exactness: summaries and gate queries are fp64 sums of activation-dtype
// values in ascending index order, rounded once to the activation dtype;
// scores are sequential fp64 FMA chains over ascending j (each product of two
// bf16/fp32 values is exact in fp64, so FMA equals multiply-then-add).  The
// ranking key is the exact score with ties going to the lower block index,
// so the selected indices are an integer function of the input bits.
#include <float.h>

#include "common.h"
#include "kernels.h"

namespace sas {

// ---------------------------------------------------------------------------
// Block summaries: thread per (b, g, m, j).
template <typename T>
__global__ void summaries_kernel(const T* __restrict__ K, T* __restrict__ out, int n, int Hkv, int dh,
                                 int B, int NB, size_t total) {
  size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  int j = (int)(idx % dh);
  size_t r = idx / dh;
  int m = (int)(r % NB);
  r /= NB;
  int g = (int)(r % Hkv);
  int bi = (int)(r / Hkv);
  if ((m + 1) * B > n) {  // incomplete block: no summary
    out[idx] = Act<T>::from_f32(0.f);
    return;
  }
  const T* p = K + (((size_t)bi * n + (size_t)m * B) * Hkv + g) * dh + j;
  const size_t stride = (size_t)Hkv * dh;
  double acc = 0.0;
  for (int i = 0; i < B; ++i) acc += (double)Act<T>::to_f32(p[(size_t)i * stride]);
  out[idx] = Act<T>::from_f64(acc / (double)B);
}

// Per-group projection out[.., g, m, k] = rho(sum_j W[g, k, j] * in[.., g, m, j]).
template <typename T>
__global__ void project_kernel(const T* __restrict__ in, const T* __restrict__ W, T* __restrict__ out,
                               int Hkv, int rows_per_group, int dh, size_t total) {
  size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  int k = (int)(idx % dh);
  size_t r = idx / dh;
  int g = (int)((r / rows_per_group) % Hkv);
  const T* v = in + r * dh;
  const T* w = W + ((size_t)g * dh + k) * dh;
  double acc = 0.0;
  for (int j = 0; j < dh; ++j)
    acc = fma((double)Act<T>::to_f32(w[j]), (double)Act<T>::to_f32(v[j]), acc);
  out[idx] = Act<T>::from_f64(acc);
}

hipError_t launch_block_summaries(int dtype, const void* K, int b, int n, int Hkv, int dh, int B,
                                  const void* w_gk, void* kplain, void* ksum, hipStream_t s) {
  const int NB = cdiv(n, B);
  const size_t total = (size_t)b * Hkv * NB * dh;
  if (total == 0) return hipSuccess;
  const unsigned grid = (unsigned)((total + 255) / 256);
  void* dst = w_gk ? kplain : ksum;
  if (dtype == SAS_BF16)
    summaries_kernel<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)K, (bf16_t*)dst, n, Hkv, dh, B, NB, total);
  else
    summaries_kernel<float><<<grid, 256, 0, s>>>((const float*)K, (float*)dst, n, Hkv, dh, B, NB, total);
  if (w_gk) {
    // rows of incomplete blocks are zero and project to zero
    if (dtype == SAS_BF16)
      project_kernel<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)kplain, (const bf16_t*)w_gk,
                                                  (bf16_t*)ksum, Hkv, NB, dh, total);
    else
      project_kernel<float><<<grid, 256, 0, s>>>((const float*)kplain, (const float*)w_gk,
                                                 (float*)ksum, Hkv, NB, dh, total);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Selection: one wave per 64 consecutive query rows of one (batch, group).
constexpr int SEL_MC = 16;  // summaries staged in LDS per step

template <typename T, int DH>
__device__ __forceinline__ double dot_f64(const float (&q)[DH], const float* __restrict__ kb) {
  double acc = 0.0;
#pragma unroll
  for (int j = 0; j < DH; j += 4) {
    float4 k4 = *(const float4*)(kb + j);
    acc = fma((double)q[j + 0], (double)k4.x, acc);
    acc = fma((double)q[j + 1], (double)k4.y, acc);
    acc = fma((double)q[j + 2], (double)k4.z, acc);
    acc = fma((double)q[j + 3], (double)k4.w, acc);
  }
  return acc;
}

template <typename T, int DH, int KMAX>
__global__ void __launch_bounds__(64) select_kernel(SelectArgs P) {
  __shared__ __align__(16) float kb[SEL_MC][DH];
  extern __shared__ __align__(16) float qs_dyn[];  // [WAVE][DH + 4]: pre-projection gate query (W_gq only)
  const int lane = threadIdx.x;
  const int g = blockIdx.y, bi = blockIdx.z;
  const int t = blockIdx.x * WAVE + lane;
  const bool valid = t < P.n;
  const int G = P.H / P.Hkv;
  const int ct = valid ? t / P.B : 0;
  const int t_last = min(P.n - 1, (int)blockIdx.x * WAVE + WAVE - 1);
  const int cmax = t_last / P.B;  // wave-uniform loop bound
  const double inv_scale = 1.0 / ((double)G * sqrt((double)DH));

  // gate query: rho(sum of the group's query heads), optionally projected
  float q[DH];
  {
    const T* Qr = (const T*)P.Q + (((size_t)bi * P.n + (valid ? t : 0)) * P.H + (size_t)g * G) * DH;
#pragma unroll
    for (int j = 0; j < DH; ++j) {
      double acc = 0.0;
      for (int h = 0; h < G; ++h) acc += (double)Act<T>::to_f32(Qr[(size_t)h * DH + j]);
      q[j] = Act<T>::to_f32(Act<T>::from_f64(acc));
    }
    if (P.w_gq) {
#pragma unroll
      for (int j = 0; j < DH; ++j) qs_dyn[lane * (DH + 4) + j] = q[j];
      const T* W = (const T*)P.w_gq + (size_t)g * DH * DH;
#pragma unroll
      for (int k = 0; k < DH; ++k) {
        double acc = 0.0;
        for (int j = 0; j < DH; ++j)
          acc = fma((double)Act<T>::to_f32(W[(size_t)k * DH + j]), (double)qs_dyn[lane * (DH + 4) + j], acc);
        q[k] = Act<T>::to_f32(Act<T>::from_f64(acc));
      }
    }
  }

  double tr[KMAX];
  int tm[KMAX];
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    tr[i] = -DBL_MAX;
    tm[i] = 0x7fffffff;
  }
  double mrun = -DBL_MAX;  // running max of s
  float lrun = 0.f;        // running sum of exp(s - mrun)

  const T* kbar = (const T*)P.kbar + ((size_t)bi * P.Hkv + g) * (size_t)P.NB * DH;
  for (int m0 = 0; m0 < cmax; m0 += SEL_MC) {
    const int mc = min(SEL_MC, cmax - m0);
    __syncthreads();
    for (int e = lane; e < mc * DH; e += WAVE) kb[e / DH][e % DH] = Act<T>::load(kbar, (size_t)m0 * DH + e);
    __syncthreads();
    for (int mm = 0; mm < mc; ++mm) {
      const int m = m0 + mm;
      if (m >= ct) continue;
      double r = dot_f64<T, DH>(q, kb[mm]);
      double sv = r * inv_scale;
      if (sv > mrun) {
        lrun = lrun * expf((float)(mrun - sv)) + 1.f;
        mrun = sv;
      } else {
        lrun += expf((float)(sv - mrun));
      }
      if (r > tr[KMAX - 1]) {
        double cr = r;
        int cm = m;
#pragma unroll
        for (int i = 0; i < KMAX; ++i) {
          bool better = cr > tr[i];  // strict: an equal key keeps the lower index ahead
          double orr = tr[i];
          int om = tm[i];
          tr[i] = better ? cr : orr;
          tm[i] = better ? cm : om;
          cr = better ? orr : cr;
          cm = better ? om : cm;
        }
      }
    }
  }
  if (!valid) return;
  const double lse = (ct > 0) ? mrun + log((double)lrun) : 0.0;
  const int K = P.K;
  const int kk = min(K, ct);
  const size_t row = ((size_t)bi * P.Hkv + g) * P.n + t;

  if (P.tau) {
    float tau;
    if (ct <= K) tau = -INFINITY;
    else if (K == 0) tau = INFINITY;
    else {
      double rk = tr[0];
#pragma unroll
      for (int i = 0; i < KMAX; ++i)
        if (i == K - 1) rk = tr[i];
      tau = (float)(rk * inv_scale - lse);
    }
    P.tau[row] = tau;
  }

  // order the kept blocks by index (odd-even transposition; empty slots last)
#pragma unroll
  for (int i = 0; i < KMAX; ++i)
    if (i >= kk) { tm[i] = 0x7fffffff; }
#pragma unroll
  for (int pass = 0; pass < KMAX; ++pass) {
#pragma unroll
    for (int i = (pass & 1); i + 1 < KMAX; i += 2) {
      bool sw = tm[i] > tm[i + 1];
      int a = tm[i], c = tm[i + 1];
      double ra = tr[i], rc = tr[i + 1];
      tm[i] = sw ? c : a;
      tm[i + 1] = sw ? a : c;
      tr[i] = sw ? rc : ra;
      tr[i + 1] = sw ? ra : rc;
    }
  }
  int32_t* sel = P.sel + row * K;
  float* sb = P.sel_bias + row * K;
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    if (i < K) {
      sel[i] = (i < kk) ? tm[i] : -1;
      sb[i] = (i < kk) ? (float)(tr[i] * inv_scale - lse) : 0.f;
    }
  }

  if (P.log_gate) {
    float* lg = P.log_gate + row * P.NB;
    for (int m = 0; m < P.NB; ++m) {
      float v = -INFINITY;
      if (m < ct) {
        const T* kr = kbar + (size_t)m * DH;
        double acc = 0.0;
#pragma unroll
        for (int j = 0; j < DH; ++j) acc = fma((double)q[j], (double)Act<T>::to_f32(kr[j]), acc);
        v = (float)(acc * inv_scale - lse);
      }
      lg[m] = v;
    }
  }
}

template <typename T, int DH>
static void run_select(const SelectArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.n, WAVE), a.Hkv, a.b);
  const size_t lds = a.w_gq ? (size_t)WAVE * (DH + 4) * sizeof(float) : 0;
  if (a.K <= 8) select_kernel<T, DH, 8><<<grid, WAVE, lds, s>>>(a);
  else if (a.K <= 16) select_kernel<T, DH, 16><<<grid, WAVE, lds, s>>>(a);
  else select_kernel<T, DH, 32><<<grid, WAVE, lds, s>>>(a);
}

hipError_t launch_select(int dtype, const SelectArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.b <= 0) return hipSuccess;
  if (dtype == SAS_BF16) {
    if (a.dh == 128) run_select<bf16_t, 128>(a, s);
    else run_select<bf16_t, 64>(a, s);
  } else {
    if (a.dh == 128) run_select<float, 128>(a, s);
    else run_select<float, 64>(a, s);
  }
  return hipGetLastError();
}

}  // namespace sas
