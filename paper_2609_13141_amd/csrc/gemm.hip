// C = A[M, K] * B[N, K]^T on MFMA (bf16 in, fp32 accumulate) with fused
// epilogues: QKV projection + RoPE, SwiGLU (gate and up in one pass),
// residual add.  A fp32 variant (plain FMA) serves the fp32 dtype.
//
// Epilogues that combine two output columns (RoPE rotates the pair
// (i, i + dh/2) of a head; SwiGLU multiplies gate column f by up column f)
// get both columns into the same lane by permuting the B rows as they are
// loaded: logical column J of the tile maps to pair p = (J/64)*32 + J%32 and
// half (J/32)%2.  A 32x32 MFMA output tile holds column J%32 in lane J%32, so
// the two halves of a pair sit in neighbouring 32-column subtiles of the same
// lane.  Plain (residual) GEMMs use the identity mapping.
#include "common.h"
#include "kernels.h"

namespace sas {

struct GemmParams {
  int epi, M, K, N;  // N = logical columns of the tiling
  int npairs;        // pair epilogues: number of output column pairs
  const bf16_t* A;
  const bf16_t* B0;
  const bf16_t* B1;
  const bf16_t* B2;
  const bf16_t* resid;
  bf16_t* out;
  bf16_t* out1;
  bf16_t* out2;
  int H, Hkv, dh, seq_len;
  const float2* rope;
  const int32_t* row_pos;
};

// Source row (in units of K elements) of logical column J, or null past the
// last column (RESID: J >= N; pair epilogues: pair index >= npairs).
template <typename T>
__device__ __forceinline__ const T* b_row(int epi, int J, int N, int npairs, int K, const T* B0,
                                          const T* B1, const T* B2, int H, int Hkv, int dh) {
  if (epi == EPI_RESID) return (J < N) ? B0 + (size_t)J * K : nullptr;
  int p = (J >> 6) * 32 + (J & 31);
  int half = (J >> 5) & 1;
  if (p >= npairs) return nullptr;
  if (epi == EPI_SWIGLU) return (half ? B1 : B0) + (size_t)p * K;
  int hh = dh >> 1;
  int hd = p / hh, ir = p % hh;
  int c = hd * dh + ir + half * hh;
  if (c < H * dh) return B0 + (size_t)c * K;
  c -= H * dh;
  if (c < Hkv * dh) return B1 + (size_t)c * K;
  return B2 + (size_t)(c - Hkv * dh) * K;
}

__device__ __forceinline__ float silu_f(float x) { return x / (1.0f + __expf(-x)); }

constexpr int BK = 64;

template <int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_bf16_kernel(GemmParams P) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int ACH = BM * 8 / NT;  // 16-byte A chunks per thread per k-tile
  constexpr int BCH = BN * 8 / NT;
  static_assert(ACH * NT == BM * 8 && BCH * NT == BN * 8, "tile/threads mismatch");
  static_assert(TN % 64 == 0, "pair epilogues need 64-column wave tiles");

  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* As = (bf16_t*)smem;                 // [2][BM][64]
  bf16_t* Bs = As + 2 * BM * BK;              // [2][BN][64]

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  const int Mt = (P.M + BM - 1) / BM;
  const int tile = blockIdx.x;
  const int mt = tile % Mt, nt = tile / Mt;
  const int m0 = mt * BM, n0 = nt * BN;

  // per-thread global source pointers (fixed along K)
  const bf16_t* a_src[ACH];
  const bf16_t* b_src[BCH];
  int a_lds[ACH], b_lds[BCH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    int c = tid + i * NT;
    int row = c >> 3, c16 = c & 7;
    int gr = m0 + row;
    a_src[i] = (gr < P.M) ? P.A + (size_t)gr * P.K + c16 * 8 : nullptr;
    a_lds[i] = row * BK + ((c16 ^ (row & 7)) << 3);
  }
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    int c = tid + i * NT;
    int row = c >> 3, c16 = c & 7;
    const bf16_t* r = b_row<bf16_t>(P.epi, n0 + row, P.N, P.npairs, P.K, P.B0, P.B1, P.B2, P.H,
                                    P.Hkv, P.dh);
    b_src[i] = r ? r + c16 * 8 : nullptr;
    b_lds[i] = row * BK + ((c16 ^ (row & 7)) << 3);
  }

  floatx16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  uint4 ra[ACH], rb[BCH];
  const int nk = (P.K + BK - 1) / BK;
  const bool k_full = (P.K % BK) == 0;

  auto gload = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      int kc = k0 + (((tid + i * NT) & 7) << 3);
      bool ok = a_src[i] && (k_full || kc < P.K);
      ra[i] = ok ? *(const uint4*)(a_src[i] + k0) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      int kc = k0 + (((tid + i * NT) & 7) << 3);
      bool ok = b_src[i] && (k_full || kc < P.K);
      rb[i] = ok ? *(const uint4*)(b_src[i] + k0) : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int buf) {
    bf16_t* a = As + buf * BM * BK;
    bf16_t* b = Bs + buf * BN * BK;
#pragma unroll
    for (int i = 0; i < ACH; ++i) *(uint4*)(a + a_lds[i]) = ra[i];
#pragma unroll
    for (int i = 0; i < BCH; ++i) *(uint4*)(b + b_lds[i]) = rb[i];
  };

  gload(0);
  lstore(0);
  __syncthreads();

  const int lr = lane & 31, lk = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload(kt + 1);
    const bf16_t* a = As + (kt & 1) * BM * BK;
    const bf16_t* b = Bs + (kt & 1) * BN * BK;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int kc = kk * 2 + lk;
      bf16x8_t fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        int row = wm * TM + i * 32 + lr;
        fa[i] = *(const bf16x8_t*)(a + row * BK + ((kc ^ (row & 7)) << 3));
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        int row = wn * TN + j * 32 + lr;
        fb[j] = *(const bf16x8_t*)(b + row * BK + ((kc ^ (row & 7)) << 3));
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore((kt + 1) & 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds column lr of each 32x32 subtile, rows
  // 8*(v/4) + 4*lk + (v%4) ----
  const int colbase = n0 + wn * TN;
  if (P.epi == EPI_RESID) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        int col = colbase + j * 32 + lr;
        if (col >= P.N) continue;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          int row = m0 + wm * TM + i * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
          if (row < P.M) {
            size_t o = (size_t)row * P.N + col;
            P.out[o] = f32_to_bf16(acc[i][j][v] + bf16_to_f32(P.resid[o]));
          }
        }
      }
    return;
  }
  const int hh = P.dh >> 1;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int jp = 0; jp < FN / 2; ++jp) {
      int J = colbase + jp * 64 + lr;  // half-0 logical column
      int p = (J >> 6) * 32 + (J & 31);
      if (p >= P.npairs) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        int row = m0 + wm * TM + i * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
        if (row >= P.M) continue;
        float x1 = acc[i][2 * jp][v], x2 = acc[i][2 * jp + 1][v];
        if (P.epi == EPI_SWIGLU) {
          P.out[(size_t)row * P.npairs + p] = f32_to_bf16(silu_f(x1) * x2);
        } else {
          int hd = p / hh, ir = p % hh;
          bf16_t* dst;
          if (hd < P.H) {
            dst = P.out + ((size_t)row * P.H + hd) * P.dh;
          } else if (hd < P.H + P.Hkv) {
            dst = P.out1 + ((size_t)row * P.Hkv + (hd - P.H)) * P.dh;
          } else {
            dst = P.out2 + ((size_t)row * P.Hkv + (hd - P.H - P.Hkv)) * P.dh;
          }
          if (hd < P.H + P.Hkv) {
            int pos = P.row_pos ? P.row_pos[row] : row % P.seq_len;
            float2 cs = P.rope[(size_t)pos * hh + ir];
            float o1 = x1 * cs.x - x2 * cs.y;
            float o2 = x2 * cs.x + x1 * cs.y;
            x1 = o1;
            x2 = o2;
          }
          dst[ir] = f32_to_bf16(x1);
          dst[ir + hh] = f32_to_bf16(x2);
        }
      }
    }
}

// ---- fp32 path: one thread per (row, logical pair or column) ----------------
__global__ void gemm_f32_kernel(int epi, int M, int K, int N, int npairs, const float* __restrict__ A,
                                const float* __restrict__ B0, const float* __restrict__ B1,
                                const float* __restrict__ B2, const float* __restrict__ resid,
                                float* out, float* out1, float* out2, int H, int Hkv, int dh,
                                int seq_len, const float2* __restrict__ rope,
                                const int32_t* __restrict__ row_pos) {
  const int cols = (epi == EPI_RESID) ? N : npairs;  // columns or pairs
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)M * cols) return;
  const int row = (int)(idx / cols), c = (int)(idx % cols);
  const float* a = A + (size_t)row * K;
  if (epi == EPI_RESID) {
    const float* b = B0 + (size_t)c * K;
    float s = 0.f;
    for (int k = 0; k < K; ++k) s = fmaf(a[k], b[k], s);
    out[(size_t)row * N + c] = resid[(size_t)row * N + c] + s;
    return;
  }
  // logical pair c -> the two logical columns of the tile mapping
  const int J = (c / 32) * 64 + (c % 32);
  const float* b1 = b_row<float>(epi, J, N, npairs, K, B0, B1, B2, H, Hkv, dh);
  const float* b2 = b_row<float>(epi, J + 32, N, npairs, K, B0, B1, B2, H, Hkv, dh);
  float x1 = 0.f, x2 = 0.f;
  for (int k = 0; k < K; ++k) {
    x1 = fmaf(a[k], b1[k], x1);
    x2 = fmaf(a[k], b2[k], x2);
  }
  if (epi == EPI_SWIGLU) {
    out[(size_t)row * npairs + c] = silu_f(x1) * x2;
    return;
  }
  const int hh = dh / 2;
  const int hd = c / hh, ir = c % hh;
  float* dst;
  if (hd < H) dst = out + ((size_t)row * H + hd) * dh;
  else if (hd < H + Hkv) dst = out1 + ((size_t)row * Hkv + (hd - H)) * dh;
  else dst = out2 + ((size_t)row * Hkv + (hd - H - Hkv)) * dh;
  if (hd < H + Hkv) {
    int pos = row_pos ? row_pos[row] : row % seq_len;
    float2 cs = rope[(size_t)pos * hh + ir];
    float o1 = x1 * cs.x - x2 * cs.y;
    float o2 = x2 * cs.x + x1 * cs.y;
    x1 = o1;
    x2 = o2;
  }
  dst[ir] = x1;
  dst[ir + hh] = x2;
}

template <int BM, int BN, int WM, int WN>
static hipError_t run_bf16(const GemmParams& P, hipStream_t s) {
  constexpr int NT = WM * WN * 64;
  const int tiles = ((P.M + BM - 1) / BM) * ((P.N + BN - 1) / BN);
  const size_t lds = (size_t)2 * (BM + BN) * BK * sizeof(bf16_t);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN>), dim3(tiles), dim3(NT), lds, s, P);
  return hipGetLastError();
}

static bool attrs_done = false;

hipError_t launch_gemm(int dtype, const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0) return hipSuccess;
  // pair epilogues: SWIGLU has F pairs, QKV has (H + 2 Hkv) dh / 2 pairs
  const int npairs = g.epi == EPI_SWIGLU ? g.N : (g.epi == EPI_QKV_ROPE ? g.N / 2 : 0);
  const int nlog = g.epi == EPI_RESID ? g.N : (npairs + 31) / 32 * 64;
  if (dtype == SAS_F32) {
    const int cols = (g.epi == EPI_RESID) ? g.N : npairs;
    size_t tot = (size_t)g.M * cols;
    gemm_f32_kernel<<<(unsigned)((tot + 255) / 256), 256, 0, s>>>(
        g.epi, g.M, g.K, nlog, npairs, (const float*)g.A, (const float*)g.B0, (const float*)g.B1,
        (const float*)g.B2, (const float*)g.resid, (float*)g.out, (float*)g.out1, (float*)g.out2,
        g.n_heads, g.n_kv_heads, g.head_dim, g.seq_len, g.rope, g.row_pos);
    return hipGetLastError();
  }
  if (!attrs_done) {
    hipFuncSetAttribute((const void*)gemm_bf16_kernel<256, 256, 2, 4>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, 2 * (256 + 256) * BK * 2);
    hipFuncSetAttribute((const void*)gemm_bf16_kernel<128, 128, 2, 2>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, 2 * (128 + 128) * BK * 2);
    attrs_done = true;
  }
  GemmParams P;
  P.epi = g.epi;
  P.M = g.M;
  P.K = g.K;
  P.N = nlog;
  P.npairs = npairs;
  P.A = (const bf16_t*)g.A;
  P.B0 = (const bf16_t*)g.B0;
  P.B1 = (const bf16_t*)g.B1;
  P.B2 = (const bf16_t*)g.B2;
  P.resid = (const bf16_t*)g.resid;
  P.out = (bf16_t*)g.out;
  P.out1 = (bf16_t*)g.out1;
  P.out2 = (bf16_t*)g.out2;
  P.H = g.n_heads;
  P.Hkv = g.n_kv_heads;
  P.dh = g.head_dim;
  P.seq_len = g.seq_len;
  P.rope = g.rope;
  P.row_pos = g.row_pos;
  const long big_tiles = (long)((g.M + 255) / 256) * ((nlog + 255) / 256);
  if (big_tiles >= 256) return run_bf16<256, 256, 2, 4>(P, s);
  return run_bf16<128, 128, 2, 2>(P, s);
}

}  // namespace sas
