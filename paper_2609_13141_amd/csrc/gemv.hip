// Skinny GEMM for decode: out = A[M, K] W^T with M <= 16 rows (the batch of
// new tokens), bound by streaming W from HBM.
//
// One workgroup per 16 output columns; its waves split K.  v_mfma_f32_16x16x32_bf16
// takes A (activations, 16 rows, rows >= M zero) and W^T (16 columns).  The
// MFMA only needs A and B to enumerate k the same way, so the k slice of MFMA
// j of a 128-wide chunk is chosen to make each load instruction contiguous per
// row: lane l reads the 16 bytes at k = kb + 32 j + 8 (l/16) of row l % 16, so
// one instruction covers 16 rows x 64 contiguous bytes (half a cache line each)
// and the chunk's four instructions cover 16 rows x 256 bytes.  Partial sums of
// the waves are added in LDS.
//
// Column groups of the pair epilogues hold 8 first-half and 8 second-half
// columns (RoPE: i and i + dh/2 of a head; SwiGLU: gate f and up f); a lane's
// partner is lane ^ 8 after the reduction.
#include "common.h"
#include "kernels.h"

namespace sas {

struct GemvParams {
  int epi, M, K, N, npairs;
  const bf16_t* A;
  const bf16_t* B0;
  const bf16_t* B1;
  const bf16_t* B2;
  const bf16_t* resid;
  void* out;
  bf16_t* out1;
  bf16_t* out2;
  int H, Hkv, dh;
  const float2* rope;  // [M, dh/2] per-row rotary table
  const int32_t* pos;  // [M] positions (cache append)
  // cache append (QKV epilogue): K/V rows into their pages, and the summary of
  // a block completed by this position (NULL k_pages: no append)
  void* k_pages;
  void* v_pages;
  void* k_summary;
  PageGeom geom;
  int B, max_blocks;
};

// weight row of local column c (0..15) of column group gi
__device__ __forceinline__ const bf16_t* gemv_row(const GemvParams& P, int gi, int c, bool& valid) {
  if (P.epi == EPI_RESID || P.epi == EPI_F32OUT) {
    const int col = gi * 16 + c;
    valid = col < P.N;
    return P.B0 + (size_t)min(col, P.N - 1) * P.K;
  }
  const int p = gi * 8 + (c & 7), half = c >> 3;
  valid = p < P.npairs;
  const int pc = min(p, P.npairs - 1);
  if (P.epi == EPI_SWIGLU) return (half ? P.B1 : P.B0) + (size_t)pc * P.K;
  const int hh = P.dh >> 1;
  const int hd = pc / hh, ir = pc % hh;
  int cc = hd * P.dh + ir + half * hh;
  if (cc < P.H * P.dh) return P.B0 + (size_t)cc * P.K;
  cc -= P.H * P.dh;
  if (cc < P.Hkv * P.dh) return P.B1 + (size_t)cc * P.K;
  return P.B2 + (size_t)(cc - P.Hkv * P.dh) * P.K;
}

template <int NW>
__global__ void __launch_bounds__(NW * 64) gemv_kernel(GemvParams P) {
  __shared__ floatx4_t part[NW][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int gi = blockIdx.x;
  const int c = lane & 15, kg = lane >> 4;
  bool cvalid;
  const bf16_t* wr = gemv_row(P, gi, c, cvalid);
  const int arow = min(c, P.M - 1);
  const bool avalid = c < P.M;
  const bf16_t* ar = P.A + (size_t)arow * P.K;

  // QKV epilogue inputs of this lane (pair gi * 8 + c % 8, rows 4 kg + v), read before the
  // weight stream so their latency (the page offset is a dependent lookup) is hidden by it
  const int hh = P.dh >> 1;
  float2 cs_pre[4];
  long long off_pre[4];
  int ps_pre[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    cs_pre[v] = make_float2(1.f, 0.f);
    off_pre[v] = -1;
    ps_pre[v] = 0;
  }
  if (P.epi == EPI_QKV_ROPE && wave == 0) {
    const int p = min(gi * 8 + (c & 7), P.npairs - 1);
    const int hd = p / hh, ir = p % hh;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = 4 * kg + v;
      if (row >= P.M) continue;
      if (hd < P.H + P.Hkv) cs_pre[v] = P.rope[(size_t)row * hh + ir];
      if (P.k_pages && hd >= P.H) {
        const int g = hd < P.H + P.Hkv ? hd - P.H : hd - P.H - P.Hkv;
        ps_pre[v] = P.pos[row];
        off_pre[v] = P.geom.offset(row, g, ps_pre[v], P.Hkv, P.dh);
      }
    }
  }

  // this wave's k range, in chunks of 128
  const int nchunk = P.K / 128;
  const int per = (nchunk + NW - 1) / NW;
  const int c0 = wave * per, c1 = min(nchunk, c0 + per);

  floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
  int ch = c0;
  for (; ch + 2 <= c1; ch += 2) {
    uint4 w[8], a[8];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int k = (ch + u) * 128 + j * 32 + kg * 8;
        w[u * 4 + j] = *(const uint4*)(wr + k);
        a[u * 4 + j] = *(const uint4*)(ar + k);
      }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (!avalid) a[q] = make_uint4(0, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(bf16x8_t*)&a[q], *(bf16x8_t*)&w[q], acc, 0, 0, 0);
    }
  }
  for (; ch < c1; ++ch) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = ch * 128 + j * 32 + kg * 8;
      uint4 w = *(const uint4*)(wr + k);
      uint4 a = avalid ? *(const uint4*)(ar + k) : make_uint4(0, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(bf16x8_t*)&a, *(bf16x8_t*)&w, acc, 0, 0, 0);
    }
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
  floatx4_t tot = part[0][lane];
#pragma unroll
  for (int wv = 1; wv < NW; ++wv) {
    const floatx4_t p = part[wv][lane];
#pragma unroll
    for (int v = 0; v < 4; ++v) tot[v] += p[v];
  }
  // lane holds column c, rows 4*kg + v
  if (P.epi == EPI_RESID || P.epi == EPI_F32OUT) {
    const int col = gi * 16 + c;
    if (!cvalid) return;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = 4 * kg + v;
      if (row >= P.M) continue;
      const size_t o = (size_t)row * P.N + col;
      if (P.epi == EPI_RESID)
        ((bf16_t*)P.out)[o] = f32_to_bf16(tot[v] + bf16_to_f32(P.resid[o]));
      else
        ((float*)P.out)[o] = tot[v];
    }
    return;
  }
  float partner[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) partner[v] = __shfl_xor(tot[v], 8, 64);
  if (c >= 8 || !cvalid) return;
  const int p = gi * 8 + c;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int row = 4 * kg + v;
    if (row >= P.M) continue;
    float x1 = tot[v], x2 = partner[v];
    if (P.epi == EPI_SWIGLU) {
      ((bf16_t*)P.out)[(size_t)row * P.npairs + p] = f32_to_bf16(x1 / (1.0f + __expf(-x1)) * x2);
      continue;
    }
    const int hd = p / hh, ir = p % hh;
    bf16_t* dst;
    if (hd < P.H) dst = (bf16_t*)P.out + ((size_t)row * P.H + hd) * P.dh;
    else if (hd < P.H + P.Hkv) dst = P.out1 + ((size_t)row * P.Hkv + (hd - P.H)) * P.dh;
    else dst = P.out2 + ((size_t)row * P.Hkv + (hd - P.H - P.Hkv)) * P.dh;
    if (hd < P.H + P.Hkv) {
      const float2 cs = cs_pre[v];
      const float o1 = x1 * cs.x - x2 * cs.y;
      const float o2 = x2 * cs.x + x1 * cs.y;
      x1 = o1;
      x2 = o2;
    }
    const bf16_t b1 = f32_to_bf16(x1), b2 = f32_to_bf16(x2);
    dst[ir] = b1;
    dst[ir + hh] = b2;
    if (P.k_pages && hd >= P.H) {
      // cache append of this row's K or V, dimensions ir and ir + dh/2
      const bool isk = hd < P.H + P.Hkv;
      const int g = isk ? hd - P.H : hd - P.H - P.Hkv;
      const int ps = ps_pre[v];
      const long long off = off_pre[v];
      if (off < 0) continue;
      bf16_t* pg = (bf16_t*)(isk ? P.k_pages : P.v_pages) + off;
      pg[ir] = b1;
      pg[ir + hh] = b2;
      if (!isk || (ps + 1) % P.B != 0 || ps / P.B >= P.max_blocks) continue;
      // this position completes block m: its summary in these two dimensions
      // (fp64 sum over ascending positions, the new key last)
      const int m = ps / P.B;
      double s1 = 0.0, s2 = 0.0;
      for (int q = m * P.B; q < ps; ++q) {
        const long long o = P.geom.offset(row, g, q, P.Hkv, P.dh);
        float k1 = 0.f, k2 = 0.f;  // a position without a page adds zero
        if (o >= 0) {
          k1 = bf16_to_f32(((const bf16_t*)P.k_pages)[o + ir]);
          k2 = bf16_to_f32(((const bf16_t*)P.k_pages)[o + ir + hh]);
        }
        s1 += (double)k1;
        s2 += (double)k2;
      }
      s1 += (double)bf16_to_f32(b1);
      s2 += (double)bf16_to_f32(b2);
      bf16_t* sm = (bf16_t*)P.k_summary + (((size_t)row * P.Hkv + g) * P.max_blocks + m) * P.dh;
      sm[ir] = Act<bf16_t>::from_f64(s1 / (double)P.B);
      sm[ir + hh] = Act<bf16_t>::from_f64(s2 / (double)P.B);
    }
  }
}

hipError_t launch_gemv(const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0) return hipSuccess;
  if (g.M > 16 || g.K % 128 != 0) return hipErrorInvalidValue;
  GemvParams P;
  P.epi = g.epi;
  P.M = g.M;
  P.K = g.K;
  P.N = g.N;
  P.npairs = g.epi == EPI_SWIGLU ? g.N : (g.epi == EPI_QKV_ROPE ? g.N / 2 : 0);
  P.A = (const bf16_t*)g.A;
  P.B0 = (const bf16_t*)g.B0;
  P.B1 = (const bf16_t*)g.B1;
  P.B2 = (const bf16_t*)g.B2;
  P.resid = (const bf16_t*)g.resid;
  P.out = g.out;
  P.out1 = (bf16_t*)g.out1;
  P.out2 = (bf16_t*)g.out2;
  P.H = g.n_heads;
  P.Hkv = g.n_kv_heads;
  P.dh = g.head_dim;
  P.rope = g.rope;
  P.pos = g.row_pos;
  P.k_pages = nullptr;
  P.v_pages = nullptr;
  P.k_summary = nullptr;
  P.geom = PageGeom{nullptr, 0, 1, 0};
  P.B = 1;
  P.max_blocks = 0;
  if (g.epi == EPI_QKV_ROPE) {
    if (!g.rope) return hipErrorInvalidValue;
    if (g.append) {
      if (!g.row_pos) return hipErrorInvalidValue;
      const DecodeArgs& c = *g.append;
      P.k_pages = c.k_pages;
      P.v_pages = c.v_pages;
      P.k_summary = c.k_summary;
      P.geom = PageGeom{c.block_table, c.num_pages, c.page_size, c.max_pages};
      P.B = c.B;
      P.max_blocks = c.max_blocks;
    }
  }
  const int groups = (g.epi == EPI_RESID || g.epi == EPI_F32OUT) ? (g.N + 15) / 16 : (P.npairs + 7) / 8;
  // fewer column groups -> more waves per group, to keep enough loads in flight
  if (groups < 1024) gemv_kernel<8><<<groups, 512, 0, s>>>(P);
  else gemv_kernel<4><<<groups, 256, 0, s>>>(P);
  return hipGetLastError();
}

}  // namespace sas
