// Skinny GEMM for decode: out = A[M, K] W^T with M <= 16 rows (the batch of
// new tokens), bound by streaming W from HBM.
//
// One workgroup per 16 output columns; its 4 waves split K into contiguous
// ranges of 32-wide steps.  v_mfma_f32_16x16x32_bf16 takes A (activations, 16
// rows, rows >= M zero) and W^T (16 columns).  The MFMA only needs A and B to
// enumerate k the same way, so the k slice of a step is chosen to make each
// load instruction contiguous: lane l reads the 16 bytes at k = 32 st +
// 8 (l/16) of row l % 16, so that with row-major weights one instruction
// covers 16 rows x 64 contiguous bytes, and with the packed decode layout
// (sas_pack_decode_weights) 1 KB of consecutive bytes.  Partial sums of the
// waves are added in LDS.
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
  const bf16_t* packed;  // the weights in the packed decode layout, or NULL
  // cache append (QKV epilogue): K/V rows into their pages, and the summary of
  // a block completed by this position (NULL k_pages: no append)
  void* k_pages;
  void* v_pages;
  void* k_summary;
  PageGeom geom;
  int B, max_blocks;
};

// weight row of local column c (0..15) of column group gi (EPI < 0: the
// epilogue kind is read from P at run time)
template <int EPI = -1>
__device__ __forceinline__ const bf16_t* gemv_row(const GemvParams& P, int gi, int c, bool& valid) {
  const int epi = EPI >= 0 ? EPI : P.epi;
  if (epi == EPI_RESID || epi == EPI_F32OUT) {
    const int col = gi * 16 + c;
    valid = col < P.N;
    return P.B0 + (size_t)min(col, P.N - 1) * P.K;
  }
  const int p = gi * 8 + (c & 7), half = c >> 3;
  valid = p < P.npairs;
  const int pc = min(p, P.npairs - 1);
  if (epi == EPI_SWIGLU) return (half ? P.B1 : P.B0) + (size_t)pc * P.K;
  const int hh = P.dh >> 1;
  const int hd = pc / hh, ir = pc % hh;
  int cc = hd * P.dh + ir + half * hh;
  if (cc < P.H * P.dh) return P.B0 + (size_t)cc * P.K;
  cc -= P.H * P.dh;
  if (cc < P.Hkv * P.dh) return P.B1 + (size_t)cc * P.K;
  return P.B2 + (size_t)(cc - P.Hkv * P.dh) * P.K;
}

// Epilogue inputs of a lane for column group gi (pair gi * 8 + c % 8, rows
// 4 kg + v): the QKV epilogue's rotary entries and cache offsets, the RESID
// epilogue's residual values; loaded before the weights they follow so that
// their latency is hidden by the weight stream.
struct GemvPre {
  float2 cs[4];
  long long off[4];
  int ps[4];
  float res[4];
};

template <int EPI = -1>
__device__ __forceinline__ void gemv_prepare(const GemvParams& P, int gi, int c, int kg, GemvPre& e) {
  const int epi = EPI >= 0 ? EPI : P.epi;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    e.cs[v] = make_float2(1.f, 0.f);
    e.off[v] = -1;
    e.ps[v] = 0;
    e.res[v] = 0.f;
  }
  if (epi == EPI_RESID) {
    const int col = min(gi * 16 + c, P.N - 1);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = min(4 * kg + v, P.M - 1);
      e.res[v] = bf16_to_f32(P.resid[(size_t)row * P.N + col]);
    }
    return;
  }
  if (epi != EPI_QKV_ROPE) return;
  const int hh = P.dh >> 1;
  const int p = min(gi * 8 + (c & 7), P.npairs - 1);
  const int hd = p / hh, ir = p % hh;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int row = 4 * kg + v;
    if (row >= P.M) continue;
    if (hd < P.H + P.Hkv) e.cs[v] = P.rope[(size_t)row * hh + ir];
    if (P.k_pages && hd >= P.H) {
      const int g = hd < P.H + P.Hkv ? hd - P.H : hd - P.H - P.Hkv;
      e.ps[v] = P.pos[row];
      e.off[v] = P.geom.offset(row, g, e.ps[v], P.Hkv, P.dh);
    }
  }
}

// The fused epilogue of column group gi; `tot` holds column c, rows 4 kg + v.
template <int EPI = -1>
__device__ __forceinline__ void gemv_epilogue(const GemvParams& P, int gi, int c, int kg, const floatx4_t& tot,
                                              const GemvPre& e) {
  const int epi = EPI >= 0 ? EPI : P.epi;
  bool cvalid;
  (void)gemv_row<EPI>(P, gi, c, cvalid);
  if (epi == EPI_RESID || epi == EPI_F32OUT) {
    const int col = gi * 16 + c;
    if (!cvalid) return;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = 4 * kg + v;
      if (row >= P.M) continue;
      const size_t o = (size_t)row * P.N + col;
      if (epi == EPI_RESID)
        ((bf16_t*)P.out)[o] = f32_to_bf16(tot[v] + e.res[v]);
      else
        ((float*)P.out)[o] = tot[v];
    }
    return;
  }
  const int hh = P.dh >> 1;
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
    if (epi == EPI_SWIGLU) {
      ((bf16_t*)P.out)[(size_t)row * P.npairs + p] = f32_to_bf16(x1 * __builtin_amdgcn_rcpf(1.0f + __expf(-x1)) * x2);
      continue;
    }
    const int hd = p / hh, ir = p % hh;
    bf16_t* dst;
    if (hd < P.H) dst = (bf16_t*)P.out + ((size_t)row * P.H + hd) * P.dh;
    else if (hd < P.H + P.Hkv) dst = P.out1 + ((size_t)row * P.Hkv + (hd - P.H)) * P.dh;
    else dst = P.out2 + ((size_t)row * P.Hkv + (hd - P.H - P.Hkv)) * P.dh;
    if (hd < P.H + P.Hkv) {
      const float2 cs = e.cs[v];
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
      const int ps = e.ps[v];
      const long long off = e.off[v];
      if (off < 0) continue;
      bf16_t* pg = (bf16_t*)(isk ? P.k_pages : P.v_pages) + off;
      pg[ir] = b1;
      pg[ir + hh] = b2;
      if (!isk || (ps + 1) % P.B != 0 || ps / P.B >= P.max_blocks) continue;
      // this position completes block m: its summary in these two dimensions
      // (fp64 sum over ascending positions, the new key last).  Positions go
      // in chunks of SUMC: the chunk's page ids, then its keys, are loaded
      // unconditionally from clamped addresses and masked afterwards, so each
      // chunk costs two memory round trips instead of two per position.
      constexpr int SUMC = 16;
      const int m = ps / P.B;
      const bf16_t* kp = (const bf16_t*)P.k_pages;
      const int32_t* trow = P.geom.table + (size_t)row * P.geom.max_pages;
      double s1 = 0.0, s2 = 0.0;
      for (int q0 = m * P.B; q0 < ps; q0 += SUMC) {
        long long o[SUMC];
#pragma unroll
        for (int j = 0; j < SUMC; ++j) {
          const int q = q0 + j, pi = q / P.geom.ps;
          const int page = trow[min(pi, P.geom.max_pages - 1)];
          const bool ok = q < ps && pi < P.geom.max_pages && page >= 0 && page < P.geom.num_pages;
          o[j] = ok ? (((long long)page * P.Hkv + g) * P.geom.ps + (q % P.geom.ps)) * P.dh : -1;
        }
        float k1[SUMC], k2[SUMC];
#pragma unroll
        for (int j = 0; j < SUMC; ++j) {
          const long long oc = o[j] >= 0 ? o[j] : 0;
          const float a = bf16_to_f32(kp[oc + ir]), b = bf16_to_f32(kp[oc + ir + hh]);
          k1[j] = o[j] >= 0 ? a : 0.f;  // a position without a page adds zero
          k2[j] = o[j] >= 0 ? b : 0.f;
        }
#pragma unroll
        for (int j = 0; j < SUMC; ++j) {
          if (q0 + j < ps) {
            s1 += (double)k1[j];
            s2 += (double)k2[j];
          }
        }
      }
      s1 += (double)bf16_to_f32(b1);
      s2 += (double)bf16_to_f32(b2);
      bf16_t* sm = (bf16_t*)P.k_summary + (((size_t)row * P.Hkv + g) * P.max_blocks + m) * P.dh;
      sm[ir] = Act<bf16_t>::from_f64(s1 / (double)P.B);
      sm[ir + hh] = Act<bf16_t>::from_f64(s2 / (double)P.B);
    }
  }
}

// The packed decode layout: the 16 columns x 32 k of step st of column group
// gi form one 1-KB block at element ((gi * K/32 + st) * 64 + l) * 8 for lane
// l, holding row(gi, l % 16)[st * 32 + (l / 16) * 8 ..+8]: the fragment lane l
// of the 16x16x32 MFMA takes, so a wave's load is 1 KB of consecutive bytes.
__global__ void gemv_pack_kernel(GemvParams P, bf16_t* __restrict__ out, size_t chunks) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;  // one 16-byte chunk
  if (idx >= chunks) return;
  const int nsteps = P.K / 32;
  const int l = (int)(idx % 64);
  const size_t r = idx / 64;
  const int st = (int)(r % nsteps), gi = (int)(r / nsteps);
  bool valid;
  const bf16_t* row = gemv_row(P, gi, l & 15, valid);  // clamped: columns past the end repeat the last row
  *(uint4*)(out + idx * 8) = *(const uint4*)(row + st * 32 + (l >> 4) * 8);
}

// One workgroup per 16-column group, its waves splitting K.  Lane (c, kg)
// multiplies step st's weights -- row-major:
// row(gi, c)[st * 32 + kg * 8 ..]; packed: its 16 bytes of block (gi, st) --
// by the activation rows' elements st * 32 + kg * 8 ..; both layouts give
// the same products in the same order.
template <int NW, int EPI>
__global__ void __launch_bounds__(NW * 64) gemv_kernel(GemvParams P) {
  __shared__ floatx4_t part[NW][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int gi = blockIdx.x;
  const int c = lane & 15, kg = lane >> 4;
  const bf16_t* wr;
  size_t wstep;
  if (P.packed) {
    wr = P.packed + ((size_t)gi * (P.K / 32) * 64 + lane) * 8;
    wstep = 512;
  } else {
    bool cvalid;
    wr = gemv_row<EPI>(P, gi, c, cvalid) + kg * 8;
    wstep = 32;
  }
  const int arow = min(c, P.M - 1);
  const bool avalid = c < P.M;
  const bf16_t* ar = P.A + (size_t)arow * P.K + kg * 8;
  GemvPre pre;
  if (wave == 0) gemv_prepare<EPI>(P, gi, c, kg, pre);

  // this wave's range of 32-wide k steps
  const int steps = P.K / 32;
  const int per = (steps + NW - 1) / NW;
  const int s0 = wave * per, s1 = min(steps, s0 + per);

  floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
  int st = s0;
  for (; st + 8 <= s1; st += 8) {
    uint4 w[8], a[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      w[q] = *(const uint4*)(wr + (size_t)(st + q) * wstep);
      a[q] = *(const uint4*)(ar + (st + q) * 32);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (!avalid) a[q] = make_uint4(0, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(bf16x8_t*)&a[q], *(bf16x8_t*)&w[q], acc, 0, 0, 0);
    }
  }
  for (; st < s1; ++st) {
    uint4 w = *(const uint4*)(wr + (size_t)st * wstep);
    uint4 a = avalid ? *(const uint4*)(ar + st * 32) : make_uint4(0, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(bf16x8_t*)&a, *(bf16x8_t*)&w, acc, 0, 0, 0);
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
  gemv_epilogue<EPI>(P, gi, c, kg, tot, pre);
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
  P.packed = (const bf16_t*)g.packed;
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
  // 4 waves per group: as fast as or faster than 8 or 16 waves at the decode
  // shapes (measured: QKV 22.6 vs 23.8 us, down 21.9 vs 22.7 us, O equal)
  constexpr int NW = 4;
  const dim3 grid(groups), block(NW * 64);
  switch (g.epi) {
    case EPI_QKV_ROPE: return launch_ext(gemv_kernel<NW, EPI_QKV_ROPE>, grid, block, 0, s, P);
    case EPI_SWIGLU: return launch_ext(gemv_kernel<NW, EPI_SWIGLU>, grid, block, 0, s, P);
    case EPI_F32OUT: return launch_ext(gemv_kernel<NW, EPI_F32OUT>, grid, block, 0, s, P);
    default: return launch_ext(gemv_kernel<NW, EPI_RESID>, grid, block, 0, s, P);
  }
}

static GemvParams pack_params(const GemmArgs& g) {
  GemvParams P = {};
  P.epi = g.epi;
  P.M = 1;
  P.K = g.K;
  P.N = g.N;
  P.npairs = g.epi == EPI_SWIGLU ? g.N : (g.epi == EPI_QKV_ROPE ? g.N / 2 : 0);
  P.B0 = (const bf16_t*)g.B0;
  P.B1 = (const bf16_t*)g.B1;
  P.B2 = (const bf16_t*)g.B2;
  P.H = g.n_heads;
  P.Hkv = g.n_kv_heads;
  P.dh = g.head_dim;
  return P;
}

size_t gemv_packed_elems(const GemmArgs& g) {
  const GemvParams P = pack_params(g);
  const size_t groups = (P.epi == EPI_RESID || P.epi == EPI_F32OUT) ? (P.N + 15) / 16 : (P.npairs + 7) / 8;
  return groups * (size_t)(g.K / 32) * 512;
}

hipError_t launch_gemv_pack(const GemmArgs& g, void* out, hipStream_t s) {
  if (g.K % 128 != 0 || g.N <= 0) return hipErrorInvalidValue;
  const GemvParams P = pack_params(g);
  const size_t chunks = gemv_packed_elems(g) / 8;
  gemv_pack_kernel<<<(unsigned)((chunks + 255) / 256), 256, 0, s>>>(P, (bf16_t*)out, chunks);
  return hipGetLastError();
}

}  // namespace sas
