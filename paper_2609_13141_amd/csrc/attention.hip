// SAS attention forward (Eq. ours_train for GATED, Alg. 2's attended set for
// SPARSE, causal Eq. fula for DENSE), fused with the block gate and the
// block mask in a tiled online softmax (the kernel described in App. E of
// the paper, redesigned for CDNA4 wave64 MFMA).
//
// bf16 kernel layout: one workgroup = 4 waves = 128 consecutive queries of
// one (batch, head); each wave owns 32 queries.  Scores are computed
// transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: lane l then holds
// query l%32 and 16 of the tile's keys, so the softmax max/sum need only the
// partner lane l^32.  The exponentiated scores P^T stay in registers and are
// fed straight back as the B operand of O^T = V^T P^T: the key order in which
// the accumulator holds P^T is a fixed permutation of the key index, and V^T
// is read from LDS in that same permutation, so no shuffle is needed.  KV
// tiles of 64 keys are staged in LDS (K row-major, V transposed); a tile
// that no query of the workgroup attends to is skipped.
//
// Per (query t, key i) with m = block(i) = i / B and beta = block(t):
//   m == beta : current block, causal (i <= t), bias 0 (unit gate);
//   m <  beta : DENSE -> bias 0; SPARSE/GATED -> kept iff m is in the
//               query group's selected list, bias log g_m (GATED) or 0;
//   m >  beta : masked.
// The selection list of a query is ascending, so each lane walks it with a
// cursor while the KV tiles advance.
#include <float.h>

#include "common.h"
#include "kernels.h"

namespace sas {

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

template <int DH, bool SINGLE>
__global__ void __launch_bounds__(256, 2) attn_bf16_kernel(AttnArgs P) {
  constexpr int KP = DH + 8;  // K tile row pitch (elements)
  constexpr int VP = 64 + 4;  // V^T tile row pitch (elements)
  constexpr int KPG = DH / 32;  // keys per V-staging group (4 for DH=128, 2 for DH=64)
  __shared__ __align__(16) bf16_t Ks[64 * KP];
  __shared__ __align__(16) bf16_t Vt[DH * VP];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  const int qtile = gridDim.x - 1 - blockIdx.x;  // heavy (late) tiles first
  const int h = blockIdx.y, bi = blockIdx.z;
  const int G = P.H / P.Hkv, g = h / G;
  const int n = P.n, B = P.B, Kn = P.K;
  const int t = qtile * 128 + wave * 32 + lr;
  const bool qvalid = t < n;
  const int beta = qvalid ? t / B : -1;
  const int bshift = 31 - __clz(B < 64 ? B : 64);  // log2 of keys per SAS block inside a tile

  // Q^T as the B operand: lane supplies Q[t][ks*16 + lk*8 + 0..7]
  bf16x8_t qb[DH / 16];
  {
    const bf16_t* qp = (const bf16_t*)P.Q + (((size_t)bi * n + (qvalid ? t : 0)) * P.H + h) * DH;
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) {
      uint4 u = qvalid ? *(const uint4*)(qp + ks * 16 + lk * 8) : make_uint4(0, 0, 0, 0);
      qb[ks] = *(bf16x8_t*)&u;
    }
  }

  // selection cursor over the ascending list of kept blocks
  const int32_t* selp = nullptr;
  const float* biasp = nullptr;
  int cur = 0, next_sel = 0x7fffffff;
  if (P.mode != SAS_MODE_DENSE && qvalid && Kn > 0) {
    const size_t row = (((size_t)bi * P.Hkv + g) * n + t) * Kn;
    selp = P.sel + row;
    biasp = P.sel_bias + row;
    const int s0 = selp[0];
    next_sel = s0 >= 0 ? s0 : 0x7fffffff;
  }
  const bool gated = P.mode == SAS_MODE_GATED;
  const bool dense = P.mode == SAS_MODE_DENSE;

  floatx16_t o[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[dt][v] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float qk_scale = P.sm_scale * LOG2E;

  const int t_hi = min(n, qtile * 128 + 128) - 1;  // last query of the workgroup
  const int last_tile = t_hi / 64;
  const bf16_t* Kg = (const bf16_t*)P.Kt + (size_t)g * DH;
  const bf16_t* Vg = (const bf16_t*)P.V + (size_t)g * DH;
  const size_t kstride = (size_t)P.Hkv * DH;  // elements between consecutive keys
  const size_t kbase = (size_t)bi * n;

  for (int kt = 0; kt <= last_tile; ++kt) {
    const int k0 = kt * 64;
    // bias (base-2 domain) of each SAS block of this tile for this lane's
    // query, -inf when masked; one block per tile when B >= 64
    constexpr int NSUB = SINGLE ? 1 : 4;
    float bsub[NSUB];
    bool need = false;
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) {
      bsub[sb] = -INFINITY;
      const int kstart = k0 + (sb << bshift);
      if (!qvalid || kstart > t || (!SINGLE && (sb << bshift) >= 64)) continue;
      const int m = kstart / B;
      if (m == beta || dense) {
        bsub[sb] = 0.f;
      } else if (m == next_sel) {
        bsub[sb] = gated ? biasp[cur] * LOG2E : 0.f;
        // a block wider than a tile is consumed at its last tile
        if (kstart + (1 << bshift) >= (m + 1) * B) {
          ++cur;
          const int s1 = cur < Kn ? selp[cur] : -1;
          next_sel = s1 >= 0 ? s1 : 0x7fffffff;
        }
      }
      need |= bsub[sb] != -INFINITY;
    }
    // also orders this tile's LDS writes after the previous tile's reads
    if (!__syncthreads_or(need)) continue;

    // stage K row-major and V transposed; each lane transposes KPG keys x 8 dims
    {
#pragma unroll
      for (int i = 0; i < (64 * DH / 8) / 256; ++i) {
        const int c = tid + i * 256;
        const int kr = c / (DH / 8), c8 = c % (DH / 8);
        const int key = k0 + kr;
        uint4 ku = key < n ? *(const uint4*)(Kg + (kbase + key) * kstride + c8 * 8) : make_uint4(0, 0, 0, 0);
        *(uint4*)(Ks + kr * KP + c8 * 8) = ku;
      }
      const int c8 = tid % (DH / 8), kg = tid / (DH / 8);
      uint32_t w[KPG][4];
#pragma unroll
      for (int q = 0; q < KPG; ++q) {
        const int key = k0 + kg * KPG + q;
        uint4 vu = key < n ? *(const uint4*)(Vg + (kbase + key) * kstride + c8 * 8) : make_uint4(0, 0, 0, 0);
        w[q][0] = vu.x; w[q][1] = vu.y; w[q][2] = vu.z; w[q][3] = vu.w;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int sh = (e & 1) * 16;
        bf16_t* dst = Vt + (c8 * 8 + e) * VP + kg * KPG;
        if constexpr (KPG == 4) {
          uint2 pk;
          pk.x = ((w[0][e >> 1] >> sh) & 0xffffu) | (((w[1][e >> 1] >> sh) & 0xffffu) << 16);
          pk.y = ((w[2][e >> 1] >> sh) & 0xffffu) | (((w[3][e >> 1] >> sh) & 0xffffu) << 16);
          *(uint2*)dst = pk;
        } else {
          *(uint32_t*)dst = ((w[0][e >> 1] >> sh) & 0xffffu) | (((w[1][e >> 1] >> sh) & 0xffffu) << 16);
        }
      }
    }
    __syncthreads();

    // S^T = K Q^T for keys [0,32) and [32,64) of the tile
    floatx16_t s[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int v = 0; v < 16; ++v) s[st][v] = 0.f;
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) {
        const bf16x8_t a = *(const bf16x8_t*)(Ks + (st * 32 + lr) * KP + ks * 16 + lk * 8);
        s[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qb[ks], s[st], 0, 0, 0);
      }
    }
    // scale, bias, mask; row max over this lane's 32 keys and the partner's
    const int lim = t - k0;  // keys kl <= lim are causal for this lane
    float mx = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int kl = st * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
        float bb;
        if constexpr (SINGLE) {
          bb = bsub[0];
        } else {
          const int sb = kl >> bshift;
          bb = sb == 0 ? bsub[0] : sb == 1 ? bsub[1] : sb == 2 ? bsub[2] : bsub[3];
        }
        const float x = (kl <= lim) ? s[st][v] * qk_scale + bb : -INFINITY;
        s[st][v] = x;
        mx = fmaxf(mx, x);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float rs = 0.f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(s[st][v] - m_use);
        s[st][v] = p;
        rs += p;
      }
    rs += __shfl_xor(rs, 32, 64);
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[dt][v] *= alpha;

    // O^T += V^T P^T, 16 keys per step in the accumulator's key permutation
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      bf16x8_t pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf16_t hb = f32_to_bf16(s[ks >> 1][8 * (ks & 1) + e]);
        pb[e] = *(__bf16*)&hb;
      }
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt) {
        const bf16_t* vr = Vt + (dt * 32 + lr) * VP + 16 * ks + 4 * lk;
        const uint2 lo = *(const uint2*)vr;
        const uint2 hi = *(const uint2*)(vr + 8);
        uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(bf16x8_t*)&u, pb, o[dt], 0, 0, 0);
      }
    }
  }

  if (!qvalid) return;
  const float inv_l = 1.0f / l_run;
  bf16_t* op = (bf16_t*)P.O + (((size_t)bi * n + t) * P.H + h) * DH;
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int d0 = dt * 32 + 8 * v4 + 4 * lk;
      const uint32_t w0 = (uint32_t)f32_to_bf16(o[dt][4 * v4 + 0] * inv_l) |
                          ((uint32_t)f32_to_bf16(o[dt][4 * v4 + 1] * inv_l) << 16);
      const uint32_t w1 = (uint32_t)f32_to_bf16(o[dt][4 * v4 + 2] * inv_l) |
                          ((uint32_t)f32_to_bf16(o[dt][4 * v4 + 3] * inv_l) << 16);
      *(uint2*)(op + d0) = make_uint2(w0, w1);
    }
  if (P.lse && lk == 0) P.lse[((size_t)bi * P.H + h) * n + t] = (m_run + log2f(l_run)) * LN2;
}

// ---- fp32: one thread per (batch, head, query), online softmax in fp32 ----
template <int DH>
__global__ void attn_f32_kernel(AttnArgs P) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = P.n;
  if (idx >= (size_t)P.b * P.H * n) return;
  const int t = (int)(idx % n);
  const int h = (int)((idx / n) % P.H);
  const int bi = (int)(idx / ((size_t)n * P.H));
  const int G = P.H / P.Hkv, g = h / G, B = P.B;
  const float* q = (const float*)P.Q + (((size_t)bi * n + t) * P.H + h) * DH;
  const float* Kg = (const float*)P.Kt;
  const float* Vg = (const float*)P.V;
  float qv[DH], acc[DH];
#pragma unroll
  for (int j = 0; j < DH; ++j) {
    qv[j] = q[j];
    acc[j] = 0.f;
  }
  float mrun = -INFINITY, lrun = 0.f;
  auto visit = [&](int i, float bias) {
    const float* k = Kg + (((size_t)bi * n + i) * P.Hkv + g) * DH;
    const float* v = Vg + (((size_t)bi * n + i) * P.Hkv + g) * DH;
    float z = 0.f;
#pragma unroll
    for (int j = 0; j < DH; ++j) z = fmaf(qv[j], k[j], z);
    z = z * P.sm_scale + bias;
    float mn = fmaxf(mrun, z);
    float a = expf(mrun - mn), p = expf(z - mn);
    lrun = lrun * a + p;
#pragma unroll
    for (int j = 0; j < DH; ++j) acc[j] = acc[j] * a + p * v[j];
    mrun = mn;
  };
  const int beta = t / B;
  if (P.mode == SAS_MODE_DENSE) {
    for (int i = 0; i <= t; ++i) visit(i, 0.f);
  } else {
    const size_t row = (((size_t)bi * P.Hkv + g) * n + t) * P.K;
    for (int k = 0; k < P.K; ++k) {
      int m = P.sel[row + k];
      if (m < 0) break;
      float bias = P.mode == SAS_MODE_GATED ? P.sel_bias[row + k] : 0.f;
      for (int i = m * B; i < (m + 1) * B; ++i) visit(i, bias);
    }
    for (int i = beta * B; i <= t; ++i) visit(i, 0.f);
  }
  float* o = (float*)P.O + (((size_t)bi * n + t) * P.H + h) * DH;
#pragma unroll
  for (int j = 0; j < DH; ++j) o[j] = acc[j] / lrun;
  if (P.lse) P.lse[((size_t)bi * P.H + h) * n + t] = mrun + logf(lrun);
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.b <= 0) return hipSuccess;
  if (dtype == SAS_BF16) {
    dim3 grid(cdiv(a.n, 128), a.H, a.b);
    const bool single = a.B >= 64;
    if (a.dh == 128) {
      if (single) attn_bf16_kernel<128, true><<<grid, 256, 0, s>>>(a);
      else attn_bf16_kernel<128, false><<<grid, 256, 0, s>>>(a);
    } else {
      if (single) attn_bf16_kernel<64, true><<<grid, 256, 0, s>>>(a);
      else attn_bf16_kernel<64, false><<<grid, 256, 0, s>>>(a);
    }
  } else {
    size_t tot = (size_t)a.b * a.H * a.n;
    unsigned grid = (unsigned)((tot + 127) / 128);
    if (a.dh == 128) attn_f32_kernel<128><<<grid, 128, 0, s>>>(a);
    else attn_f32_kernel<64><<<grid, 128, 0, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace sas
