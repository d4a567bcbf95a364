// SAS attention forward (Eq. ours_train for GATED, Alg. 2's attended set for
// SPARSE, causal Eq. fula for DENSE), fused with the block gate and the
// block mask in a tiled online softmax (the kernel described in App. E of
// the paper, redesigned for CDNA4 wave64 MFMA), with the gating
// formulations of Table 1 as flags (outer gate, full scope).
//
// bf16 kernel layout: one workgroup = 4 waves = 128 query rows of one (batch,
// kv group): 128 / G consecutive positions x the group's G heads (the heads of
// a group share the selection at a position); each wave owns 32 rows.  Scores are computed
// transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: lane l then holds
// query l%32 and 16 of the tile's keys, so the softmax max/sum need only the
// partner lane l^32.  The exponentiated scores P^T stay in registers and are
// fed straight back as the B operand of O^T = V^T P^T: the key order in which
// the accumulator holds P^T is a fixed permutation of the key index, and V^T
// is read from LDS in that same permutation, so no shuffle is needed.
//
// The 64-key tiles that any query of the workgroup attends are flagged in an
// LDS bitmask first (every query's current block and selected blocks, or
// every earlier tile for DENSE and the full scope); each flagged tile's K and
// V are loaded into registers while the previous tile is multiplied, then
// written to LDS (K row-major, V transposed).  The selection rows of the
// workgroup's queries are staged in LDS, and each lane walks its ascending
// list with a cursor while the tiles advance.
//
// Per (query t, key i) with m = block(i) = i / B and beta = block(t):
//   m == beta : current block, causal (i <= t), unit gate;
//   m <  beta : DENSE -> unit gate; SPARSE/GATED -> kept iff m is selected
//               (every m for the full scope), gate g_m (GATED) or 1;
//   m >  beta : masked.
// The gate enters as the logit bias log g_m (inner) or as a weight g_m on
// the block's values (outer; the softmax then normalizes unbiased logits).
#include <float.h>
#include <stdint.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace sas {

__global__ void fill_u32_kernel(uint32_t* p, int n, uint32_t v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

template <int DH, int LSB, bool OUTER, bool SKIP>
__device__ __forceinline__ void attn_bf16_job(const AttnArgs& P, const int qtile, const int g, const int bi,
                                              const int tlo, const int thi, const int slot) {
  constexpr int KP = DH + 8;    // K tile row pitch (elements)
  // V^T tile: head dimension d starts at (d / 8) * VGS + (d % 8) * VP
  // elements (rows 96 apart, groups of 8 rows 776 apart).  A row holds the
  // tile's 64 keys in 8 pairs of 4-key chunks: pair 2 j + h holds keys
  // 16 j + 4 h + 0..3 and 16 j + 8 + 4 h + 0..3, the 8 keys one lane group
  // (h) feeds to the PV product's MFMA step j, so an operand is one 16-byte
  // read.  The strides were chosen by measuring the LDS bank-conflict
  // counter for these exact access patterns: the operand reads run without
  // conflicts and the staging writes (rows 8 apart) with two-way ones.
  constexpr int VP = 96;
  constexpr int VGS = 8 * VP + 8;
  constexpr int KPG = DH / 32;  // keys per thread in the tile staging
  constexpr int C8 = DH / 8;
  constexpr int NSUB = 64 >> LSB;  // sub-blocks of min(B, 64) keys in a tile
  constexpr int KMAX = 32;
  __shared__ __align__(16) bf16_t Ks[64 * KP];
  __shared__ __align__(16) bf16_t Vt[DH / 8 * VGS];
  // selection slots of the workgroup's queries, slot-major ([KMAX][128]):
  // the lanes of a wave read consecutive words
  __shared__ int sel_s[128 * KMAX];
  __shared__ float sbias_s[128 * KMAX];
  __shared__ uint32_t need[ATTN_MAX_SEQ / 64 / 32];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lk = lane >> 5;
  // the workgroup's 128 rows: QPT consecutive positions x the G heads of kv
  // group g (the heads of a group share the selection at a position, so the
  // key tiles the rows attend are the union over QPT positions, not 128)
  const int G = P.H / P.Hkv, QPT = 128 / G;
  const int n = P.n, B = P.B;
  const int qrow = wave * 32 + lr;
  const int pl = qrow / G, h = g * G + (qrow - pl * G);
  const int t0 = qtile * QPT;  // first position of the tile
  const int t = t0 + pl;
  const bool qvalid = pl < QPT && t < n;
  const int beta = qvalid ? t / B : -1;
  const bool gated = P.mode == SAS_MODE_GATED;
  const bool full = gated && P.full;  // every historical block, gates from the table
  const bool every = P.mode == SAS_MODE_DENSE || full;
  const bool outer = OUTER;  // the launch picks OUTER = GATED with the outer gate
  const int Kn = every ? 0 : P.K;
  const int ntiles = (n + 63) / 64;
  const int t_hi = min(n, t0 + QPT) - 1;  // last position of the workgroup
  const int last_tile = t_hi / 64;
  const size_t grow = ((size_t)bi * P.Hkv + g) * n;  // first (b, g) row of [b, Hkv, n, ...]
  const int NB = (n + B - 1) / B;
  const int fb = qvalid ? doc_first(P.doc, bi, NB, t, B) : 0;  // first block of the query's document
  // the workgroup's earliest document start (queries are ascending): its first possible key tile
  const int first_tile = doc_first(P.doc, bi, NB, t0, B) * B / 64;

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

  // selection rows (the lane pair lk = 0, 1 splits the slots) and the tile flags
  for (int w = tid; w < (ntiles + 31) / 32; w += 256) {
    const int lo = w * 32;
    uint32_t bits = 0;
    if (every && lo <= last_tile) bits = last_tile - lo >= 31 ? 0xffffffffu : ((1u << (last_tile - lo + 1)) - 1u);
    if (every && lo + 31 >= first_tile && lo < first_tile) bits &= ~((1u << (first_tile - lo)) - 1u);
    if (lo + 31 < first_tile) bits = 0;
    need[w] = bits;
  }
  if (Kn > 0 && qvalid) {
    const size_t row = (grow + t) * Kn;
    for (int k = lk; k < Kn; k += 2) {
      sel_s[k * 128 + qrow] = P.sel[row + k];
      if (gated) sbias_s[k * 128 + qrow] = P.sel_bias[row + k];
    }
  }
  __syncthreads();
  if (!every && qvalid && lk == 0) {
    for (int tl = (beta * B) / 64; tl <= t / 64; ++tl) atomicOr(&need[tl >> 5], 1u << (tl & 31));
    for (int k = 0; k < Kn; ++k) {
      const int m = sel_s[k * 128 + qrow];
      if (m < 0 || m >= beta) break;  // slots are ascending historical blocks, -1 padded
      for (int tl = (m * B) / 64; tl <= ((m + 1) * B - 1) / 64; ++tl) atomicOr(&need[tl >> 5], 1u << (tl & 31));
    }
  }
  __syncthreads();

  floatx16_t o[DH / 32];
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[dt][v] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float qk_scale = P.sm_scale * LOG2E;

  const bf16_t* Kg = (const bf16_t*)P.Kt + (size_t)g * DH;
  const bf16_t* Vg = (const bf16_t*)P.V + (size_t)g * DH;
  const size_t kstride = (size_t)P.Hkv * DH;  // elements between consecutive keys
  const size_t kbase = (size_t)bi * n;
  const int c8 = tid % C8, kg = tid / C8;
  // this thread's 16-byte column of keys kg * KPG + q of a tile; element
  // offsets within the batch entry fit 32 bits (n * Hkv * DH < 2^31)
  const bf16_t* Kb = Kg + kbase * kstride + c8 * 8;
  const bf16_t* Vb = Vg + kbase * kstride + c8 * 8;
  const uint32_t ks32 = (uint32_t)kstride, last_off = (uint32_t)(n - 1) * ks32;
  u32x4_t rk[KPG], rv[KPG];  // native vectors: the staging stays in registers
  float r_lg[NSUB];  // full scope: this lane's log gates of the tile's blocks
  auto prefetch = [&](int kt) {
    // keys past the end load the last key's row instead (finite; their
    // scores are masked and their probabilities are zero)
    const int r0 = kt * 64 + kg * KPG;
    const uint32_t off0 = (uint32_t)r0 * ks32;
#pragma unroll
    for (int q = 0; q < KPG; ++q) {
      const uint32_t off = r0 + q < n ? off0 + q * ks32 : last_off;
      rk[q] = *(const u32x4_t*)(Kb + off);
      rv[q] = *(const u32x4_t*)(Vb + off);
    }
    if (full) {
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb) {
        const int m = (kt * 64 + (sb << LSB)) / B;
        r_lg[sb] = (qvalid && m < beta && m >= fb) ? P.gate_table[(grow + t) * NB + m] : 0.f;
      }
    }
  };
  auto commit = [&]() {
#pragma unroll
    for (int q = 0; q < KPG; ++q) *(u32x4_t*)(Ks + (kg * KPG + q) * KP + c8 * 8) = rk[q];
    // V^T: word wd of a key holds dims 2 wd (low half) and 2 wd + 1; one byte
    // permute joins the same half of two keys
#pragma unroll
    for (int wd = 0; wd < 4; ++wd) {
      uint32_t a[KPG];
#pragma unroll
      for (int q = 0; q < KPG; ++q) a[q] = rv[q][wd];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const uint32_t sel = hf ? 0x07060302u : 0x05040100u;
        // dimension d = 8 c8 + e, keys kg * KPG ..: chunk c = kg * KPG / 4 (its part kg * KPG % 4)
        const int c = (kg * KPG) >> 2;
        bf16_t* dst = Vt + c8 * VGS + (2 * wd + hf) * VP + 16 * (c >> 2) + 8 * (c & 1) + 4 * ((c >> 1) & 1) +
                      ((kg * KPG) & 3);
        if constexpr (KPG == 4) {
          *(uint2*)dst = make_uint2(__builtin_amdgcn_perm(a[1], a[0], sel), __builtin_amdgcn_perm(a[3], a[2], sel));
        } else {
          *(uint32_t*)dst = __builtin_amdgcn_perm(a[1], a[0], sel);
        }
      }
    }
  };

  // key tiles [tlo, thi) of this job (a part of the range when the query tile is split);
  // the selection cursor starts at the first block not consumed before tile tlo
  const int tend = min(thi, ntiles);
  int cur = 0, next_sel = 0x7fffffff;  // selection cursor of this lane's query
  if (Kn > 0 && qvalid) {
    const int s0 = sel_s[qrow];
    next_sel = s0 >= 0 ? s0 : 0x7fffffff;
    while (next_sel != 0x7fffffff && (next_sel + 1) * B <= tlo * 64) {
      ++cur;
      const int s1 = cur < Kn ? sel_s[cur * 128 + qrow] : -1;
      next_sel = s1 >= 0 ? s1 : 0x7fffffff;
    }
  }
  int kt = next_set(need, tlo, tend);
  if (kt < tend) prefetch(kt);
  while (kt < tend) {
    commit();
    lds_barrier();
    const int k0 = kt * 64;
    // logit offset (log2 domain; -inf: not attended) and value weight of each sub-block
    float offs[NSUB], wts[NSUB];
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) {
      offs[sb] = -INFINITY;
      wts[sb] = 1.f;
      const int kstart = k0 + (sb << LSB);
      if (!qvalid || kstart > t) continue;
      const int m = kstart / B;
      float lg = 0.f;
      bool att = false;
      if (m == beta || (P.mode == SAS_MODE_DENSE && m >= fb)) {
        att = true;
      } else if (full) {
        att = m >= fb;
        lg = r_lg[sb];
      } else if (m == next_sel) {
        att = true;
        lg = gated ? sbias_s[cur * 128 + qrow] : 0.f;
        if (kstart + (1 << LSB) >= (m + 1) * B) {  // a block wider than a tile is consumed at its last tile
          ++cur;
          const int s1 = cur < Kn ? sel_s[cur * 128 + qrow] : -1;
          next_sel = s1 >= 0 ? s1 : 0x7fffffff;
        }
      }
      if (att) {
        offs[sb] = outer ? 0.f : lg * LOG2E;
        wts[sb] = outer ? __builtin_amdgcn_exp2f(lg * LOG2E) : 1.f;
      }
    }
    const int nkt = next_set(need, kt + 1, tend);
    if (nkt < tend) prefetch(nkt);
    // SKIP (grouped queries: a wave's 32 rows span only 32 / G positions): a
    // wave none of whose rows attends a key of the tile skips its products;
    // it still stages the tiles and meets the barriers
    bool att_any = !SKIP;
    if constexpr (SKIP) {
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb) att_any = att_any || offs[sb] != -INFINITY;
    }
    if (!SKIP || __builtin_amdgcn_ballot_w64(att_any) != 0) {

    // S^T = K Q^T for keys [0,32) and [32,64) of the tile.  The MFMA phases
    // run at a raised wave priority, so that while this wave feeds the
    // matrix unit the other wave on the SIMD issues its softmax in between.
    __builtin_amdgcn_s_setprio(2);
    // The two 32-key halves alternate, so that consecutive MFMAs are
    // independent, and the K fragments of step ks + 1 are read while step ks
    // multiplies.
    floatx16_t s[2];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) s[st][v] = 0.f;
    const bf16_t* kf = Ks + lr * KP + lk * 8;
    bf16x8_t ka0 = *(const bf16x8_t*)kf, ka1 = *(const bf16x8_t*)(kf + 32 * KP);
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) {
      bf16x8_t kn0 = ka0, kn1 = ka1;
      if (ks + 1 < DH / 16) {
        kn0 = *(const bf16x8_t*)(kf + (ks + 1) * 16);
        kn1 = *(const bf16x8_t*)(kf + 32 * KP + (ks + 1) * 16);
      }
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka0, qb[ks], s[0], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka1, qb[ks], s[1], 0, 0, 0);
      ka0 = kn0;
      ka1 = kn1;
    }
    // Keep the reads one step ahead of the MFMAs (the scheduler otherwise
    // sinks each read next to its consumer to save registers).
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) {
      if (ks + 1 < DH / 16) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
    __builtin_amdgcn_s_setprio(0);
    // causal mask on the diagonal tiles (raw scores of later keys -> -inf)
    if (k0 + 63 > t0) {
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (k0 + st * 32 + 8 * (v >> 2) + 4 * lk + (v & 3) > t) s[st][v] = -INFINITY;
    }
    // row max of the logits s * scale + offset: the scale is positive, so per
    // sub-block the largest raw score gives the largest logit
    float mxs[NSUB];
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) mxs[sb] = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int sb = (st * 32 + 8 * (v >> 2)) >> LSB;
        mxs[sb] = fmaxf(mxs[sb], s[st][v]);
      }
    float mx = -INFINITY;
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) mx = fmaxf(mx, fmaf(mxs[sb], qk_scale, offs[sb]));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    // The reference max m_run moves only when a logit exceeds it by more than
    // 8 (log2 units): the exponentials stay below 2^8 and the accumulators
    // are rescaled only on those tiles.  Any reference gives the same O and
    // LSE; the partner lanes share mx and so the decision.
    const bool upd = mx > m_run + 8.f;
    float alpha = 1.f;
    if (upd) {
      alpha = __builtin_amdgcn_exp2f(m_run - mx);
      m_run = mx;
    }
    const float m_use = m_run == -INFINITY ? 0.f : m_run;
    float bias[NSUB];
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) bias[sb] = offs[sb] - m_use;
    float rs4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int sb = (st * 32 + 8 * (v >> 2)) >> LSB;
        const float p = __builtin_amdgcn_exp2f(fmaf(s[st][v], qk_scale, bias[sb]));
        rs4[v & 3] += p;
        if constexpr (OUTER) s[st][v] = p * wts[sb];
        else s[st][v] = p;
      }
    float rs = (rs4[0] + rs4[1]) + (rs4[2] + rs4[3]);
    rs += __shfl_xor(rs, 32, 64);
    l_run = l_run * alpha + rs;
    if (__builtin_amdgcn_ballot_w64(upd) != 0) {
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[dt][v] *= alpha;
    }

    // O^T += V^T P^T, 16 keys per step in the accumulator's key permutation
    __builtin_amdgcn_s_setprio(2);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int st = ks >> 1, v0 = 8 * (ks & 1);
      uint4 pu;
      pu.x = pack_bf16x2(s[st][v0 + 0], s[st][v0 + 1]);
      pu.y = pack_bf16x2(s[st][v0 + 2], s[st][v0 + 3]);
      pu.z = pack_bf16x2(s[st][v0 + 4], s[st][v0 + 5]);
      pu.w = pack_bf16x2(s[st][v0 + 6], s[st][v0 + 7]);
      const bf16x8_t pb = *(const bf16x8_t*)&pu;
#pragma unroll
      for (int dt = 0; dt < DH / 32; ++dt) {
        // pair 2 ks + lk of dimension dt * 32 + lr
        const bf16_t* vr = Vt + (4 * dt + (lr >> 3)) * VGS + (lr & 7) * VP + 16 * ks + 8 * lk;
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(const bf16x8_t*)vr, pb, o[dt], 0, 0, 0);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    }
    lds_barrier();
    kt = nkt;
  }

  if (slot >= 0) {  // a part of a split query tile: unnormalized sums and (max, sum) per row
    float* po = P.part_o + ((size_t)slot * 128 + qrow) * DH;
#pragma unroll
    for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4)
        *(float4*)(po + dt * 32 + 8 * v4 + 4 * lk) =
            make_float4(o[dt][4 * v4 + 0], o[dt][4 * v4 + 1], o[dt][4 * v4 + 2], o[dt][4 * v4 + 3]);
    if (lk == 0) *(float2*)(P.part_ml + ((size_t)slot * 128 + qrow) * 2) = make_float2(m_run, l_run);
    return;
  }
  if (!qvalid) return;
  const float inv_l = 1.0f / l_run;
  bf16_t* op = (bf16_t*)P.O + (((size_t)bi * n + t) * P.H + h) * DH;
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const int d0 = dt * 32 + 8 * v4 + 4 * lk;
      const uint32_t w0 = pack_bf16x2(o[dt][4 * v4 + 0] * inv_l, o[dt][4 * v4 + 1] * inv_l);
      const uint32_t w1 = pack_bf16x2(o[dt][4 * v4 + 2] * inv_l, o[dt][4 * v4 + 3] * inv_l);
      *(uint2*)(op + d0) = make_uint2(w0, w1);
    }
  if (P.lse && lk == 0) P.lse[((size_t)bi * P.H + h) * n + t] = (m_run + log2f(l_run)) * LN2;
}

// Splitting a query tile's key range: with fewer jobs than resident
// workgroups the longest job bounds the kernel, so a tile whose causal range
// holds more than `split_tiles` key tiles is cut into up to ATTN_MAX_SPLIT
// parts of about equal tile counts, merged afterwards by attn_combine_kernel.
// (a query tile holds QPT = 128 / G positions of every head of one kv group)
__device__ __forceinline__ int attn_tiles(int n, int qpt, int qtile) { return (min(n, qtile * qpt + qpt) - 1) / 64 + 1; }
__device__ __forceinline__ int attn_splits(int n, int qpt, int qtile, int split_tiles) {
  if (split_tiles <= 0) return 1;
  return min(ATTN_MAX_SPLIT, (attn_tiles(n, qpt, qtile) + split_tiles - 1) / split_tiles);
}
// job -> (query tile, kv group, batch entry, part); the latest query tiles first, a tile's
// parts consecutive; jbase: the job index of the tile's first job
__device__ __forceinline__ void attn_job_of(const AttnArgs& P, int job, int& qtile, int& g, int& bi, int& part,
                                            int& nparts, int& jbase) {
  const int qpt = 128 / (P.H / P.Hkv), nqt = (P.n + qpt - 1) / qpt, per = P.Hkv * P.b;
  jbase = 0;
  for (qtile = nqt - 1; qtile > 0; --qtile) {
    const int cnt = attn_splits(P.n, qpt, qtile, P.split_tiles) * per;
    if (job < jbase + cnt) break;
    jbase += cnt;
  }
  nparts = attn_splits(P.n, qpt, qtile, P.split_tiles);
  int r = job - jbase;
  part = r % nparts;
  r /= nparts;
  g = r % P.Hkv;
  bi = r / P.Hkv;
}

// Work-queue order.  The jobs that read the same keys and values are those
// of one unit (batch entry, kv head): its query tiles.  Each XCD (the workgroups
// blockIdx % ATTN_XCDS, which the dispatcher places on that die) owns a
// contiguous share of the units and a counter of its own, so that a unit's
// jobs run together on one L2.  A unit is split into `unit_parts`
// interleaved query-tile sets when there are fewer units than XCDs.  Within
// a share, groups of `unit_group` units (about 2 MB of keys and values) run
// one after another, each longest query tile first; the last `tail_units`
// units form one group, so that the share ends on short jobs.  A workgroup
// whose share is drained takes jobs from the next shares.
struct AttnQueuePos {
  int nv, cq, v0;  // units of the share, query-tile slots per unit, first unit
};
__device__ __forceinline__ AttnQueuePos attn_share(const AttnArgs& P, int x) {
  const int qpt = 128 / (P.H / P.Hkv), nqt = (P.n + qpt - 1) / qpt, V = P.b * P.Hkv * P.unit_parts;
  AttnQueuePos s;
  s.v0 = (int)((long long)x * V / ATTN_XCDS);
  s.nv = (int)((long long)(x + 1) * V / ATTN_XCDS) - s.v0;
  s.cq = (nqt + P.unit_parts - 1) / P.unit_parts;
  return s;
}
// position r of share s -> job; false for the empty slots of a ragged interleave
__device__ __forceinline__ bool attn_queue_job(const AttnArgs& P, const AttnQueuePos& s, int r, int& qtile, int& g,
                                               int& bi) {
  const int qpt = 128 / (P.H / P.Hkv), nqt = (P.n + qpt - 1) / qpt;
  const int tail = min(P.tail_units, s.nv), nh = s.nv - tail, hpos = nh * s.cq;
  int a, se;
  if (r < hpos) {
    a = r / (P.unit_group * s.cq) * P.unit_group;
    se = min(P.unit_group, nh - a);
  } else {
    a = nh;
    se = tail;
  }
  const int rr = r - a * s.cq, i = rr / se;
  const int vu = s.v0 + a + (rr - i * se);
  const int part = vu % P.unit_parts, u = vu / P.unit_parts;
  qtile = nqt - 1 - i * P.unit_parts - part;
  bi = u / P.Hkv;
  g = u % P.Hkv;
  return qtile >= 0;
}

// One job (query tile or part of it, head, batch entry) per workgroup (grid =
// job count, no queue), or the per-XCD work queues.
template <int DH, int LSB, bool OUTER, bool SKIP>
__global__ void __launch_bounds__(256, 2) attn_bf16_kernel(AttnArgs P, int njobs) {
  if (!P.queue) {
    const int job = blockIdx.x;
    int qtile, g, bi, part, nparts, jbase;
    attn_job_of(P, job, qtile, g, bi, part, nparts, jbase);
    const int nt = attn_tiles(P.n, 128 / (P.H / P.Hkv), qtile), per_part = (nt + nparts - 1) / nparts;
    attn_bf16_job<DH, LSB, OUTER, SKIP>(P, qtile, g, bi, part * per_part,
                                        nparts > 1 ? (part + 1) * per_part : 1 << 30, nparts > 1 ? job : -1);
    return;
  }
  __shared__ int3 job_s;
  const int x0 = blockIdx.x % ATTN_XCDS;
  int drained = 0;  // thread 0: shares found empty, in visiting order (they stay empty)
  for (;;) {
    __syncthreads();  // every thread has finished the previous job and read job_s
    if (threadIdx.x == 0) {
      int3 j = make_int3(-1, 0, 0);
      while (drained < ATTN_XCDS) {
        const int x = (x0 + drained) % ATTN_XCDS;
        const AttnQueuePos sh = attn_share(P, x);
        const uint32_t npos = (uint32_t)sh.nv * sh.cq;
        const uint32_t r = npos ? atomicAdd(&P.queue[x], 1u) : npos;
        if (r >= npos) {
          ++drained;
          continue;
        }
        if (attn_queue_job(P, sh, (int)r, j.x, j.y, j.z)) break;
        j.x = -1;
      }
      job_s = j;
    }
    __syncthreads();
    const int3 j = job_s;
    if (j.x < 0) break;
    attn_bf16_job<DH, LSB, OUTER, SKIP>(P, j.x, j.y, j.z, 0, 1 << 30, -1);
  }
}

// Merge of a split query tile's parts: thread per (batch, head, query, 8
// dimensions); rows of unsplit tiles are skipped.
__global__ void attn_combine_kernel(AttnArgs P) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int n = P.n, C8 = P.dh / 8;
  if (idx >= (size_t)P.b * P.H * n * C8) return;
  const int c8 = (int)(idx % C8);
  size_t r = idx / C8;
  const int t = (int)(r % n);
  r /= n;
  const int h = (int)(r % P.H), bi = (int)(r / P.H);
  const int G = P.H / P.Hkv, qpt = 128 / G, g = h / G;
  const int qtile = t / qpt, nparts = attn_splits(n, qpt, qtile, P.split_tiles);
  if (nparts <= 1) return;
  const int nqt = (n + qpt - 1) / qpt, per = P.Hkv * P.b;
  int jbase = 0;
  for (int q = nqt - 1; q > qtile; --q) jbase += attn_splits(n, qpt, q, P.split_tiles) * per;
  const int j0 = jbase + (bi * P.Hkv + g) * nparts, qrow = (t - qtile * qpt) * G + (h - g * G);
  float mx = -INFINITY;
  for (int p = 0; p < nparts; ++p) mx = fmaxf(mx, P.part_ml[((size_t)(j0 + p) * 128 + qrow) * 2]);
  const float mu = mx == -INFINITY ? 0.f : mx;
  float l = 0.f, acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int p = 0; p < nparts; ++p) {
    const size_t row = (size_t)(j0 + p) * 128 + qrow;
    const float2 ml = *(const float2*)(P.part_ml + row * 2);
    const float w = __builtin_amdgcn_exp2f(ml.x - mu);
    l += ml.y * w;
    const float4 a = *(const float4*)(P.part_o + row * P.dh + c8 * 8);
    const float4 b = *(const float4*)(P.part_o + row * P.dh + c8 * 8 + 4);
    acc[0] += a.x * w;
    acc[1] += a.y * w;
    acc[2] += a.z * w;
    acc[3] += a.w * w;
    acc[4] += b.x * w;
    acc[5] += b.y * w;
    acc[6] += b.z * w;
    acc[7] += b.w * w;
  }
  const float inv_l = 1.0f / l;
  bf16_t* op = (bf16_t*)P.O + (((size_t)bi * n + t) * P.H + h) * P.dh + c8 * 8;
  uint4 u;
  u.x = pack_bf16x2(acc[0] * inv_l, acc[1] * inv_l);
  u.y = pack_bf16x2(acc[2] * inv_l, acc[3] * inv_l);
  u.z = pack_bf16x2(acc[4] * inv_l, acc[5] * inv_l);
  u.w = pack_bf16x2(acc[6] * inv_l, acc[7] * inv_l);
  *(uint4*)op = u;
  if (P.lse && c8 == 0) P.lse[((size_t)bi * P.H + h) * n + t] = (mu + log2f(l)) * LN2;
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
  auto visit = [&](int i, float bias, float w) {
    const float* k = Kg + (((size_t)bi * n + i) * P.Hkv + g) * DH;
    const float* v = Vg + (((size_t)bi * n + i) * P.Hkv + g) * DH;
    float z = 0.f;
#pragma unroll
    for (int j = 0; j < DH; ++j) z = fmaf(qv[j], k[j], z);
    z = z * P.sm_scale + bias;
    float mn = fmaxf(mrun, z);
    float a = expf(mrun - mn), p = expf(z - mn);
    lrun = lrun * a + p;
    const float pw = p * w;
#pragma unroll
    for (int j = 0; j < DH; ++j) acc[j] = acc[j] * a + pw * v[j];
    mrun = mn;
  };
  const int beta = t / B;
  const bool gated = P.mode == SAS_MODE_GATED;
  const bool outer = gated && P.outer;
  // log gate lg of a kept historical block -> (logit bias, value weight)
  auto gate = [&](float lg, float& w) -> float {
    w = outer ? expf(lg) : 1.f;
    return outer ? 0.f : lg;
  };
  const size_t row = ((size_t)bi * P.Hkv + g) * n + t;
  const int NB = (n + B - 1) / B;
  const int fb = doc_first(P.doc, bi, NB, t, B);
  if (P.mode == SAS_MODE_DENSE) {
    for (int i = fb * B; i <= t; ++i) visit(i, 0.f, 1.f);
  } else if (gated && P.full) {
    for (int m = fb; m < beta; ++m) {
      float w;
      const float bias = gate(P.gate_table[row * NB + m], w);
      for (int i = m * B; i < (m + 1) * B; ++i) visit(i, bias, w);
    }
    for (int i = beta * B; i <= t; ++i) visit(i, 0.f, 1.f);
  } else {
    for (int k = 0; k < P.K; ++k) {
      const int m = P.sel[row * P.K + k];
      if (m < 0 || m >= beta) break;  // slots are ascending historical blocks, -1 padded
      float w = 1.f, bias = 0.f;
      if (gated) bias = gate(P.sel_bias[row * P.K + k], w);
      for (int i = m * B; i < (m + 1) * B; ++i) visit(i, bias, w);
    }
    for (int i = beta * B; i <= t; ++i) visit(i, 0.f, 1.f);
  }
  float* o = (float*)P.O + (((size_t)bi * n + t) * P.H + h) * DH;
#pragma unroll
  for (int j = 0; j < DH; ++j) o[j] = acc[j] / lrun;
  if (P.lse) P.lse[((size_t)bi * P.H + h) * n + t] = mrun + logf(lrun);
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.b <= 0) return hipSuccess;
  if (dtype == SAS_BF16) {
    if (a.n > ATTN_MAX_SEQ || a.K > 32) return hipErrorInvalidValue;
    // the kernel's key offsets within a batch entry are 32-bit
    if ((unsigned long long)a.n * a.Hkv * a.dh > 0xffffffffull) return hipErrorInvalidValue;
    const int lsb = a.B >= 64 ? 6 : (a.B == 32 ? 5 : 4);
    const bool outer = a.mode == SAS_MODE_GATED && a.outer;
    const bool skip = a.Hkv > 0 && a.H > a.Hkv;  // grouped queries
    void (*kern)(AttnArgs, int);
#define ATTN_PICK(DH, LSB)                                                                              \
  kern = outer ? (skip ? attn_bf16_kernel<DH, LSB, true, true> : attn_bf16_kernel<DH, LSB, true, false>) \
               : (skip ? attn_bf16_kernel<DH, LSB, false, true> : attn_bf16_kernel<DH, LSB, false, false>)
    if (a.dh == 128) {
      if (lsb == 6) ATTN_PICK(128, 6);
      else if (lsb == 5) ATTN_PICK(128, 5);
      else ATTN_PICK(128, 4);
    } else {
      if (lsb == 6) ATTN_PICK(64, 6);
      else if (lsb == 5) ATTN_PICK(64, 5);
      else ATTN_PICK(64, 4);
    }
#undef ATTN_PICK
    // query tiles of qpt positions x the G heads of a kv group
    if (a.Hkv <= 0 || a.H % a.Hkv != 0 || a.H / a.Hkv > 128) return hipErrorInvalidValue;
    const int qpt = 128 / (a.H / a.Hkv);
    const int nqt = cdiv(a.n, qpt), ntk = cdiv(a.n, 64), per = a.Hkv * a.b;
    const long long jobs = (long long)nqt * per;
    const int res = resident_workgroups(kern, 256);
    if (res <= 0 || jobs > INT32_MAX) return hipErrorInvalidValue;
    AttnArgs A = a;
    A.queue = nullptr;
    A.split_tiles = 0;
    long long total = jobs;
    if (jobs < res && a.part_o && a.part_ml && jobs * ATTN_MAX_SPLIT <= a.part_slots) {
      // fewer jobs than resident workgroups: split the long query tiles so that no job
      // walks much more than the average share of key tiles
      auto tiles = [&](int q) { return std::min(ntk, (std::min(a.n, q * qpt + qpt) - 1) / 64 + 1); };
      long long W = 0;
      for (int q = 0; q < nqt; ++q) W += (long long)tiles(q) * per;
      // the smallest part length whose job count still fits the resident workgroups
      for (int st = (int)std::max<long long>(2, (W + res - 1) / res); st < ntk; ++st) {
        long long tot = 0;
        for (int q = 0; q < nqt; ++q) tot += (long long)std::min(ATTN_MAX_SPLIT, cdiv(tiles(q), st)) * per;
        if (tot <= res) {
          if (tot > jobs) {
            A.split_tiles = st;
            total = tot;
          }
          break;
        }
      }
    }
    if (total > res) {
      if (!a.queue) return hipErrorInvalidValue;
      fill_u32_kernel<<<1, 64, 0, s>>>(a.queue, ATTN_XCDS, 0u);
      A.queue = a.queue;
      const int U = a.b * a.Hkv;
      A.unit_parts = U >= ATTN_XCDS ? 1 : cdiv(ATTN_XCDS, U);
      const long long unit_bytes = (long long)a.n * a.dh * 4;  // keys and values of a unit
      A.unit_group = (int)std::max<long long>(1, (2ll << 20) / std::max<long long>(1, unit_bytes));
      A.tail_units = 8;
      A.unit_group = std::min(A.unit_group, U * A.unit_parts);
    }
    kern<<<(unsigned)std::min<long long>(total, res), 256, 0, s>>>(A, (int)total);
    if (A.split_tiles > 0) {
      const size_t rows = (size_t)a.b * a.H * a.n * (a.dh / 8);
      attn_combine_kernel<<<(unsigned)cdiv(rows, 256), 256, 0, s>>>(A);
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
