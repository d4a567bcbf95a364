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
// Block summaries: thread per (b, m, g, 8-dim chunk), the chunk fastest and
// then the KV head, so that a load instruction reads a contiguous stretch of
// one key row (Hkv * dh values per position); the B keys of the block are
// read 16 at a time (independent 16-byte loads) and summed per dimension in
// fp64 in ascending token order.
template <typename T>
__global__ void summaries_kernel(const T* __restrict__ K, T* __restrict__ out, int n, int Hkv, int dh,
                                 int B, int NB, size_t total) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int nc = dh / 8;
  const int c8 = (int)(idx % nc);
  size_t r = idx / nc;
  const int g = (int)(r % Hkv);
  r /= Hkv;
  const int m = (int)(r % NB);
  const int bi = (int)(r / NB);
  T* o = out + (((size_t)bi * Hkv + g) * NB + m) * dh + c8 * 8;
  if ((m + 1) * B > n) {  // incomplete block: no summary
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = Act<T>::from_f32(0.f);
    return;
  }
  const T* p = K + (((size_t)bi * n + (size_t)m * B) * Hkv + g) * dh + c8 * 8;
  const size_t stride = (size_t)Hkv * dh;
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  for (int i0 = 0; i0 < B; i0 += 16) {  // B is a multiple of 16
    Vec8<T> v[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) v[q].load(p + (size_t)(i0 + q) * stride);
#pragma unroll
    for (int q = 0; q < 16; ++q)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += (double)v[q].get(e);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = Act<T>::from_f64(acc[e] / (double)B);
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

// Gate query qhat[b, g, t, j] = rho(sum over the group's heads of Q[b, t, h, j]),
// fp64 sum in ascending head order: thread per (b, g, t, 8-dim chunk), with
// 16-byte loads and stores.
template <typename T>
__global__ void gate_query_kernel(const T* __restrict__ Q, T* __restrict__ out, int n, int H, int Hkv, int dh,
                                  size_t chunks) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= chunks) return;
  const int nc = dh / 8;
  const int c8 = (int)(idx % nc);
  size_t r = idx / nc;
  const int t = (int)(r % n);
  r /= n;
  const int g = (int)(r % Hkv);
  const int bi = (int)(r / Hkv);
  const int G = H / Hkv;
  const T* q = Q + (((size_t)bi * n + t) * H + (size_t)g * G) * dh + c8 * 8;
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  for (int h = 0; h < G; ++h) {
    Vec8<T> v;
    v.load(q + (size_t)h * dh);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += (double)v.get(e);
  }
  alignas(16) T res[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) res[e] = Act<T>::from_f64(acc[e]);
  uint4* o = (uint4*)(out + idx * 8);  // [b, Hkv, n, dh]: chunk idx
#pragma unroll
  for (int k = 0; k < (int)(8 * sizeof(T) / 16); ++k) o[k] = ((const uint4*)res)[k];
}

hipError_t launch_gate_query(int dtype, const void* Q, int b, int n, int H, int Hkv, int dh, const void* w_gq,
                             void* qplain, void* qhat, hipStream_t s) {
  const size_t total = (size_t)b * Hkv * n * dh;
  if (total == 0) return hipSuccess;
  const unsigned grid = (unsigned)((total + 255) / 256);
  const size_t chunks = total / 8;  // dh is a multiple of 8
  const unsigned cgrid = (unsigned)((chunks + 255) / 256);
  void* dst = w_gq ? qplain : qhat;
  if (dtype == SAS_BF16)
    gate_query_kernel<bf16_t><<<cgrid, 256, 0, s>>>((const bf16_t*)Q, (bf16_t*)dst, n, H, Hkv, dh, chunks);
  else
    gate_query_kernel<float><<<cgrid, 256, 0, s>>>((const float*)Q, (float*)dst, n, H, Hkv, dh, chunks);
  if (w_gq) {
    if (dtype == SAS_BF16)
      project_kernel<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)qplain, (const bf16_t*)w_gq, (bf16_t*)qhat,
                                                  Hkv, n, dh, total);
    else
      project_kernel<float><<<grid, 256, 0, s>>>((const float*)qplain, (const float*)w_gq, (float*)qhat, Hkv,
                                                 n, dh, total);
  }
  return hipGetLastError();
}

hipError_t launch_block_summaries(int dtype, const void* K, int b, int n, int Hkv, int dh, int B,
                                  const void* w_gk, void* kplain, void* ksum, hipStream_t s) {
  const int NB = cdiv(n, B);
  const size_t total = (size_t)b * Hkv * NB * dh;
  if (total == 0) return hipSuccess;
  const unsigned grid = (unsigned)((total + 255) / 256);
  const size_t tchunks = total / 8;
  const unsigned sgrid = (unsigned)((tchunks + 63) / 64);
  void* dst = w_gk ? kplain : ksum;
  if (dtype == SAS_BF16)
    summaries_kernel<bf16_t><<<sgrid, 64, 0, s>>>((const bf16_t*)K, (bf16_t*)dst, n, Hkv, dh, B, NB, tchunks);
  else
    summaries_kernel<float><<<sgrid, 64, 0, s>>>((const float*)K, (float*)dst, n, Hkv, dh, B, NB, tchunks);
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
// Selection: one workgroup of SEL_NW waves per 64 consecutive query rows of
// one (batch, group); lane = query row.  The 64 gate queries are staged in
// LDS once (as fp32, each the rounded gate query); the waves split the
// historical blocks into contiguous ranges and walk theirs in ascending
// order, in chunks of SEL_MC = 8 summaries, one exact fp64 FMA chain per
// (row, block), j ascending.  The summary values reach the rows through DPP
// row broadcasts: for a 16-dimension group, lane n of every 16-lane row holds
// summary n % 8 at dimensions 8 (n / 8) .. + 8 (the four rows hold the same
// values), and each v_fmac_f64 takes its summary operand from one lane of its
// row, so the wave's 64 chains share one loaded copy without LDS traffic.
// Each lane keeps a register Top-K (best first) and a running LSE.  The lists
// are ordered by score, then by lower block index (the order of a single
// ascending scan with strict comparisons).  Two sorted lists are merged by
// taking the elementwise better of one and the reverse of the other, which
// holds the best K as a bitonic sequence that a half-cleaner cascade sorts:
// a chunk's candidates (sorted by a bitonic network) into a wave's list, and
// the other waves' lists into wave 0's, in wave order.
constexpr int SEL_NW = 4;  // waves per workgroup

// r[mm] += k(lane L + mm of the 16-lane row) * q, mm = 0..7, for the four
// dimensions whose summary values are k0..k3 and query values q0..q3, in that
// order (L = 0: summaries of the group's first 8 dimensions, L = 8: its last
// 8).  v_fmac_f64 with a row_newbcast DPP source: every lane of a row reads
// the source from one lane of that row.  The s_nop covers the two wait states
// a DPP read needs after a VALU write of its source.
#define SEL_F(R, K, Q, N) "v_fmac_f64_dpp %" #R ", %" #K ", %" #Q " row_newbcast:" #N " row_mask:0xf bank_mask:0xf\n\t"
#define SEL_DIM0(K, Q) \
  SEL_F(0, K, Q, 0) SEL_F(1, K, Q, 1) SEL_F(2, K, Q, 2) SEL_F(3, K, Q, 3) \
  SEL_F(4, K, Q, 4) SEL_F(5, K, Q, 5) SEL_F(6, K, Q, 6) SEL_F(7, K, Q, 7)
#define SEL_DIM8(K, Q) \
  SEL_F(0, K, Q, 8) SEL_F(1, K, Q, 9) SEL_F(2, K, Q, 10) SEL_F(3, K, Q, 11) \
  SEL_F(4, K, Q, 12) SEL_F(5, K, Q, 13) SEL_F(6, K, Q, 14) SEL_F(7, K, Q, 15)
template <int L>
__device__ __forceinline__ void sel_fma4(double (&r)[8], double k0, double k1, double k2, double k3, double q0,
                                         double q1, double q2, double q3) {
  static_assert(L == 0 || L == 8, "lane base 0 or 8");
  if constexpr (L == 0) {
    asm("s_nop 1\n\t" SEL_DIM0(8, 12) SEL_DIM0(9, 13) SEL_DIM0(10, 14) SEL_DIM0(11, 15)
        : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]), "+v"(r[7])
        : "v"(k0), "v"(k1), "v"(k2), "v"(k3), "v"(q0), "v"(q1), "v"(q2), "v"(q3));
  } else {
    asm("s_nop 1\n\t" SEL_DIM8(8, 12) SEL_DIM8(9, 13) SEL_DIM8(10, 14) SEL_DIM8(11, 15)
        : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]), "+v"(r[7])
        : "v"(k0), "v"(k1), "v"(k2), "v"(k3), "v"(q0), "v"(q1), "v"(q2), "v"(q3));
  }
}
#undef SEL_DIM8
#undef SEL_DIM0
#undef SEL_F

// Lists of up to 16 slots: three waves per SIMD (a few values spill, and the
// third wave hides more of the merge and load latency than they cost).
template <typename T, int DH, int KMAX, int SEL_MC, bool NOISY>
__global__ void __launch_bounds__(SEL_NW * WAVE, KMAX <= 16 ? 3 : 2) select_kernel(SelectArgs P) {
  static_assert((KMAX & (KMAX - 1)) == 0, "the merge network needs a power-of-two list");
  static_assert(SEL_MC == 8 && DH % 16 == 0, "chunks of 8 summaries, 16-dimension groups");
  // a list exchange region: [KMAX][WAVE] keys, [KMAX][WAVE] blocks, [WAVE]
  // running max and sum; the second region reuses the query staging when it
  // is large enough (the queries are dead once every wave has scored)
  constexpr int MG_BYTES = KMAX * WAVE * 12 + WAVE * 12;
  constexpr bool R1_IN_QS = WAVE * (DH + 4) * 4 >= MG_BYTES;
  __shared__ __align__(16) unsigned char pool[R1_IN_QS ? MG_BYTES : 2 * MG_BYTES];
  // the 64 gate queries as fp32 (exact: each is a rounded value of T); the
  // pitch of DH + 4 puts the 16-byte reads of 16 lanes in distinct banks
  __shared__ __align__(16) float qs[WAVE][DH + 4];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = blockIdx.y, bi = blockIdx.z;
  const int t0 = (gridDim.x - 1 - blockIdx.x) * WAVE;  // the late rows (more blocks to score) first
  const int t = t0 + lane;
  const bool valid = t < P.n;
  const int G = P.H / P.Hkv;
  const int ct = valid ? t / P.B : 0;
  const int fb = valid ? doc_first(P.doc, bi, P.NB, t, P.B) : 0;  // first block of the query's document
  const int t_last = min(P.n - 1, t0 + WAVE - 1);
  const int cmax = t_last / P.B;  // wave-uniform block count
  const int mlo = doc_first(P.doc, bi, P.NB, t0, P.B);  // the rows' earliest document start
  const double den = (double)G * sqrt((double)DH);  // s = r / (G sqrt(dh))
  const double inv_scale = 1.0 / den;
  const size_t row = ((size_t)bi * P.Hkv + g) * P.n + t;
  const float* noise = (NOISY && valid) ? P.noise + row * P.NB : nullptr;
  // the log-gate table row of this query: raw scores written as they are computed (softmax:
  // the LSE is subtracted at the end), the other activations' gates written directly
  float* lgrow = (P.log_gate && valid) ? P.log_gate + row * P.NB : nullptr;
  const int act = P.act;

  // stage the 64 gate queries: either the precomputed (projected) rows, or
  // the group's query heads summed here in fp64 and rounded once; a thread's
  // loads of one head are issued together
  {
    constexpr int NC = DH / 8;       // 8-value chunks per row
    constexpr int NI = NC / SEL_NW;  // chunks per thread (64 rows x NC chunks)
    const int rows = t_last - t0 + 1;
    const int nh = P.qhat ? 1 : G;
    double acc[NI][8];
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[i][e] = 0.0;
    for (int h = 0; h < nh; ++h) {
      Vec8<T> v[NI];
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int c = tid + i * SEL_NW * WAVE;
        const int r = c / NC, c8 = c % NC;
        const int rr = min(r, rows - 1);
        v[i].load(P.qhat ? (const T*)P.qhat + (((size_t)bi * P.Hkv + g) * P.n + t0 + rr) * DH + c8 * 8
                         : (const T*)P.Q + (((size_t)bi * P.n + t0 + rr) * P.H + (size_t)g * G + h) * DH + c8 * 8);
      }
#pragma unroll
      for (int i = 0; i < NI; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[i][e] += (double)v[i].get(e);
    }
    // a single row (one head, or the projected query) is already a value of
    // T, and its rounding the identity: stored as it is
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int c = tid + i * SEL_NW * WAVE;
      const int r = c / NC, c8 = c % NC;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        qs[r][c8 * 8 + e] =
            r < rows ? (nh == 1 ? (float)acc[i][e] : Act<T>::to_f32(Act<T>::from_f64(acc[i][e]))) : 0.f;
    }
  }
  __syncthreads();

  constexpr int EMPTY = 0x7fffffff;  // block id of an empty slot
  double tr[KMAX];
  int tm[KMAX];
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    tr[i] = -DBL_MAX;
    tm[i] = EMPTY;
  }
  double mrun = -DBL_MAX;  // running max of s
  float lrun = 0.f;        // running sum of exp(s - mrun)
  // does key a rank strictly ahead of the slot (b, bm)?  An equal key keeps
  // the earlier (lower) block ahead.  Without noise every key is a finite
  // exact dot product, above the empty slots' -DBL_MAX.  With noise a key can
  // be -inf (or NaN): every key then beats an empty slot (so such blocks are
  // kept when fewer than K others exist) and NaN ranks below every number.
  auto beats = [](double a, double b, int bm) -> bool {
    if constexpr (!NOISY) {
      return a > b;
    } else {
      if (bm == EMPTY) return true;
      if (a != a) return false;
      return a > b || b != b;
    }
  };
  // the total order of the lists: a ranks ahead of b (ties: lower block first)
  auto ahead = [](double a, int am, double b, int bm) -> bool {
    if constexpr (!NOISY) {
      return a > b || (a == b && am < bm);
    } else {
      const int ca = am == EMPTY ? 2 : (a != a ? 1 : 0), cb = bm == EMPTY ? 2 : (b != b ? 1 : 0);
      if (ca != cb) return ca < cb;
      return (ca == 0 && a > b) || ((ca == 1 || a == b) && am < bm);
    }
  };

  const T* kbar = (const T*)P.kbar + ((size_t)bi * P.Hkv + g) * (size_t)P.NB * DH;
  const int per = (cmax - mlo + SEL_NW - 1) / SEL_NW;
  const int mb = mlo + wave * per, me = min(cmax, mb + per);
  // this lane's part of a 16-dimension group jg of the chunk at m0: summary
  // (lane % 8) of the chunk (the last block for a ragged chunk's missing
  // ones), dimensions 16 jg + 8 ((lane % 16) / 8) .. + 8
  const int lsum = lane & 7, lhalf = (lane >> 3) & 1;
  auto group_ptr = [&](int m0, int jg) {
    return kbar + (size_t)min(m0 + lsum, me - 1) * DH + jg * 16 + lhalf * 8;
  };
  constexpr int NG = DH / 16;  // dimension groups per summary
  Vec8<T> kn;  // the next group's values, loaded one group ahead
  if (mb < me) kn.load(group_ptr(mb, 0));
  for (int m0 = mb; m0 < me; m0 += SEL_MC) {
    const int mc = min(SEL_MC, me - m0);
    // r[mm] = sum_j q_j kbar[m0+mm]_j: one fp64 FMA chain per block, j ascending
    double r[SEL_MC];
#pragma unroll
    for (int mm = 0; mm < SEL_MC; ++mm) r[mm] = 0.0;
    const float* qrow = qs[lane];
#pragma unroll
    for (int jg = 0; jg < NG; ++jg) {
      const Vec8<T> kc = kn;
      if (jg + 1 < NG) kn.load(group_ptr(m0, jg + 1));
      else if (m0 + SEL_MC < me) kn.load(group_ptr(m0 + SEL_MC, 0));
      double kd[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) kd[e] = (double)kc.get(e);
      const float4 q0 = *(const float4*)(qrow + jg * 16), q1 = *(const float4*)(qrow + jg * 16 + 4);
      const float4 q2 = *(const float4*)(qrow + jg * 16 + 8), q3 = *(const float4*)(qrow + jg * 16 + 12);
      // dimensions 16 jg + 0..7 from lanes 0..7 of the row, then 16 jg + 8..15 from lanes 8..15
      sel_fma4<0>(r, kd[0], kd[1], kd[2], kd[3], q0.x, q0.y, q0.z, q0.w);
      sel_fma4<0>(r, kd[4], kd[5], kd[6], kd[7], q1.x, q1.y, q1.z, q1.w);
      sel_fma4<8>(r, kd[0], kd[1], kd[2], kd[3], q2.x, q2.y, q2.z, q2.w);
      sel_fma4<8>(r, kd[4], kd[5], kd[6], kd[7], q3.x, q3.y, q3.z, q3.w);
    }
    // the chunk's candidates (ranking key, block; EMPTY where the block is not
    // a historical block of this row's document)
    double cr[SEL_MC];
    int cmi[SEL_MC];
    bool any = false;
#pragma unroll
    for (int mm = 0; mm < SEL_MC; ++mm) {
      const int m = m0 + mm;
      cr[mm] = -DBL_MAX;
      cmi[mm] = EMPTY;
      if (mm >= mc || m >= ct || m < fb) continue;
      // ranking key: the raw score r, or the noisy score s + noise when noise is given
      const double sv = noise ? r[mm] / den + (double)noise[m] : r[mm] * inv_scale;
      const double rv = noise ? sv : r[mm];
      if (lgrow) {
        double gv = sv;
        if (act == SAS_ACT_SIGMOID) gv = sv >= 0.0 ? -log1p(exp(-sv)) : sv - log1p(exp(sv));
        lgrow[m] = (float)gv;
      }
      // running LSE: one exponential of minus the gap to the running max, the
      // sum rescaled when sv is the new max (no divergent branch)
      {
        const float d = (float)(sv - mrun);
        const float e = __expf(-fabsf(d));
        const bool up = d > 0.f;
        lrun = up ? fmaf(lrun, e, 1.f) : lrun + e;
        mrun = up ? sv : mrun;
      }
      cr[mm] = rv;
      cmi[mm] = m;
      any = any || beats(rv, tr[KMAX - 1], tm[KMAX - 1]);
    }
    // Keep the best KMAX of the list and the chunk's candidates: sort the
    // candidates best first; the better of list slot KMAX-1-i and candidate i
    // leaves the best KMAX as a bitonic sequence, which a half-cleaner cascade
    // sorts.  The order is the total order (key descending, block ascending)
    // that inserting the blocks one by one in ascending order gives.
    if (__builtin_amdgcn_ballot_w64(any) != 0) {
      auto cas = [&](double& ra, int& ma, double& rb, int& mb) {  // the better one into (ra, ma)
        const bool sw = ahead(rb, mb, ra, ma);
        const double x = ra, y = rb;
        const int u = ma, v = mb;
        ra = sw ? y : x;
        rb = sw ? x : y;
        ma = sw ? v : u;
        mb = sw ? u : v;
      };
#pragma unroll
      for (int k = 2; k <= SEL_MC; k <<= 1)
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
          for (int i = 0; i < SEL_MC; ++i) {
            const int l = i ^ j;
            if (l > i) {
              if ((i & k) == 0) cas(cr[i], cmi[i], cr[l], cmi[l]);
              else cas(cr[l], cmi[l], cr[i], cmi[i]);
            }
          }
      static_assert(SEL_MC <= KMAX, "a chunk fits the list");
      if (!NOISY && m0 == mb) {
        // the wave's first chunk: the list is empty, so the sorted candidates
        // are the list (what the merge below would leave; the noisy variant,
        // at its register limit, takes the merge)
#pragma unroll
        for (int i = 0; i < SEL_MC; ++i) {
          tr[i] = cr[i];
          tm[i] = cmi[i];
        }
      } else {
#pragma unroll
        for (int i = 0; i < SEL_MC; ++i) {
          const int q = KMAX - 1 - i;
          if (ahead(cr[i], cmi[i], tr[q], tm[q])) {
            tr[q] = cr[i];
            tm[q] = cmi[i];
          }
        }
#pragma unroll
        for (int len = KMAX / 2; len >= 1; len >>= 1)
#pragma unroll
          for (int i = 0; i < KMAX; ++i)
            if ((i & len) == 0) cas(tr[i], tm[i], tr[i + len], tm[i + len]);
      }
    }
  }
  __syncthreads();
  // merge the waves' lists as a tree: 1 into 0 and 3 into 2, then 2 into 0.
  // The lists are ordered by a strict total order, so the best KMAX of the
  // union do not depend on the merge order.
  unsigned char* const region[2] = {pool, R1_IN_QS ? (unsigned char*)&qs[0][0] : pool + MG_BYTES};
  auto put = [&](const unsigned char* base) {  // this wave's list and LSE into a region
    double* rk = (double*)base;
    int* rb = (int*)(base + KMAX * WAVE * 8);
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      rk[i * WAVE + lane] = tr[i];
      rb[i * WAVE + lane] = tm[i];
    }
    ((double*)(base + KMAX * WAVE * 12))[lane] = mrun;
    ((float*)(base + KMAX * WAVE * 12 + WAVE * 8))[lane] = lrun;
  };
  auto take = [&](const unsigned char* base) {  // a region's list and LSE into this wave's
    const double* rk = (const double*)base;
    const int* rb = (const int*)(base + KMAX * WAVE * 8);
    // the better of slot i and the other list's slot KMAX-1-i: the best KMAX
    // of both, descending then ascending (a bitonic sequence)
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      const double ob = rk[(KMAX - 1 - i) * WAVE + lane];
      const int om = rb[(KMAX - 1 - i) * WAVE + lane];
      if (ahead(ob, om, tr[i], tm[i])) {
        tr[i] = ob;
        tm[i] = om;
      }
    }
    // bitonic sort, best first
#pragma unroll
    for (int len = KMAX / 2; len >= 1; len >>= 1)
#pragma unroll
      for (int i = 0; i < KMAX; ++i)
        if ((i & len) == 0) {
          const int j = i + len;
          const bool sw = ahead(tr[j], tm[j], tr[i], tm[i]);
          const double ri = tr[i], rj = tr[j];
          const int mi = tm[i], mj = tm[j];
          tr[i] = sw ? rj : ri;
          tr[j] = sw ? ri : rj;
          tm[i] = sw ? mj : mi;
          tm[j] = sw ? mi : mj;
        }
    const double om = ((const double*)(base + KMAX * WAVE * 12))[lane];
    const float ol = ((const float*)(base + KMAX * WAVE * 12 + WAVE * 8))[lane];
    if (om > mrun) {
      lrun = lrun * expf((float)(mrun - om)) + ol;
      mrun = om;
    } else if (ol > 0.f) {
      lrun += ol * expf((float)(om - mrun));
    }
  };
  static_assert(SEL_NW == 4, "a two-level merge tree");
  if (wave == 1) put(region[0]);
  if (wave == 3) put(region[1]);
  __syncthreads();
  if (wave == 0) take(region[0]);
  if (wave == 2) take(region[1]);
  __syncthreads();
  if (wave == 2) put(region[0]);
  __syncthreads();
  if (wave == 0) take(region[0]);
  if (wave != 0 || !valid) return;
  const double lse = (ct > fb) ? mrun + log((double)lrun) : 0.0;
  auto log_gate_of = [&](double key) -> double {  // log g of a block from its ranking key
    const double sv = noise ? key : key * inv_scale;
    if (act == SAS_ACT_SOFTMAX) return sv - lse;
    if (act == SAS_ACT_SIGMOID) return sv >= 0.0 ? -log1p(exp(-sv)) : sv - log1p(exp(sv));
    return sv;
  };
  const int K = P.K;
  const int C = ct - fb;  // historical blocks of the query (its own document)
  const int kk = min(K, C);

  if (P.tau) {
    float tau;
    if (C <= K) tau = -INFINITY;
    else if (K == 0) tau = INFINITY;
    else {
      double rk = tr[0];
#pragma unroll
      for (int i = 0; i < KMAX; ++i)
        if (i == K - 1) rk = tr[i];
      tau = (float)log_gate_of(rk);
    }
    P.tau[row] = tau;
  }

  // order the kept blocks by index (a bitonic sorting network; empty slots,
  // the largest index, last)
#pragma unroll
  for (int i = 0; i < KMAX; ++i)
    if (i >= kk) tm[i] = EMPTY;
#pragma unroll
  for (int k = 2; k <= KMAX; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < KMAX; ++i) {
        const int l = i ^ j;
        if (l > i) {
          const bool sw = (i & k) == 0 ? tm[i] > tm[l] : tm[i] < tm[l];
          const int a = tm[i], c = tm[l];
          const double ra = tr[i], rc = tr[l];
          tm[i] = sw ? c : a;
          tm[l] = sw ? a : c;
          tr[i] = sw ? rc : ra;
          tr[l] = sw ? ra : rc;
        }
      }
  int32_t* sel = P.sel + row * K;
  float* sb = P.sel_bias + row * K;
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    if (i < K) {
      const bool kept = i < kk && tm[i] != EMPTY;
      sel[i] = kept ? tm[i] : -1;
      sb[i] = kept ? (float)log_gate_of(tr[i]) : 0.f;
    }
  }

  if (lgrow) P.row_lse[row] = (float)lse;  // finish_table_kernel subtracts it (softmax)
}

// finish the log-gate table: softmax gates are the written scores minus the
// row's LSE; blocks m >= C_t are not historical (-inf)
__global__ void finish_table_kernel(float* __restrict__ table, const float* __restrict__ row_lse, size_t rows,
                                    int n, int Hkv, int B, int NB, int softmax, const int32_t* __restrict__ doc) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * NB) return;
  const size_t row = idx / NB;
  const int t = (int)(row % n), bi = (int)(row / ((size_t)n * Hkv));
  const int m = (int)(idx % NB), ct = t / B, fb = doc_first(doc, bi, NB, t, B);
  table[idx] = (m < ct && m >= fb) ? (softmax ? table[idx] - row_lse[row] : table[idx]) : -INFINITY;
}

template <typename T, int DH, bool NOISY>
static void run_select_t(const SelectArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.n, WAVE), a.Hkv, a.b);
  if (a.K <= 8) select_kernel<T, DH, 8, 8, NOISY><<<grid, SEL_NW * WAVE, 0, s>>>(a);
  else if (a.K <= 16) select_kernel<T, DH, 16, 8, NOISY><<<grid, SEL_NW * WAVE, 0, s>>>(a);
  else select_kernel<T, DH, 32, 8, NOISY><<<grid, SEL_NW * WAVE, 0, s>>>(a);
}

template <typename T, int DH>
static void run_select(const SelectArgs& a, hipStream_t s) {
  if (a.noise) run_select_t<T, DH, true>(a, s);
  else run_select_t<T, DH, false>(a, s);
}

hipError_t launch_select(int dtype, const SelectArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.b <= 0) return hipSuccess;
  if (a.log_gate && !a.row_lse) return hipErrorInvalidValue;
  if (dtype == SAS_BF16) {
    if (a.dh == 128) run_select<bf16_t, 128>(a, s);
    else run_select<bf16_t, 64>(a, s);
  } else {
    if (a.dh == 128) run_select<float, 128>(a, s);
    else run_select<float, 64>(a, s);
  }
  if (a.log_gate) {
    const size_t rows = (size_t)a.b * a.Hkv * a.n;
    finish_table_kernel<<<(unsigned)cdiv(rows * a.NB, 256), 256, 0, s>>>(a.log_gate, a.row_lse, rows, a.n, a.Hkv, a.B,
                                                                          a.NB, a.act == SAS_ACT_SOFTMAX, a.doc);
  }
  return hipGetLastError();
}

}  // namespace sas
