// C ABI of the SAS hot path: argument validation, workspace planning and the
// kernel sequence of every entry point.  No allocation happens here; all
// scratch comes from the caller's workspace.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <string>
#include <vector>

#include "../../include/sas.h"
#include "kernels.h"

using namespace sas;

namespace sas {
LaunchEvents g_launch_events = {nullptr, nullptr, 0};  // see kernels.h
}

namespace {

thread_local std::string g_err;

sas_status fail(sas_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

sas_status hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return SAS_OK;
  return fail(SAS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define SAS_TRY(expr)                         \
  do {                                        \
    sas_status _st = (expr);                  \
    if (_st != SAS_OK) return _st;            \
  } while (0)
#define HIP_TRY(expr, what) SAS_TRY(hip_check((expr), (what)))

// Opt-in kernel timing: a hipEvent pair around every launch on its stream,
// and a second pair that a single-kernel launch made through launch_ext
// records at the kernel's own start and end (used when it was recorded).
struct Profiler {
  bool on = false;
  std::vector<hipEvent_t> ev;  // 4 per record: outer begin, outer end, kernel start, kernel stop
  std::vector<const char*> names;
  std::vector<char> exact;     // the kernel pair of the record was recorded
  int used = 0;
  bool filtered = false;            // record only the families in `only`
  std::vector<std::string> only;
  int start(int capacity) {
    // the events of an earlier start are reused when there are enough of them
    if ((int)ev.size() < 4 * capacity) {
      for (auto e : ev) (void)hipEventDestroy(e);
      ev.clear();
      for (int i = 0; i < 4 * capacity; ++i) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return -1;
        ev.push_back(e);
      }
    }
    names.assign(capacity, nullptr);
    exact.assign(capacity, 0);
    used = 0;
    on = true;
    return 0;
  }
  void select(const char* families) {
    only.clear();
    filtered = families != nullptr;
    if (!families) return;
    std::string cur;
    for (const char* p = families;; ++p) {
      if (*p == ',' || *p == '\0') {
        if (!cur.empty()) only.push_back(cur);
        cur.clear();
        if (*p == '\0') break;
      } else {
        cur += *p;
      }
    }
  }
  bool wanted(const char* name) const {
    if (!filtered) return true;
    for (const auto& f : only)
      if (f == name) return true;
    return false;
  }
  int begin(const char* name, hipStream_t s) {
    if (!on || used >= (int)names.size() || !wanted(name)) return -1;
    names[used] = name;
    (void)hipEventRecord(ev[4 * used], s);
    g_launch_events = LaunchEvents{ev[4 * used + 2], ev[4 * used + 3], 0};
    return used++;
  }
  void end(int id, hipStream_t s) {
    if (id < 0) return;
    (void)hipEventRecord(ev[4 * id + 1], s);
    exact[id] = g_launch_events.taken == 1;  // recorded by the one launch that took them
    g_launch_events = LaunchEvents{nullptr, nullptr, 0};
  }
};
Profiler g_prof;

struct Timed {
  int id;
  hipStream_t s;
  Timed(const char* name, hipStream_t st) : id(g_prof.begin(name, st)), s(st) {}
  ~Timed() { g_prof.end(id, s); }
};

size_t act_bytes(const sas_config* c) { return c->dtype == SAS_BF16 ? 2 : 4; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

sas_status check_ptr(const void* p, const char* name, bool required) {
  if (!p) return required ? fail(SAS_ERR_INVALID_ARGUMENT, "%s is NULL", name) : SAS_OK;
  if (!aligned16(p)) return fail(SAS_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", name);
  return SAS_OK;
}

sas_status check_config(const sas_config* c, bool need_mlp) {
  if (!c) return fail(SAS_ERR_INVALID_ARGUMENT, "config is NULL");
  if (c->dtype != SAS_F32 && c->dtype != SAS_BF16)
    return fail(SAS_ERR_INVALID_ARGUMENT, "dtype %d is not SAS_F32 or SAS_BF16", c->dtype);
  if (c->mode < SAS_MODE_DENSE || c->mode > SAS_MODE_GATED)
    return fail(SAS_ERR_INVALID_ARGUMENT, "mode %d is not DENSE, SPARSE or GATED", c->mode);
  if (c->n_heads <= 0 || c->n_kv_heads <= 0 || c->n_heads % c->n_kv_heads != 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "n_heads %d must be a positive multiple of n_kv_heads %d",
                c->n_heads, c->n_kv_heads);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(SAS_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", c->head_dim);
  if (c->block_size != 16 && c->block_size != 32 && c->block_size != 64 && c->block_size != 128)
    return fail(SAS_ERR_UNSUPPORTED, "block_size %d (supported: 16, 32, 64, 128)", c->block_size);
  if (c->top_k < 0) return fail(SAS_ERR_INVALID_ARGUMENT, "top_k %d is negative", c->top_k);
  if (c->top_k > 32) return fail(SAS_ERR_UNSUPPORTED, "top_k %d (supported: 0..32)", c->top_k);
  if (c->gate_pos < SAS_GATE_INNER || c->gate_pos > SAS_GATE_OUTER || c->gate_act < SAS_ACT_SOFTMAX ||
      c->gate_act > SAS_ACT_RAW || c->scope < SAS_SCOPE_SPARSE || c->scope > SAS_SCOPE_FULL || c->gate_ste < 0 ||
      c->gate_ste > 1)
    return fail(SAS_ERR_INVALID_ARGUMENT, "gating fields out of range (pos %d, act %d, scope %d, ste %d)",
                c->gate_pos, c->gate_act, c->scope, c->gate_ste);
  if (c->mode == SAS_MODE_GATED && c->gate_pos == SAS_GATE_OUTER && (c->gate_act == SAS_ACT_RAW || c->gate_ste))
    return fail(SAS_ERR_UNSUPPORTED, "the outer gate supports the softmax and sigmoid activations without the "
                                     "straight-through gate");
  if (need_mlp) {
    if (c->d_model <= 0 || c->d_ff <= 0)
      return fail(SAS_ERR_INVALID_ARGUMENT, "d_model %d and d_ff %d must be positive", c->d_model, c->d_ff);
    if (c->d_model % 8 || c->d_ff % 8)
      return fail(SAS_ERR_UNSUPPORTED, "d_model %d and d_ff %d must be multiples of 8", c->d_model, c->d_ff);
    if (!(c->rms_eps >= 0.f)) return fail(SAS_ERR_INVALID_ARGUMENT, "rms_eps must be >= 0");
    if (!(c->rope_base > 0.f)) return fail(SAS_ERR_INVALID_ARGUMENT, "rope_base must be > 0");
  }
  return SAS_OK;
}

float sm_scale_of(const sas_config* c) {
  return c->sm_scale > 0.f ? c->sm_scale : 1.0f / sqrtf((float)c->head_dim);
}

bool gated_of(const sas_config* c) { return c->mode == SAS_MODE_GATED; }
// the forward attends every historical block with its gate (needs the log-gate table)
bool full_fwd(const sas_config* c) { return gated_of(c) && c->scope == SAS_SCOPE_FULL && !c->gate_ste; }
// the backward produces a gradient for every historical block
bool full_grad(const sas_config* c) { return gated_of(c) && c->scope == SAS_SCOPE_FULL; }

// Bump allocator over the caller's workspace (offsets aligned to 256 bytes).
struct Carve {
  char* base;
  size_t off = 0;
  explicit Carve(void* b) : base((char*)b) {}
  void* take(size_t bytes) {
    void* p = base ? base + off : nullptr;
    off += align_up(bytes, 256);
    return p;
  }
};

struct AttnWs {
  void* kplain;
  void* ksum;
  void* qplain;
  void* qhat;
  int32_t* sel;
  float* sel_bias;
  float* gate_table;  // log gates of every block (full scope, when the caller does not ask for them)
  float* row_lse;     // per-row LSE of the scores while the log-gate table is finished
  uint32_t* queue;    // job counter of the attention kernel
  float* part_o;      // parts of split query tiles (short sequences)
  float* part_ml;
  long long part_slots;
};

AttnWs carve_attention(Carve& cv, const sas_config* c, int b, int n) {
  const size_t ab = act_bytes(c);
  const int NB = cdiv(n, c->block_size);
  const size_t kb = (size_t)b * c->n_kv_heads * NB * c->head_dim * ab;
  const size_t rows = (size_t)b * c->n_kv_heads * n * (size_t)(c->top_k > 0 ? c->top_k : 1);
  AttnWs w;
  w.kplain = cv.take(kb);
  w.ksum = cv.take(kb);
  const size_t qb = (size_t)b * c->n_kv_heads * n * c->head_dim * ab;
  w.qplain = cv.take(qb);
  w.qhat = cv.take(qb);
  w.sel = (int32_t*)cv.take(rows * 4);
  w.sel_bias = (float*)cv.take(rows * 4);
  w.gate_table = full_fwd(c) ? (float*)cv.take((size_t)b * c->n_kv_heads * n * NB * 4) : nullptr;
  w.row_lse = (float*)cv.take((size_t)b * c->n_kv_heads * n * 4);
  w.queue = (uint32_t*)cv.take(256);
  // split query tiles: only when the jobs are few (then at most ATTN_MAX_SPLIT parts each)
  const long long jobs = (long long)cdiv(n, 128) * c->n_heads * b;
  w.part_slots = jobs < 1024 ? jobs * ATTN_MAX_SPLIT : 0;
  w.part_o = w.part_slots ? (float*)cv.take((size_t)w.part_slots * 128 * c->head_dim * 4) : nullptr;
  w.part_ml = w.part_slots ? (float*)cv.take((size_t)w.part_slots * 128 * 2 * 4) : nullptr;
  return w;
}

struct MlpWs {
  void* u2;
  void* a;
};

MlpWs carve_mlp(Carve& cv, const sas_config* c, size_t T) {
  const size_t ab = act_bytes(c);
  MlpWs w;
  w.u2 = cv.take(T * c->d_model * ab);
  w.a = cv.take(T * c->d_ff * ab);
  return w;
}

struct LayerWs {
  void* u1;
  float2* rope;
  void* q;
  void* k;
  void* v;
  void* o;
  float* lse;
  void* h1;
  AttnWs att;
  MlpWs mlp;
};

LayerWs carve_layer(Carve& cv, const sas_config* c, int b, int n) {
  const size_t ab = act_bytes(c);
  const size_t T = (size_t)b * n;
  const size_t H = c->n_heads, Hkv = c->n_kv_heads, dh = c->head_dim;
  LayerWs w;
  w.u1 = cv.take(T * c->d_model * ab);
  w.rope = (float2*)cv.take((size_t)n * (dh / 2) * sizeof(float2));
  w.q = cv.take(T * H * dh * ab);
  w.k = cv.take(T * Hkv * dh * ab);
  w.v = cv.take(T * Hkv * dh * ab);
  w.o = cv.take(T * H * dh * ab);
  w.lse = (float*)cv.take(T * H * 4);
  w.h1 = cv.take(T * c->d_model * ab);
  w.att = carve_attention(cv, c, b, n);
  w.mlp = carve_mlp(cv, c, T);
  return w;
}

// Selector + attention given Q/K/V already in device memory.
sas_status run_attention(const sas_config* c, int b, int n, const void* q, const void* k, const void* v,
                         const void* w_gq, const void* w_gk, void* o, float* lse, void* k_summary,
                         int32_t* sel_idx, float* log_gate, float* tau, const AttnWs& ws,
                         hipStream_t s, bool need_summary = false, const float* noise = nullptr,
                         const int32_t* doc = nullptr) {
  const int NB = cdiv(n, c->block_size);
  const int H = c->n_heads, Hkv = c->n_kv_heads, dh = c->head_dim;
  // DENSE attention reads no selection: score and select only when a selector output is asked for;
  // the block summaries alone are needed when the caller or the KV cache wants them
  const bool need_sel = c->mode != SAS_MODE_DENSE || sel_idx || log_gate || tau;
  const bool need_ksum = need_sel || k_summary || need_summary;
  if (full_fwd(c) && !log_gate) log_gate = ws.gate_table;
  void* ksum = k_summary ? k_summary : ws.ksum;
  int32_t* sel = sel_idx ? sel_idx : ws.sel;
  if (need_ksum) {
    Timed tm("summaries", s);
    HIP_TRY(launch_block_summaries(c->dtype, k, b, n, Hkv, dh, c->block_size, w_gk, ws.kplain, ksum, s),
            "block summaries");
  }
  if (need_sel) {
    if (w_gq) {  // projected gate queries are computed first; otherwise the select kernel sums the heads
      Timed tm("gate_query", s);
      HIP_TRY(launch_gate_query(c->dtype, q, b, n, H, Hkv, dh, w_gq, ws.qplain, ws.qhat, s), "gate query");
    }
    SelectArgs sa;
    sa.b = b;
    sa.n = n;
    sa.H = H;
    sa.Hkv = Hkv;
    sa.dh = dh;
    sa.B = c->block_size;
    sa.K = c->top_k;
    sa.NB = NB;
    sa.Q = q;
    sa.qhat = w_gq ? ws.qhat : nullptr;
    sa.kbar = ksum;
    sa.sel = sel;
    sa.sel_bias = ws.sel_bias;
    sa.log_gate = log_gate;
    sa.tau = tau;
    sa.noise = noise;
    sa.act = gated_of(c) ? c->gate_act : SAS_ACT_SOFTMAX;
    sa.row_lse = ws.row_lse;
    sa.doc = doc;
    {
      Timed tm("select", s);
      HIP_TRY(launch_select(c->dtype, sa, s), "select");
    }
  }
  AttnArgs aa;
  aa.b = b;
  aa.n = n;
  aa.H = H;
  aa.Hkv = Hkv;
  aa.dh = dh;
  aa.B = c->block_size;
  aa.K = c->top_k;
  // the straight-through gate's forward attends the Top-K blocks with unit gates
  aa.mode = gated_of(c) && c->gate_ste ? SAS_MODE_SPARSE : c->mode;
  aa.sm_scale = sm_scale_of(c);
  aa.Q = q;
  aa.Kt = k;
  aa.V = v;
  aa.sel = sel;
  aa.sel_bias = ws.sel_bias;
  aa.O = o;
  aa.lse = lse;
  aa.outer = gated_of(c) && c->gate_pos == SAS_GATE_OUTER;
  aa.full = full_fwd(c);
  aa.gate_table = log_gate;
  aa.doc = doc;
  aa.queue = ws.queue;
  aa.part_o = c->dtype == SAS_BF16 ? ws.part_o : nullptr;
  aa.part_ml = c->dtype == SAS_BF16 ? ws.part_ml : nullptr;
  aa.part_slots = ws.part_slots;
  aa.split_tiles = 0;
  {
    Timed tm("attention", s);
    HIP_TRY(launch_attention(c->dtype, aa, s), "attention");
  }
  return SAS_OK;
}

sas_status run_mlp(const sas_config* c, size_t T, const void* x, const sas_layer_weights* w, void* y,
                   const MlpWs& ws, hipStream_t s) {
  {
    Timed tm("rmsnorm", s);
    HIP_TRY(launch_rmsnorm(c->dtype, x, w->rms2, ws.u2, (int)T, c->d_model, c->rms_eps, s), "rmsnorm");
  }
  GemmArgs g = {};
  g.epi = EPI_SWIGLU;
  g.M = (int)T;
  g.K = c->d_model;
  g.A = ws.u2;
  g.B0 = w->w_gate;
  g.B1 = w->w_up;
  g.N = c->d_ff;
  g.out = ws.a;
  {
    Timed tm("gemm_gate_up", s);
    HIP_TRY(launch_gemm(c->dtype, g, s), "gate/up gemm");
  }
  GemmArgs d = {};
  d.epi = EPI_RESID;
  d.M = (int)T;
  d.K = c->d_ff;
  d.A = ws.a;
  d.B0 = w->w_down;
  d.N = c->d_model;
  d.resid = x;
  d.out = y;
  {
    Timed tm("gemm_down", s);
    HIP_TRY(launch_gemm(c->dtype, d, s), "down gemm");
  }
  return SAS_OK;
}

sas_status check_weights(const sas_layer_weights* w, bool attn, bool mlp) {
  if (!w) return fail(SAS_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (attn) {
    SAS_TRY(check_ptr(w->rms1, "w.rms1", true));
    SAS_TRY(check_ptr(w->wq, "w.wq", true));
    SAS_TRY(check_ptr(w->wk, "w.wk", true));
    SAS_TRY(check_ptr(w->wv, "w.wv", true));
    SAS_TRY(check_ptr(w->wo, "w.wo", true));
    SAS_TRY(check_ptr(w->w_gq, "w.w_gq", false));
    SAS_TRY(check_ptr(w->w_gk, "w.w_gk", false));
    SAS_TRY(check_ptr(w->decode_packed, "w.decode_packed", false));
  }
  if (mlp) {
    SAS_TRY(check_ptr(w->rms2, "w.rms2", true));
    SAS_TRY(check_ptr(w->w_gate, "w.w_gate", true));
    SAS_TRY(check_ptr(w->w_up, "w.w_up", true));
    SAS_TRY(check_ptr(w->w_down, "w.w_down", true));
  }
  return SAS_OK;
}

sas_status check_cache(const sas_config* c, const sas_paged_kv* kv) {
  SAS_TRY(check_ptr(kv->k_pages, "cache.k_pages", true));
  SAS_TRY(check_ptr(kv->v_pages, "cache.v_pages", true));
  SAS_TRY(check_ptr(kv->block_table, "cache.block_table", true));
  SAS_TRY(check_ptr(kv->k_summary, "cache.k_summary", true));
  if (kv->page_size <= 0 || kv->num_pages <= 0 || kv->max_pages_per_seq <= 0 || kv->max_blocks <= 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "cache geometry must be positive (page_size %d, num_pages %d, "
                "max_pages_per_seq %d, max_blocks %d)", kv->page_size, kv->num_pages, kv->max_pages_per_seq,
                kv->max_blocks);
  if (c->block_size % kv->page_size != 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "block_size %d is not a multiple of page_size %d", c->block_size,
                kv->page_size);
  if (c->block_size / kv->page_size > 64)
    return fail(SAS_ERR_UNSUPPORTED, "block_size / page_size = %d (supported: <= 64)", c->block_size / kv->page_size);
  if (kv->max_blocks > DSEL_MAX_BLOCKS)
    return fail(SAS_ERR_UNSUPPORTED, "max_blocks %d (supported: <= %d)", kv->max_blocks, DSEL_MAX_BLOCKS);
  return SAS_OK;
}

DecodeArgs decode_args(const sas_config* c, int b, const int32_t* pos, const sas_paged_kv* kv,
                       const sas_layer_weights* w) {
  DecodeArgs d;
  d.b = b;
  d.H = c->n_heads;
  d.Hkv = c->n_kv_heads;
  d.dh = c->head_dim;
  d.B = c->block_size;
  d.K = c->top_k;
  d.d = c->d_model;
  d.F = c->d_ff;
  d.sm_scale = sm_scale_of(c);
  d.eps = c->rms_eps;
  d.rope_base = c->rope_base;
  d.pos = pos;
  d.k_pages = kv->k_pages;
  d.v_pages = kv->v_pages;
  d.block_table = kv->block_table;
  d.k_summary = kv->k_summary;
  d.num_pages = kv->num_pages;
  d.page_size = kv->page_size;
  d.max_pages = kv->max_pages_per_seq;
  d.max_blocks = kv->max_blocks;
  d.w_gq = w ? w->w_gq : nullptr;
  d.w_gk = w ? w->w_gk : nullptr;
  return d;
}

// Linear layer of a few rows (decode): the streaming kernel when it applies,
// else the tiled GEMM (rope table indexed by row).
hipError_t small_gemm(int dtype, GemmArgs g, hipStream_t s) {
  if (dtype == SAS_BF16 && g.M <= 16 && g.K % 128 == 0) return launch_gemv(g, s);
  g.seq_len = g.M;
  g.row_pos = nullptr;
  return launch_gemm(dtype, g, s);
}

struct DecodeWs {
  void* u1;
  float2* rope;
  void* q;
  void* k;
  void* v;
  void* kplain;
  int32_t* sel;
  float* part_ml;
  float* part_o;
  void* o;
  void* h1;
  double* scores;
  MlpWs mlp;
};

// selector scores of the long-context path: b * Hkv * max_blocks doubles
double* carve_scores(Carve& cv, const sas_config* c, int b, int max_blocks) {
  if (max_blocks <= DSEL_WAVE_MAX_BLOCKS) return nullptr;
  return (double*)cv.take((size_t)b * c->n_kv_heads * max_blocks * sizeof(double));
}

// max context (tokens) -> summary blocks the workspace must cover
int blocks_of(const sas_config* c, int max_context) {
  return max_context > 0 ? (int)cdiv(max_context, c->block_size) : 0;
}

DecodeWs carve_decode(Carve& cv, const sas_config* c, int b, int max_blocks) {
  const size_t ab = act_bytes(c);
  const size_t H = c->n_heads, Hkv = c->n_kv_heads, dh = c->head_dim, K = c->top_k;
  DecodeWs w;
  w.u1 = cv.take((size_t)b * c->d_model * ab);
  w.rope = (float2*)cv.take((size_t)b * (dh / 2) * sizeof(float2));
  w.q = cv.take((size_t)b * H * dh * ab);
  w.k = cv.take((size_t)b * Hkv * dh * ab);
  w.v = cv.take((size_t)b * Hkv * dh * ab);
  w.kplain = cv.take((size_t)b * Hkv * dh * ab);
  w.sel = (int32_t*)cv.take((size_t)b * Hkv * (K > 0 ? K : 1) * 4);
  w.part_ml = (float*)cv.take((size_t)b * H * (K + 1) * 2 * 4);
  w.part_o = (float*)cv.take((size_t)b * H * (K + 1) * dh * 4);
  w.o = cv.take((size_t)b * H * dh * ab);
  w.h1 = cv.take((size_t)b * c->d_model * ab);
  w.scores = carve_scores(cv, c, b, max_blocks);
  w.mlp = carve_mlp(cv, c, (size_t)b);
  return w;
}

struct BwdWs {
  float* delta;
  float* dlg_head;
  uint32_t* selmask;
  int* tile_cnt;
  int* tile_off;
  int* tile_rows;
  float* sel_bias;
  float* dlg_head_full;  // [b, H, n, NB] (full scope)
  float* dlg_slots;      // [b, Hkv, n, K] per-slot gradient when only the table is asked for
  uint32_t* queue;       // job counters of the pass kernels
};

BwdWs carve_backward(Carve& cv, const sas_config* c, int b, int n) {
  const size_t H = c->n_heads, Hkv = c->n_kv_heads, K = c->top_k > 0 ? c->top_k : 0;
  const size_t NB = cdiv(n, c->block_size);
  BwdWs w;
  w.delta = (float*)cv.take((size_t)b * H * n * 4);
  w.dlg_head = (float*)cv.take((size_t)b * H * n * K * 4);
  const size_t ntk = cdiv(n, 64);
  w.tile_cnt = (int*)cv.take((size_t)b * Hkv * ntk * 4);
  w.tile_off = (int*)cv.take((size_t)b * Hkv * ntk * 4);
  w.tile_rows = (int*)cv.take(K > 0 ? (size_t)b * Hkv * n * 2 * (K + 1) * 4 : 0);
  w.selmask = (uint32_t*)cv.take((size_t)b * Hkv * n * cdiv(NB, (size_t)32) * 4);
  w.sel_bias = (float*)cv.take((size_t)b * Hkv * n * K * 4);
  w.dlg_head_full = full_grad(c) ? (float*)cv.take((size_t)b * H * n * NB * 4) : nullptr;
  w.dlg_slots = (float*)cv.take((size_t)b * Hkv * n * K * 4);
  w.queue = (uint32_t*)cv.take(256);
  return w;
}

// Selector backward scratch.  The reductions over t (dkbar, dW_gq) and over
// the batch (dW) go through split partials summed in a fixed order.
struct SelBwdWs {
  void* kplain;
  void* ksum;
  void* qplain;
  void* qhat;
  float* ds;
  float* dqhat;
  float* dkbar;
  float* part;
};

// k splits of a reduction of length K feeding `tiles` output tiles per batch
// entry, for Z entries: enough workgroups to fill the chip, each split >= 256
int sel_bwd_splits(int tiles, int Z, int K) {
  const int want = cdiv(1024, tiles * Z);
  return std::max(1, std::min(want, cdiv(K, 256)));
}

struct SelBwdShape {
  int NB, Z, s_dkbar, s_dwq, s_dwk;
  size_t part_floats;
};

SelBwdShape sel_bwd_shape(const sas_config* c, int b, int n) {
  SelBwdShape h;
  const int dh = c->head_dim, Hkv = c->n_kv_heads;
  h.NB = cdiv(n, c->block_size);
  h.Z = b * Hkv;
  const int tdh = cdiv(dh, 64);
  h.s_dkbar = sel_bwd_splits(cdiv(h.NB, 64) * tdh, h.Z, n);
  h.s_dwq = sel_bwd_splits(tdh * tdh, h.Z, n);
  h.s_dwk = sel_bwd_splits(tdh * tdh, h.Z, h.NB);
  const size_t z = h.Z;
  h.part_floats = std::max({z * h.s_dkbar * h.NB * dh, z * h.s_dwq * dh * dh, z * h.s_dwk * dh * dh});
  return h;
}

SelBwdWs carve_selector_backward(Carve& cv, const sas_config* c, int b, int n) {
  const size_t ab = act_bytes(c), Hkv = c->n_kv_heads, dh = c->head_dim;
  const SelBwdShape h = sel_bwd_shape(c, b, n);
  SelBwdWs w;
  w.kplain = cv.take((size_t)b * Hkv * h.NB * dh * ab);
  w.ksum = cv.take((size_t)b * Hkv * h.NB * dh * ab);
  w.qplain = cv.take((size_t)b * Hkv * n * dh * ab);
  w.qhat = cv.take((size_t)b * Hkv * n * dh * ab);
  w.ds = (float*)cv.take((size_t)b * Hkv * n * h.NB * 4);
  w.dqhat = (float*)cv.take((size_t)b * Hkv * n * dh * 4);
  w.dkbar = (float*)cv.take((size_t)b * Hkv * h.NB * dh * 4);
  w.part = (float*)cv.take(h.part_floats * 4);
  return w;
}

struct StatsWs {
  float* lvn;
  float* blk_lse;
  uint32_t* head_mask;
  uint32_t* queue;  // job counter of the statistics kernel
};

StatsWs carve_stats(Carve& cv, const sas_config* c, int b, int n) {
  const size_t H = c->n_heads, Hkv = c->n_kv_heads, NB = cdiv(n, c->block_size);
  StatsWs w;
  w.lvn = (float*)cv.take((size_t)b * n * Hkv * 4);
  w.blk_lse = (float*)cv.take((size_t)b * H * n * NB * 4);
  w.head_mask = (uint32_t*)cv.take((size_t)b * H * n * cdiv(NB, (size_t)32) * 4);
  w.queue = (uint32_t*)cv.take(256);
  return w;
}

constexpr int ARGMAX_SLICES = 64;

struct LmWs {
  void* u;
  float* logits;
  float* pv;
  int32_t* pi;
};

LmWs carve_lm(Carve& cv, const sas_config* c, int b, int vocab) {
  LmWs w;
  w.u = cv.take((size_t)b * c->d_model * act_bytes(c));
  w.logits = (float*)cv.take((size_t)b * vocab * 4);
  w.pv = (float*)cv.take((size_t)b * ARGMAX_SLICES * 4);
  w.pi = (int32_t*)cv.take((size_t)b * ARGMAX_SLICES * 4);
  return w;
}

sas_status check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return SAS_OK;
  if (!ws) return fail(SAS_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (ws_bytes < need) return fail(SAS_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  if (!aligned16(ws)) return fail(SAS_ERR_INVALID_ARGUMENT, "workspace is not 16-byte aligned");
  return SAS_OK;
}

// Byte offsets of the four products in a layer's packed decode copy (each
// 256-byte aligned), or false when the configuration has none.
struct PackedLayout {
  size_t qkv, o, gu, down, total;
};
bool packed_layout(const sas_config* c, PackedLayout& L) {
  if (c->dtype != SAS_BF16) return false;
  const int d = c->d_model, H = c->n_heads, Hkv = c->n_kv_heads, dh = c->head_dim, F = c->d_ff;
  if (d % 128 != 0 || (H * dh) % 128 != 0 || F % 128 != 0) return false;
  auto bytes = [](int epi, int N, int K) {
    GemmArgs a = {};
    a.epi = epi;
    a.N = N;
    a.K = K;
    return (gemv_packed_elems(a) * 2 + 255) / 256 * 256;
  };
  L.qkv = 0;
  L.o = bytes(EPI_QKV_ROPE, (H + 2 * Hkv) * dh, d);
  L.gu = L.o + bytes(EPI_RESID, d, H * dh);
  L.down = L.gu + bytes(EPI_SWIGLU, F, d);
  L.total = L.down + bytes(EPI_RESID, d, F);
  return true;
}

}  // namespace

namespace sas {
int set_error(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return status;
}
}  // namespace sas

extern "C" {

const char* sas_last_error(void) { return g_err.c_str(); }

const char* sas_version(void) { return "sas-mi355x 0.1 (gfx950)"; }

int32_t sas_profiler_start(int32_t capacity) {
  if (capacity <= 0) return fail(SAS_ERR_INVALID_ARGUMENT, "capacity must be positive");
  return g_prof.start(capacity) == 0 ? SAS_OK : fail(SAS_ERR_HIP, "hipEventCreate failed");
}

int32_t sas_profiler_select(const char* families) {
  g_prof.select(families);
  return SAS_OK;
}

int32_t sas_profiler_stop(void) {
  g_prof.on = false;
  return g_prof.used;
}

int32_t sas_profiler_record(int32_t i, const char** name, float* ms) {
  if (i < 0 || i >= g_prof.used) return fail(SAS_ERR_INVALID_ARGUMENT, "record %d out of range", i);
  *name = g_prof.names[i];
  const int k = g_prof.exact[i] ? 2 : 0;
  return hip_check(hipEventElapsedTime(ms, g_prof.ev[4 * i + k], g_prof.ev[4 * i + k + 1]), "hipEventElapsedTime");
}

size_t sas_workspace_size(const sas_config* c, int32_t op, int32_t batch, int32_t seq_len) {
  if (!c || batch <= 0) return 0;
  Carve cv(nullptr);
  switch (op) {
    case SAS_OP_ATTENTION:
      if (seq_len <= 0 || check_config(c, false) != SAS_OK) return 0;
      carve_attention(cv, c, batch, seq_len);
      break;
    case SAS_OP_ATTENTION_BACKWARD:
      if (seq_len <= 0 || check_config(c, false) != SAS_OK) return 0;
      carve_backward(cv, c, batch, seq_len);
      break;
    case SAS_OP_SELECTOR_BACKWARD:
      if (seq_len <= 0 || check_config(c, false) != SAS_OK) return 0;
      carve_selector_backward(cv, c, batch, seq_len);
      break;
    case SAS_OP_SELECTION_STATS:
      if (seq_len <= 0 || check_config(c, false) != SAS_OK) return 0;
      carve_stats(cv, c, batch, seq_len);
      break;
    case SAS_OP_MLP:
      if (check_config(c, true) != SAS_OK) return 0;
      carve_mlp(cv, c, (size_t)batch);
      break;
    case SAS_OP_LAYER:
      if (seq_len <= 0 || check_config(c, true) != SAS_OK) return 0;
      carve_layer(cv, c, batch, seq_len);
      break;
    case SAS_OP_DECODE:
      if (check_config(c, true) != SAS_OK || blocks_of(c, seq_len) > DSEL_MAX_BLOCKS) return 0;
      carve_decode(cv, c, batch, blocks_of(c, seq_len));
      break;
    case SAS_OP_DECODE_SELECT:
      if (check_config(c, false) != SAS_OK || blocks_of(c, seq_len) > DSEL_MAX_BLOCKS) return 0;
      cv.take(1);
      carve_scores(cv, c, batch, blocks_of(c, seq_len));
      break;
    case SAS_OP_LM_HEAD:
      if (seq_len <= 0 || !c || (c->dtype != SAS_F32 && c->dtype != SAS_BF16) || c->d_model <= 0) return 0;
      carve_lm(cv, c, batch, seq_len);
      break;
    default:
      return 0;
  }
  g_err.clear();
  return cv.off;
}

sas_status sas_attention_backward(const sas_config* c, int32_t batch, int32_t seq_len, const sas_bwd_in* in,
                                  sas_bwd_out* out, void* ws, size_t ws_bytes, void* stream) {
  SAS_TRY(check_config(c, false));
  if (batch <= 0 || seq_len <= 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "batch %d and seq_len %d must be positive", batch, seq_len);
  if (!in || !out) return fail(SAS_ERR_INVALID_ARGUMENT, "in/out is NULL");
  const bool gated = gated_of(c), fullf = full_fwd(c), fullg = full_grad(c);
  const int K = c->top_k > 0 ? c->top_k : 0;
  // the walk over selected blocks: SPARSE, GATED with the sparse scope, and the straight-through gate
  const bool walk = c->mode != SAS_MODE_DENSE && K > 0 && !fullf;
  SAS_TRY(check_ptr(in->q, "in.q", true));
  SAS_TRY(check_ptr(in->k, "in.k", true));
  SAS_TRY(check_ptr(in->v, "in.v", true));
  SAS_TRY(check_ptr(in->o, "in.o", true));
  SAS_TRY(check_ptr(in->d_o, "in.d_o", true));
  SAS_TRY(check_ptr(in->lse, "in.lse", true));
  SAS_TRY(check_ptr(in->sel_idx, "in.sel_idx", walk));
  SAS_TRY(check_ptr(in->log_gate, "in.log_gate", gated && (walk || fullg)));
  SAS_TRY(check_ptr(out->dq, "out.dq", true));
  SAS_TRY(check_ptr(out->dk, "out.dk", true));
  SAS_TRY(check_ptr(out->dv, "out.dv", true));
  SAS_TRY(check_ptr(out->dlog_gate, "out.dlog_gate", false));
  SAS_TRY(check_ptr(out->dlog_gate_full, "out.dlog_gate_full", fullg));
  if (fullg && out->dlog_gate)
    return fail(SAS_ERR_INVALID_ARGUMENT, "scope FULL has no per-slot gradient: pass dlog_gate_full only");
  if (c->dtype == SAS_BF16 && seq_len > BWD_MAX_SEQ)
    return fail(SAS_ERR_UNSUPPORTED, "seq_len %d (the bf16 backward supports <= %d)", seq_len, BWD_MAX_SEQ);
  Carve cv(ws);
  BwdWs bw = carve_backward(cv, c, batch, seq_len);
  SAS_TRY(check_ws(ws, ws_bytes, cv.off));
  hipStream_t s = (hipStream_t)stream;
  const int Hkv = c->n_kv_heads;
  const int NB = (int)cdiv(seq_len, c->block_size);
  const size_t rows = (size_t)batch * Hkv * seq_len;
  if (walk && gated) {
    Timed tm("bwd_gather_gate", s);
    HIP_TRY(launch_gather_gate(in->sel_idx, in->log_gate, batch, seq_len, Hkv, K, NB, bw.sel_bias, s),
            "gather gate");
  }
  // per-slot gradient: asked for, or needed to build the table of the sparse scope
  float* slots = nullptr;
  if (gated && walk && !fullg) slots = out->dlog_gate ? out->dlog_gate : (out->dlog_gate_full ? bw.dlg_slots : nullptr);
  BwdArgs a = {};
  a.b = batch;
  a.n = seq_len;
  a.H = c->n_heads;
  a.Hkv = Hkv;
  a.dh = c->head_dim;
  a.B = c->block_size;
  a.K = walk ? K : 0;
  a.mode = c->mode;
  a.sm_scale = sm_scale_of(c);
  a.Q = in->q;
  a.Kt = in->k;
  a.V = in->v;
  a.O = in->o;
  a.dO = in->d_o;
  a.lse = in->lse;
  a.sel = walk ? in->sel_idx : nullptr;
  a.sel_bias = bw.sel_bias;
  a.dQ = out->dq;
  a.dK = out->dk;
  a.dV = out->dv;
  a.dlog_gate = slots;
  a.delta = bw.delta;
  a.dlg_head = bw.dlg_head;
  a.selmask = bw.selmask;
  a.tile_cnt = bw.tile_cnt;
  a.tile_off = bw.tile_off;
  a.tile_rows = bw.tile_rows;
  a.queue = bw.queue;
  a.log_gate = gated ? in->log_gate : nullptr;
  a.outer = gated && c->gate_pos == SAS_GATE_OUTER;
  a.full = fullg;
  a.ste = gated && c->gate_ste;
  a.dlog_gate_full = fullg ? out->dlog_gate_full : nullptr;
  a.dlg_head_full = bw.dlg_head_full;
  a.doc = in->doc_first_block;
  {
    Timed tm("bwd_zero", s);
    if (out->dlog_gate && !slots) HIP_TRY(launch_fill_f32(out->dlog_gate, rows * K, 0.f, s), "zero dlog_gate");
    if (out->dlog_gate_full && !fullg && !slots)
      HIP_TRY(launch_fill_f32(out->dlog_gate_full, rows * NB, 0.f, s), "zero dlog_gate_full");
  }
  {
    Timed tm("attention_bwd", s);
    HIP_TRY(launch_attention_backward(c->dtype, a, s), "attention backward");
  }
  if (slots && out->dlog_gate_full) {
    Timed tm("bwd_scatter", s);
    HIP_TRY(launch_scatter_slots(in->sel_idx, slots, batch, seq_len, Hkv, K, NB, out->dlog_gate_full, s),
            "scatter slots");
  }
  return SAS_OK;
}

sas_status sas_selector_backward(const sas_config* c, int32_t batch, int32_t seq_len, const sas_sel_bwd_in* in,
                                 sas_sel_bwd_out* out, void* ws, size_t ws_bytes, void* stream) {
  SAS_TRY(check_config(c, false));
  if (batch <= 0 || seq_len <= 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "batch %d and seq_len %d must be positive", batch, seq_len);
  if (!in || !out) return fail(SAS_ERR_INVALID_ARGUMENT, "in/out is NULL");
  const int K = c->top_k;
  const float* dfull = in->dlog_gate_full;
  const bool slots = K > 0 && !dfull;  // per-slot input
  SAS_TRY(check_ptr(in->q, "in.q", true));
  SAS_TRY(check_ptr(in->k, "in.k", true));
  SAS_TRY(check_ptr(in->w_gq, "in.w_gq", false));
  SAS_TRY(check_ptr(in->w_gk, "in.w_gk", false));
  SAS_TRY(check_ptr(in->sel_idx, "in.sel_idx", slots));
  SAS_TRY(check_ptr(in->log_gate, "in.log_gate", slots || dfull));
  SAS_TRY(check_ptr(in->dlog_gate, "in.dlog_gate", slots));
  SAS_TRY(check_ptr(dfull, "in.dlog_gate_full", false));
  SAS_TRY(check_ptr(out->ds, "out.ds", false));
  SAS_TRY(check_ptr(out->dqhat, "out.dqhat", false));
  SAS_TRY(check_ptr(out->dkbar, "out.dkbar", false));
  SAS_TRY(check_ptr(out->dw_gq, "out.dw_gq", in->w_gq != nullptr));
  SAS_TRY(check_ptr(out->dw_gk, "out.dw_gk", in->w_gk != nullptr));
  Carve cv(ws);
  SelBwdWs w = carve_selector_backward(cv, c, batch, seq_len);
  SAS_TRY(check_ws(ws, ws_bytes, cv.off));
  hipStream_t s = (hipStream_t)stream;
  const int n = seq_len, H = c->n_heads, Hkv = c->n_kv_heads, dh = c->head_dim, B = c->block_size;
  const SelBwdShape h = sel_bwd_shape(c, batch, n);
  const int NB = h.NB;
  const size_t rows = (size_t)batch * Hkv * n;
  float* dw_gq = in->w_gq ? out->dw_gq : nullptr;
  float* dw_gk = in->w_gk ? out->dw_gk : nullptr;
  if (K == 0 && !dfull) {  // no selected block: every gradient is zero
    Timed tm("sel_bwd_zero", s);
    HIP_TRY(launch_fill_f32(out->ds, out->ds ? rows * NB : 0, 0.f, s), "zero ds");
    HIP_TRY(launch_fill_f32(out->dqhat, out->dqhat ? rows * dh : 0, 0.f, s), "zero dqhat");
    HIP_TRY(launch_fill_f32(out->dkbar, out->dkbar ? (size_t)batch * Hkv * NB * dh : 0, 0.f, s), "zero dkbar");
    HIP_TRY(launch_fill_f32(dw_gq, dw_gq ? (size_t)Hkv * dh * dh : 0, 0.f, s), "zero dw_gq");
    HIP_TRY(launch_fill_f32(dw_gk, dw_gk ? (size_t)Hkv * dh * dh : 0, 0.f, s), "zero dw_gk");
    return SAS_OK;
  }
  {
    Timed tm("summaries", s);
    HIP_TRY(launch_block_summaries(c->dtype, in->k, batch, n, Hkv, dh, B, in->w_gk, w.kplain, w.ksum, s),
            "block summaries");
  }
  {
    Timed tm("gate_query", s);
    HIP_TRY(launch_gate_query(c->dtype, in->q, batch, n, H, Hkv, dh, in->w_gq, w.qplain, w.qhat, s), "gate query");
  }
  float* ds = out->ds ? out->ds : w.ds;
  {
    Timed tm("sel_bwd_ds", s);
    HIP_TRY(launch_selector_ds(slots ? in->sel_idx : nullptr, in->log_gate, in->dlog_gate, dfull,
                               gated_of(c) ? c->gate_act : SAS_ACT_SOFTMAX, batch, n, Hkv, slots ? K : 0, B, ds,
                               in->doc_first_block, s),
            "ds");
  }
  // s = r / (G sqrt(dh)) with r = qhat . kbar
  const float dr_scale = 1.0f / ((float)(H / Hkv) * sqrtf((float)dh));
  float* dqhat = out->dqhat ? out->dqhat : w.dqhat;
  float* dkbar = out->dkbar ? out->dkbar : w.dkbar;
  Timed tm("sel_bwd_gemm", s);
  if (out->dqhat || dw_gq) {  // dqhat[t] = c sum_m ds[t, m] kbar[m]
    SmallGemm g = {};
    g.M = n, g.N = dh, g.K = NB, g.Z = h.Z, g.splits = 1, g.alpha = dr_scale;
    g.A = ds, g.sAz = (long long)n * NB, g.sAi = NB, g.sAk = 1;
    g.Bm = w.ksum, g.sBz = (long long)NB * dh, g.sBk = dh, g.sBj = 1;
    g.C = dqhat, g.sCz = (long long)n * dh, g.sCs = 0, g.sCi = dh;
    HIP_TRY(launch_small_gemm(c->dtype, g, s), "dqhat");
  }
  if (out->dkbar || dw_gk) {  // dkbar[m] = c sum_t ds[t, m] qhat[t]
    const size_t E = (size_t)NB * dh;
    SmallGemm g = {};
    g.M = NB, g.N = dh, g.K = n, g.Z = h.Z, g.splits = h.s_dkbar, g.alpha = dr_scale;
    g.A = ds, g.sAz = (long long)n * NB, g.sAi = 1, g.sAk = NB;
    g.Bm = w.qhat, g.sBz = (long long)n * dh, g.sBk = dh, g.sBj = 1;
    const bool direct = h.s_dkbar == 1;
    g.C = direct ? dkbar : w.part, g.sCz = direct ? (long long)E : (long long)(E * h.s_dkbar), g.sCs = E, g.sCi = dh;
    HIP_TRY(launch_small_gemm(c->dtype, g, s), "dkbar");
    if (!direct) HIP_TRY(launch_partial_sum(w.part, 1, h.Z, h.s_dkbar, E, dkbar, s), "dkbar sum");
  }
  const size_t E = (size_t)dh * dh;
  if (dw_gq) {  // dW_gq[g] = sum_b sum_t dqhat[t]^T qhat0[t]
    SmallGemm g = {};
    g.M = dh, g.N = dh, g.K = n, g.Z = h.Z, g.splits = h.s_dwq, g.alpha = 1.f;
    g.A = dqhat, g.sAz = (long long)n * dh, g.sAi = 1, g.sAk = dh;
    g.Bm = w.qplain, g.sBz = (long long)n * dh, g.sBk = dh, g.sBj = 1;
    g.C = w.part, g.sCz = (long long)(E * h.s_dwq), g.sCs = E, g.sCi = dh;
    HIP_TRY(launch_small_gemm(c->dtype, g, s), "dw_gq");
    HIP_TRY(launch_partial_sum(w.part, batch, Hkv, h.s_dwq, E, dw_gq, s), "dw_gq sum");
  }
  if (dw_gk) {  // dW_gk[g] = sum_b sum_m dkbar[m]^T kbar0[m]
    SmallGemm g = {};
    g.M = dh, g.N = dh, g.K = NB, g.Z = h.Z, g.splits = h.s_dwk, g.alpha = 1.f;
    g.A = dkbar, g.sAz = (long long)NB * dh, g.sAi = 1, g.sAk = dh;
    g.Bm = w.kplain, g.sBz = (long long)NB * dh, g.sBk = dh, g.sBj = 1;
    g.C = w.part, g.sCz = (long long)(E * h.s_dwk), g.sCs = E, g.sCi = dh;
    HIP_TRY(launch_small_gemm(c->dtype, g, s), "dw_gk");
    HIP_TRY(launch_partial_sum(w.part, batch, Hkv, h.s_dwk, E, dw_gk, s), "dw_gk sum");
  }
  return SAS_OK;
}

sas_status sas_selection_stats(const sas_config* c, int32_t batch, int32_t seq_len, const sas_stats_in* in,
                               sas_stats_out* out, void* ws, size_t ws_bytes, void* stream) {
  SAS_TRY(check_config(c, false));
  if (batch <= 0 || seq_len <= 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "batch %d and seq_len %d must be positive", batch, seq_len);
  if (!in || !out) return fail(SAS_ERR_INVALID_ARGUMENT, "in/out is NULL");
  const bool walk = c->mode != SAS_MODE_DENSE && c->top_k > 0;
  SAS_TRY(check_ptr(in->q, "in.q", true));
  SAS_TRY(check_ptr(in->k, "in.k", true));
  SAS_TRY(check_ptr(in->v, "in.v", out->cov_v != nullptr));
  SAS_TRY(check_ptr(in->sel_idx, "in.sel_idx", walk && (out->cov || out->cov_v || out->sel_union)));
  SAS_TRY(check_ptr(out->cov, "out.cov", false));
  SAS_TRY(check_ptr(out->cov_v, "out.cov_v", false));
  SAS_TRY(check_ptr(out->sel_union, "out.sel_union", false));
  SAS_TRY(check_ptr(out->ref_union, "out.ref_union", false));
  if (seq_len > ATTN_MAX_SEQ) return fail(SAS_ERR_UNSUPPORTED, "seq_len %d (supported <= %d)", seq_len, ATTN_MAX_SEQ);
  Carve cv(ws);
  StatsWs w = carve_stats(cv, c, batch, seq_len);
  SAS_TRY(check_ws(ws, ws_bytes, cv.off));
  hipStream_t s = (hipStream_t)stream;
  const int n = seq_len, Hkv = c->n_kv_heads, NB = (int)cdiv(n, c->block_size);
  const int K = c->top_k > 0 ? c->top_k : 0;
  if (out->sel_union && walk) {
    Timed tm("stats_union", s);
    HIP_TRY(launch_sel_union(in->sel_idx, (size_t)batch * Hkv * n, K, NB, out->sel_union, s), "selection union");
  }
  if (!out->cov && !out->cov_v && !out->ref_union) return SAS_OK;
  if (out->cov_v) {
    Timed tm("stats_vnorm", s);
    HIP_TRY(launch_vnorm(c->dtype, in->v, (size_t)batch * n * Hkv, c->head_dim, w.lvn, s), "value norms");
  } else {
    HIP_TRY(launch_fill_f32(w.lvn, (size_t)batch * n * Hkv, 0.f, s), "value norms");
  }
  StatsArgs a = {};
  a.b = batch;
  a.n = n;
  a.H = c->n_heads;
  a.Hkv = Hkv;
  a.dh = c->head_dim;
  a.B = c->block_size;
  a.K = walk ? K : 0;
  a.mode = c->mode;
  a.sm_scale = sm_scale_of(c);
  a.Q = in->q;
  a.Kt = in->k;
  a.sel = walk ? in->sel_idx : nullptr;
  a.lvn = w.lvn;
  a.cov = out->cov;
  a.cov_v = out->cov_v;
  a.blk_lse = out->ref_union ? w.blk_lse : nullptr;
  a.doc = in->doc_first_block;
  a.queue = w.queue;
  {
    Timed tm("stats", s);
    HIP_TRY(launch_stats(c->dtype, a, s), "selection stats");
  }
  if (out->ref_union) {
    Timed tm("stats_reference", s);
    HIP_TRY(launch_ref_sets(w.blk_lse, batch, n, c->n_heads, Hkv, c->block_size, K, w.head_mask, out->ref_union,
                            in->doc_first_block, s),
            "reference sets");
  }
  return SAS_OK;
}

sas_status sas_overlap_recall(int64_t words, const uint32_t* sel_union, const uint32_t* ref_union, uint64_t* counts,
                              void* stream) {
  if (words < 0) return fail(SAS_ERR_INVALID_ARGUMENT, "words %lld is negative", (long long)words);
  SAS_TRY(check_ptr(sel_union, "sel_union", words > 0));
  SAS_TRY(check_ptr(ref_union, "ref_union", words > 0));
  SAS_TRY(check_ptr(counts, "counts", true));
  HIP_TRY(launch_overlap_count(sel_union, ref_union, (size_t)words, (unsigned long long*)counts, (hipStream_t)stream),
          "overlap counts");
  return SAS_OK;
}

sas_status sas_attention_prefill(const sas_config* c, int32_t batch, int32_t seq_len, const sas_attn_in* in,
                                 sas_attn_out* out, void* ws, size_t ws_bytes, void* stream) {
  SAS_TRY(check_config(c, false));
  if (batch <= 0 || seq_len <= 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "batch %d and seq_len %d must be positive", batch, seq_len);
  if (!in || !out) return fail(SAS_ERR_INVALID_ARGUMENT, "in/out is NULL");
  SAS_TRY(check_ptr(in->q, "in.q", true));
  SAS_TRY(check_ptr(in->k, "in.k", true));
  SAS_TRY(check_ptr(in->v, "in.v", true));
  SAS_TRY(check_ptr(in->w_gq, "in.w_gq", false));
  SAS_TRY(check_ptr(in->w_gk, "in.w_gk", false));
  SAS_TRY(check_ptr(in->score_noise, "in.score_noise", false));
  SAS_TRY(check_ptr(in->doc_first_block, "in.doc_first_block", false));
  SAS_TRY(check_ptr(out->o, "out.o", true));
  SAS_TRY(check_ptr(out->lse, "out.lse", false));
  SAS_TRY(check_ptr(out->k_summary, "out.k_summary", false));
  SAS_TRY(check_ptr(out->sel_idx, "out.sel_idx", false));
  SAS_TRY(check_ptr(out->log_gate, "out.log_gate", false));
  SAS_TRY(check_ptr(out->tau, "out.tau", false));
  Carve cv(ws);
  AttnWs aw = carve_attention(cv, c, batch, seq_len);
  SAS_TRY(check_ws(ws, ws_bytes, cv.off));
  SAS_TRY(run_attention(c, batch, seq_len, in->q, in->k, in->v, in->w_gq, in->w_gk, out->o, out->lse,
                        out->k_summary, out->sel_idx, out->log_gate, out->tau, aw, (hipStream_t)stream, false,
                        in->score_noise, in->doc_first_block));
  return SAS_OK;
}

sas_status sas_mlp_forward(const sas_config* c, int32_t tokens, const void* x, const sas_layer_weights* w,
                           void* y, void* ws, size_t ws_bytes, void* stream) {
  SAS_TRY(check_config(c, true));
  if (tokens <= 0) return fail(SAS_ERR_INVALID_ARGUMENT, "tokens %d must be positive", tokens);
  SAS_TRY(check_ptr(x, "x", true));
  SAS_TRY(check_ptr(y, "y", true));
  SAS_TRY(check_weights(w, false, true));
  Carve cv(ws);
  MlpWs mw = carve_mlp(cv, c, (size_t)tokens);
  SAS_TRY(check_ws(ws, ws_bytes, cv.off));
  return run_mlp(c, (size_t)tokens, x, w, y, mw, (hipStream_t)stream);
}

sas_status sas_layer_forward(const sas_config* c, int32_t batch, int32_t seq_len, const void* x,
                             const sas_layer_weights* w, void* y, sas_attn_out* stats, sas_layer_taps* taps,
                             sas_paged_kv* cache, void* ws, size_t ws_bytes, void* stream) {
  SAS_TRY(check_config(c, true));
  if (batch <= 0 || seq_len <= 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "batch %d and seq_len %d must be positive", batch, seq_len);
  SAS_TRY(check_ptr(x, "x", true));
  SAS_TRY(check_ptr(y, "y", true));
  SAS_TRY(check_weights(w, true, true));
  sas_attn_out st = {};
  if (stats) {
    st = *stats;
    SAS_TRY(check_ptr(st.o, "stats.o", false));
    SAS_TRY(check_ptr(st.lse, "stats.lse", false));
    SAS_TRY(check_ptr(st.k_summary, "stats.k_summary", false));
    SAS_TRY(check_ptr(st.sel_idx, "stats.sel_idx", false));
    SAS_TRY(check_ptr(st.log_gate, "stats.log_gate", false));
    SAS_TRY(check_ptr(st.tau, "stats.tau", false));
  }
  sas_layer_taps tp = {};
  if (taps) {
    tp = *taps;
    SAS_TRY(check_ptr(tp.q, "taps.q", false));
    SAS_TRY(check_ptr(tp.k, "taps.k", false));
    SAS_TRY(check_ptr(tp.v, "taps.v", false));
    SAS_TRY(check_ptr(tp.h1, "taps.h1", false));
  }
  if (cache) SAS_TRY(check_cache(c, cache));
  Carve cv(ws);
  LayerWs lw = carve_layer(cv, c, batch, seq_len);
  SAS_TRY(check_ws(ws, ws_bytes, cv.off));
  hipStream_t s = (hipStream_t)stream;
  const size_t T = (size_t)batch * seq_len;
  void* q = tp.q ? tp.q : lw.q;
  void* k = tp.k ? tp.k : lw.k;
  void* v = tp.v ? tp.v : lw.v;
  void* o = st.o ? st.o : lw.o;
  void* h1 = tp.h1 ? tp.h1 : lw.h1;

  {
    // the first norm also writes the rotary table of positions 0 .. seq_len - 1 (rows of the first sequence)
    Timed tm("rmsnorm", s);
    HIP_TRY(launch_rmsnorm_rope(c->dtype, x, w->rms1, lw.u1, (int)T, c->d_model, c->rms_eps, nullptr, lw.rope,
                                c->head_dim, c->rope_base, seq_len, s),
            "rmsnorm");
  }
  GemmArgs g = {};
  g.epi = EPI_QKV_ROPE;
  g.M = (int)T;
  g.K = c->d_model;
  g.A = lw.u1;
  g.B0 = w->wq;
  g.B1 = w->wk;
  g.B2 = w->wv;
  g.N = (c->n_heads + 2 * c->n_kv_heads) * c->head_dim;
  g.out = q;
  g.out1 = k;
  g.out2 = v;
  g.n_heads = c->n_heads;
  g.n_kv_heads = c->n_kv_heads;
  g.head_dim = c->head_dim;
  g.seq_len = seq_len;
  g.rope = lw.rope;
  // with a cache, the QKV product writes the K/V pages itself where it can
  const DecodeArgs da = cache ? decode_args(c, batch, nullptr, cache, w) : DecodeArgs{};
  g.prefill_cache = (cache && gemm_fills_cache(c->dtype, g)) ? &da : nullptr;
  {
    Timed tm("gemm_qkv", s);
    HIP_TRY(launch_gemm(c->dtype, g, s), "qkv gemm");
  }
  SAS_TRY(run_attention(c, batch, seq_len, q, k, v, w->w_gq, w->w_gk, o, st.lse, st.k_summary, st.sel_idx,
                        st.log_gate, st.tau, lw.att, s, cache != nullptr));
  if (cache) {
    Timed tm("cache_fill", s);
    HIP_TRY(launch_cache_fill(c->dtype, k, v, st.k_summary ? st.k_summary : lw.att.ksum, batch, seq_len,
                              c->n_kv_heads, c->head_dim, c->block_size, cdiv(seq_len, c->block_size), da, s,
                              g.prefill_cache == nullptr),
            "cache fill");
  }
  GemmArgs og = {};
  og.epi = EPI_RESID;
  og.M = (int)T;
  og.K = c->n_heads * c->head_dim;
  og.A = o;
  og.B0 = w->wo;
  og.N = c->d_model;
  og.resid = x;
  og.out = h1;
  {
    Timed tm("gemm_o", s);
    HIP_TRY(launch_gemm(c->dtype, og, s), "o-proj gemm");
  }
  return run_mlp(c, T, h1, w, y, lw.mlp, s);
}

size_t sas_decode_packed_bytes(const sas_config* c) {
  PackedLayout L;
  if (!c || check_config(c, true) != SAS_OK || !packed_layout(c, L)) return 0;
  return L.total;
}

sas_status sas_pack_decode_weights(const sas_config* c, const sas_layer_weights* w, void* packed,
                                   size_t packed_bytes, void* stream) {
  SAS_TRY(check_config(c, true));
  PackedLayout L;
  if (!packed_layout(c, L))
    return fail(SAS_ERR_UNSUPPORTED, "no packed decode layout for this configuration (bf16 with d, H*dh and "
                                     "d_ff multiples of 128)");
  if (!w) return fail(SAS_ERR_INVALID_ARGUMENT, "weights are NULL");
  SAS_TRY(check_ptr(w->wq, "wq", true));
  SAS_TRY(check_ptr(w->wk, "wk", true));
  SAS_TRY(check_ptr(w->wv, "wv", true));
  SAS_TRY(check_ptr(w->wo, "wo", true));
  SAS_TRY(check_ptr(w->w_gate, "w_gate", true));
  SAS_TRY(check_ptr(w->w_up, "w_up", true));
  SAS_TRY(check_ptr(w->w_down, "w_down", true));
  SAS_TRY(check_ptr(packed, "packed", true));
  if (((uintptr_t)packed & 255u) != 0) return fail(SAS_ERR_INVALID_ARGUMENT, "packed is not 256-byte aligned");
  if (packed_bytes < L.total)
    return fail(SAS_ERR_WORKSPACE, "packed holds %zu bytes, the layer's packed copy needs %zu", packed_bytes,
                L.total);
  hipStream_t s = (hipStream_t)stream;
  const int d = c->d_model, H = c->n_heads, Hkv = c->n_kv_heads, dh = c->head_dim, F = c->d_ff;
  char* out = (char*)packed;
  auto pack = [&](int epi, int N, int K, const void* b0, const void* b1, const void* b2, size_t off) {
    GemmArgs a = {};
    a.epi = epi;
    a.N = N;
    a.K = K;
    a.B0 = b0;
    a.B1 = b1;
    a.B2 = b2;
    a.n_heads = H;
    a.n_kv_heads = Hkv;
    a.head_dim = dh;
    return launch_gemv_pack(a, out + off, s);
  };
  HIP_TRY(pack(EPI_QKV_ROPE, (H + 2 * Hkv) * dh, d, w->wq, w->wk, w->wv, L.qkv), "pack qkv");
  HIP_TRY(pack(EPI_RESID, d, H * dh, w->wo, nullptr, nullptr, L.o), "pack o");
  HIP_TRY(pack(EPI_SWIGLU, F, d, w->w_gate, w->w_up, nullptr, L.gu), "pack gate/up");
  HIP_TRY(pack(EPI_RESID, d, F, w->w_down, nullptr, nullptr, L.down), "pack down");
  return SAS_OK;
}

sas_status sas_decode_step(const sas_config* c, int32_t batch, const void* x, const int32_t* pos,
                           const sas_layer_weights* w, sas_paged_kv* cache, void* y, int32_t* sel_idx,
                           sas_layer_taps* taps, void* ws, size_t ws_bytes, void* stream) {
  SAS_TRY(check_config(c, true));
  if (batch <= 0) return fail(SAS_ERR_INVALID_ARGUMENT, "batch %d must be positive", batch);
  SAS_TRY(check_ptr(x, "x", true));
  SAS_TRY(check_ptr(pos, "pos", true));
  SAS_TRY(check_ptr(y, "y", true));
  SAS_TRY(check_ptr(sel_idx, "sel_idx", false));
  SAS_TRY(check_weights(w, true, true));
  if (!cache) return fail(SAS_ERR_INVALID_ARGUMENT, "cache is NULL");
  SAS_TRY(check_cache(c, cache));
  sas_layer_taps tp = {};
  if (taps) {
    tp = *taps;
    SAS_TRY(check_ptr(tp.q, "taps.q", false));
    SAS_TRY(check_ptr(tp.k, "taps.k", false));
    SAS_TRY(check_ptr(tp.v, "taps.v", false));
    SAS_TRY(check_ptr(tp.h1, "taps.h1", false));
  }
  Carve cv(ws);
  DecodeWs dw = carve_decode(cv, c, batch, cache->max_blocks);
  SAS_TRY(check_ws(ws, ws_bytes, cv.off));
  // the taps, when given, take the place of the step's own scratch rows
  if (tp.q) dw.q = tp.q;
  if (tp.k) dw.k = tp.k;
  if (tp.v) dw.v = tp.v;
  if (tp.h1) dw.h1 = tp.h1;
  hipStream_t s = (hipStream_t)stream;
  const DecodeArgs da = decode_args(c, batch, pos, cache, w);
  const int H = c->n_heads, Hkv = c->n_kv_heads, dh = c->head_dim;
  int32_t* sel = sel_idx ? sel_idx : dw.sel;
  // The first RMSNorm launch also writes the rotary rows of the positions.  On
  // the skinny-GEMM path the QKV product appends K/V to the cache itself
  // (unless a summary projection follows the append).
  const bool gemv = c->dtype == SAS_BF16 && batch <= 16 && c->d_model % 128 == 0;
  const bool fused_append = gemv && !da.w_gk;
  // the packed copy of the weights, streamed by the skinny-GEMM path when given
  PackedLayout pl;
  const char* pk = (gemv && w->decode_packed && packed_layout(c, pl)) ? (const char*)w->decode_packed : nullptr;
  {
    Timed tm("rmsnorm", s);
    HIP_TRY(launch_rmsnorm_rope(c->dtype, x, w->rms1, dw.u1, batch, c->d_model, c->rms_eps, pos, dw.rope, dh,
                                c->rope_base, batch, s),
            "rmsnorm");
  }
  GemmArgs g = {};
  g.epi = EPI_QKV_ROPE;
  g.M = batch;
  g.K = c->d_model;
  g.A = dw.u1;
  g.B0 = w->wq;
  g.B1 = w->wk;
  g.B2 = w->wv;
  g.N = (H + 2 * Hkv) * dh;
  g.out = dw.q;
  g.out1 = dw.k;
  g.out2 = dw.v;
  g.n_heads = H;
  g.n_kv_heads = Hkv;
  g.head_dim = dh;
  g.rope = dw.rope;
  g.row_pos = fused_append ? pos : nullptr;
  g.append = fused_append ? &da : nullptr;
  g.packed = pk ? pk + pl.qkv : nullptr;
  {
    Timed tm("dec_qkv", s);
    HIP_TRY(small_gemm(c->dtype, g, s), "qkv gemm");
  }
  if (!fused_append) {
    Timed tm("dec_append", s);
    HIP_TRY(launch_kv_append(c->dtype, dw.k, dw.v, da, dw.kplain, s), "kv append");
  }
  {
    Timed tm("dec_select", s);
    HIP_TRY(launch_decode_select(c->dtype, dw.q, da, sel, dw.scores, s), "decode select");
  }
  {
    Timed tm("dec_attention", s);
    HIP_TRY(launch_decode_attention(c->dtype, dw.q, da, sel, dw.part_ml, dw.part_o, dw.o, s), "decode attention");
  }
  GemmArgs og = {};
  og.epi = EPI_RESID;
  og.M = batch;
  og.K = H * dh;
  og.A = dw.o;
  og.B0 = w->wo;
  og.N = c->d_model;
  og.resid = x;
  og.out = dw.h1;
  og.packed = pk ? pk + pl.o : nullptr;
  {
    Timed tm("dec_o", s);
    HIP_TRY(small_gemm(c->dtype, og, s), "o-proj gemm");
  }
  {
    Timed tm("rmsnorm", s);
    HIP_TRY(launch_rmsnorm(c->dtype, dw.h1, w->rms2, dw.mlp.u2, batch, c->d_model, c->rms_eps, s), "rmsnorm");
  }
  GemmArgs gu = {};
  gu.epi = EPI_SWIGLU;
  gu.M = batch;
  gu.K = c->d_model;
  gu.A = dw.mlp.u2;
  gu.B0 = w->w_gate;
  gu.B1 = w->w_up;
  gu.N = c->d_ff;
  gu.out = dw.mlp.a;
  gu.packed = pk ? pk + pl.gu : nullptr;
  {
    Timed tm("dec_gate_up", s);
    HIP_TRY(small_gemm(c->dtype, gu, s), "gate/up gemm");
  }
  GemmArgs dg = {};
  dg.epi = EPI_RESID;
  dg.M = batch;
  dg.K = c->d_ff;
  dg.A = dw.mlp.a;
  dg.B0 = w->w_down;
  dg.N = c->d_model;
  dg.resid = dw.h1;
  dg.out = y;
  dg.packed = pk ? pk + pl.down : nullptr;
  {
    Timed tm("dec_down", s);
    HIP_TRY(small_gemm(c->dtype, dg, s), "down gemm");
  }
  return SAS_OK;
}

sas_status sas_decode_select(const sas_config* c, int32_t batch, const void* q, const int32_t* pos,
                             const void* w_gq, const sas_paged_kv* cache, int32_t* sel_idx, void* ws,
                             size_t ws_bytes, void* stream) {
  SAS_TRY(check_config(c, false));
  if (batch <= 0) return fail(SAS_ERR_INVALID_ARGUMENT, "batch %d must be positive", batch);
  SAS_TRY(check_ptr(q, "q", true));
  SAS_TRY(check_ptr(pos, "pos", true));
  SAS_TRY(check_ptr(w_gq, "w_gq", false));
  SAS_TRY(check_ptr(sel_idx, "sel_idx", true));
  if (!cache) return fail(SAS_ERR_INVALID_ARGUMENT, "cache is NULL");
  SAS_TRY(check_ptr(cache->k_summary, "cache.k_summary", true));
  if (cache->max_blocks <= 0 || cache->max_blocks > DSEL_MAX_BLOCKS)
    return fail(SAS_ERR_UNSUPPORTED, "max_blocks %d (supported: 1..%d)", cache->max_blocks, DSEL_MAX_BLOCKS);
  Carve cv(ws);
  cv.take(1);
  double* scores = carve_scores(cv, c, batch, cache->max_blocks);
  SAS_TRY(check_ws(ws, ws_bytes, cv.off));
  sas_layer_weights w = {};
  w.w_gq = w_gq;
  const DecodeArgs da = decode_args(c, batch, pos, cache, &w);
  hipStream_t s = (hipStream_t)stream;
  {
    Timed tm("dec_select", s);
    HIP_TRY(launch_decode_select(c->dtype, q, da, sel_idx, scores, s), "decode select");
  }
  return SAS_OK;
}

sas_status sas_embed(const sas_config* c, int32_t batch, int32_t seq_len, const int32_t* ids, const void* table,
                     int32_t vocab, const void* img_embed, int32_t n_img, void* x, void* stream) {
  if (!c || (c->dtype != SAS_F32 && c->dtype != SAS_BF16) || c->d_model <= 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "config is NULL or invalid");
  if (batch <= 0 || seq_len <= 0 || vocab <= 0 || n_img < 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "batch %d, seq_len %d, vocab %d must be positive, n_img %d >= 0", batch,
                seq_len, vocab, n_img);
  SAS_TRY(check_ptr(ids, "ids", true));
  SAS_TRY(check_ptr(table, "table", true));
  SAS_TRY(check_ptr(img_embed, "img_embed", false));
  SAS_TRY(check_ptr(x, "x", true));
  hipStream_t s = (hipStream_t)stream;
  Timed tm("embed", s);
  HIP_TRY(launch_embed(c->dtype, batch, seq_len, ids, table, vocab, img_embed, n_img, x, c->d_model, s), "embed");
  return SAS_OK;
}

sas_status sas_lm_head_argmax(const sas_config* c, int32_t batch, const void* h, const void* gamma,
                              const void* w_lm, int32_t vocab, float* logits, int32_t* tokens, void* ws,
                              size_t ws_bytes, void* stream) {
  if (!c || (c->dtype != SAS_F32 && c->dtype != SAS_BF16) || c->d_model <= 0 || c->d_model % 8)
    return fail(SAS_ERR_INVALID_ARGUMENT, "config is NULL or invalid");
  if (batch <= 0 || vocab <= 0)
    return fail(SAS_ERR_INVALID_ARGUMENT, "batch %d and vocab %d must be positive", batch, vocab);
  if (c->dtype == SAS_BF16 && (batch > 16 || c->d_model % 128))
    return fail(SAS_ERR_UNSUPPORTED, "bf16 LM head needs batch <= 16 and d_model %% 128 == 0");
  SAS_TRY(check_ptr(h, "h", true));
  SAS_TRY(check_ptr(gamma, "gamma", true));
  SAS_TRY(check_ptr(w_lm, "w_lm", true));
  SAS_TRY(check_ptr(logits, "logits", false));
  SAS_TRY(check_ptr(tokens, "tokens", true));
  Carve cv(ws);
  LmWs lw = carve_lm(cv, c, batch, vocab);
  SAS_TRY(check_ws(ws, ws_bytes, cv.off));
  hipStream_t s = (hipStream_t)stream;
  float* lg = logits ? logits : lw.logits;
  {
    Timed tm("rmsnorm", s);
    HIP_TRY(launch_rmsnorm(c->dtype, h, gamma, lw.u, batch, c->d_model, c->rms_eps, s), "rmsnorm");
  }
  GemmArgs g = {};
  g.epi = EPI_F32OUT;
  g.M = batch;
  g.K = c->d_model;
  g.A = lw.u;
  g.B0 = w_lm;
  g.N = vocab;
  g.out = lg;
  {
    Timed tm("lm_head", s);
    HIP_TRY(small_gemm(c->dtype, g, s), "lm head");
  }
  {
    Timed tm("argmax", s);
    HIP_TRY(launch_argmax(lg, batch, vocab, lw.pv, lw.pi, ARGMAX_SLICES, tokens, s), "argmax");
  }
  return SAS_OK;
}

}  // extern "C"
