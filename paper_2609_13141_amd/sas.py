"""ctypes binding of ``libsas.so`` (the C ABI declared in ``include/sas.h``).

Argument marshalling only: torch tensors provide device memory and the
current HIP stream; every computation runs in the library's HIP kernels.
The library is loaded on first use; if it is missing or was built without a
GPU target the call raises instead of computing anything another way.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import torch

from .configs import Workload

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsas.so")

SAS_OK, SAS_ERR_INVALID_ARGUMENT, SAS_ERR_UNSUPPORTED, SAS_ERR_WORKSPACE, SAS_ERR_HIP = 0, -1, -2, -3, -4
SAS_F32, SAS_BF16 = 0, 1
MODES = {"dense": 0, "sparse": 1, "gated": 2}
GATE_POS = {"inner": 0, "outer": 1}
GATE_ACT = {"softmax": 0, "sigmoid": 1, "raw": 2}
SCOPES = {"sparse": 0, "full": 1}
(OP_ATTENTION, OP_MLP, OP_LAYER, OP_DECODE, OP_LM_HEAD, OP_DECODE_SELECT, OP_ATTENTION_BACKWARD,
 OP_SELECTOR_BACKWARD, OP_SELECTION_STATS) = range(9)
TORCH_DTYPE = {"bf16": torch.bfloat16, "f32": torch.float32}

EXPORTS = ("sas_workspace_size", "sas_attention_prefill", "sas_mlp_forward", "sas_layer_forward",
           "sas_decode_step", "sas_decode_step_noalloc", "sas_decode_select", "sas_attention_backward", "sas_selector_backward", "sas_selection_stats", "sas_overlap_recall", "sas_embed", "sas_lm_head_argmax", "sas_last_error", "sas_version",
           "sas_profiler_start", "sas_profiler_select", "sas_profiler_stop", "sas_profiler_record",
           "sas_decode_packed_bytes", "sas_pack_decode_weights")


class SasError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"sas status {status}: {msg}")
        self.status = status


class Config(C.Structure):
    _fields_ = [("d_model", C.c_int32), ("n_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("d_ff", C.c_int32), ("block_size", C.c_int32),
                ("top_k", C.c_int32), ("rope_base", C.c_float), ("rms_eps", C.c_float),
                ("sm_scale", C.c_float), ("dtype", C.c_int32), ("mode", C.c_int32),
                ("gate_pos", C.c_int32), ("gate_act", C.c_int32), ("scope", C.c_int32), ("gate_ste", C.c_int32)]


class AttnIn(C.Structure):
    _fields_ = [("q", C.c_void_p), ("k", C.c_void_p), ("v", C.c_void_p), ("w_gq", C.c_void_p),
                ("w_gk", C.c_void_p), ("score_noise", C.c_void_p), ("doc_first_block", C.c_void_p)]


class AttnOut(C.Structure):
    _fields_ = [("o", C.c_void_p), ("lse", C.c_void_p), ("k_summary", C.c_void_p),
                ("sel_idx", C.c_void_p), ("log_gate", C.c_void_p), ("tau", C.c_void_p)]


class BwdIn(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in ("q", "k", "v", "o", "d_o", "lse", "sel_idx", "log_gate", "doc_first_block")]


class BwdOut(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in ("dq", "dk", "dv", "dlog_gate", "dlog_gate_full")]


class StatsIn(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in ("q", "k", "v", "sel_idx", "doc_first_block")]


class StatsOut(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in ("cov", "cov_v", "sel_union", "ref_union")]


class SelBwdIn(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in ("q", "k", "w_gq", "w_gk", "sel_idx", "log_gate", "dlog_gate",
                                          "dlog_gate_full", "doc_first_block")]


class SelBwdOut(C.Structure):
    _fields_ = [(f, C.c_void_p) for f in ("ds", "dqhat", "dkbar", "dw_gq", "dw_gk")]


class LayerWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("rms1", "wq", "wk", "wv", "wo", "rms2", "w_gate", "w_up",
                                          "w_down", "w_gq", "w_gk", "decode_packed")]


class LayerTaps(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("q", "k", "v", "h1")]


class PagedKV(C.Structure):
    _fields_ = [("k_pages", C.c_void_p), ("v_pages", C.c_void_p), ("block_table", C.c_void_p),
                ("k_summary", C.c_void_p), ("num_pages", C.c_int32), ("page_size", C.c_int32),
                ("max_pages_per_seq", C.c_int32), ("max_blocks", C.c_int32)]


_lib = None


def lib() -> C.CDLL:
    """Load libsas.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_13141_amd.build`")
    L = C.CDLL(LIB_PATH)
    vp, i32, sz = C.c_void_p, C.c_int32, C.c_size_t
    L.sas_workspace_size.restype = sz
    L.sas_workspace_size.argtypes = [C.POINTER(Config), i32, i32, i32]
    L.sas_attention_prefill.restype = i32
    L.sas_attention_prefill.argtypes = [C.POINTER(Config), i32, i32, C.POINTER(AttnIn), C.POINTER(AttnOut),
                                        vp, sz, vp]
    L.sas_mlp_forward.restype = i32
    L.sas_mlp_forward.argtypes = [C.POINTER(Config), i32, vp, C.POINTER(LayerWeights), vp, vp, sz, vp]
    L.sas_layer_forward.restype = i32
    L.sas_layer_forward.argtypes = [C.POINTER(Config), i32, i32, vp, C.POINTER(LayerWeights), vp,
                                    C.POINTER(AttnOut), C.POINTER(LayerTaps), C.POINTER(PagedKV), vp, sz, vp]
    L.sas_decode_step.restype = i32
    L.sas_decode_step.argtypes = [C.POINTER(Config), i32, vp, vp, C.POINTER(LayerWeights), C.POINTER(PagedKV),
                                  vp, vp, C.POINTER(LayerTaps), vp, sz, vp]
    L.sas_decode_step_noalloc.restype = i32
    L.sas_decode_step_noalloc.argtypes = [C.POINTER(Config), i32, vp, vp, C.POINTER(LayerWeights),
                                          C.POINTER(PagedKV), vp, vp, vp]
    L.sas_decode_select.restype = i32
    L.sas_decode_select.argtypes = [C.POINTER(Config), i32, vp, vp, vp, C.POINTER(PagedKV), vp, vp, sz, vp]
    L.sas_attention_backward.restype = i32
    L.sas_attention_backward.argtypes = [C.POINTER(Config), i32, i32, C.POINTER(BwdIn), C.POINTER(BwdOut), vp, sz,
                                         vp]
    L.sas_selector_backward.restype = i32
    L.sas_selector_backward.argtypes = [C.POINTER(Config), i32, i32, C.POINTER(SelBwdIn), C.POINTER(SelBwdOut), vp,
                                        sz, vp]
    L.sas_selection_stats.restype = i32
    L.sas_selection_stats.argtypes = [C.POINTER(Config), i32, i32, C.POINTER(StatsIn), C.POINTER(StatsOut), vp, sz,
                                      vp]
    L.sas_overlap_recall.restype = i32
    L.sas_overlap_recall.argtypes = [C.c_int64, vp, vp, vp, vp]
    L.sas_embed.restype = i32
    L.sas_embed.argtypes = [C.POINTER(Config), i32, i32, vp, vp, i32, vp, i32, vp, vp]
    L.sas_lm_head_argmax.restype = i32
    L.sas_lm_head_argmax.argtypes = [C.POINTER(Config), i32, vp, vp, vp, i32, vp, vp, vp, sz, vp]
    L.sas_last_error.restype = C.c_char_p
    L.sas_last_error.argtypes = []
    L.sas_version.restype = C.c_char_p
    L.sas_version.argtypes = []
    L.sas_profiler_start.restype = i32
    L.sas_profiler_start.argtypes = [i32]
    L.sas_profiler_select.restype = i32
    L.sas_profiler_select.argtypes = [C.c_char_p]
    L.sas_decode_packed_bytes.restype = sz
    L.sas_decode_packed_bytes.argtypes = [C.POINTER(Config)]
    L.sas_pack_decode_weights.restype = i32
    L.sas_pack_decode_weights.argtypes = [C.POINTER(Config), C.POINTER(LayerWeights), vp, sz, vp]
    L.sas_profiler_stop.restype = i32
    L.sas_profiler_stop.argtypes = []
    L.sas_profiler_record.restype = i32
    L.sas_profiler_record.argtypes = [i32, C.POINTER(C.c_char_p), C.POINTER(C.c_float)]
    _lib = L
    return L


def _check(status: int):
    if status != SAS_OK:
        raise SasError(status, lib().sas_last_error().decode())


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def make_config(w: Workload, mode: str | None = None, sm_scale: float = 0.0, *, gate_pos: str = "inner",
                gate_act: str = "softmax", scope: str = "sparse", ste: bool = False) -> Config:
    """Library config of a workload; the gating keywords select one of the
    training formulations of Table 1 (GATED mode only)."""
    return Config(w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.d_ff, w.block_size, w.top_k,
                  w.rope_base, w.rms_eps, sm_scale, SAS_BF16 if w.dtype == "bf16" else SAS_F32,
                  MODES[mode or w.mode], GATE_POS[gate_pos], GATE_ACT[gate_act], SCOPES[scope], int(ste))


def workspace_size(cfg: Config, op: int, batch: int, seq_len: int) -> int:
    return int(lib().sas_workspace_size(C.byref(cfg), op, batch, seq_len))


class Workspace:
    """Grow-only device scratch buffer reused across calls."""

    def __init__(self, device="cuda"):
        self.device = device
        self.buf = None

    def get(self, nbytes: int):
        if nbytes == 0:
            return None, 0
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self.buf, self.buf.numel()


_default_ws: dict = {}


def _ws(ws: Workspace | None, nbytes: int):
    if ws is None:
        dev = torch.cuda.current_device()
        ws = _default_ws.setdefault(dev, Workspace(f"cuda:{dev}"))
    buf, n = ws.get(nbytes)
    return _ptr(buf), n


def weights_struct(W: dict) -> LayerWeights:
    return LayerWeights(*[_ptr(W.get(k)) for k in ("rms1", "wq", "wk", "wv", "wo", "rms2", "w_gate",
                                                   "w_up", "w_down", "w_gq", "w_gk", "decode_packed")])


def attention_prefill(cfg: Config, q, k, v, w_gq=None, w_gk=None, *, lse=True, k_summary=True,
                      sel_idx=True, log_gate=False, tau=False, noise=None, doc=None,
                      ws: Workspace | None = None) -> dict:
    """Selector + SAS attention.  q [b,n,H,dh], k/v [b,n,Hkv,dh] on the GPU;
    noise [b,Hkv,n,NB] fp32 (optional) is added to the selector scores; doc
    [b,NB] int32 (optional) packs several block-aligned documents per row."""
    b, n, H, dh = q.shape
    Hkv = k.shape[2]
    B, K = cfg.block_size, cfg.top_k
    NB = -(-n // B)
    dev = q.device
    out = {"o": torch.empty_like(q)}
    if lse:
        out["lse"] = torch.empty(b, H, n, dtype=torch.float32, device=dev)
    if k_summary:
        out["k_summary"] = torch.empty(b, Hkv, NB, dh, dtype=q.dtype, device=dev)
    if sel_idx:
        out["sel_idx"] = torch.empty(b, Hkv, n, K, dtype=torch.int32, device=dev)
    if log_gate:
        out["log_gate"] = torch.empty(b, Hkv, n, NB, dtype=torch.float32, device=dev)
    if tau:
        out["tau"] = torch.empty(b, Hkv, n, dtype=torch.float32, device=dev)
    ain = AttnIn(_ptr(q), _ptr(k), _ptr(v), _ptr(w_gq), _ptr(w_gk), _ptr(noise), _ptr(doc))
    aout = AttnOut(*[_ptr(out.get(f)) for f in ("o", "lse", "k_summary", "sel_idx", "log_gate", "tau")])
    wsp, wsn = _ws(ws, workspace_size(cfg, OP_ATTENTION, b, n))
    _check(lib().sas_attention_prefill(C.byref(cfg), b, n, C.byref(ain), C.byref(aout), wsp, wsn, _stream()))
    return out


def attention_backward(cfg: Config, q, k, v, o, d_o, lse, sel_idx=None, log_gate=None, *, dlog_gate: bool = True,
                       dlog_gate_full: bool = False, doc=None, ws: Workspace | None = None) -> dict:
    """dQ, dK, dV and the log-gate gradient of the attention given the
    forward's inputs, its output o, LSE and selection, and d_o: per selection
    slot (dlog_gate, sparse scope) and/or per block (dlog_gate_full; the only
    form for the full scope)."""
    b, n, H, dh = q.shape
    Hkv, K = cfg.n_kv_heads, max(cfg.top_k, 0)
    NB = -(-n // cfg.block_size)
    full = cfg.mode == MODES["gated"] and cfg.scope == SCOPES["full"]
    out = {"dq": torch.empty_like(q), "dk": torch.empty_like(k), "dv": torch.empty_like(v)}
    if dlog_gate and not full:
        out["dlog_gate"] = torch.empty(b, Hkv, n, K, dtype=torch.float32, device=q.device)
    if dlog_gate_full or full:
        out["dlog_gate_full"] = torch.empty(b, Hkv, n, NB, dtype=torch.float32, device=q.device)
    bi = BwdIn(*[_ptr(t) for t in (q, k, v, o, d_o, lse, sel_idx, log_gate, doc)])
    bo = BwdOut(*[_ptr(out.get(f)) for f in ("dq", "dk", "dv", "dlog_gate", "dlog_gate_full")])
    wsp, wsn = _ws(ws, workspace_size(cfg, OP_ATTENTION_BACKWARD, b, n))
    _check(lib().sas_attention_backward(C.byref(cfg), b, n, C.byref(bi), C.byref(bo), wsp, wsn, _stream()))
    return out


def selector_backward(cfg: Config, q, k, sel_idx, log_gate, dlog_gate, w_gq=None, w_gk=None, *, ds: bool = True,
                      dqhat: bool = True, dkbar: bool = True, dlog_gate_full=None, doc=None,
                      ws: Workspace | None = None) -> dict:
    """Selector gradients from the selected blocks' log-gate gradient: ds
    [b,Hkv,n,NB], dqhat [b,Hkv,n,dh], dkbar [b,Hkv,NB,dh] and, for given
    projections, dw_gq / dw_gk [Hkv,dh,dh] (all fp32)."""
    b, n, H, dh = q.shape
    Hkv = cfg.n_kv_heads
    NB = -(-n // cfg.block_size)
    dev = q.device
    out = {}
    if ds:
        out["ds"] = torch.empty(b, Hkv, n, NB, dtype=torch.float32, device=dev)
    if dqhat:
        out["dqhat"] = torch.empty(b, Hkv, n, dh, dtype=torch.float32, device=dev)
    if dkbar:
        out["dkbar"] = torch.empty(b, Hkv, NB, dh, dtype=torch.float32, device=dev)
    if w_gq is not None:
        out["dw_gq"] = torch.empty(Hkv, dh, dh, dtype=torch.float32, device=dev)
    if w_gk is not None:
        out["dw_gk"] = torch.empty(Hkv, dh, dh, dtype=torch.float32, device=dev)
    si = SelBwdIn(*[_ptr(t) for t in (q, k, w_gq, w_gk, sel_idx, log_gate, dlog_gate, dlog_gate_full, doc)])
    so = SelBwdOut(*[_ptr(out.get(f)) for f in ("ds", "dqhat", "dkbar", "dw_gq", "dw_gk")])
    wsp, wsn = _ws(ws, workspace_size(cfg, OP_SELECTOR_BACKWARD, b, n))
    _check(lib().sas_selector_backward(C.byref(cfg), b, n, C.byref(si), C.byref(so), wsp, wsn, _stream()))
    return out


def union_words(cfg: Config, n: int) -> int:
    """uint32 words per (query, group) row of a block bitmask."""
    return -(-(-(-n // cfg.block_size)) // 32)


def alloc_union(cfg: Config, b: int, n: int, device="cuda"):
    """Zeroed block bitmask [b, Hkv, n, W] (int32 storage of uint32 words)."""
    return torch.zeros(b, cfg.n_kv_heads, n, union_words(cfg, n), dtype=torch.int32, device=device)


def selection_stats(cfg: Config, q, k, v=None, sel_idx=None, *, cov: bool = True, cov_v: bool = True,
                    sel_union=None, ref_union=None, doc=None, ws: Workspace | None = None) -> dict:
    """Mass coverage (cov, cov_v [b,H,n]) of the attended sets and OR-accumulation
    of the selected / full-attention reference block sets into the given
    bitmasks (see alloc_union)."""
    b, n, H, dh = q.shape
    out = {}
    if cov:
        out["cov"] = torch.empty(b, H, n, dtype=torch.float32, device=q.device)
    if cov_v:
        out["cov_v"] = torch.empty(b, H, n, dtype=torch.float32, device=q.device)
    si = StatsIn(*[_ptr(t) for t in (q, k, v, sel_idx, doc)])
    so = StatsOut(_ptr(out.get("cov")), _ptr(out.get("cov_v")), _ptr(sel_union), _ptr(ref_union))
    wsp, wsn = _ws(ws, workspace_size(cfg, OP_SELECTION_STATS, b, n))
    _check(lib().sas_selection_stats(C.byref(cfg), b, n, C.byref(si), C.byref(so), wsp, wsn, _stream()))
    return out


def overlap_recall(sel_union, ref_union):
    """Eq. overlap_recall of two accumulated bitmasks: (|I n I*|, |I*|, recall)."""
    counts = torch.empty(2, dtype=torch.int64, device=sel_union.device)
    _check(lib().sas_overlap_recall(C.c_int64(sel_union.numel()), _ptr(sel_union), _ptr(ref_union), _ptr(counts),
                                    _stream()))
    inter, tot = (int(x) for x in counts.cpu())
    return inter, tot, (inter / tot if tot else float("nan"))


def mlp_forward(cfg: Config, x, W: dict, ws: Workspace | None = None):
    """y = x + SwiGLU(RMSNorm(x)); x [..., d]."""
    T = x.numel() // x.shape[-1]
    y = torch.empty_like(x)
    wsp, wsn = _ws(ws, workspace_size(cfg, OP_MLP, T, 0))
    _check(lib().sas_mlp_forward(C.byref(cfg), T, _ptr(x), C.byref(weights_struct(W)), _ptr(y), wsp, wsn,
                                 _stream()))
    return y


@dataclass
class PagedCache:
    """Paged KV cache of one layer (device tensors)."""
    k_pages: torch.Tensor
    v_pages: torch.Tensor
    block_table: torch.Tensor
    k_summary: torch.Tensor
    page_size: int

    def struct(self) -> PagedKV:
        return PagedKV(_ptr(self.k_pages), _ptr(self.v_pages), _ptr(self.block_table), _ptr(self.k_summary),
                       self.k_pages.shape[0], self.page_size, self.block_table.shape[1],
                       self.k_summary.shape[2])

    def max_context(self, cfg: Config) -> int:
        """Tokens the summary cache covers (what the workspace is sized for)."""
        return self.k_summary.shape[2] * cfg.block_size


def layer_forward(cfg: Config, x, W: dict, *, stats: bool = True, lse=True, sel_idx=True, log_gate=False,
                  tau=False, k_summary=False, taps: bool = False, cache: PagedCache | None = None,
                  ws: Workspace | None = None) -> dict:
    """One decoder layer over x [b, n, d]."""
    b, n, d = x.shape
    H, Hkv, dh, B, K = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.block_size, cfg.top_k
    NB = -(-n // B)
    dev = x.device
    out = {"y": torch.empty_like(x)}
    st = None
    if stats:
        out["o"] = torch.empty(b, n, H, dh, dtype=x.dtype, device=dev)
        if lse:
            out["lse"] = torch.empty(b, H, n, dtype=torch.float32, device=dev)
        if sel_idx:
            out["sel_idx"] = torch.empty(b, Hkv, n, K, dtype=torch.int32, device=dev)
        if log_gate:
            out["log_gate"] = torch.empty(b, Hkv, n, NB, dtype=torch.float32, device=dev)
        if tau:
            out["tau"] = torch.empty(b, Hkv, n, dtype=torch.float32, device=dev)
        if k_summary:
            out["k_summary"] = torch.empty(b, Hkv, NB, dh, dtype=x.dtype, device=dev)
        st = AttnOut(*[_ptr(out.get(f)) for f in ("o", "lse", "k_summary", "sel_idx", "log_gate", "tau")])
    tp = None
    if taps:
        out["q"] = torch.empty(b, n, H, dh, dtype=x.dtype, device=dev)
        out["k"] = torch.empty(b, n, Hkv, dh, dtype=x.dtype, device=dev)
        out["v"] = torch.empty(b, n, Hkv, dh, dtype=x.dtype, device=dev)
        out["h1"] = torch.empty_like(x)
        tp = LayerTaps(*[_ptr(out[f]) for f in ("q", "k", "v", "h1")])
    cs = cache.struct() if cache is not None else None
    wsp, wsn = _ws(ws, workspace_size(cfg, OP_LAYER, b, n))
    _check(lib().sas_layer_forward(C.byref(cfg), b, n, _ptr(x), C.byref(weights_struct(W)), _ptr(out["y"]),
                                   C.byref(st) if st is not None else None,
                                   C.byref(tp) if tp is not None else None,
                                   C.byref(cs) if cs is not None else None, wsp, wsn, _stream()))
    return out


def profiler_start(capacity: int = 4096):
    _check(lib().sas_profiler_start(capacity))


def profiler_select(families):
    """Record only these kernel families (an iterable of names; None = all)."""
    arg = None if families is None else ",".join(families).encode()
    _check(lib().sas_profiler_select(arg))


def profiler_stop() -> list:
    """Stop recording; synchronise; return [(kernel family, ms), ...]."""
    n = lib().sas_profiler_stop()
    torch.cuda.synchronize()
    out = []
    name, ms = C.c_char_p(), C.c_float()
    for i in range(n):
        _check(lib().sas_profiler_record(i, C.byref(name), C.byref(ms)))
        out.append((name.value.decode(), float(ms.value)))
    return out


def alloc_cache(cfg: Config, batch: int, max_len: int, page_size: int = 16, device="cuda",
                shuffle_pages: bool = True, seed: int = 0) -> PagedCache:
    """Zeroed paged KV cache for `batch` sequences of up to `max_len` tokens.
    Pages are handed out in a seeded random order so that logical and
    physical order differ."""
    dt = torch.bfloat16 if cfg.dtype == SAS_BF16 else torch.float32
    per_seq = -(-max_len // page_size)
    num_pages = batch * per_seq
    Hkv, dh = cfg.n_kv_heads, cfg.head_dim
    k_pages = torch.zeros(num_pages, Hkv, page_size, dh, dtype=dt, device=device)
    v_pages = torch.zeros_like(k_pages)
    order = torch.randperm(num_pages, generator=torch.Generator().manual_seed(seed)) if shuffle_pages \
        else torch.arange(num_pages)
    block_table = order.to(torch.int32).reshape(batch, per_seq).to(device)
    nblk = -(-max_len // cfg.block_size)
    k_summary = torch.zeros(batch, Hkv, nblk, dh, dtype=dt, device=device)
    return PagedCache(k_pages, v_pages, block_table, k_summary, page_size)


def pack_decode_weights(cfg: Config, W: dict):
    """The layer's linear weights in the packed decode layout (a new uint8
    tensor on W's device); returns W with "decode_packed" set to it, so that
    decode steps stream the packed copy."""
    n = lib().sas_decode_packed_bytes(C.byref(cfg))
    if n == 0:
        raise SasError("no packed decode layout for this configuration")
    out = torch.empty(n + 256, dtype=torch.uint8, device=W["wq"].device)
    off = (-out.data_ptr()) % 256  # 256-byte aligned view
    buf = out[off:off + n]
    ws = weights_struct(W)
    _check(lib().sas_pack_decode_weights(C.byref(cfg), C.byref(ws), _ptr(buf), n, _stream()))
    W2 = dict(W)
    W2["decode_packed"] = buf
    return W2


def decode_step(cfg: Config, x, pos, W: dict, cache: PagedCache, *, sel_idx: bool = True,
                taps: bool = False, ws: Workspace | None = None):
    """One SAS decode step of one layer.  x [b, d]; pos [b] int32 (device).
    Returns (y, sel) or, with taps, (y, sel, {"q", "k", "v", "h1"})."""
    b = x.shape[0]
    H, Hkv, dh = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    y = torch.empty_like(x)
    sel = torch.empty(b, Hkv, cfg.top_k, dtype=torch.int32, device=x.device) if sel_idx else None
    tap = None
    tp = None
    if taps:
        tap = {"q": torch.empty(b, H, dh, dtype=x.dtype, device=x.device),
               "k": torch.empty(b, Hkv, dh, dtype=x.dtype, device=x.device),
               "v": torch.empty(b, Hkv, dh, dtype=x.dtype, device=x.device),
               "h1": torch.empty_like(x)}
        tp = LayerTaps(*[_ptr(tap[f]) for f in ("q", "k", "v", "h1")])
    cs = cache.struct()
    wsp, wsn = _ws(ws, workspace_size(cfg, OP_DECODE, b, cache.max_context(cfg)))
    _check(lib().sas_decode_step(C.byref(cfg), b, _ptr(x), _ptr(pos), C.byref(weights_struct(W)), C.byref(cs),
                                 _ptr(y), _ptr(sel), C.byref(tp) if tp is not None else None, wsp, wsn,
                                 _stream()))
    return (y, sel, tap) if taps else (y, sel)


def decode_step_noalloc(cfg: Config, x, pos, W: dict, cache: PagedCache, *, sel_idx: bool = True):
    """sas_decode_step_noalloc: the decode step with the library's static
    scratch (no workspace, nothing allocated by the library)."""
    b = x.shape[0]
    y = torch.empty_like(x)
    sel = torch.empty(b, cfg.n_kv_heads, cfg.top_k, dtype=torch.int32, device=x.device) if sel_idx else None
    cs = cache.struct()
    _check(lib().sas_decode_step_noalloc(C.byref(cfg), b, _ptr(x), _ptr(pos), C.byref(weights_struct(W)),
                                         C.byref(cs), _ptr(y), _ptr(sel), _stream()))
    return y, sel


def decode_select(cfg: Config, q, pos, cache: PagedCache, w_gq=None, ws: Workspace | None = None):
    """Top-K blocks per KV group for the new tokens' query heads q [b, H, dh]
    at positions pos [b] (device int32) against the cache's summaries."""
    b = q.shape[0]
    sel = torch.empty(b, cfg.n_kv_heads, cfg.top_k, dtype=torch.int32, device=q.device)
    cs = cache.struct()
    wsp, wsn = _ws(ws, workspace_size(cfg, OP_DECODE_SELECT, b, cache.max_context(cfg)))
    _check(lib().sas_decode_select(C.byref(cfg), b, _ptr(q), _ptr(pos), _ptr(w_gq), C.byref(cs), _ptr(sel), wsp,
                                   wsn, _stream()))
    return sel


def embed(cfg: Config, ids, table, img=None):
    """x [b, n, d] from token ids [b, n] (int32, -1 = next image row)."""
    b, n = ids.shape
    n_img = 0 if img is None else img.shape[1]
    x = torch.empty(b, n, table.shape[1], dtype=table.dtype, device=table.device)
    _check(lib().sas_embed(C.byref(cfg), b, n, _ptr(ids), _ptr(table), table.shape[0], _ptr(img), n_img, _ptr(x),
                           _stream()))
    return x


def lm_head_argmax(cfg: Config, h, gamma, w_lm, *, logits: bool = False, ws: Workspace | None = None):
    """Greedy next tokens [b] (int32) and optionally the fp32 logits."""
    b = h.shape[0]
    V = w_lm.shape[0]
    tok = torch.empty(b, dtype=torch.int32, device=h.device)
    lg = torch.empty(b, V, dtype=torch.float32, device=h.device) if logits else None
    wsp, wsn = _ws(ws, workspace_size(cfg, OP_LM_HEAD, b, V))
    _check(lib().sas_lm_head_argmax(C.byref(cfg), b, _ptr(h), _ptr(gamma), _ptr(w_lm), V, _ptr(lg), _ptr(tok),
                                    wsp, wsn, _stream()))
    return tok, lg


def to_device(arr, dtype: str, device="cuda"):
    """float32 NumPy array (values exact in `dtype`) -> device tensor."""
    t = torch.from_numpy(arr)
    return t.to(TORCH_DTYPE[dtype]).to(device)


def weights_to_device(W: dict, dtype: str, device="cuda") -> dict:
    return {k: (None if v is None else to_device(v, dtype, device)) for k, v in W.items()}
