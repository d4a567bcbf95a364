"""Decoder layer, MLP, attention prefill, decode step and model ends around
SAS attention, in float64.

Materialisation points (rounded to the activation dtype, exactly where the
GPU path writes a tensor to HBM; everything else stays float64):
u1 = RMSNorm(x); Q, K (after RoPE), V; the selector's kbar / qhat; O;
h1 = x + O Wo^T; u2 = RMSNorm(h1); a = silu(u2 Wg^T) * (u2 Wu^T);
y = h1 + a Wd^T.  Linear layers use the nn.Linear convention y = x W^T
without biases; query head h reads KV head h // G.

Inference (Alg. 2, Sec. 5.1): prefill is dense and fills the KV cache; every
decode step scores the cached block summaries, selects Top-K per KV group and
attends to the selected blocks plus the current block, without gate bias.

TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
from dataclasses import dataclass

import numpy as np

from .attention import causal_attention, sas_attention
from .numerics import rho, rmsnorm, rope, silu
from .selector import (block_summaries, gate_query, project_summaries,
                       select, selector_scores, topk_blocks)


@dataclass(frozen=True)
class Spec:
    n_heads: int
    n_kv_heads: int
    head_dim: int
    block_size: int
    top_k: int
    mode: str               # "dense" | "sparse" | "gated"
    dtype: str              # "bf16" | "f32"
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    sm_scale: float = 0.0   # <= 0: 1/sqrt(head_dim)

    @property
    def group(self):
        return self.n_heads // self.n_kv_heads


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def attention_prefill(Q, K, V, spec, rows=None, w_gq=None, w_gk=None):
    """Selector + SAS attention for a batch.  K/V[b, n, Hkv, dh]; Q[b, R, H,
    dh] holds the rows listed in ``rows`` (all n when None).  Returns O[b, R,
    H, dh] (rounded), LSE[b, H, R], sel[b, Hkv, R, K], log_gate[b, Hkv, R, NB],
    tau[b, Hkv, R], k_summary[b, Hkv, n//B, dh] (the selector's key summaries,
    after the optional projection)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    b, n = K.shape[0], K.shape[1]
    rows = np.arange(n) if rows is None else np.asarray(rows)
    outs = {k: [] for k in ("O", "O_exact", "LSE", "sel", "log_gate", "tau", "k_summary", "r")}
    for bi in range(b):
        st = select(Q[bi], K[bi], spec.block_size, spec.top_k, spec.dtype, rows=rows,
                    w_gq=_f64(w_gq), w_gk=_f64(w_gk))
        O, Oe, L = sas_attention(Q[bi], K[bi], V[bi], spec.block_size, spec.mode, spec.dtype,
                                 sel=st["sel"], log_gate=st["log_gate"],
                                 sm_scale=spec.sm_scale, rows=rows)
        outs["O"].append(O)
        outs["O_exact"].append(Oe)
        outs["LSE"].append(L)
        outs["sel"].append(st["sel"])
        outs["log_gate"].append(st["log_gate"])
        outs["tau"].append(st["tau"])
        outs["k_summary"].append(st["kbar_proj"])
        outs["r"].append(st["r"])
    return {k: np.stack(v) for k, v in outs.items()}


def qkv_projection(x, W, spec, rows):
    """u1 = rho(RMSNorm(x)); Q at ``rows`` and K, V at every position.
    x[b, n, d] -> Q[b, R, H, dh], K/V[b, n, Hkv, dh] (rounded)."""
    x = _f64(x)
    b, n, d = x.shape
    H, Hkv, dh = spec.n_heads, spec.n_kv_heads, spec.head_dim
    u1 = rho(rmsnorm(x, _f64(W["rms1"]), spec.rms_eps), spec.dtype)
    pos = np.arange(n)
    K = rho(rope((u1 @ _f64(W["wk"]).T).reshape(b, n, Hkv, dh), pos, spec.rope_base), spec.dtype)
    V = rho((u1 @ _f64(W["wv"]).T).reshape(b, n, Hkv, dh), spec.dtype)
    ur = u1[:, rows]
    Q = rho(rope((ur @ _f64(W["wq"]).T).reshape(b, len(rows), H, dh), rows, spec.rope_base),
            spec.dtype)
    return Q, K, V


def mlp_forward(h1, W, spec):
    """y = rho(h1 + a Wd^T) with a = rho(silu(u2 Wg^T) * (u2 Wu^T)) and
    u2 = rho(RMSNorm(h1)).  h1[..., d] (already in the activation dtype)."""
    h1 = _f64(h1)
    u2 = rho(rmsnorm(h1, _f64(W["rms2"]), spec.rms_eps), spec.dtype)
    a = rho(silu(u2 @ _f64(W["w_gate"]).T) * (u2 @ _f64(W["w_up"]).T), spec.dtype)
    return rho(h1 + a @ _f64(W["w_down"]).T, spec.dtype)


def layer_forward(x, W, spec, rows=None):
    """One decoder layer over x[b, n, d]; outputs at ``rows`` (all when None):
    y[b, R, d] and the attention statistics of ``attention_prefill``."""
    x = _f64(x)
    b, n, d = x.shape
    rows = np.arange(n) if rows is None else np.asarray(rows)
    Q, K, V = qkv_projection(x, W, spec, rows)
    att = attention_prefill(Q, K, V, spec, rows=rows, w_gq=W.get("w_gq"), w_gk=W.get("w_gk"))
    R = len(rows)
    O = att["O"].reshape(b, R, spec.n_heads * spec.head_dim)
    h1 = rho(x[:, rows] + O @ _f64(W["wo"]).T, spec.dtype)
    y = mlp_forward(h1, W, spec)
    out = dict(att)
    out.update({"y": y, "h1": h1, "Q": Q, "K": K, "V": V})
    return out


def dense_prefill_layer(x, W, spec):
    """One decoder layer of the serving prefill (Sec. 5.1: the prompt is
    attended densely) over one sequence x[n, d], every row: u1, Q/K/V with
    RoPE, causal attention, h1, MLP.  Returns y[n, d] and what the KV cache
    holds for the decode steps that follow: K, V [n, Hkv, dh] and the block
    summaries k_summary [Hkv, n // B, dh] (after W_gk when given)."""
    x = _f64(x)
    n, d = x.shape
    Q, K, V = qkv_projection(x[None], W, spec, np.arange(n))
    O, O_exact, _ = causal_attention(Q[0], K[0], V[0], spec.dtype, spec.sm_scale)
    h1 = rho(x + O.reshape(n, spec.n_heads * spec.head_dim) @ _f64(W["wo"]).T, spec.dtype)
    y = mlp_forward(h1, W, spec)
    kbar = project_summaries(block_summaries(K[0], spec.block_size, spec.dtype), _f64(W.get("w_gk")), spec.dtype)
    return {"y": y, "h1": h1, "O": O, "O_exact": O_exact, "K": K[0], "V": V[0], "k_summary": kbar}


class DecodeCache:
    """Logical KV cache of one layer for a batch of sequences: K/V at every
    position written so far and the selector's summary of every complete
    block (after the optional W_gk projection)."""

    def __init__(self, b, max_len, spec):
        self.spec = spec
        Hkv, dh, B = spec.n_kv_heads, spec.head_dim, spec.block_size
        self.K = np.zeros((b, max_len, Hkv, dh))
        self.V = np.zeros((b, max_len, Hkv, dh))
        self.kbar = np.zeros((b, Hkv, -(-max_len // B), dh))
        self.length = np.zeros(b, dtype=np.int64)

    def fill_prefill(self, bi, K, V, k_summary):
        n = K.shape[0]
        self.K[bi, :n] = K
        self.V[bi, :n] = V
        self.kbar[bi, :, :k_summary.shape[1]] = k_summary
        self.length[bi] = n


def decode_step(x, pos, W, cache, spec, taps=False):
    """One SAS inference step (Alg. 2) of one layer for a batch.
    x[b, d] (activation dtype), pos[b] = position of each new token.
    Appends K/V at pos, completes the block summary when pos + 1 is a
    multiple of B, selects the Top-K historical blocks per KV group against
    the cached summaries and attends to them plus the current block without
    gate bias.  Returns y[b, d] and sel[b, Hkv, K] (and, with taps, the
    post-RoPE query heads q[b, H, dh])."""
    x = _f64(x)
    b, d = x.shape
    H, Hkv, dh, B, Kb = spec.n_heads, spec.n_kv_heads, spec.head_dim, spec.block_size, spec.top_k
    G = spec.group
    y = np.zeros((b, d))
    q_all = np.zeros((b, H, dh))
    sel_all = np.full((b, Hkv, max(Kb, 0)), -1, dtype=np.int64)
    for bi in range(b):
        t = int(pos[bi])
        p = np.array([t])
        u1 = rho(rmsnorm(x[bi:bi + 1], _f64(W["rms1"]), spec.rms_eps), spec.dtype)
        q = rho(rope((u1 @ _f64(W["wq"]).T).reshape(1, H, dh), p, spec.rope_base), spec.dtype)
        k = rho(rope((u1 @ _f64(W["wk"]).T).reshape(1, Hkv, dh), p, spec.rope_base), spec.dtype)
        v = rho((u1 @ _f64(W["wv"]).T).reshape(1, Hkv, dh), spec.dtype)
        q_all[bi] = q[0]
        cache.K[bi, t] = k[0]
        cache.V[bi, t] = v[0]
        cache.length[bi] = t + 1
        if (t + 1) % B == 0:
            m = t // B
            kb = block_summaries(cache.K[bi, m * B:(m + 1) * B], B, spec.dtype)   # [Hkv,1,dh]
            cache.kbar[bi, :, m] = project_summaries(kb, _f64(W.get("w_gk")), spec.dtype)[:, 0]
        ct = t // B
        qhat = gate_query(q, G, spec.dtype, _f64(W.get("w_gq")))                  # [Hkv,1,dh]
        r = selector_scores(qhat, cache.kbar[bi][:, :ct])                         # [Hkv,1,ct]
        sel = np.full((Hkv, 1, max(Kb, 0)), -1, dtype=np.int64)
        for g in range(Hkv):
            chosen, _ = topk_blocks(r[g, 0], ct, Kb)
            sel[g, 0, :len(chosen)] = chosen
        sel_all[bi] = sel[:, 0]
        O, _, _ = sas_attention(q, cache.K[bi, :t + 1], cache.V[bi, :t + 1], B, "sparse",
                                spec.dtype, sel=sel, rows=np.array([t]),
                                sm_scale=spec.sm_scale)
        h1 = rho(x[bi] + O.reshape(H * dh) @ _f64(W["wo"]).T, spec.dtype)
        y[bi] = mlp_forward(h1[None], W, spec)[0]
    return (y, sel_all, q_all) if taps else (y, sel_all)


def decode_select(q, pos, kbar, spec, w_gq=None):
    """The selection of a decode step (Alg. 2) alone: q[b, H, dh] query heads
    of the new tokens at positions pos[b]; kbar[b, Hkv, M, dh] the cached
    block summaries.  Each group's gate query scores the floor(pos/B)
    complete blocks and keeps the Top-K under (r desc, m asc).  Returns
    sel[b, Hkv, K] ascending, -1 padded, and r[b][Hkv, C]."""
    q = _f64(q)
    b = q.shape[0]
    Hkv, Kb, B = spec.n_kv_heads, spec.top_k, spec.block_size
    sel = np.full((b, Hkv, max(Kb, 0)), -1, dtype=np.int64)
    rs = []
    for bi in range(b):
        ct = min(int(pos[bi]) // B, kbar.shape[2]) if pos[bi] >= 0 else 0
        qhat = gate_query(q[bi:bi + 1], spec.group, spec.dtype, _f64(w_gq))     # [Hkv,1,dh]
        r = selector_scores(qhat, _f64(kbar[bi])[:, :ct])                        # [Hkv,1,ct]
        for g in range(Hkv):
            chosen, _ = topk_blocks(r[g, 0], ct, Kb)
            sel[bi, g, :len(chosen)] = chosen
        rs.append(r[:, 0])
    return sel, rs


def embed_tokens(ids, table, img_embed=None):
    """x[b, n, d]: row table[id] for id >= 0; image slots (id < 0) take the
    next row of img_embed[b, n_img, d] in order."""
    ids = np.asarray(ids)
    table = _f64(table)
    out = np.zeros(ids.shape + (table.shape[1],))
    for bi in range(ids.shape[0]):
        j = 0
        for t in range(ids.shape[1]):
            if ids[bi, t] >= 0:
                out[bi, t] = table[ids[bi, t]]
            else:
                out[bi, t] = img_embed[bi, j]
                j += 1
    return out


def lm_head_argmax(h, gamma, w_lm, eps, dtype):
    """Greedy next token: logits = rho(RMSNorm(h)) W_lm^T in fp64, argmax with
    the lowest token id winning ties.  h[b, d] -> (tokens[b], logits[b, V])."""
    u = rho(rmsnorm(_f64(h), _f64(gamma), eps), dtype)
    logits = u @ _f64(w_lm).T
    return np.argmax(logits, axis=1), logits
