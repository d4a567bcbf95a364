"""Seeded synthetic inputs, shared by the HIP path, the tests and the oracle.

This module only draws random numbers and stores them in the activation
dtype; it holds none of the method's arithmetic.  Every tensor comes from its
own stream ``PCG64(SeedSequence(seed, spawn_key=(workload, tensor, layer)))``:
float32 standard normals, times ``std`` in float32, then rounded once
(round-to-nearest-even) to bfloat16 when the dtype is bf16.  Arrays are
returned as float32 NumPy arrays whose values are exactly representable in
the activation dtype, so both sides read identical bits.
"""
from __future__ import annotations

import zlib

import numpy as np

from .configs import Workload


def _key(name: str) -> int:
    return zlib.crc32(name.encode()) & 0x7FFFFFFF


def stream(w: Workload | int, name: str, layer: int = 0, seed: int = 0) -> np.random.Generator:
    idx = w if isinstance(w, int) else w.index
    ss = np.random.SeedSequence(entropy=seed, spawn_key=(idx, _key(name), layer))
    return np.random.Generator(np.random.PCG64(ss))


def bf16_bits(x32: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    b = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    r = (b + (((b >> 16) & 1) + 0x7FFF)) >> 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def as_dtype(x32: np.ndarray, dtype: str) -> np.ndarray:
    """Store float32 values in the activation dtype (values stay float32)."""
    if dtype == "f32":
        return np.ascontiguousarray(x32, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_to_f32(bf16_bits(x32))
    raise ValueError(dtype)


def normal(w: Workload, name: str, shape, std: float = 1.0, layer: int = 0,
           seed: int = 0, dtype: str | None = None) -> np.ndarray:
    g = stream(w, name, layer, seed)
    z = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        z *= np.float32(std)
    return as_dtype(z, dtype or w.dtype)


def token_kinds(w: Workload) -> np.ndarray:
    """Per-position kind of one sequence: 1 = image/video token, 0 = text."""
    kinds = []
    for kind, cnt in w.segments:
        kinds += [1 if kind == "img" else 0] * cnt
    k = np.array(kinds, dtype=np.int8)
    if len(k) != w.seq_len:
        raise ValueError(f"segments cover {len(k)} tokens, seq_len is {w.seq_len}")
    return k


def embeddings(w: Workload, seed: int = 0) -> np.ndarray:
    """Layer input x[b, n, d]: text tokens N(0,1), image tokens N(0,1)*img_scale."""
    z = stream(w, "x", 0, seed).standard_normal(
        size=(w.batch, w.seq_len, w.d_model), dtype=np.float32)
    scale = np.where(token_kinds(w) == 1, np.float32(w.img_scale), np.float32(1.0))
    z *= scale[None, :, None].astype(np.float32)
    return as_dtype(z, w.dtype)


def layer_weights(w: Workload, layer: int = 0, seed: int = 0, selector_proj: bool = False) -> dict:
    """nn.Linear-layout ([out, in]) weights of one decoder layer, N(0, std).
    RMSNorm gains are 1.  ``w_gq``/``w_gk`` ([Hkv, dh, dh]) are drawn only when
    ``selector_proj`` is set (otherwise the selector uses the identity)."""
    d, H, Hkv, dh, f = w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.d_ff
    s = w.weight_std
    out = {
        "rms1": as_dtype(np.ones(d, np.float32), w.dtype),
        "wq": normal(w, "wq", (H * dh, d), s, layer, seed),
        "wk": normal(w, "wk", (Hkv * dh, d), s, layer, seed),
        "wv": normal(w, "wv", (Hkv * dh, d), s, layer, seed),
        "wo": normal(w, "wo", (d, H * dh), s, layer, seed),
        "rms2": as_dtype(np.ones(d, np.float32), w.dtype),
        "w_gate": normal(w, "w_gate", (f, d), s, layer, seed),
        "w_up": normal(w, "w_up", (f, d), s, layer, seed),
        "w_down": normal(w, "w_down", (d, f), s, layer, seed),
        "w_gq": None,
        "w_gk": None,
    }
    if selector_proj:
        # a projection near the identity keeps the selector's ranking close to
        # the plain pooled-key dot product while still exercising the matmul
        eye = np.eye(dh, dtype=np.float32)[None]
        out["w_gq"] = as_dtype(eye + normal(w, "w_gq", (Hkv, dh, dh), 0.05, layer, seed,
                                            dtype="f32"), w.dtype)
        out["w_gk"] = as_dtype(eye + normal(w, "w_gk", (Hkv, dh, dh), 0.05, layer, seed,
                                            dtype="f32"), w.dtype)
    return out


def qkv(w: Workload, seed: int = 0, scale: float = 1.0):
    """Attention inputs for the attention-only entry point: Q[b,n,H,dh],
    K,V[b,n,Hkv,dh], N(0, scale) (post-RoPE values as they would sit in HBM)."""
    b, n, H, Hkv, dh = w.batch, w.seq_len, w.n_heads, w.n_kv_heads, w.head_dim
    q = normal(w, "q", (b, n, H, dh), scale, 0, seed)
    k = normal(w, "k", (b, n, Hkv, dh), scale, 0, seed)
    v = normal(w, "v", (b, n, Hkv, dh), 1.0, 0, seed)
    return q, k, v


def model_ends(w: Workload, seed: int = 0) -> dict:
    """Embedding table and LM head ([vocab, d], N(0,1) and N(0, std)), final
    RMSNorm gain, prompt token ids and image embeddings of every sequence."""
    d, V = w.d_model, w.vocab
    kinds = token_kinds(w)
    n_img = int(kinds.sum())
    ids = stream(w, "tokens", 0, seed).integers(0, V, size=(w.batch, w.seq_len), dtype=np.int64)
    ids = np.where(kinds[None, :] == 1, -1, ids).astype(np.int32)  # -1: image slot
    img = normal(w, "img_embed", (w.batch, n_img, d), w.img_scale, 0, seed)
    return {
        "embed": normal(w, "embed", (V, d), 1.0, 0, seed),
        "w_lm": normal(w, "w_lm", (V, d), w.weight_std, 0, seed),
        "rms_final": as_dtype(np.ones(d, np.float32), w.dtype),
        "token_ids": ids,
        "img_embed": img,
    }


def layer_weights_device(w: Workload, layer: int = 0, seed: int = 0, device="cuda"):
    """Layer weights drawn on the GPU, for stacks too large to draw on the host
    (32 layers of the 7B shape are 6.5 G values): N(0, weight_std) from
    torch's Philox generator seeded per (workload, tensor, layer), rounded to
    the activation dtype; RMSNorm gains 1.  Same shapes and distribution as
    layer_weights(); the values differ (the oracle receives these ones by copying
    them to the host)."""
    import torch

    d, H, Hkv, dh, F = w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.d_ff
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    shapes = {"wq": (H * dh, d), "wk": (Hkv * dh, d), "wv": (Hkv * dh, d), "wo": (d, H * dh),
              "w_gate": (F, d), "w_up": (F, d), "w_down": (d, F)}
    out = {"rms1": torch.ones(d, dtype=dt, device=device), "rms2": torch.ones(d, dtype=dt, device=device),
           "w_gq": None, "w_gk": None}
    for name, shape in shapes.items():
        g = torch.Generator(device=device)
        g.manual_seed(int(np.random.SeedSequence(entropy=seed, spawn_key=(w.index, _key(name), layer))
                          .generate_state(1, np.uint64)[0] & 0x7FFFFFFFFFFFFFFF))
        out[name] = (torch.randn(shape, generator=g, device=device, dtype=torch.float32) * w.weight_std).to(dt)
    return out


def model_ends_device(w: Workload, seed: int = 0, device="cuda") -> dict:
    """model_ends() for large vocabularies: the embedding table and LM head
    ([vocab, d]) drawn on the GPU as in layer_weights_device(); prompt token
    ids and image embeddings drawn on the host exactly as model_ends()."""
    import torch

    d, V = w.d_model, w.vocab
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    kinds = token_kinds(w)
    n_img = int(kinds.sum())
    ids = stream(w, "tokens", 0, seed).integers(0, V, size=(w.batch, w.seq_len), dtype=np.int64)
    ids = np.where(kinds[None, :] == 1, -1, ids).astype(np.int32)
    img = normal(w, "img_embed", (w.batch, n_img, d), w.img_scale, 0, seed)

    def draw(name, shape, std):
        g = torch.Generator(device=device)
        g.manual_seed(int(np.random.SeedSequence(entropy=seed, spawn_key=(w.index, _key(name), 0))
                          .generate_state(1, np.uint64)[0] & 0x7FFFFFFFFFFFFFFF))
        return (torch.randn(shape, generator=g, device=device, dtype=torch.float32) * std).to(dt)

    return {
        "embed": draw("embed", (V, d), 1.0),
        "w_lm": draw("w_lm", (V, d), w.weight_std),
        "rms_final": torch.ones(d, dtype=dt, device=device),
        "token_ids": torch.from_numpy(ids).to(device),
        "img_embed": torch.from_numpy(img).to(device=device, dtype=dt),
    }
