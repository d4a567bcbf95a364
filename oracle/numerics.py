"""Elementwise pieces of the decoder layer around SAS, in float64.

The paper works with text LLM backbones (Qwen3, OLMo3) and does not restate
their layer; the layer here is the usual pre-norm decoder block: RMSNorm,
rotary position embedding (rotate-half pairing, base 10000), SwiGLU MLP.
TEST INFRASTRUCTURE ONLY (see the package docstring).
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127

# elementwise work on large arrays is split into chunks run on threads (NumPy
# releases the GIL inside its loops); every element is computed the same way
_POOL = ThreadPoolExecutor(max_workers=min(16, len(os.sched_getaffinity(0))))
_CHUNK = 1 << 19


def elementwise(f, x):
    """f applied to the float64 array x, in chunks of its flattened elements
    (f must act on each element independently)."""
    x = np.asarray(x, dtype=np.float64)
    if x.size <= _CHUNK:
        return f(x)
    flat = x.reshape(-1)
    out = np.empty_like(flat)

    def run(i):
        out[i:i + _CHUNK] = f(flat[i:i + _CHUNK])
    list(_POOL.map(run, range(0, flat.size, _CHUNK)))
    return out.reshape(x.shape)


def _round_bf16(x):
    out = np.array(x, dtype=np.float64, copy=True)
    fin = np.isfinite(x) & (x != 0.0)
    if np.any(fin):
        xf = x[fin]
        _, e = np.frexp(xf)                 # |x| in [2^(e-1), 2^e)
        q = np.maximum(e - 8, -133)         # exponent of one unit in the last place
        r = np.ldexp(np.rint(np.ldexp(xf, -q)), q)   # rint: ties to even
        r = np.where(np.abs(r) > BF16_MAX, np.copysign(np.inf, r), r)
        out[fin] = r
    return out


def round_bf16(x):
    """Round float64 values to the nearest bfloat16 value, ties to even,
    directly from float64 (8 significant bits; subnormal spacing 2^-133;
    overflow to +-inf).  Returns float64 holding the bfloat16 values."""
    return elementwise(_round_bf16, x)


def round_f32(x):
    """Round float64 values to float32 (IEEE round to nearest even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def rho(x, dtype):
    """Materialise a tensor in the activation dtype ("bf16" or "f32")."""
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return round_f32(x)
    raise ValueError(dtype)


def rmsnorm(x, gamma, eps):
    """u = x / sqrt(mean(x^2) + eps) * gamma over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gamma, dtype=np.float64)


def rope(x, pos, base):
    """Rotary embedding, rotate-half pairing (i, i + dh/2), angle pos*theta_i
    with theta_i = base^(-2i/dh).  x[..., n, heads, dh]; pos[n]."""
    x = np.asarray(x, dtype=np.float64)
    dh = x.shape[-1]
    half = dh // 2
    i = np.arange(half, dtype=np.float64)
    theta = np.power(float(base), -2.0 * i / dh)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * theta[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def _silu(x):
    with np.errstate(over="ignore"):
        return x / (1.0 + np.exp(-x))


def silu(x):
    """silu(x) = x / (1 + exp(-x))."""
    return elementwise(_silu, x)
