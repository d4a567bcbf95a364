"""Pins of the oracle's elementwise pieces against library routines,
hand-derived rounding cases and the invariants of rotary embeddings."""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_round_bf16_matches_torch_on_float32_inputs():
    rng = np.random.default_rng(1)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(5000) * 1e30).astype(np.float32),
        (rng.standard_normal(5000) * 1e-38).astype(np.float32),   # bf16 subnormals
        (rng.standard_normal(5000) * 1e-42).astype(np.float32),   # fp32 subnormals
        np.array([0.0, -0.0, 3.3895314e38, -3.3895314e38], dtype=np.float32),
    ])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = oracle.round_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_round_bf16_golden_cases():
    # hand-derived ties and a case that double rounding through float32 gets wrong
    with open(os.path.join(GOLDEN, "bf16_rounding.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        x = float.fromhex(c["x"])
        want = float.fromhex(c["bf16"]) if c["bf16"] not in ("inf", "-inf") else float(c["bf16"])
        got = oracle.round_bf16(np.array([x]))[0]
        assert got == want, (c, got.hex())


def test_round_f32_is_ieee():
    x = np.array([1.0 + 2.0 ** -24, 1.0 + 3 * 2.0 ** -24, 0.1])
    np.testing.assert_array_equal(oracle.round_f32(x), [1.0, 1.0 + 2.0 ** -22, float(np.float32(0.1))])


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((7, 96)) * 3
    g = rng.standard_normal(96)
    ref = F.rms_norm(torch.from_numpy(x), (96,), weight=torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1e-6), ref, rtol=1e-13, atol=1e-13)


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(oracle.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-14, atol=1e-300)


def test_rope_identity_at_position_zero_and_closed_form():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((1, 3, 8))
    np.testing.assert_allclose(oracle.rope(x, np.array([0]), 10000.0), x, rtol=0, atol=0)
    # dh = 2: a single pair rotated by pos * 1 radian
    y = oracle.rope(np.array([[[1.0, 0.0]]]), np.array([5]), 10000.0)
    np.testing.assert_allclose(y[0, 0], [math.cos(5.0), math.sin(5.0)], rtol=1e-15)
    # theta_i = base^(-2i/dh): pair i = 1 of dh = 4 turns at 1/base^(1/2) rad per position
    y = oracle.rope(np.array([[[0.0, 1.0, 0.0, 0.0]]]), np.array([3]), 100.0)
    np.testing.assert_allclose(y[0, 0], [0.0, math.cos(0.3), 0.0, math.sin(0.3)], atol=1e-15)


def test_rope_preserves_pair_norms_and_is_relative():
    rng = np.random.default_rng(4)
    dh = 64
    q = rng.standard_normal((1, 1, dh))
    k = rng.standard_normal((1, 1, dh))
    rq = oracle.rope(q, np.array([37]), 10000.0)
    pn = q[..., :32] ** 2 + q[..., 32:] ** 2
    np.testing.assert_allclose(rq[..., :32] ** 2 + rq[..., 32:] ** 2, pn, rtol=1e-12)
    # <rope(q, p1), rope(k, p2)> depends only on p1 - p2
    dots = []
    for shift in (0, 5, 1000):
        a = oracle.rope(q, np.array([40 + shift]), 10000.0)
        b = oracle.rope(k, np.array([13 + shift]), 10000.0)
        dots.append(float((a * b).sum()))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-10)
    # and it is not the identity away from position 0
    assert abs(float((rq - q).sum())) > 1e-3


def test_rope_batched_shape_broadcast():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 5, 3, 16))
    pos = np.arange(5)
    y = oracle.rope(x, pos, 10000.0)
    for bi in range(2):
        for t in range(5):
            np.testing.assert_allclose(y[bi, t], oracle.rope(x[bi, t][None], np.array([t]), 10000.0)[0])
