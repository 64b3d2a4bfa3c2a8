"""Pins of oracle.numerics against the bf16 format definition, a library
conversion (torch's fp32 -> bf16), and closed forms."""
import math

import numpy as np
import pytest
import scipy.special
import torch

from oracle.numerics import round_bf16, silu, softmax_rows


def test_round_bf16_matches_torch_on_fp32_inputs():
    rng = np.random.default_rng(1)
    mags = 10.0 ** rng.uniform(-38, 38, size=20000)
    x = (rng.choice([-1.0, 1.0], size=mags.size) * mags).astype(np.float32)
    # also exact ties and values close to them
    base = np.float32(1.0) + np.float32(2.0 ** -8) * np.arange(-64, 64, dtype=np.float32)
    x = np.concatenate([x, base, np.float32([3.39e38, 3.4e38, -3.4e38, 1e-40, 2.0 ** -130])])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = round_bf16(x.astype(np.float64))
    assert np.array_equal(got, ref)


def test_round_bf16_hand_ties():
    # spacing on [1, 2) is 2^-7
    assert round_bf16(1 + 2.0 ** -8) == 1.0                    # tie -> even (128)
    assert round_bf16(1 + 3 * 2.0 ** -8) == 1 + 2.0 ** -6      # tie -> even (130)
    assert round_bf16(-(1 + 2.0 ** -8)) == -1.0
    # fp64 input just above a tie rounds up (rounding through fp32 first would not)
    assert round_bf16(1 + 2.0 ** -8 + 2.0 ** -40) == 1 + 2.0 ** -7
    # subnormal range: fixed spacing 2^-133
    assert round_bf16(2.0 ** -130) == 2.0 ** -130
    assert round_bf16(2.0 ** -134) == 0.0                      # tie -> even (0)
    assert round_bf16(3 * 2.0 ** -134) == 2 * 2.0 ** -133      # tie -> even (2)
    assert round_bf16(0.0) == 0.0
    assert math.isinf(float(round_bf16(1e39)))
    # representable values are fixed points
    v = np.array([1.0, 1.5, 255 * 2.0 ** 120, -3.0, 2.0 ** -126])
    assert np.array_equal(round_bf16(v), v)


def test_silu_closed_forms():
    v = np.linspace(-30, 30, 1001)
    assert np.allclose(silu(v), v * scipy.special.expit(v), rtol=1e-14, atol=1e-300)
    assert silu(np.array([0.0]))[0] == 0.0
    assert abs(silu(np.array([40.0]))[0] - 40.0) < 1e-12


def test_softmax_against_scipy_and_invariants():
    rng = np.random.default_rng(2)
    z = rng.normal(size=(50, 17)) * 5
    p = softmax_rows(z)
    assert np.allclose(p, scipy.special.softmax(z, axis=1), rtol=1e-13)
    assert np.allclose(p.sum(1), 1.0)
    assert np.allclose(softmax_rows(np.zeros((1, 8))), 1 / 8)
    # shift invariance
    assert np.allclose(softmax_rows(z + 123.0), p, rtol=1e-12)
