"""Pins for the oracle's elementary pieces: closed forms, special cases, library routines."""

import math

import numpy as np
import pytest
import torch

import oracle


# ------------------------------------------------------------------ bf16 rounding

def test_bf16_round_hand_cases():
    # bf16 spacing just above 1.0 is 2**-7; halfway cases round to the even mantissa.
    cases = {
        1.0: 1.0,
        1.0 + 2 ** -8: 1.0,                       # tie -> even (mantissa 0)
        1.0 + 3 * 2 ** -8: 1.0 + 2 ** -6,         # tie -> even (mantissa 2)
        1.0 + 2 ** -8 + 2 ** -30: 1.0 + 2 ** -7,  # just above the tie -> up
        -1.0 - 2 ** -8 - 2 ** -30: -1.0 - 2 ** -7,
        0.1: 0.10009765625,
    }
    for x, want in cases.items():
        assert oracle.bf16_round(np.array([x]))[0] == want, x


def test_bf16_round_matches_torch_on_fp32_values():
    # For float32 inputs torch's float32 -> bfloat16 conversion is round-to-nearest-even.
    rng = np.random.default_rng(7)
    x32 = (rng.standard_normal(200000) * np.exp(rng.uniform(-20, 20, 200000))).astype(np.float32)
    # add exact halfway points: float32 values whose low 16 bits are 0x8000
    u = x32.view(np.uint32).copy()
    u[:5000] = (u[:5000] & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    x32 = u.view(np.float32)
    ref = torch.from_numpy(x32).to(torch.bfloat16).float().numpy().astype(np.float64)
    got = oracle.bf16_round(x32.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


# ------------------------------------------------------------------ RMSNorm

def test_rmsnorm_closed_forms():
    g = np.linspace(0.5, 1.5, 8)
    c = -3.0
    x = np.full(8, c)
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 0.0), -g, rtol=1e-15)
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1.0), c / math.sqrt(c * c + 1.0) * g, rtol=1e-15)
    # scale invariance (eps = 0) and unit mean square of the output with g = 1
    rng = np.random.default_rng(1)
    y = rng.standard_normal((3, 64))
    a = oracle.rmsnorm(y, np.ones(64), 0.0)
    np.testing.assert_allclose(oracle.rmsnorm(7.5 * y, np.ones(64), 0.0), a, rtol=1e-13)
    np.testing.assert_allclose(np.mean(a * a, axis=-1), 1.0, rtol=1e-13)


# ------------------------------------------------------------------ RoPE

def test_rope_position_zero_is_identity():
    x = np.random.default_rng(2).standard_normal((5, 64))
    np.testing.assert_array_equal(oracle.rope(x, np.zeros(5), 1e4), x)


def test_rope_two_dim_is_plane_rotation():
    # Dh = 2: one pair, frequency theta**0 = 1, so position p rotates by p radians.
    for p in (1.0, 2.5, -0.75):
        got = oracle.rope(np.array([1.0, 0.0]), np.array(p), 1e4)
        np.testing.assert_allclose(got, [math.cos(p), math.sin(p)], rtol=0, atol=1e-15)
        got = oracle.rope(np.array([0.0, 1.0]), np.array(p), 1e4)
        np.testing.assert_allclose(got, [-math.sin(p), math.cos(p)], rtol=0, atol=1e-15)


def test_rope_pairing_and_frequency_dh4():
    # Dh = 4: pairs (0, 2) at frequency 1 and (1, 3) at frequency theta**-0.5.
    theta, p = 100.0, 3.0
    got = oracle.rope(np.array([0.0, 1.0, 0.0, 0.0]), np.array(p), theta)
    a = p * theta ** -0.5
    np.testing.assert_allclose(got, [0.0, math.cos(a), 0.0, math.sin(a)], atol=1e-15)
    got = oracle.rope(np.array([1.0, 0.0, 0.0, 0.0]), np.array(p), theta)
    np.testing.assert_allclose(got, [math.cos(p), 0.0, math.sin(p), 0.0], atol=1e-15)


def test_rope_relative_positions():
    # Scores depend on the position difference only, and norms are preserved.
    rng = np.random.default_rng(3)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    for a, b, shift in ((5, 2, 100), (0, 511, 1000), (37, 37, 4096)):
        s0 = oracle.rope(q, np.array(a), 1e4) @ oracle.rope(k, np.array(b), 1e4)
        s1 = oracle.rope(q, np.array(a + shift), 1e4) @ oracle.rope(k, np.array(b + shift), 1e4)
        assert abs(s0 - s1) < 1e-10 * (1 + abs(s0))
    r = oracle.rope(q, np.array(123), 1e4)
    assert abs(np.linalg.norm(r) - np.linalg.norm(q)) < 1e-12


# ------------------------------------------------------------------ SiLU / attention

def test_silu_values():
    assert oracle.silu(0.0) == 0.0
    assert abs(oracle.silu(1.0) - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16
    assert abs(oracle.silu(40.0) - 40.0) < 1e-12
    assert abs(oracle.silu(-40.0)) < 1e-15
    np.testing.assert_allclose(oracle.silu(np.array([2.0])), torch.nn.functional.silu(
        torch.tensor([2.0], dtype=torch.float64)).numpy(), rtol=1e-15)


def test_attend_special_cases():
    from oracle.model import attend

    rng = np.random.default_rng(4)
    H, Dh = 3, 16
    q = rng.standard_normal((H, Dh))
    v = rng.standard_normal((1, H, Dh))
    k = rng.standard_normal((1, H, Dh))
    np.testing.assert_allclose(attend(q, k, v), v[0], rtol=1e-15)
    # identical keys -> uniform weights -> mean of the values
    k5 = np.repeat(k, 5, axis=0)
    v5 = rng.standard_normal((5, H, Dh))
    np.testing.assert_allclose(attend(q, k5, v5), v5.mean(axis=0), rtol=1e-13)
    # against torch's scaled-dot-product attention in float64 on the CPU
    T = 9
    kk, vv = rng.standard_normal((T, H, Dh)), rng.standard_normal((T, H, Dh))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[:, None, :], torch.from_numpy(kk).transpose(0, 1),
        torch.from_numpy(vv).transpose(0, 1))[:, 0, :].numpy()
    np.testing.assert_allclose(attend(q, kk, vv), ref, rtol=1e-12, atol=1e-14)
