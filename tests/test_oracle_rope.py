"""Pins for the oracle's rotation (§2.4; Theorem "Chunked RoPE Injection",
§5.1): identity at p = 0, an independent complex-multiplication form,
pair-norm preservation, composition, relative-position scores, shift
equivalence and the frequency ladder recovered from outputs."""
import math

import numpy as np
import pytest

import oracle

THETA = 500000.0


def _x(rng, D):
    return rng.standard_normal(D)


def test_p0_is_identity_bit_exact():
    rng = np.random.default_rng(20)
    for D in (16, 64, 128, 256):
        bits = oracle.f64_to_bf16(_x(rng, D))
        assert np.array_equal(oracle.rope_bf16(bits, 0, THETA, D), bits)


@pytest.mark.parametrize("p", [1, 7, 128, 2000, 3327, 131071])
def test_complex_multiplication_form(p):
    # pair j is the complex number x_j + i x_{j+D/2}; R_p multiplies it by
    # e^{i p w_j} with w_j = theta^(-2j/D)
    rng = np.random.default_rng(21 + p)
    D = 128
    x = _x(rng, D)
    z = x[: D // 2] + 1j * x[D // 2:]
    w = THETA ** (-np.arange(D // 2) * 2.0 / D)
    zr = z * np.exp(1j * (p * w))
    want = np.concatenate([zr.real, zr.imag])
    got = oracle.rope_f64(x, p, THETA, D)
    assert np.max(np.abs(got - want)) <= 1e-12 * (1 + p * 1e-5) * np.max(np.abs(x))


def test_lowest_pair_turns_by_p_radians():
    D = 128
    x = np.zeros(D)
    x[0], x[D // 2] = 1.0, 0.0
    for p in (1, 2, 3):
        y = oracle.rope_f64(x, p, THETA, D)
        assert abs(y[0] - math.cos(p)) < 1e-15 and abs(y[D // 2] - math.sin(p)) < 1e-15


def test_pairing_is_rotate_half():
    # a unit vector at index j < D/2 only moves into index j + D/2
    D = 64
    for j in (0, 5, 31):
        x = np.zeros(D)
        x[j] = 1.0
        y = oracle.rope_f64(x, 11, 10000.0, D)
        nz = set(np.nonzero(np.abs(y) > 1e-300)[0].tolist())
        assert nz <= {j, j + D // 2}
        assert abs(y[j] ** 2 + y[j + D // 2] ** 2 - 1) < 1e-14


def test_frequency_ladder_from_outputs():
    # recover the angle of each pair at p = 1: w_0 = 1, a geometric ladder
    # with ratio theta^(-2/D), ending at theta^(-(D-2)/D)
    D = 128
    ang = []
    for j in range(D // 2):
        x = np.zeros(D)
        x[j] = 1.0
        y = oracle.rope_f64(x, 1, THETA, D)
        ang.append(math.atan2(y[j + D // 2], y[j]))
    ang = np.array(ang)
    assert abs(ang[0] - 1.0) < 1e-15
    ratio = ang[1:] / ang[:-1]
    assert np.allclose(ratio, math.exp(-2.0 / D * math.log(THETA)), rtol=1e-12, atol=0)
    assert abs(ang[-1] / math.exp(-(D - 2) / D * math.log(THETA)) - 1) < 1e-12


def test_pair_norms_preserved():
    rng = np.random.default_rng(22)
    D = 128
    x = _x(rng, D)
    y = oracle.rope_f64(x, 54321, THETA, D)
    nx = np.hypot(x[: D // 2], x[D // 2:])
    ny = np.hypot(y[: D // 2], y[D // 2:])
    assert np.max(np.abs(nx - ny) / nx) < 1e-14


@pytest.mark.parametrize("a,b", [(3, 5), (128, 2000), (4000, 9000), (0, 77)])
def test_composition(a, b):
    rng = np.random.default_rng(23)
    D = 128
    x = _x(rng, D)
    twice = oracle.rope_f64(oracle.rope_f64(x, a, THETA, D), b, THETA, D)
    once = oracle.rope_f64(x, a + b, THETA, D)
    assert np.max(np.abs(twice - once)) < 1e-11


@pytest.mark.parametrize("a,b", [(10, 3), (128, 2000), (2500, 130)])
def test_scores_depend_on_relative_position(a, b):
    rng = np.random.default_rng(24)
    D = 128
    q, k = _x(rng, D), _x(rng, D)
    lhs = oracle.rope_f64(q, a, THETA, D) @ oracle.rope_f64(k, b, THETA, D)
    rhs = q @ oracle.rope_f64(k, b - a, THETA, D)
    assert abs(lhs - rhs) < 1e-10


def test_shift_equivalence():
    # <R_N q, R_{v0+j} k> = <R_{N'} q, R_{p0+j} k> with N' = N - (v0 - p0)
    rng = np.random.default_rng(25)
    D = 128
    q = _x(rng, D)
    N, v0, p0 = 2128, 1500, 37
    Np = N - (v0 - p0)
    for j in range(0, 40, 7):
        k = _x(rng, D)
        lhs = oracle.rope_f64(q, N, THETA, D) @ oracle.rope_f64(k, v0 + j, THETA, D)
        rhs = oracle.rope_f64(q, Np, THETA, D) @ oracle.rope_f64(k, p0 + j, THETA, D)
        assert abs(lhs - rhs) < 1e-10


def test_bf16_rotation_is_rounded_f64_rotation():
    rng = np.random.default_rng(26)
    D = 128
    bits = oracle.f64_to_bf16(_x(rng, D))
    for p in (1, 999, 3000):
        want = oracle.f64_to_bf16(oracle.rope_f64(oracle.bf16_to_f64(bits), p, THETA, D))
        assert np.array_equal(oracle.rope_bf16(bits, p, THETA, D), want)
