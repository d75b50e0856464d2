"""Pins for the oracle's rotation with a model's own rotary table and pair
layout (§3.3: composition rotates with the model's rotary tables; §6.1: the
evaluated models differ in their RoPE parameterisation): independent complex
forms for both layouts with arbitrary tables, the permutation that relates
the two layouts (also through the whole inject), zero-frequency pairs,
composition and relative-position scores with a scaled table, and the
default table's geometric ladder."""
import math

import numpy as np
import pytest

import oracle
import workloads


def _table(rng, D):
    # an arbitrary positive table, far from the default ladder
    return np.sort(rng.uniform(1e-6, 1.5, D // 2))[::-1].copy()


@pytest.mark.parametrize("interleaved", [False, True])
@pytest.mark.parametrize("p", [0, 1, 129, 4096, 100000])
def test_complex_form_with_an_arbitrary_table(interleaved, p):
    rng = np.random.default_rng(300 + p + 7 * interleaved)
    D = 64
    x = rng.standard_normal(D)
    f = _table(rng, D)
    if interleaved:
        z = x[0::2] + 1j * x[1::2]
    else:
        z = x[: D // 2] + 1j * x[D // 2:]
    zr = z * np.exp(1j * (p * f))
    want = np.empty(D)
    if interleaved:
        want[0::2], want[1::2] = zr.real, zr.imag
    else:
        want[: D // 2], want[D // 2:] = zr.real, zr.imag
    got = oracle.rope_table_f64(x, p, f, D, interleaved)
    assert np.max(np.abs(got - want)) <= 1e-12 * (1 + p * 1e-4) * np.max(np.abs(x))


def _deinterleave(D):
    # position of interleaved element i in the half-split layout
    q = np.empty(D, dtype=np.int64)
    q[0::2] = np.arange(D // 2)
    q[1::2] = np.arange(D // 2) + D // 2
    return q


def test_layouts_are_related_by_a_permutation_bit_exact():
    rng = np.random.default_rng(310)
    for D in (16, 128, 256):
        q = _deinterleave(D)
        f = workloads.llama31_inv_freq(D)
        for p in (3, 777, 65000):
            x = rng.standard_normal(D)
            xs = np.empty(D)
            xs[q] = x  # the same pairs laid out half-split
            yi = oracle.rope_table_f64(x, p, f, D, True)
            ys = oracle.rope_table_f64(xs, p, f, D, False)
            assert np.array_equal(yi, ys[q])


def test_zero_frequency_pairs_do_not_move():
    rng = np.random.default_rng(311)
    D = 32
    f = _table(rng, D)
    f[[0, 5, 15]] = 0.0
    x = rng.standard_normal(D)
    for interleaved in (False, True):
        y = oracle.rope_table_f64(x, 12345, f, D, interleaved)
        for j in (0, 5, 15):
            i0, i1 = (2 * j, 2 * j + 1) if interleaved else (j, j + D // 2)
            assert y[i0] == x[i0] and y[i1] == x[i1]


@pytest.mark.parametrize("interleaved", [False, True])
def test_composition_and_relative_scores_with_a_scaled_table(interleaved):
    rng = np.random.default_rng(312 + interleaved)
    D = 128
    f = workloads.llama31_inv_freq(D)
    x, qv = rng.standard_normal(D), rng.standard_normal(D)
    for a, b in ((5, 9), (300, 1700), (4000, 60000)):
        ab = oracle.rope_table_f64(oracle.rope_table_f64(x, b, f, D, interleaved), a, f, D,
                                   interleaved)
        direct = oracle.rope_table_f64(x, a + b, f, D, interleaved)
        assert np.max(np.abs(ab - direct)) <= 1e-11 * np.max(np.abs(x)) * (1 + (a + b) * 1e-4)
        # <R_a q, R_b k> = <q, R_{b-a} k>: only the relative position matters
        lhs = oracle.rope_table_f64(qv, a, f, D, interleaved) @ oracle.rope_table_f64(
            x, b, f, D, interleaved)
        rhs = qv @ oracle.rope_table_f64(x, b - a, f, D, interleaved)
        assert abs(lhs - rhs) <= 1e-10 * (1 + (a + b) * 1e-4) * np.linalg.norm(qv) * np.linalg.norm(x)


def test_pair_norms_preserved_with_a_table():
    rng = np.random.default_rng(313)
    D = 64
    f = _table(rng, D)
    x = rng.standard_normal(D)
    for interleaved in (False, True):
        y = oracle.rope_table_f64(x, 98765, f, D, interleaved)
        if interleaved:
            nx, ny = x[0::2] ** 2 + x[1::2] ** 2, y[0::2] ** 2 + y[1::2] ** 2
        else:
            nx = x[: D // 2] ** 2 + x[D // 2:] ** 2
            ny = y[: D // 2] ** 2 + y[D // 2:] ** 2
        assert np.max(np.abs(nx - ny) / nx) < 1e-13


def test_default_table_is_a_geometric_ladder_from_one():
    for theta, D in ((10000.0, 64), (500000.0, 128), (1000000.0, 256)):
        f = oracle.default_inv_freq(theta, D)
        assert f[0] == 1.0
        ratio = f[1:] / f[:-1]
        assert np.max(np.abs(ratio / ratio[0] - 1)) < 1e-13
        # D/2 ratios of theta^(-2/D) multiply to 1/theta
        assert abs(math.log(ratio[0]) * D / 2 + math.log(theta)) < 1e-10


def test_llama31_table_bands():
    D = 128
    base = oracle.default_inv_freq(500000.0, D)
    f = workloads.llama31_inv_freq(D)
    wl = 2 * math.pi / base
    hi = wl < 8192 / 4
    lo = wl > 8192 / 1
    assert np.allclose(f[hi], base[hi], rtol=4e-16, atol=0)  # equal up to the pow ulp
    assert np.allclose(f[lo], base[lo] / 8, rtol=1e-15)
    mid = ~hi & ~lo
    assert mid.any() and np.all((f[mid] >= base[mid] / 8) & (f[mid] <= base[mid]))
    assert np.all(np.diff(f) < 0)  # still strictly decreasing


def test_inject_layouts_related_by_the_same_permutation():
    # through the whole oracle inject: storing every head de-interleaved and
    # injecting half-split gives the de-interleaved pages of the interleaved run
    rng = np.random.default_rng(314)
    L, H, D, T = 2, 3, 32, 40
    k, n = 3, 6
    lens = np.array([[4, 7, 3, 5, 6, 2]], dtype=np.int32)
    offs = np.array([[0, 4, 11, 14, 19, 25]], dtype=np.int64)
    ids = np.array([[4, 1, 2]], dtype=np.int32)
    K = oracle.f64_to_bf16(rng.standard_normal((L, T, H, D)))
    V = oracle.f64_to_bf16(rng.standard_normal((L, T, H, D)))
    m_tok = int(lens[0, ids[0]].sum())
    slots = np.arange(m_tok, dtype=np.int64)[None, :] * 2 + 1
    pos = (np.arange(m_tok, dtype=np.int32) + 1000)[None, :]
    m = np.array([m_tok], dtype=np.int32)
    f = workloads.llama31_inv_freq(D)
    q = _deinterleave(D)
    Ks = np.empty_like(K)
    Ks[..., q] = K
    Vs = np.empty_like(V)
    Vs[..., q] = V
    outs = []
    for KK, VV, inter in ((K, V, True), (Ks, Vs, False)):
        pk = np.zeros((L, 2 * m_tok + 2, H, D), dtype=np.uint16)
        pv = np.zeros_like(pk)
        st = oracle.inject(ids, KK, VV, slots, pos, 500000.0, pk, pv, offs, lens, m, k, 1, n, 0,
                           1, m_tok, L, H, D, T, pk.shape[1], inv_freq=f, interleaved=inter)
        assert st == 0
        outs.append((pk, pv))
    assert np.array_equal(outs[0][0], outs[1][0][..., q])
    assert np.array_equal(outs[0][1], outs[1][1][..., q])
    assert (outs[0][0][:, 1::2] != 0).any()
