"""Pins for the oracle's retrieval step (§3.2: top-k by inner product over
fact embeddings): exact rational arithmetic, closed-form special cases,
numpy lexsort and brute force over all k-subsets on tiny banks."""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import oracle


def _unit(rng, rows, d):
    x = rng.standard_normal((rows, d)).astype(np.float32)
    return (x / np.linalg.norm(x, axis=1, keepdims=True)).astype(np.float32)


def test_scores_exact_rational_small():
    rng = np.random.default_rng(3)
    d, n = 16, 40
    bank = _unit(rng, n, d)
    q = _unit(rng, 1, d)
    got = oracle.scores(q, bank, n, d, 1)[0]
    for j in range(n):
        exact = sum(Fraction(float(q[0, t])) * Fraction(float(bank[j, t])) for t in range(d))
        mag = sum(abs(Fraction(float(q[0, t])) * Fraction(float(bank[j, t]))) for t in range(d))
        # binary64 summation of exact products: error at most (d-1) u sum|terms|
        assert abs(Fraction(got[j]) - exact) <= Fraction(d) * Fraction(2) ** -53 * mag


def test_scores_one_hot_query_reads_a_column():
    rng = np.random.default_rng(4)
    d, n = 384, 64
    bank = _unit(rng, n, d)
    for t in (0, 7, 383):
        q = np.zeros((1, d), dtype=np.float32)
        q[0, t] = 1.0
        got = oracle.scores(q, bank, n, d, 1)[0]
        assert np.array_equal(got, bank[:, t].astype(np.float64))


def test_scores_orthonormal_bank_closed_form():
    # bank rows = scaled standard basis vectors: s_j = q[j] * c_j exactly
    d = n = 32
    c = np.arange(1, n + 1, dtype=np.float32) / 8
    bank = np.diag(c).astype(np.float32)
    q = np.linspace(-1, 1, d, dtype=np.float32)[None, :]
    got = oracle.scores(q, bank, n, d, 1)[0]
    assert np.array_equal(got, q[0].astype(np.float64) * c.astype(np.float64))


def test_query_equal_to_a_row_wins_with_its_norm():
    rng = np.random.default_rng(5)
    d, n = 768, 500
    bank = _unit(rng, n, d)
    jstar = 123
    q = bank[jstar:jstar + 1].copy()
    ids, vals, _ = oracle.retrieve(q, bank, n, d, k=3)
    assert ids[0, 0] == jstar  # Cauchy-Schwarz: no unit row scores above |e|^2
    exact = float(sum(Fraction(float(v)) ** 2 for v in q[0]))
    assert abs(vals[0, 0] - exact) <= d * 2.0 ** -53


def test_bf16_bank_decodes_exactly():
    rng = np.random.default_rng(6)
    d, n = 64, 50
    x = _unit(rng, n + 1, d)
    bits = np.array(
        __import__("torch").from_numpy(x).to(__import__("torch").bfloat16)
        .view(__import__("torch").int16).numpy().view(np.uint16))
    as_f32 = oracle.bf16_to_f64(bits).astype(np.float32)
    s_bf16 = oracle.scores(bits[:1], bits[1:], n, d, 1, dtype=oracle.BF16)
    s_f32 = oracle.scores(as_f32[:1], as_f32[1:], n, d, 1, dtype=oracle.F32)
    assert np.array_equal(s_bf16, s_f32)


def test_per_query_banks_use_their_own_bank():
    rng = np.random.default_rng(7)
    d, n, nq = 32, 20, 3
    banks = _unit(rng, nq * n, d).reshape(nq, n, d)
    qs = _unit(rng, nq, d)
    got = oracle.scores(qs, banks, n, d, nq, bank_stride=n * d)
    for r in range(nq):
        assert np.array_equal(got[r], oracle.scores(qs[r:r + 1], banks[r], n, d, 1)[0])


def test_topk_matches_lexsort_with_ties():
    rng = np.random.default_rng(8)
    n, nq, k = 3000, 4, 64
    sc = rng.standard_normal((nq, n))
    sc[:, 100:400] = np.round(sc[:, 100:400], 1)   # plenty of exact ties
    ids, vals = oracle.topk(sc, k)
    for r in range(nq):
        order = np.lexsort((np.arange(n), -sc[r]))
        assert np.array_equal(ids[r], order[:k].astype(np.int32))
        assert np.array_equal(vals[r], sc[r][order[:k]])


def test_topk_duplicate_rows_lower_id_first():
    rng = np.random.default_rng(9)
    d, n = 48, 30
    bank = _unit(rng, n, d)
    bank[17] = bank[4]
    bank[29] = bank[4]
    q = bank[4:5].copy()
    ids, _, _ = oracle.retrieve(q, bank, n, d, k=3)
    assert list(ids[0]) == [4, 17, 29]


def test_topk_k_equals_n_is_a_full_permutation():
    rng = np.random.default_rng(10)
    sc = rng.standard_normal((1, 257))
    ids, vals = oracle.topk(sc, 257)
    assert sorted(ids[0].tolist()) == list(range(257))
    assert np.all(np.diff(vals[0]) <= 0)


@pytest.mark.parametrize("seed", range(6))
def test_topk_bruteforce_over_subsets(seed):
    rng = np.random.default_rng(100 + seed)
    n, k = 8, 3
    sc = np.round(rng.standard_normal(n), 1)[None, :]   # ties likely
    ids, _ = oracle.topk(sc, k)
    best = None
    for sub in itertools.combinations(range(n), k):
        outside = [j for j in range(n) if j not in sub]
        # a valid top-k set: nothing outside beats anything inside under
        # (score desc, id asc)
        ok = all((sc[0, o], -o) < (sc[0, i], -i) for o in outside for i in sub)
        if ok:
            assert best is None, "the top-k set must be unique"
            best = sub
    ordered = sorted(best, key=lambda j: (-sc[0, j], j))
    assert list(ids[0]) == ordered
