"""Pins of the graph-ANN oracle (oracle/ann.c) against what the paper and the
mathematics fix, independently of the oracle itself:

* hand-worked graphs and searches (tests/golden/ann_worked_example.json,
  §2.6 / §6.1 with the readings stated in the oracle's header);
* a closed form of the exact neighbour lists on banded indicator vectors;
* special cases that reduce to exact top-k by brute force: no iterations
  (the best seeds), a complete graph, and a beam that holds the whole bank
  on a ring (every fact expanded exactly once);
* invariants: the forward half, reverse entries and fill of every final
  list; beam results are valid, ordered and only improve with iterations.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                    "ann_worked_example.json")


def golden():
    with open(GOLD) as f:
        return json.load(f)


def exact_topk(query, bank, k):
    """Brute force: sort every fact by (score desc, id asc) with numpy."""
    s = bank.astype(np.float64) @ query.astype(np.float64)
    order = np.lexsort((np.arange(len(s)), -s))
    return order[:k], s[order[:k]]


def test_worked_pairwise_scores():
    g = golden()
    X = np.array(g["points"], dtype=np.float64)
    for i, row in g["pairwise_scores"].items():
        if i == "note":
            continue
        for j, v in row.items():
            assert X[int(i)] @ X[int(j)] == v


@pytest.mark.parametrize("which", [0, 1])
def test_worked_graph(which):
    g = golden()
    X = np.array(g["points"], dtype=np.float32)
    case = g["graphs"][which]
    F, G = oracle.ann_build(X, len(X), 2, case["degree"])
    assert F.tolist() == case["F"]
    assert G.tolist() == case["G"]


def test_worked_merge_ordering():
    m = golden()["merge_only"]
    G = oracle.ann_merge(np.array(m["F"], dtype=np.int32))
    assert G.tolist() == m["G"]


@pytest.mark.parametrize("which", [0, 1, 2, 3])
def test_worked_search(which):
    g = golden()
    X = np.array(g["points"], dtype=np.float32)
    case = g["searches"][which]
    graph = [gr for gr in g["graphs"] if gr["degree"] == case["graph_degree"]][0]["G"]
    r = oracle.ann_search(np.array(case["query"], np.float32), X, len(X), 2,
                          np.array(graph, np.int32), np.array(case["seeds"], np.int32),
                          case["beam"], case["k"], case["max_iters"], width=case["width"])
    assert r["ids"][0].tolist() == case["ids"]
    assert r["scores"][0].tolist() == case["scores"]
    assert int(r["iters"][0]) == case["iters"]
    assert r["status"] == 0


def banded(n, w):
    """x_i = e_i + ... + e_{i+w-1}: <x_i, x_j> = max(0, w - |i - j|)."""
    X = np.zeros((n, n + w - 1), dtype=np.float32)
    for i in range(n):
        X[i, i:i + w] = 1.0
    return X


@pytest.mark.parametrize("n,w,R", [(12, 4, 5), (30, 3, 9), (9, 9, 8)])
def test_knn_banded_closed_form(n, w, R):
    # the nearest facts are the ones at distance 1, 2, ..., w-1 (the lower id
    # first at equal distance), then every other fact by id (score 0)
    X = banded(n, w)
    F = oracle.ann_knn(X, n, X.shape[1], R)
    for i in range(n):
        near = []
        for r in range(1, w):
            near += [j for j in (i - r, i + r) if 0 <= j < n]
        rest = [j for j in range(n) if j != i and j not in near]
        assert F[i].tolist() == (near + rest)[:R], i


def test_knn_bf16_decode():
    # small integers are exact in bf16: the bf16 path gives the same lists
    rng = np.random.default_rng(5)
    X = rng.integers(-3, 4, size=(40, 24)).astype(np.float32)
    F32 = oracle.ann_knn(X, 40, 24, 7)
    Fb = oracle.ann_knn(oracle.f64_to_bf16(X.astype(np.float64)), 40, 24, 7, dtype=oracle.BF16)
    assert np.array_equal(F32, Fb)


def random_forward(rng, n, R):
    F = np.empty((n, R), dtype=np.int32)
    for i in range(n):
        others = np.array([j for j in range(n) if j != i])
        F[i] = rng.permutation(others)[:R]
    return F


@pytest.mark.parametrize("n,R,seed", [(30, 8, 0), (50, 5, 1), (9, 8, 2), (64, 16, 3)])
def test_merge_invariants(n, R, seed):
    rng = np.random.default_rng(seed)
    F = random_forward(rng, n, R)
    G = oracle.ann_merge(F)
    h = R // 2
    for i in range(n):
        row = G[i].tolist()
        assert len(set(row)) == R and i not in row
        assert row[:h] == F[i, :h].tolist()  # forward half first
        rev = [j for j in range(n) if i in F[j, :h].tolist()]
        pos = {j: F[j, :h].tolist().index(i) for j in rev}
        # what follows: reverse entries in (position, id) order, then the
        # forward tail in order
        t = h
        taken = []
        while t < R and row[t] in pos and row[t] not in F[i, :h]:
            taken.append(row[t])
            t += 1
        avail = sorted((j for j in rev if j not in F[i, :h]), key=lambda j: (pos[j], j))
        assert taken == avail[:min(len(avail), R - h)]
        tail = [j for j in F[i, h:].tolist() if j not in taken]
        assert row[t:] == tail[:R - t]


def test_max_iters_zero_is_best_seeds():
    rng = np.random.default_rng(7)
    n, d = 200, 16
    X = rng.standard_normal((n, d)).astype(np.float32)
    q = rng.standard_normal(d).astype(np.float32)
    G = random_forward(rng, n, 6)
    seeds = np.arange(0, n, 9, dtype=np.int32)
    r = oracle.ann_search(q, X, n, d, G, seeds, beam=10, k=10, max_iters=0)
    ids, s = exact_topk(q, X[seeds], 10)
    assert r["ids"][0].tolist() == seeds[ids].tolist()
    assert np.allclose(r["scores"][0], s, rtol=1e-12, atol=1e-12)
    assert r["iters"][0] == 0


@pytest.mark.parametrize("width", [1, 3])
def test_complete_graph_is_exact(width):
    rng = np.random.default_rng(8)
    n, d = 60, 12
    X = rng.standard_normal((n, d)).astype(np.float32)
    G = np.array([[j for j in range(n) if j != i] for i in range(n)], dtype=np.int32)
    Q = rng.standard_normal((5, d)).astype(np.float32)
    r = oracle.ann_search(Q, X, n, d, G, np.array([17], np.int32), beam=8, k=8, max_iters=100,
                          width=width)
    for t in range(5):
        ids, s = exact_topk(Q[t], X, 8)
        assert r["ids"][t].tolist() == ids.tolist()
        assert np.allclose(r["scores"][t], s, rtol=1e-12, atol=1e-12)


def test_full_beam_on_a_ring_expands_every_fact_once():
    rng = np.random.default_rng(9)
    n, d = 40, 10
    X = rng.standard_normal((n, d)).astype(np.float32)
    G = np.array([[(i + 1) % n, (i - 1) % n] for i in range(n)], dtype=np.int32)
    q = rng.standard_normal(d).astype(np.float32)
    r = oracle.ann_search(q, X, n, d, G, np.array([3], np.int32), beam=n, k=12,
                          max_iters=10 * n)
    ids, s = exact_topk(q, X, 12)
    assert r["ids"][0].tolist() == ids.tolist()
    assert r["iters"][0] == n


def test_results_valid_and_improve_with_iterations():
    rng = np.random.default_rng(10)
    n, d, R = 300, 32, 8
    X = rng.standard_normal((n, d)).astype(np.float32)
    G = random_forward(rng, n, R)
    Q = rng.standard_normal((4, d)).astype(np.float32)
    seeds = np.arange(0, n, 37, dtype=np.int32)
    prev = None
    for T in (0, 1, 2, 4, 8, 1000):
        r = oracle.ann_search(Q, X, n, d, G, seeds, beam=16, k=10, max_iters=T, width=2)
        for t in range(4):
            ids, sc = r["ids"][t], r["scores"][t]
            m = int((ids >= 0).sum())  # the beam holds fewer than k facts only
            assert (ids[m:] == -1).all() and (sc[m:] == -np.inf).all()  # at the end
            ids, sc = ids[:m], sc[:m]
            assert len(set(ids.tolist())) == m
            exact = X[ids].astype(np.float64) @ Q[t].astype(np.float64)
            assert np.allclose(sc, exact, rtol=1e-12, atol=1e-12)
            key = list(zip(-sc, ids))
            assert key == sorted(key)
            if prev is not None:
                assert (r["scores"][t] >= prev[t]).all()  # order statistics only improve
        assert (r["iters"] <= T).all()
        prev = r["scores"]


def test_short_beam_pads_and_bad_ids_flag():
    X = np.eye(4, dtype=np.float32)
    G = np.array([[1], [2], [3], [7]], dtype=np.int32)  # 7 is out of range
    r = oracle.ann_search(X[3], X, 4, 4, G, np.array([0], np.int32), beam=4, k=4, max_iters=0)
    assert r["ids"][0].tolist() == [0, -1, -1, -1]
    assert r["scores"][0][1] == -np.inf
    r = oracle.ann_search(X[3], X, 4, 4, G, np.array([0], np.int32), beam=4, k=4, max_iters=10)
    assert r["status"] == 1
    assert r["ids"][0].tolist() == [3, 0, 1, 2]
