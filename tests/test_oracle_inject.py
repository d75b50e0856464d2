"""Pins for the oracle's composition + injection (§3.3, §3.4): reading the
pages back through the block table gives the contiguous concatenation of the
chosen facts, each rotated at its own positions; V is a bit copy; nothing
else is written; permuting the facts only moves them (Appendix F: cost and
content depend on the set, not the order)."""
import numpy as np

import oracle

SENT = 0x7FA5


def _store(rng, L, H, D, n, lo, hi):
    lens = rng.integers(lo, hi + 1, size=n).astype(np.int32)
    offs = (np.cumsum(lens) - lens).astype(np.int64)
    T = int(lens.sum())
    K = oracle.f64_to_bf16(rng.standard_normal((L, T, H, D)))
    V = oracle.f64_to_bf16(rng.standard_normal((L, T, H, D)))
    return lens, offs, T, K, V


def _inject(ids, lens, offs, K, V, bt, start, P, theta, num_blocks, reverse=1):
    L, T, H, D = K.shape
    k = ids.shape[1]
    n = lens.size
    mt = k * int(lens.max())
    mb = bt.shape[1]
    sm = oracle.slot_map(ids, lens[None], start, bt, P, k, 1, n, n, mb, mt, reverse)
    num_slots = num_blocks * P
    pk = np.full((L, num_slots, H, D), SENT, dtype=np.uint16)
    pv = np.full((L, num_slots, H, D), SENT, dtype=np.uint16)
    st = oracle.inject(ids, K, V, sm["slots"], sm["positions"], theta, pk, pv, offs[None],
                       lens[None], sm["m"], k, 1, n, n, reverse, mt, L, H, D, T, num_slots)
    return sm, pk, pv, st


def _read_back(pages, bt, start, m, P):
    pos = start + np.arange(m)
    slots = bt[0][pos // P].astype(np.int64) * P + pos % P
    return pages[:, slots]


def test_pages_equal_rotated_concatenation():
    rng = np.random.default_rng(30)
    L, H, D, n, k, P, start, theta = 3, 2, 16, 40, 6, 4, 9, 10000.0
    lens, offs, T, K, V = _store(rng, L, H, D, n, 0, 7)
    ids = rng.permutation(n)[:k].astype(np.int32)[None]
    mb = -(-(start + k * 7) // P)
    num_blocks = mb + 5
    bt = rng.permutation(num_blocks)[:mb].astype(np.int32)[None]
    sm, pk, pv, st = _inject(ids, lens, offs, K, V, bt, start, P, theta, num_blocks)
    assert st == 0
    m = int(sm["m"][0])
    order = ids[0][::-1]                         # most relevant fact last
    rows = np.concatenate([offs[c] + np.arange(lens[c]) for c in order]).astype(np.int64)
    assert rows.size == m
    gotK = _read_back(pk, bt, start, m, P)
    gotV = _read_back(pv, bt, start, m, P)
    for l in range(L):
        assert np.array_equal(gotV[l], V[l, rows])
        want = oracle.rope_rows_bf16(K[l, rows].reshape(m, H * D), start + np.arange(m), theta, H, D)
        assert np.array_equal(gotK[l].reshape(m, H * D), want)
    # nothing else written
    touched = np.zeros(num_blocks * P, dtype=bool)
    pos = start + np.arange(m)
    touched[bt[0][pos // P].astype(np.int64) * P + pos % P] = True
    assert (pk[:, ~touched] == SENT).all() and (pv[:, ~touched] == SENT).all()
    assert (pk[:, touched] != SENT).any(axis=(2, 3)).all()


def test_permuting_facts_moves_them_only():
    rng = np.random.default_rng(31)
    L, H, D, n, k, P, start, theta = 2, 1, 32, 25, 5, 8, 0, 500000.0
    lens, offs, T, K, V = _store(rng, L, H, D, n, 1, 9)
    ids = rng.permutation(n)[:k].astype(np.int32)[None]
    mb = -(-(start + k * 9) // P)
    bt = np.arange(mb, dtype=np.int32)[None]
    for perm_seed in range(3):
        order = np.random.default_rng(perm_seed).permutation(k)
        pid = ids[:, order]
        sm, pk, pv, _ = _inject(pid, lens, offs, K, V, bt, start, P, theta, mb, reverse=0)
        b = start
        for c in pid[0]:
            c = int(c)
            pos = b + np.arange(lens[c])
            for l in range(L):
                want = oracle.rope_rows_bf16(K[l, offs[c] + np.arange(lens[c])].reshape(-1, H * D),
                                             pos, theta, H, D)
                assert np.array_equal(pk[l, pos].reshape(-1, H * D), want)
                assert np.array_equal(pv[l, pos], V[l, offs[c] + np.arange(lens[c])])
            b += lens[c]


def test_bad_slots_and_sources_are_skipped_and_flagged():
    rng = np.random.default_rng(32)
    L, H, D, n, k, P = 1, 1, 16, 10, 3, 4
    lens, offs, T, K, V = _store(rng, L, H, D, n, 2, 4)
    ids = np.array([[1, 2, 3]], dtype=np.int32)
    mt = k * 4
    m = np.array([int(lens[[1, 2, 3]].sum())], dtype=np.int32)
    slots = np.full((1, mt), -1, dtype=np.int64)
    slots[0, :m[0]] = np.arange(m[0])
    slots[0, 0] = 10 ** 6                                  # outside the pool
    pos = np.zeros((1, mt), dtype=np.int32)
    num_slots = 64
    pk = np.full((L, num_slots, H, D), SENT, dtype=np.uint16)
    pv = pk.copy()
    st = oracle.inject(ids, K, V, slots, pos, 1e4, pk, pv, offs[None], lens[None], m, k, 1, n, n,
                       1, mt, L, H, D, T, num_slots)
    assert st & oracle.SLOT_RANGE
    assert (pk[0, 1:m[0]] != SENT).any()
    offs2 = offs.copy()
    offs2[2] = T                                           # fact 2 runs past the store
    pk[:] = SENT
    st = oracle.inject(ids, K, V, slots, pos, 1e4, pk, pv, offs2[None], lens[None], m, k, 1, n,
                       n, 1, mt, L, H, D, T, num_slots)
    assert st & oracle.SRC_RANGE


def test_storage_formula_worked_example():
    import json
    import os
    import workloads
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "storage_formula.json")))
    w = workloads.LLAMA8B
    assert (w.L, w.H, w.D) == (g["L"], g["h"], g["d"])
    per_token = workloads.kv_bytes_per_token(w)
    assert per_token * g["tokens"] == g["bytes_exact"]
    assert abs(per_token * g["tokens"] / 2 ** 20 - g["paper_megabytes_approx"]) < 1e-9
    # the inject step moves each stored byte once in and once out
    assert workloads.inject_algorithmic_bytes(w, g["tokens"]) == 2 * g["bytes_exact"]
