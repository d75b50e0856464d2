"""Pins for the oracle's placement and slot map (§5.2 Position policy; paged
blocks of §2.2): properties that fix the formulas without restating them."""
import numpy as np
import pytest

import oracle


def _case(rng, n=200, k=7, lo=0, hi=20, start=37, P=16, nq=1, perm=True):
    lens = rng.integers(lo, hi + 1, size=(nq, n)).astype(np.int32)
    ids = np.stack([rng.permutation(n)[:k] for _ in range(nq)]).astype(np.int32)
    max_tokens = k * hi
    max_blocks = -(-(start + max_tokens) // P)
    pool = nq * max_blocks
    order = rng.permutation(pool) if perm else np.arange(pool)
    bt = order.reshape(nq, max_blocks).astype(np.int32)
    return lens, ids, bt, max_tokens, max_blocks


def _run(lens, ids, bt, start, P, max_tokens, max_blocks, reverse=1):
    nq, k = ids.shape
    n = lens.shape[1]
    return oracle.slot_map(ids, lens, start, bt, P, k, nq, n, n, max_blocks, max_tokens, reverse)


def test_identity_block_table_gives_slot_equal_position():
    rng = np.random.default_rng(11)
    lens, ids, bt, mt, mb = _case(rng, perm=False)
    out = _run(lens, ids, bt, 37, 16, mt, mb)
    m = out["m"][0]
    assert m > 0 and out["status"] == 0
    assert np.array_equal(out["slots"][0, :m], out["positions"][0, :m].astype(np.int64))


@pytest.mark.parametrize("P", [1, 16, 32])
def test_permuted_table_inverts_back_to_contiguous_positions(P):
    rng = np.random.default_rng(12 + P)
    start = 37
    lens, ids, bt, mt, mb = _case(rng, P=P, start=start)
    out = _run(lens, ids, bt, start, P, mt, mb)
    m = out["m"][0]
    slots = out["slots"][0, :m]
    inv = {int(b): i for i, b in enumerate(bt[0])}
    back = np.array([inv[int(s) // P] * P + int(s) % P for s in slots])
    assert np.array_equal(back, start + np.arange(m))
    assert np.array_equal(out["positions"][0, :m], start + np.arange(m))
    assert len(set(slots.tolist())) == m


def test_reverse_proximity_order_and_runs():
    rng = np.random.default_rng(13)
    lens, ids, bt, mt, mb = _case(rng, lo=1, hi=9, k=9)
    out = _run(lens, ids, bt, 5, 16, mt, mb)
    m = out["m"][0]
    fact, tok = out["fact"][0, :m], out["tok"][0, :m]
    assert m == lens[0, ids[0]].sum()
    # the facts appear as consecutive runs, least relevant first, and the most
    # relevant fact (rank 0) is the last run, adjacent to the query at start+m
    runs = [fact[0]] + [f for a, f in zip(fact[:-1], fact[1:]) if f != a]
    assert runs == list(ids[0][::-1])
    assert fact[-1] == ids[0, 0]
    for f in set(runs):
        sel = tok[fact == f]
        assert np.array_equal(sel, np.arange(lens[0, f]))


def test_forward_order_when_reverse_is_off():
    rng = np.random.default_rng(14)
    lens, ids, bt, mt, mb = _case(rng, lo=1, hi=9, k=6)
    out = _run(lens, ids, bt, 0, 16, mt, mb, reverse=0)
    m = out["m"][0]
    fact = out["fact"][0, :m]
    runs = [fact[0]] + [f for a, f in zip(fact[:-1], fact[1:]) if f != a]
    assert runs == list(ids[0])


def test_zero_length_facts_and_k1():
    rng = np.random.default_rng(15)
    lens, ids, bt, mt, mb = _case(rng, k=1, lo=0, hi=0)
    out = _run(lens, ids, bt, 3, 16, mt, mb)
    assert out["m"][0] == 0 and out["status"] == 0
    lens[0, ids[0, 0]] = 5
    out = _run(lens, ids, bt, 3, 16, 5, mb)
    assert out["m"][0] == 5


def test_multi_request_rows_are_independent():
    rng = np.random.default_rng(16)
    lens, ids, bt, mt, mb = _case(rng, nq=4)
    out = _run(lens, ids, bt, 20, 16, mt, mb)
    for r in range(4):
        one = _run(lens[r:r + 1], ids[r:r + 1], bt[r:r + 1], 20, 16, mt, mb)
        m = one["m"][0]
        assert out["m"][r] == m
        assert np.array_equal(out["slots"][r, :m], one["slots"][0, :m])
    allslots = np.concatenate([out["slots"][r, :out["m"][r]] for r in range(4)])
    assert len(set(allslots.tolist())) == allslots.size


def test_error_flags_and_skipped_requests():
    rng = np.random.default_rng(17)
    lens, ids, bt, mt, mb = _case(rng, nq=2, lo=1, hi=9)
    bad = ids.copy()
    bad[0, 2] = 10_000                       # id out of range
    out = _run(lens, bad, bt, 0, 16, mt, mb)
    assert out["status"] & oracle.ID_RANGE and out["m"][0] == 0 and out["m"][1] > 0
    out = _run(lens, ids, bt, 0, 16, 3, mb)  # capacity
    assert out["status"] & oracle.CAPACITY and (out["m"] == 0).all()
    out = _run(lens, ids, bt[:, :1], 100, 16, mt, 1)   # block table too short
    assert out["status"] & oracle.BT_SHORT
    bt2 = bt.copy()
    bt2[1, :] = -1
    out = _run(lens, ids, bt2, 0, 16, mt, mb)
    assert out["status"] & oracle.BAD_BLOCK and out["m"][1] == 0 and out["m"][0] > 0
    l2 = lens.copy()
    l2[0, ids[0, 0]] = -3
    out = _run(l2, ids, bt, 0, 16, mt, mb)
    assert out["status"] & oracle.BAD_LEN and out["m"][0] == 0
