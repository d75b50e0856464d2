"""The oracle's OpenMP loops compute every output (one score, one query's
ranking, one (layer, head) sweep over the placed tokens) on one thread in
the written order, so its results must not depend on the thread count:
one thread is the plain serial program, and a team of any size reproduces
it bit for bit, including a slot written twice (the later placed token
wins, as in a serial run)."""
import numpy as np
import pytest

import oracle


def _bf16_unit(rng, rows, d):
    x = rng.standard_normal((rows, d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    return oracle.f64_to_bf16(x)


@pytest.mark.parametrize("dtype", [oracle.F32, oracle.BF16])
@pytest.mark.parametrize("shared", [True, False])
def test_scores_and_topk_independent_of_threads(dtype, shared):
    rng = np.random.default_rng(71)
    n, d, nq, k = 1500, 40, 5, 17
    banks = 1 if shared else nq
    x = rng.standard_normal((banks * n, d)).astype(np.float32)
    q = rng.standard_normal((nq, d)).astype(np.float32)
    if dtype == oracle.BF16:
        x, q = oracle.f64_to_bf16(x), oracle.f64_to_bf16(q)
    # planted exact ties: a duplicated row in every bank
    xb = x.reshape(banks, n, d)
    xb[:, 900] = xb[:, 3]
    stride = 0 if shared else n * d
    with oracle.using_threads(1):
        s1 = oracle.scores(q, x, n, d, nq, stride, dtype)
        i1, v1 = oracle.topk(s1, k)
    for t in (2, 3, 8):
        with oracle.using_threads(t):
            st = oracle.scores(q, x, n, d, nq, stride, dtype)
            it, vt = oracle.topk(st, k)
        assert np.array_equal(st, s1)
        assert np.array_equal(it, i1) and np.array_equal(vt, v1)
    # the serial program, written out: one row at a time, sum over t in order
    for r in range(nq):
        qd = (oracle.bf16_to_f64(q[r]) if dtype == oracle.BF16 else q[r].astype(np.float64))
        for j in (0, 3, 900, n - 1):
            row = xb[0 if shared else r, j]
            ed = oracle.bf16_to_f64(row) if dtype == oracle.BF16 else row.astype(np.float64)
            acc = 0.0
            for t in range(d):
                acc += float(qd[t]) * float(ed[t])
            assert s1[r, j] == acc


def test_inject_independent_of_threads_with_a_slot_written_twice():
    rng = np.random.default_rng(72)
    L, H, D, n, k, theta = 5, 3, 8, 30, 7, 10000.0
    lens = rng.integers(1, 6, size=n).astype(np.int32)
    offs = (np.cumsum(lens) - lens).astype(np.int64)
    T = int(lens.sum())
    K = oracle.f64_to_bf16(rng.standard_normal((L, T, H, D)))
    V = oracle.f64_to_bf16(rng.standard_normal((L, T, H, D)))
    ids = np.stack([rng.permutation(n)[:k] for _ in range(2)]).astype(np.int32)
    mt = k * 6
    m = np.array([lens[ids[r]].sum() for r in range(2)], dtype=np.int32)
    num_slots = 200
    slots = np.full((2, mt), -1, dtype=np.int64)
    pos = np.full((2, mt), -1, dtype=np.int32)
    for r in range(2):
        slots[r, :m[r]] = rng.permutation(num_slots)[:m[r]]
        pos[r, :m[r]] = 11 + np.arange(m[r])
    slots[1, 0] = slots[0, 2]          # request 1 rewrites a slot of request 0
    slots[0, m[0] - 1] = slots[0, 0]   # and request 0 one of its own

    def run(threads):
        pk = np.full((L, num_slots, H, D), 0x7FA5, dtype=np.uint16)
        pv = pk.copy()
        with oracle.using_threads(threads):
            st = oracle.inject(ids, K, V, slots, pos, theta, pk, pv, offs[None], lens[None], m,
                               k, 2, n, 0, 1, mt, L, H, D, T, num_slots)
        return pk, pv, st

    pk1, pv1, st1 = run(1)
    # the later placed token wins a twice-written slot
    r1_first = offs[ids[1, k - 1]]  # request 1's first placed token (reverse rank)
    assert np.array_equal(pv1[:, slots[1, 0]], V[:, r1_first])
    for t in (2, 4, 8):
        pkt, pvt, stt = run(t)
        assert np.array_equal(pkt, pk1) and np.array_equal(pvt, pv1) and stt == st1
