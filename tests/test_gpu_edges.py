"""GPU edge cases: retrieval sizes that hit every scan/select shape (single
and multi chunk, multi-level merge, k = n, k = 1, the largest k, bf16 and
fp32, shared and per-query banks), exact ties, signed zeros, unusual head
shapes and page sizes, zero-length facts, forward order, and the device
error flags."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2607_27090_amd import (IS_DEV_BAD_BLOCK, IS_DEV_BT_SHORT, IS_DEV_CAPACITY,
                                  IS_DEV_ID_RANGE, IS_DEV_SLOT_RANGE, IS_DEV_SRC_RANGE,
                                  is_inject, is_slot_map)
from paper_2607_27090_amd.pipeline import RequestBuffers
from tests import parity
from tests.gpu_harness import Instance, host_emb, log, u16

pytestmark = pytest.mark.gpu


def _ret_case(n, d, k, nq, dt, shared, seed):
    return workloads.TINY.with_(n=n, d_e=d, k=k, nq=nq, emb_dtype=dt, shared_bank=shared,
                                index=100 + seed)


@pytest.mark.parametrize("n,d,k,nq,dt,shared", [
    (1, 8, 1, 1, "f32", True),
    (300, 64, 300, 1, "f32", True),          # k = n: the full permutation
    (16384, 32, 7, 1, "f32", True),          # exactly one full select chunk
    (16385, 32, 7, 1, "f32", True),          # one key into a second chunk
    (20000, 32, 1024, 2, "f32", True),       # largest k, two chunks
    (300000, 16, 1024, 1, "f32", True),      # multi-level candidate merge
    (65536, 16, 1024, 1, "f32", True),       # 4 x 1024 chunk winners: merged by rank
    (65537, 16, 1024, 1, "f32", True),       # 5 x 1024: one list past the rank merge
    (100000, 16, 100, 8, "bf16", True),      # 8 queries per row load, rows of 2 units
    (30000, 1000, 20, 5, "f32", True),       # 4 queries per row load, ragged row, 4 + 1
    (5000, 1024, 100, 3, "bf16", True),      # several queries share each row load
    (2000, 768, 50, 5, "f32", False),        # one bank per query
    (777, 264, 7, 9, "bf16", True),          # ragged d, 9 queries over 2 groups
    (1000, 4096, 10, 2, "f32", True),        # long rows
    (3000, 8, 1, 4, "bf16", False),
    # the single-chunk select's bound from offered wave maxima (k <= 96) and
    # its radix fallback: too few rows to offer k maxima, k at the limit of
    # the offered-maxima bound and one past it
    (100, 32, 40, 1, "f32", True),
    (64, 8, 63, 1, "f32", True),
    (1000, 32, 96, 2, "f32", True),
    (1000, 32, 97, 1, "f32", True),
    (16384, 32, 96, 1, "f32", True),
    (10000, 768, 50, 2, "f32", True),
    # matrix-core scan (shared bf16 bank, >= 32 queries): ragged rows, ragged
    # reduction chunks, partial query tiles and more queries than one tile
    (1000, 64, 10, 32, "bf16", True),
    (257, 72, 5, 33, "bf16", True),
    (70000, 1024, 100, 100, "bf16", True),
    (4099, 200, 64, 300, "bf16", True),
])
def test_retrieve_shapes(n, d, k, nq, dt, shared):
    w = _ret_case(n, d, k, nq, dt, shared, seed=n % 97)
    bank = workloads.make_bank(w, "cuda")
    q = workloads.make_queries(w, "cuda")
    buf = RequestBuffers(n=n, d=d, k=k, nq=nq, emb_dtype=bank.dtype, max_tokens=1)
    buf.retrieve(q, bank, bank_stride=0 if shared else n * d)
    torch.cuda.synchronize()
    gids, gsc = buf.ids.cpu().numpy(), buf.scores.cpu().numpy()
    near = 0
    for r in range(nq):
        qh, odt = host_emb(q[r:r + 1])
        bh, _ = host_emb(bank if shared else bank[r])
        ids_o, _, s_all = oracle.retrieve(qh, bh, n, d, k, 1, 0, odt)
        near += parity.check_ids(gids[r], ids_o[0], s_all[0], n)
        qd = oracle.bf16_to_f64(qh) if odt == oracle.BF16 else qh.astype(np.float64)
        rows = bh[gids[r]]
        rd = oracle.bf16_to_f64(rows) if odt == oracle.BF16 else rows.astype(np.float64)
        parity.check_scores(gsc[r], s_all[0][gids[r]], np.abs(rd * qd).sum(axis=1))
    log(f"retrieve n={n} d={d} k={k} nq={nq} {dt} shared={shared}: near-tie swaps {near}")


def test_retrieve_exact_ties_go_to_lower_id():
    w = _ret_case(4000, 128, 6, 1, "f32", True, seed=1)
    bank = workloads.make_bank(w, "cuda")
    for j in (5, 9, 3000, 3999):
        bank[j] = bank[3]
    q = bank[3:4].clone()
    buf = RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=1, emb_dtype=bank.dtype, max_tokens=1)
    buf.retrieve(q, bank)
    torch.cuda.synchronize()
    assert buf.ids[0, :5].tolist() == [3, 5, 9, 3000, 3999]


@pytest.mark.parametrize("n,k", [(3000, 10), (16384, 40), (700, 700)])
def test_retrieve_many_tied_scores(n, k):
    # a few rows above a block of thousands of exactly tied rows: more tied
    # candidates than the pairwise ranking takes, so the single-chunk select
    # falls back to its general radix path; ties go to the lower id
    d = 16
    bank = torch.zeros(n, d, device="cuda")
    bank[:, 0] = 0.25
    top = {7: 0.75, n // 2: 0.5, n - 1: 0.5, 100: 0.625, 3: 1.0}
    for j, v in top.items():
        bank[j, 0] = v
    q = torch.zeros(1, d, device="cuda")
    q[0, 0] = 1.0
    buf = RequestBuffers(n=n, d=d, k=k, nq=1, emb_dtype=torch.float32, max_tokens=1)
    buf.retrieve(q, bank)
    torch.cuda.synchronize()
    ranked = sorted(range(n), key=lambda j: (-top.get(j, 0.25), j))[:k]
    assert buf.ids[0].tolist() == ranked
    qh, odt = host_emb(q)
    bh, _ = host_emb(bank)
    ids_o, _, _ = oracle.retrieve(qh, bh, n, d, k, 1, 0, odt)
    assert buf.ids[0].tolist() == ids_o[0].tolist()
    assert buf.scores[0].tolist() == [top.get(j, 0.25) for j in ranked]


def test_retrieve_exact_ties_matrix_core_path():
    w = _ret_case(5000, 256, 8, 64, "bf16", True, seed=2)
    bank = workloads.make_bank(w, "cuda")
    for j in (17, 900, 4999):
        bank[j] = bank[11]
    q = workloads.make_queries(w, "cuda")
    q[5] = bank[11]
    buf = RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=bank.dtype, max_tokens=1)
    buf.retrieve(q, bank)
    torch.cuda.synchronize()
    assert buf.ids[5, :4].tolist() == [11, 17, 900, 4999]
    assert len(set(buf.scores[5, :4].tolist())) == 1


def _ranked_against_oracle(q, bank, k):
    nq, d = q.shape
    n = bank.shape[0]
    buf = RequestBuffers(n=n, d=d, k=k, nq=nq, emb_dtype=bank.dtype, max_tokens=1)
    buf.retrieve(q, bank)
    torch.cuda.synchronize()
    gids, gsc = buf.ids.cpu().numpy(), buf.scores.cpu().numpy()
    qh, odt = host_emb(q)
    bh, _ = host_emb(bank)
    ids_o, _, s_all = oracle.retrieve(qh, bh, n, d, k, nq, 0, odt)
    near = 0
    for r in range(nq):
        near += parity.check_ids(gids[r], ids_o[r], s_all[r], n)
        rows = oracle.bf16_to_f64(bh[gids[r]])
        qd = oracle.bf16_to_f64(qh[r])
        parity.check_scores(gsc[r], s_all[r][gids[r]], np.abs(rows * qd).sum(axis=1))
    return gids, near


def test_retrieve_filtered_scan_every_row_survives():
    # matrix-core path with a row sample: the rows after the sample all equal
    # query 0, so for it every one of them scores at or above the sample's
    # k-th best. Every survivor region fills to capacity and the final ranking
    # runs over several chunks; exact ties go to the lower ids.
    g = torch.Generator(device="cuda").manual_seed(91)
    n, d, k, nq, S = 100_000, 64, 50, 32, 16384
    bank = torch.randn(n, d, generator=g, device="cuda")
    bank = (bank / bank.norm(dim=1, keepdim=True)).to(torch.bfloat16)
    v = bank[7].clone()
    bank[S:] = v
    q = (torch.randn(nq, d, generator=g, device="cuda"))
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.bfloat16)
    q[0] = v
    gids, near = _ranked_against_oracle(q, bank, k)
    assert gids[0][0] == 7 and list(gids[0][1:]) == list(range(S, S + k - 1))
    log(f"filtered scan, all rows survive for one query: near-tie swaps {near}")


def test_retrieve_filtered_scan_four_chunk_sample():
    # a bank of 300,000 rows takes a sample of four select chunks (65,536
    # rows), whose chunk winners are merged by rank into the bound; the
    # rows after the sample all equal query 0, so for it every one of them
    # survives the filter, and its ties go to the lower ids
    g = torch.Generator(device="cuda").manual_seed(93)
    n, d, k, nq, S = 300_000, 64, 50, 32, 4 * 16384
    bank = torch.randn(n, d, generator=g, device="cuda")
    bank = (bank / bank.norm(dim=1, keepdim=True)).to(torch.bfloat16)
    v = bank[7].clone()
    bank[S:] = v
    q = (torch.randn(nq, d, generator=g, device="cuda"))
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.bfloat16)
    q[0] = v
    gids, near = _ranked_against_oracle(q, bank, k)
    assert gids[0][0] == 7 and list(gids[0][1:]) == list(range(S, S + k - 1))
    log(f"filtered scan, four-chunk sample, all rows survive for one query: near-tie swaps {near}")


def test_retrieve_filtered_scan_negative_scores():
    # every score is negative, so the sample threshold is below the zero
    # scores of the padding rows of partial tiles: they must not be ranked
    g = torch.Generator(device="cuda").manual_seed(92)
    n, d, k, nq = 40_000, 128, 20, 40
    bank = torch.rand(n, d, generator=g, device="cuda") + 0.01
    bank = (bank / bank.norm(dim=1, keepdim=True)).to(torch.bfloat16)
    q = -(torch.rand(nq, d, generator=g, device="cuda") + 0.01)
    q = (q / q.norm(dim=1, keepdim=True)).to(torch.bfloat16)
    gids, near = _ranked_against_oracle(q, bank, k)
    assert (gids >= 0).all() and (gids < n).all()
    log(f"filtered scan, negative scores: near-tie swaps {near}")


def test_retrieve_ties_across_select_chunks():
    # 30 rows at the start of each of four 16,384-score select chunks share
    # the top score, every other row scores 0: the chunks' winner lists are
    # merged by rank, and the tied keys order by id across the lists
    n, d, k = 4 * 16384, 8, 100
    bank = torch.zeros(n, d, device="cuda")
    top = [c * 16384 + j for c in range(4) for j in range(30)]
    bank[top, 0] = 1.0
    q = torch.zeros(2, d, device="cuda")
    q[:, 0] = 1.0
    buf = RequestBuffers(n=n, d=d, k=k, nq=2, emb_dtype=torch.float32, max_tokens=1)
    buf.retrieve(q, bank)
    torch.cuda.synchronize()
    for r in range(2):
        assert buf.ids[r].tolist() == top[:k]
        assert (buf.scores[r] == 1.0).all()


def test_retrieve_signed_zero_scores_tie():
    # every score is +0 or -0: they are equal, so ranks follow the ids
    n, d = 500, 16
    bank = torch.zeros(n, d, device="cuda")
    bank[::2, 0] = -0.0
    bank[:, 1] = 1.0
    q = torch.zeros(1, d, device="cuda")
    q[0, 0] = 1.0
    buf = RequestBuffers(n=n, d=d, k=20, nq=1, emb_dtype=torch.float32, max_tokens=1)
    buf.retrieve(q, bank)
    torch.cuda.synchronize()
    assert buf.ids[0].tolist() == list(range(20))
    assert (buf.scores == 0).all()


@pytest.mark.parametrize("H,D,L,P,start,lo,hi,k,rev", [
    (8, 128, 2, 1, 37, 0, 9, 12, 1),    # page size 1, zero-length facts
    (3, 64, 3, 32, 5, 1, 40, 9, 1),     # odd head count, page 32
    (1, 16, 1, 16, 0, 0, 3, 30, 0),     # smallest head, forward order
    (2, 256, 2, 16, 130, 16, 48, 5, 1), # widest supported-by-test head
    (8, 512, 1, 8, 3, 1, 5, 4, 1),      # IS_MAX_HEAD_DIM
])
def test_place_inject_shapes(H, D, L, P, start, lo, hi, k, rev):
    w = workloads.TINY.with_(H=H, D=D, L=L, page_size=P, start_pos=start, len_lo=lo,
                             len_hi=hi, k=k, n=200, index=7 + D)
    inst = Instance(w)
    inst.run(reverse_rank=rev)
    if rev:
        inst.check_slot_map()
        floor = inst.check_inject_full()
    else:
        # forward order: compare against the oracle's forward placement
        gids = inst.buf.ids.cpu().numpy()
        lens = inst.store["fact_lens"].cpu().numpy()
        bt = inst.bt.cpu().numpy()
        o = oracle.slot_map(gids, lens, w.start_pos, bt, w.page_size, w.k, 1, w.n, 0,
                            bt.shape[1], inst.max_tokens, 0)
        assert int(inst.buf.m[0]) == int(o["m"][0])
        inst._place = o
        _, floor = inst.check_inject_sampled(frac=1.0)
    log(f"H={H} D={D} L={L} P={P} start={start} rev={rev}: floor-rescued {floor}")


def test_place_inject_largest_k():
    # k = IS_MAX_K facts: the inject workgroup's set-up threads own two facts
    # each of the placement prefix (the first 512 threads busy, the rest
    # empty); zero-length facts mixed in
    w = workloads.TINY.with_(L=2, n=2000, k=1024, len_lo=0, len_hi=3, index=71)
    inst = Instance(w)
    inst.run()
    inst.check_slot_map()
    floor = inst.check_inject_full()
    log(f"k=1024: m={int(inst.buf.m[0])}, floor-rescued {floor}")


def test_place_inject_more_requests_than_cus():
    # 300 requests in one slot-map and one inject launch: one inject
    # workgroup per request, more workgroups than CUs
    w = workloads.TINY.with_(L=2, nq=300, n=200, k=3, len_lo=1, len_hi=5, index=72)
    inst = Instance(w)
    inst.run()
    inst.check_slot_map()
    floor = inst.check_inject_full()
    log(f"nq=300: m total={int(inst.buf.m.sum())}, floor-rescued {floor}")


def _small_setup(max_tokens=64, max_blocks=8):
    w = workloads.TINY.with_(L=2, n=50, k=4, len_lo=2, len_hi=6, index=55)
    inst = Instance(w, max_tokens=max_tokens)
    inst.buf.ids.copy_(torch.tensor([[3, 7, 11, 19]], dtype=torch.int32))
    return w, inst


def _slot_map_call(w, inst, max_tokens, max_blocks, bt=None):
    b = inst.buf
    b.status.zero_()
    bt = inst.bt if bt is None else bt
    is_slot_map(b.ids, inst.store["fact_lens"], w.start_pos, bt, w.page_size, b.slots,
                b.positions, b.m, k=w.k, nq=1, n=w.n, lens_stride=0, max_blocks=max_blocks,
                max_tokens=max_tokens, status=b.status)
    torch.cuda.synchronize()
    return int(b.status.item()), int(b.m.item())


def test_slot_map_flags():
    w, inst = _small_setup()
    st, m = _slot_map_call(w, inst, 64, inst.bt.shape[1])
    assert st == 0 and m > 0
    inst.buf.ids[0, 2] = w.n                       # out of range
    st, m = _slot_map_call(w, inst, 64, inst.bt.shape[1])
    assert st & IS_DEV_ID_RANGE and m == 0
    inst.buf.ids[0, 2] = 11
    st, m = _slot_map_call(w, inst, 3, inst.bt.shape[1])
    assert st & IS_DEV_CAPACITY and m == 0
    st, m = _slot_map_call(w, inst, 64, 1)         # the table ends at the prefix
    assert st & IS_DEV_BT_SHORT and m == 0
    bad = inst.bt.clone()
    bad[0, -3:] = -1
    bad[0, :] = -1
    st, m = _slot_map_call(w, inst, 64, inst.bt.shape[1], bt=bad)
    assert st & IS_DEV_BAD_BLOCK and m == 0


def test_inject_flags_skip_only_the_bad_items():
    w, inst = _small_setup()
    st, m = _slot_map_call(w, inst, 64, inst.bt.shape[1])
    assert st == 0
    b = inst.buf
    L, T, H, D = inst.store["preK"].shape
    # 1) a slot beyond the pool: that token is skipped, the others land
    good_slots = b.slots.clone()
    b.slots[0, 0] = inst.num_slots + 5
    b.status.zero_()
    b.inject(inst.store["preK"], inst.store["V"], w.theta, inst.pk, inst.pv,
             fact_offsets=inst.store["fact_offsets"], fact_lens=inst.store["fact_lens"],
             lens_stride=0)
    torch.cuda.synchronize()
    assert int(b.status.item()) & IS_DEV_SLOT_RANGE
    sl = good_slots[0, :m]
    kv = inst.pk[:, sl].view(torch.int16)
    assert (kv[:, 0] == workloads.SENTINEL_BITS).all()
    assert (kv[:, 1:] != workloads.SENTINEL_BITS).any()
    # 2) a fact whose rows run past the store: its tokens are skipped
    workloads.fill_sentinel(inst.pk)
    b.slots.copy_(good_slots)
    offs = inst.store["fact_offsets"].clone()
    offs[0, 11] = T - 1
    b.status.zero_()
    b.inject(inst.store["preK"], inst.store["V"], w.theta, inst.pk, inst.pv, fact_offsets=offs,
             fact_lens=inst.store["fact_lens"], lens_stride=0)
    torch.cuda.synchronize()
    assert int(b.status.item()) & IS_DEV_SRC_RANGE
    # 3) m = 0 writes nothing
    workloads.fill_sentinel(inst.pk)
    b.m.zero_()
    b.inject(inst.store["preK"], inst.store["V"], w.theta, inst.pk, inst.pv,
             fact_offsets=inst.store["fact_offsets"], fact_lens=inst.store["fact_lens"],
             lens_stride=0)
    torch.cuda.synchronize()
    assert (inst.pk.view(torch.int16) == workloads.SENTINEL_BITS).all()
    # 4) an id out of range skips the whole request
    st, m = _slot_map_call(w, inst, 64, inst.bt.shape[1])
    b.ids[0, 1] = -4
    b.status.zero_()
    b.inject(inst.store["preK"], inst.store["V"], w.theta, inst.pk, inst.pv,
             fact_offsets=inst.store["fact_offsets"], fact_lens=inst.store["fact_lens"],
             lens_stride=0)
    torch.cuda.synchronize()
    assert int(b.status.item()) & IS_DEV_ID_RANGE
    assert (inst.pk.view(torch.int16) == workloads.SENTINEL_BITS).all()


@pytest.mark.parametrize("fused", [True, False])
def test_largest_request_count_per_launch(fused):
    # 65,535 requests in one launch (the largest the library accepts): every
    # per-request offset into ids, slots, positions, m and the block tables
    # is at its largest. Placement of every request is checked against the
    # oracle, retrieval and pages of a sample of requests.
    w = workloads.TINY.with_(n=64, d_e=8, k=1, nq=65535, L=1, H=1, D=16, page_size=4,
                             start_pos=0, len_lo=1, len_hi=2, index=401)
    inst = Instance(w)
    inst.run(fused=fused)
    assert int(inst.buf.status.item()) == 0
    inst.check_slot_map()
    gids = inst.buf.ids.cpu().numpy()
    qh, odt = host_emb(inst.query)
    bh, _ = host_emb(inst.bank)
    rng = np.random.default_rng(401)
    near = 0
    for r in [0, 1, 32767, w.nq - 1] + list(rng.integers(0, w.nq, 60)):
        ids_o, _, s_all = oracle.retrieve(qh[r:r + 1], bh, w.n, w.d_e, w.k, 1, 0, odt)
        near += parity.check_ids(gids[r], ids_o[0], s_all[0], w.n)
    rows, floor = inst.check_inject_sampled(frac=0.05)
    log(f"65,535 requests ({'one launch' if fused else 'separate calls'}): m total "
        f"{int(inst.buf.m.sum())}, {rows} sampled rows, near-tie swaps {near}, floor {floor}")
