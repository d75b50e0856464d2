"""The one-launch placement + injection (is_place_inject) against the oracle
and against the two separate calls it replaces (is_slot_map followed by
is_inject_rotary): on the same inputs both must leave bit-identical pages,
slots, positions, m and status words, on unusual shapes, both pair layouts,
every device error condition, mixed batches where only some requests are
bad, and block tables longer than the part each thread loads up front."""
import numpy as np
import pytest
import torch

import workloads
from paper_2607_27090_amd import (IS_DEV_BAD_BLOCK, IS_DEV_BAD_LEN, IS_DEV_BT_SHORT,
                                  IS_DEV_CAPACITY, IS_DEV_ID_RANGE, IS_DEV_SLOT_RANGE,
                                  IS_DEV_SRC_RANGE, IS_ROPE_HALF_SPLIT, IS_ROPE_INTERLEAVED,
                                  is_inject_rotary, is_place_inject, is_slot_map)
from tests.gpu_harness import Instance, log

pytestmark = pytest.mark.gpu


def _outputs(inst, nq, max_tokens):
    mt = max(max_tokens, 1)
    pk, pv = torch.empty_like(inst.pk), torch.empty_like(inst.pv)
    workloads.fill_sentinel(pk)
    workloads.fill_sentinel(pv)
    return dict(slots=torch.full((nq, mt), -1, dtype=torch.int64, device="cuda"),
                positions=torch.full((nq, mt), -1, dtype=torch.int32, device="cuda"),
                m=torch.full((nq,), -7, dtype=torch.int32, device="cuda"),
                status=torch.zeros(1, dtype=torch.int32, device="cuda"), pk=pk, pv=pv)


def _both(inst, *, ids=None, lens=None, offs=None, bt=None, max_tokens=None, max_blocks=None,
          rev=1, inv_freq=None, pairing=IS_ROPE_HALF_SPLIT):
    """Separate calls and the fused call on the same inputs; every output
    must be identical. Returns the fused outputs."""
    w = inst.w
    ids = inst.buf.ids if ids is None else ids
    lens = inst.store["fact_lens"] if lens is None else lens
    offs = inst.store["fact_offsets"] if offs is None else offs
    bt = inst.bt if bt is None else bt
    mt = inst.max_tokens if max_tokens is None else max_tokens
    mb = bt.shape[1] if max_blocks is None else max_blocks
    lens_stride = 0 if lens.shape[0] == 1 else w.n
    preK, V = inst.store["preK"], inst.store["V"]
    L, T, H, D = preK.shape
    a, b = _outputs(inst, w.nq, mt), _outputs(inst, w.nq, mt)
    is_slot_map(ids, lens, w.start_pos, bt, w.page_size, a["slots"], a["positions"], a["m"],
                k=w.k, nq=w.nq, n=w.n, lens_stride=lens_stride, max_blocks=mb, max_tokens=mt,
                reverse_rank=rev, status=a["status"])
    is_inject_rotary(ids, preK, V, a["slots"], a["positions"], w.theta, a["pk"], a["pv"],
                     fact_offsets=offs, fact_lens=lens, m=a["m"], k=w.k, nq=w.nq, n=w.n,
                     lens_stride=lens_stride, reverse_rank=rev, max_tokens=mt, L=L, H=H, D=D,
                     T_store=T, num_slots=inst.num_slots, inv_freq=inv_freq, pairing=pairing,
                     status=a["status"])
    is_place_inject(ids, preK, V, w.theta, b["pk"], b["pv"], b["slots"], b["positions"], b["m"],
                    fact_offsets=offs, fact_lens=lens, start_pos=w.start_pos, block_table=bt,
                    page_size=w.page_size, max_blocks=mb, k=w.k, nq=w.nq, n=w.n,
                    lens_stride=lens_stride, reverse_rank=rev, max_tokens=mt, L=L, H=H, D=D,
                    T_store=T, num_slots=inst.num_slots, inv_freq=inv_freq, pairing=pairing,
                    status=b["status"])
    torch.cuda.synchronize()
    for key in ("status", "m", "slots", "positions"):
        assert torch.equal(a[key], b[key]), key
    for key in ("pk", "pv"):
        assert torch.equal(a[key].view(torch.int16), b[key].view(torch.int16)), key
    return b


def _untouched(out):
    return bool((out["pk"].view(torch.int16) == workloads.SENTINEL_BITS).all() and
                (out["pv"].view(torch.int16) == workloads.SENTINEL_BITS).all())


@pytest.mark.parametrize("H,D,L,P,start,lo,hi,k,rev,pairing", [
    (8, 128, 2, 1, 37, 0, 9, 12, 1, IS_ROPE_HALF_SPLIT),
    (3, 64, 3, 32, 5, 1, 40, 9, 1, IS_ROPE_INTERLEAVED),
    (1, 16, 1, 16, 0, 0, 3, 30, 0, IS_ROPE_HALF_SPLIT),
    (2, 256, 2, 16, 130, 16, 48, 5, 1, IS_ROPE_HALF_SPLIT),
    (8, 512, 1, 8, 3, 1, 5, 4, 1, IS_ROPE_INTERLEAVED),
    (8, 128, 5, 7, 21, 2, 30, 17, 0, IS_ROPE_INTERLEAVED),
])
def test_fused_equals_separate_and_oracle(H, D, L, P, start, lo, hi, k, rev, pairing):
    w = workloads.TINY.with_(H=H, D=D, L=L, page_size=P, start_pos=start, len_lo=lo,
                             len_hi=hi, k=k, n=200, index=300 + D + P)
    inst = Instance(w)
    inst.run(reverse_rank=rev)  # retrieval (and the separate path, into inst's pools)
    interleaved = pairing == IS_ROPE_INTERLEAVED
    # a model rotary table (Llama 3.1-style scaled frequencies) on the interleaved cases
    inv = None
    if interleaved:
        j = np.arange(D // 2, dtype=np.float64)
        inv = w.theta ** (-2.0 * j / D) / np.where(j >= D // 4, 8.0, 1.0)
    tinv = None if inv is None else torch.from_numpy(inv).cuda()
    out = _both(inst, rev=rev, inv_freq=tinv, pairing=pairing)
    assert int(out["status"].item()) == 0 and int(out["m"][0]) > 0
    if rev:
        # the fused path through the request pipeline, checked by the oracle
        workloads.fill_sentinel(inst.pk)
        workloads.fill_sentinel(inst.pv)
        inst.buf.m.fill_(-7)
        inst.run(reverse_rank=rev, inv_freq=inv, interleaved=interleaved, fused=True)
        inst.check_slot_map()
        floor = inst.check_inject_full()
        log(f"fused H={H} D={D} L={L} P={P} start={start}: m={int(out['m'][0])}, "
            f"floor-rescued {floor}")


def test_fused_error_conditions_equal_separate():
    w = workloads.TINY.with_(L=2, n=50, k=4, len_lo=2, len_hi=6, index=355)
    inst = Instance(w, max_tokens=64)
    inst.buf.ids.copy_(torch.tensor([[3, 7, 11, 19]], dtype=torch.int32))
    ids, bt = inst.buf.ids, inst.bt
    lens, offs = inst.store["fact_lens"], inst.store["fact_offsets"]
    L, T, H, D = inst.store["preK"].shape
    out = _both(inst)
    m = int(out["m"][0])
    assert int(out["status"].item()) == 0 and m > 0
    # request-level: skipped as a whole, m = 0, no page written
    bad_ids = ids.clone()
    bad_ids[0, 2] = w.n
    out = _both(inst, ids=bad_ids)
    assert int(out["status"].item()) == IS_DEV_ID_RANGE and int(out["m"][0]) == 0
    assert _untouched(out)
    bad_lens = lens.clone()
    bad_lens[0, 7] = -3
    out = _both(inst, lens=bad_lens)
    assert int(out["status"].item()) == IS_DEV_BAD_LEN and int(out["m"][0]) == 0
    out = _both(inst, max_tokens=m - 1)
    assert int(out["status"].item()) == IS_DEV_CAPACITY and int(out["m"][0]) == 0
    assert _untouched(out)
    out = _both(inst, max_blocks=(w.start_pos + m - 1) // w.page_size)  # one block short
    assert int(out["status"].item()) == IS_DEV_BT_SHORT and int(out["m"][0]) == 0
    last_blk = (w.start_pos + m - 1) // w.page_size
    bad_bt = bt.clone()
    bad_bt[0, last_blk] = -1
    out = _both(inst, bt=bad_bt)
    assert int(out["status"].item()) == IS_DEV_BAD_BLOCK and int(out["m"][0]) == 0
    assert _untouched(out)
    # a negative entry past the last used block, or in the prefix, is not used
    ok_bt = bt.clone()
    ok_bt[0, last_blk + 1:] = -1
    ok_bt[0, :w.start_pos // w.page_size] = -1
    out = _both(inst, bt=ok_bt)
    assert int(out["status"].item()) == 0 and int(out["m"][0]) == m
    # token-level: a block beyond the pool skips its tokens only
    far_bt = bt.clone()
    far_bt[0, w.start_pos // w.page_size] = inst.num_blocks + 3
    out = _both(inst, bt=far_bt)
    assert int(out["status"].item()) == IS_DEV_SLOT_RANGE and int(out["m"][0]) == m
    if last_blk > w.start_pos // w.page_size:
        assert not _untouched(out)
    # fact-level: rows past the store skip that fact's tokens only
    bad_offs = offs.clone()
    bad_offs[0, 11] = T - 1
    out = _both(inst, offs=bad_offs)
    assert int(out["status"].item()) == IS_DEV_SRC_RANGE and int(out["m"][0]) == m
    assert not _untouched(out)
    # an id error wins over everything else, as in the slot map
    out = _both(inst, ids=bad_ids, bt=bad_bt, max_tokens=m - 1)
    assert int(out["status"].item()) == IS_DEV_ID_RANGE and int(out["m"][0]) == 0
    # nothing fits: m = 0 everywhere, the launch still validates
    out = _both(inst, max_tokens=0)
    assert int(out["status"].item()) == IS_DEV_CAPACITY and int(out["m"][0]) == 0
    assert _untouched(out)


def test_fused_mixed_batch_skips_only_the_bad_requests():
    # per-request banks; request 1 has an id out of range, 2 a negative block,
    # 3 too many tokens, 4 a block beyond the pool, 5 a fact past the store
    w = workloads.TINY.with_(L=3, nq=7, shared_bank=False, n=120, k=6, len_lo=3, len_hi=20,
                             index=356)
    inst = Instance(w)
    inst.run()
    base = _both(inst)
    m0 = base["m"].cpu().numpy()
    assert int(base["status"].item()) == 0 and (m0 > 0).all()
    ids = inst.buf.ids.clone()
    ids[1, 0] = -1
    bt = inst.bt.clone()
    bt[2, (w.start_pos + int(m0[2]) - 1) // w.page_size] = -5
    bt[4, w.start_pos // w.page_size] = inst.num_blocks + 1
    lens = inst.store["fact_lens"].clone()
    lens[3, inst.buf.ids[3, 0]] = inst.max_tokens  # alone exceeds the capacity
    offs = inst.store["fact_offsets"].clone()
    offs[5, inst.buf.ids[5, 2]] = inst.store["preK"].shape[1] - 1
    out = _both(inst, ids=ids, bt=bt, lens=lens, offs=offs)
    st = int(out["status"].item())
    assert st == (IS_DEV_ID_RANGE | IS_DEV_BAD_BLOCK | IS_DEV_CAPACITY | IS_DEV_SLOT_RANGE |
                  IS_DEV_SRC_RANGE)
    m = out["m"].cpu().numpy()
    assert m[1] == m[2] == m[3] == 0
    assert m[0] == m0[0] and m[4] == m0[4] and m[5] == m0[5] and m[6] == m0[6]
    # the good requests' pages equal those of the clean batch
    for r in (0, 6):
        sl = base["slots"][r, :int(m0[r])]
        assert torch.equal(out["pk"][:, sl].view(torch.int16), base["pk"][:, sl].view(torch.int16))
        assert torch.equal(out["pv"][:, sl].view(torch.int16), base["pv"][:, sl].view(torch.int16))


def test_fused_long_block_table_beyond_the_preloaded_part():
    # page_size 1: ~3000 blocks per request, more than the 2 x 1024 entries
    # each thread loads before the scan, so the rest is checked after it
    w = workloads.TINY.with_(L=2, page_size=1, n=300, k=64, len_lo=40, len_hi=60, index=357)
    inst = Instance(w)
    inst.run()
    out = _both(inst)
    m = int(out["m"][0])
    assert int(out["status"].item()) == 0 and w.start_pos + m > 2048 + 400
    bad = inst.bt.clone()
    bad[0, w.start_pos + m - 1] = -2          # the last used block, checked after the scan
    out = _both(inst, bt=bad)
    assert int(out["status"].item()) == IS_DEV_BAD_BLOCK and int(out["m"][0]) == 0
    bad = inst.bt.clone()
    bad[0, w.start_pos + 5] = -2              # a preloaded one
    out = _both(inst, bt=bad)
    assert int(out["status"].item()) == IS_DEV_BAD_BLOCK and int(out["m"][0]) == 0
    workloads.fill_sentinel(inst.pk)
    workloads.fill_sentinel(inst.pv)
    inst.run(fused=True)
    inst.check_slot_map()
    inst.check_inject_full()
    log(f"page_size 1: m={m} tokens over {m} blocks")


@pytest.mark.parametrize("case", ["k1024", "nq300"])
def test_fused_large_k_and_many_requests(case):
    if case == "k1024":
        w = workloads.TINY.with_(L=2, n=2000, k=1024, len_lo=0, len_hi=3, index=358)
    else:
        w = workloads.TINY.with_(L=2, nq=300, n=200, k=3, len_lo=1, len_hi=5, index=359)
    inst = Instance(w)
    inst.run()
    _both(inst)
    workloads.fill_sentinel(inst.pk)
    workloads.fill_sentinel(inst.pv)
    inst.run(fused=True)
    inst.check_slot_map()
    floor = inst.check_inject_full()
    log(f"fused {case}: m total={int(inst.buf.m.sum())}, floor-rescued {floor}")
