"""is_inject_rotary on the GPU: the model's own rotary table and pair layout
(§3.3, §6.1) against the oracle, and the default table through the new entry
point bit-identical to is_inject."""
import ctypes

import pytest
import torch

import oracle
import workloads
from paper_2607_27090_amd import (IS_ERR_INVALID, IS_ROPE_INTERLEAVED, is_inject_rotary,
                                  load_library)
from tests.gpu_harness import Instance, log

pytestmark = pytest.mark.gpu

W = workloads.LLAMA8B.with_(n=1500, k=12, L=3, index=31)


def test_default_table_through_rotary_entry_equals_is_inject():
    a = Instance(W)
    a.run()
    b = Instance(W, store=a.store, bank=a.bank)
    b.run(inv_freq=None, interleaved=False)  # same as a.run(): is_inject
    c = Instance(W, store=a.store, bank=a.bank)
    c.run(inv_freq=oracle.default_inv_freq(W.theta, W.D), interleaved=False)
    # the explicit default table differs from the in-kernel one by at most an
    # ulp of the frequency: compare against the oracle, and a against b exactly
    assert torch.equal(a.pk.view(torch.int16), b.pk.view(torch.int16))
    c.check_slot_map()
    floor = c.check_inject_full()
    log(f"default table via is_inject_rotary: oracle parity, floor-rescued {floor}")


@pytest.mark.parametrize("table,interleaved,D", [
    ("llama3.1", False, 128),
    ("default", True, 128),
    ("llama3.1", True, 128),
    ("llama3.1", True, 64),
    ("default", True, 512),
])
def test_rotary_table_and_layout_match_oracle(table, interleaved, D):
    w = W.with_(D=D, H=8 if D <= 128 else 2, index=40 + D + interleaved)
    inst = Instance(w)
    f = workloads.llama31_inv_freq(D, w.theta) if table == "llama3.1" else \
        oracle.default_inv_freq(w.theta, D)
    inst.run(inv_freq=f, interleaved=interleaved)
    inst.check_slot_map()
    floor = inst.check_inject_full()
    log(f"table={table} interleaved={interleaved} D={D}: m={int(inst.buf.m.sum())}, "
        f"floor-rescued {floor}")


def test_rotary_argument_checks():
    inst = Instance(W)
    b = inst.buf
    L, T, H, D = inst.store["preK"].shape
    kw = dict(fact_offsets=inst.store["fact_offsets"], fact_lens=inst.store["fact_lens"], m=b.m,
              k=W.k, nq=1, n=W.n, lens_stride=0, max_tokens=inst.max_tokens, L=L, H=H, D=D,
              T_store=T, num_slots=inst.num_slots, status=b.status)
    with pytest.raises(Exception) as e:
        is_inject_rotary(b.ids, inst.store["preK"], inst.store["V"], b.slots, b.positions,
                         W.theta, inst.pk, inst.pv, pairing=2, **kw)
    assert "pairing" in str(e.value)
    # a misaligned table is refused before anything is enqueued
    raw = torch.zeros(D // 2 + 1, dtype=torch.float64, device="cuda")
    lib = load_library()
    rc = lib.is_inject_rotary(
        b.ids.data_ptr(), inst.store["preK"].data_ptr(), inst.store["V"].data_ptr(),
        b.slots.data_ptr(), b.positions.data_ptr(), ctypes.c_float(W.theta), inst.pk.data_ptr(),
        inst.pv.data_ptr(), inst.store["fact_offsets"].data_ptr(),
        inst.store["fact_lens"].data_ptr(), b.m.data_ptr(), W.k, 1, W.n, 0, 1, inst.max_tokens,
        L, H, D, T, inst.num_slots, raw.data_ptr() + 4, IS_ROPE_INTERLEAVED, None, None)
    torch.cuda.synchronize()
    assert rc == IS_ERR_INVALID
