"""Requests in flight together on different streams: every call keeps no state
between invocations, so passes on separate streams with disjoint outputs may
overlap. Two requests write disjoint blocks of one shared page pool and a
third (a batch of four, other k) its own pool, all enqueued before any is
waited for; each is then checked against the oracle in full."""
import numpy as np
import pytest
import torch

import workloads
from tests.gpu_harness import Instance, log

pytestmark = pytest.mark.gpu


def _placed(inst):
    m = inst.buf.m.cpu().numpy()
    s = inst.buf.slots.cpu().numpy()
    return np.concatenate([s[r, :m[r]] for r in range(inst.w.nq)])


def test_three_streams_in_flight():
    w = workloads.LLAMA8B.with_(n=3000, k=20, index=61)
    store = workloads.make_store(w, "cuda")
    bank = workloads.make_bank(w, "cuda")
    a = Instance(w, store=store, bank=bank, variant=1)
    b = Instance(w, store=store, bank=bank, variant=2)
    # one pool for a and b: a keeps blocks [0, nb_a), b moves to [nb_a, nb_a + nb_b)
    nb = a.num_blocks + b.num_blocks
    pk, pv, ns = workloads.make_pages(w, nb, "cuda")
    b.bt = (b.bt + a.num_blocks).contiguous()
    for inst in (a, b):
        inst.pk, inst.pv, inst.num_blocks, inst.num_slots = pk, pv, nb, ns
    wc = workloads.CONCURRENCY.with_(nq=4, k=50, index=62)
    c = Instance(wc, variant=3)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(3)]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    log("three passes enqueued on three streams before any wait")
    for inst, s in zip((a, b, c), streams):
        inst.run(stream=s, sync=False)
    torch.cuda.synchronize()
    for name, inst, other in (("a", a, b), ("b", b, a), ("c", c, None)):
        inst.check_retrieve()
        inst.check_slot_map()
        foreign = None if other is None else _placed(other)
        floor = inst.check_inject_full(foreign_slots=foreign)
        log(f"stream request {name}: m={inst.buf.m.tolist()}, floor-rescued {floor}")
