"""GPU parity: the HIP path through the C ABI against the oracle, on the
seeded workloads (full comparison where the oracle can afford it, sampled
rows at the large shapes)."""
import numpy as np
import pytest
import torch

import workloads
from tests.gpu_harness import Instance, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def llama_store():
    w = workloads.LLAMA8B
    log("generating the Llama-3.1-8B-shaped store (n=10000, L=32) on the device")
    store = workloads.make_store(w, "cuda")
    bank = workloads.make_bank(w, "cuda")
    torch.cuda.synchronize()
    yield store, bank
    del store, bank
    torch.cuda.empty_cache()


def test_tiny_full_chain():
    inst = Instance(workloads.TINY)
    inst.run()
    near = inst.check_retrieve()
    inst.check_slot_map()
    floor = inst.check_inject_full()
    log(f"tiny: near-tie rank swaps {near}, floor-rescued K elements {floor}")


@pytest.mark.parametrize("k", [5, 10, 20, 50])
def test_llama8b_full_chain(llama_store, k):
    store, bank = llama_store
    w = workloads.LLAMA8B.with_(k=k)
    inst = Instance(w, store=store, bank=bank, variant=k)
    inst.run()
    near = inst.check_retrieve()
    o = inst.check_slot_map()
    floor = inst.check_inject_full()
    log(f"llama8b k={k}: m={int(o['m'][0])}, near-tie swaps {near}, floor-rescued {floor}")


@pytest.mark.parametrize("k", [5, 50])
def test_llama8b_fused_place_inject(llama_store, k):
    # retrieval, then placement and injection in one launch
    store, bank = llama_store
    w = workloads.LLAMA8B.with_(k=k)
    inst = Instance(w, store=store, bank=bank, variant=100 + k)
    inst.buf.m.fill_(-7)
    inst.run(fused=True)
    near = inst.check_retrieve()
    o = inst.check_slot_map()
    floor = inst.check_inject_full()
    log(f"llama8b fused k={k}: m={int(o['m'][0])}, near-tie swaps {near}, floor-rescued {floor}")


def test_llama8b_deterministic(llama_store):
    store, bank = llama_store
    w = workloads.LLAMA8B
    inst = Instance(w, store=store, bank=bank, variant=3)
    inst.run()
    first_k, first_v = inst.pk.clone(), inst.pv.clone()
    ids = inst.buf.ids.clone()
    workloads.fill_sentinel(inst.pk)
    workloads.fill_sentinel(inst.pv)
    inst.run()
    assert torch.equal(ids, inst.buf.ids)
    assert torch.equal(first_k.view(torch.int16), inst.pk.view(torch.int16))
    assert torch.equal(first_v.view(torch.int16), inst.pv.view(torch.int16))
