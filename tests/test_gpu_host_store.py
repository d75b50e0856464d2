"""The pre-RoPE store kept in pinned host memory (§6.8, App. C: the KV store
offloaded to host DRAM, the retrieved facts streamed over PCIe). The inject
kernel reads the store over the host link; its pages must equal the oracle's
and, bit for bit, those of the same request served from a device store."""
import ctypes

import numpy as np
import pytest
import torch

import workloads
from paper_2607_27090_amd import IS_ERR_INVALID, load_library
from tests.gpu_harness import Instance, log

pytestmark = pytest.mark.gpu

W = workloads.LLAMA8B.with_(n=2000, k=20, L=4, payloads=96, index=21)


def test_inject_from_pinned_host_store_matches_oracle_and_device_store():
    host = workloads.make_store(W, "cuda", host=True)
    assert not host["preK"].is_cuda and host["preK"].is_pinned()
    a = Instance(W, store=host)
    a.run()
    a.check_slot_map()
    floor = a.check_inject_full()
    dev = workloads.make_store(W, "cuda")
    b = Instance(W, store=dev, bank=a.bank)
    b.run()
    assert torch.equal(a.buf.ids, b.buf.ids) and torch.equal(a.buf.slots, b.buf.slots)
    assert torch.equal(a.pk.view(torch.int16), b.pk.view(torch.int16))
    assert torch.equal(a.pv.view(torch.int16), b.pv.view(torch.int16))
    # the one-launch placement + inject reading the same host store
    c = Instance(W, store=host, bank=a.bank)
    c.run(fused=True)
    assert torch.equal(a.buf.m, c.buf.m) and torch.equal(a.buf.slots, c.buf.slots)
    assert torch.equal(a.buf.positions, c.buf.positions)
    assert torch.equal(a.pk.view(torch.int16), c.pk.view(torch.int16))
    assert torch.equal(a.pv.view(torch.int16), c.pv.view(torch.int16))
    log(f"host store: m={int(a.buf.m.sum())} tokens, pages equal to the device-store run "
        f"and to the one-launch path, floor-rescued {floor}")


def test_pageable_host_store_is_rejected_before_launch():
    # m = 0, so even a launch would return before touching the store
    lib = load_library()
    dev = workloads.make_store(W, "cuda")
    L, T, H, D = dev["preK"].shape
    pageable = np.zeros(L * T * H * D, dtype=np.uint16)
    ids = torch.zeros(1, W.k, dtype=torch.int32, device="cuda")
    slots = torch.zeros(1, 8, dtype=torch.int64, device="cuda")
    pos = torch.zeros(1, 8, dtype=torch.int32, device="cuda")
    m = torch.zeros(1, dtype=torch.int32, device="cuda")
    pk = torch.zeros(L, 64, H, D, dtype=torch.bfloat16, device="cuda")
    rc = lib.is_inject(ids.data_ptr(), pageable.ctypes.data, dev["V"].data_ptr(),
                       slots.data_ptr(), pos.data_ptr(), ctypes.c_float(W.theta), pk.data_ptr(),
                       pk.data_ptr(), dev["fact_offsets"].data_ptr(), dev["fact_lens"].data_ptr(),
                       m.data_ptr(), W.k, 1, W.n, 0, 1, 8, L, H, D, T, 64, None, None)
    torch.cuda.synchronize()
    assert rc == IS_ERR_INVALID
    assert b"preK" in lib.is_last_error()
    bt = torch.zeros(1, 8, dtype=torch.int32, device="cuda")
    rc = lib.is_place_inject(ids.data_ptr(), pageable.ctypes.data, dev["V"].data_ptr(),
                             dev["fact_offsets"].data_ptr(), dev["fact_lens"].data_ptr(), 0,
                             bt.data_ptr(), 16, 8, ctypes.c_float(W.theta), None, 0,
                             pk.data_ptr(), pk.data_ptr(), slots.data_ptr(), pos.data_ptr(),
                             m.data_ptr(), W.k, 1, W.n, 0, 1, 8, L, H, D, T, 64, None, None)
    torch.cuda.synchronize()
    assert rc == IS_ERR_INVALID
    assert b"preK" in lib.is_last_error()


def test_host_store_at_the_llama_k50_shape_sampled_against_oracle():
    # the bench's host-store configuration: Llama-3.1-8B KV shapes, 10,000
    # facts aliased onto 2,048 payloads in pinned host memory (~10.5 GB), one
    # request with k=50 placed and injected in one launch over PCIe; checked
    # against the oracle on sampled rows (1% plus every fact's first and last
    # token) and, bit for bit, against the same request from a device store
    w = workloads.LLAMA8B.with_(payloads=2048)
    host = workloads.make_store(w, "cuda", host=True)
    a = Instance(w, store=host)
    a.run(fused=True)
    near = a.check_retrieve()
    a.check_slot_map()
    rows, floor = a.check_inject_sampled(frac=0.01, seed=5)
    pk_host, pv_host = a.pk.clone(), a.pv.clone()
    del host
    dev = workloads.make_store(w, "cuda")
    b = Instance(w, store=dev, bank=a.bank)
    b.run(fused=True)
    assert torch.equal(a.buf.ids, b.buf.ids) and torch.equal(a.buf.slots, b.buf.slots)
    assert torch.equal(pk_host.view(torch.int16), b.pk.view(torch.int16))
    assert torch.equal(pv_host.view(torch.int16), b.pv.view(torch.int16))
    log(f"host store at k=50: m={int(a.buf.m.sum())} tokens, near-tie swaps {near}, {rows} "
        f"sampled rows against the oracle (floor-rescued {floor}), pages equal to the "
        f"device-store run")

