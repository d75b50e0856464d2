"""is_retrieve_noalloc (the retrieval entry point for callers that cannot
allocate) against is_retrieve with a caller workspace, called through the C
ABI: two calls in a row on the same GPU, the second with a smaller input,
each checked bit for bit against is_retrieve's ids and scores on the same
inputs, and the ids against the oracle's ranking (near-tie rule)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2607_27090_amd as isl
import workloads
from tests import parity
from tests.gpu_harness import host_emb, log

pytestmark = pytest.mark.gpu


def _raw_stream():
    return torch.cuda.current_stream().cuda_stream


def _with_workspace(q, bank, n, d, k, nq, dt):
    ids = torch.full((nq, k), -7, dtype=torch.int32, device="cuda")
    sc = torch.full((nq, k), float("nan"), dtype=torch.float32, device="cuda")
    size = ctypes.c_size_t(0)
    lib = isl.load_library()
    assert lib.is_retrieve_workspace_size(n, d, k, nq, dt, ctypes.byref(size)) == 0
    ws = torch.empty(max(size.value, 256), dtype=torch.uint8, device="cuda")
    rc = lib.is_retrieve(q.data_ptr(), bank.data_ptr(), n, d, k, ids.data_ptr(), sc.data_ptr(),
                         nq, 0, dt, ws.data_ptr(), ws.numel(), _raw_stream())
    assert rc == 0, lib.is_last_error()
    return ids, sc


def _noalloc(q, bank, n, d, k, nq, dt):
    ids = torch.full((nq, k), -7, dtype=torch.int32, device="cuda")
    sc = torch.full((nq, k), float("nan"), dtype=torch.float32, device="cuda")
    lib = isl.load_library()
    rc = lib.is_retrieve_noalloc(q.data_ptr(), bank.data_ptr(), n, d, k, ids.data_ptr(),
                                 sc.data_ptr(), nq, 0, dt, _raw_stream())
    assert rc == 0, lib.is_last_error()
    return ids, sc


def _case(w, k, variant):
    bank = workloads.make_bank(w, "cuda")
    q = workloads.make_queries(w, "cuda", variant)
    n, d, nq = w.n, w.d_e, w.nq
    dt = isl.IS_DTYPE_F32 if bank.dtype == torch.float32 else isl.IS_DTYPE_BF16
    log(f"noalloc case: n={n} d={d} nq={nq} k={k} dtype={bank.dtype}")
    ids_n, sc_n = _noalloc(q, bank, n, d, k, nq, dt)
    ids_w, sc_w = _with_workspace(q, bank, n, d, k, nq, dt)
    torch.cuda.synchronize()
    assert torch.equal(ids_n, ids_w)
    assert torch.equal(sc_n.view(torch.int32), sc_w.view(torch.int32))
    # and to the oracle's ranking, as for is_retrieve
    qh, odt = host_emb(q)
    bh, _ = host_emb(bank)
    ids_o, _, s_all = oracle.retrieve(qh, bh, n, d, k, nq, 0, odt)
    g = ids_n.cpu().numpy()
    gs = sc_n.cpu().numpy()
    qd = oracle.bf16_to_f64(qh) if odt == oracle.BF16 else qh.astype(np.float64)
    for r in range(nq):
        parity.check_ids(g[r], ids_o[r], s_all[r], n)
        rows = bh[g[r]]
        rd = oracle.bf16_to_f64(rows) if odt == oracle.BF16 else rows.astype(np.float64)
        parity.check_scores(gs[r], s_all[r][g[r]], np.abs(rd * qd[r]).sum(axis=1))


def test_noalloc_equals_workspace_path_two_calls_second_smaller():
    # first: 8 queries over 20,000 bf16 facts (d=1024, k=100; 0.66 MB of
    # scratch); second, smaller: the Llama-3.1-8B retrieval (one query over
    # 10,000 fp32 facts, d=768, k=50; 40 KB). The array keeps the first
    # call's contents, which the second must not depend on.
    _case(workloads.LLAMA70B.with_(n=20_000, nq=8, k=100), 100, 1)
    _case(workloads.LLAMA8B, 50, 3)


def test_noalloc_refuses_sizes_beyond_its_array():
    lib = isl.load_library()
    q = torch.zeros(64, 64, dtype=torch.float32, device="cuda")
    ids = torch.empty(64, 10, dtype=torch.int32, device="cuda")
    rc = lib.is_retrieve_noalloc(q.data_ptr(), q.data_ptr(), 100_000, 64, 10, ids.data_ptr(),
                                 None, 64, 0, isl.IS_DTYPE_F32, _raw_stream())
    assert rc == isl.IS_ERR_WORKSPACE
    assert b"is_retrieve_noalloc" in lib.is_last_error()
