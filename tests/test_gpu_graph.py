"""The whole request (retrieve -> slot map -> inject) captured once in a HIP
graph and replayed with new queries: every replay must equal an eager run of
the same query (ids, scores, slots, positions, m and both page pools), with
eager work and synchronisation between the replays. Also for the filtered
matrix-core retrieval, whose four kernels share one workspace."""
import pytest
import torch

import workloads
from paper_2607_27090_amd.pipeline import RequestBuffers, run_request
from tests.gpu_harness import log

pytestmark = pytest.mark.gpu


def _setup(w):
    bank = workloads.make_bank(w, "cuda")
    store = workloads.make_store(w, "cuda")
    bt, nb = workloads.make_block_tables(w, "cuda")
    return bank, store, bt, nb


def _pages(w, nb):
    return workloads.make_pages(w, nb, "cuda")[:2]


@pytest.mark.parametrize("fused", [False, True])
def test_request_graph_replays_match_eager(fused):
    # fused: the graph holds retrieve + one place + inject launch, compared
    # with the eager three-call path
    w = workloads.LLAMA8B.with_(n=3000, k=20, L=4, index=51)
    bank, store, bt, nb = _setup(w)
    q_in = workloads.make_queries(w, "cuda", variant=0).clone()
    gbuf = RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=bank.dtype,
                          max_tokens=w.max_tokens)
    gpk, gpv = _pages(w, nb)
    kw = dict(start_pos=w.start_pos, page_size=w.page_size, rope_theta=w.theta)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm-up on the capture stream
        run_request(gbuf, q_in, bank, store, bt, gpk, gpv, fused=fused, **kw)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run_request(gbuf, q_in, bank, store, bt, gpk, gpv, fused=fused, **kw)
    torch.cuda.synchronize()
    for v in (1, 2, 3, 1):
        q = workloads.make_queries(w, "cuda", variant=v)
        workloads.fill_sentinel(gpk)
        workloads.fill_sentinel(gpv)
        q_in.copy_(q)
        g.replay()
        torch.cuda.synchronize()
        ebuf = RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=bank.dtype,
                              max_tokens=w.max_tokens)
        epk, epv = _pages(w, nb)
        run_request(ebuf, q, bank, store, bt, epk, epv, **kw)
        torch.cuda.synchronize()
        for name in ("ids", "scores", "m", "status"):
            assert torch.equal(getattr(gbuf, name), getattr(ebuf, name)), (v, name)
        m = int(ebuf.m[0])
        assert torch.equal(gbuf.slots[:, :m], ebuf.slots[:, :m])
        assert torch.equal(gbuf.positions[:, :m], ebuf.positions[:, :m])
        assert torch.equal(gpk.view(torch.int16), epk.view(torch.int16)), v
        assert torch.equal(gpv.view(torch.int16), epv.view(torch.int16)), v
        log(f"graph replay (fused={fused}), query variant {v}: m={m}, equal to eager")


def test_filtered_retrieval_graph_replays_match_eager():
    w = workloads.TINY.with_(n=60000, d_e=256, k=40, nq=64, emb_dtype="bf16", index=52)
    bank = workloads.make_bank(w, "cuda")
    q_in = workloads.make_queries(w, "cuda", variant=0).clone()
    gbuf = RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=bank.dtype, max_tokens=1)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        gbuf.retrieve(q_in, bank)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        gbuf.retrieve(q_in, bank)
    for v in (1, 2, 1):
        q = workloads.make_queries(w, "cuda", variant=v)
        q_in.copy_(q)
        g.replay()
        torch.cuda.synchronize()
        ebuf = RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=bank.dtype,
                              max_tokens=1)
        ebuf.retrieve(q, bank)
        torch.cuda.synchronize()
        assert torch.equal(gbuf.ids, ebuf.ids) and torch.equal(gbuf.scores, ebuf.scores), v
    log("filtered matrix-core retrieval: graph replays equal to eager")
