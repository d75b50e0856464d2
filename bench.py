"""Benchmark of the InferScale serving-time hot path on one MI355X.

Default (the headline): one step = one request on the Llama-3.1-8B-shaped
workload: exact top-k (k=50) over a 10,000-fact fp32 embedding bank
(d=768), placement + slot map, and the fused gather + RoPE + scatter of the
chosen facts' bf16 K/V (32 layers, 8 KV heads, head dim 128) into a paged
cache with 16-token pages. Every step uses a different query (so different
facts) and a different region of the page pool; all inputs are resident in
HBM before the timed region starts.

--workload selects one of the other seeded shapes (64 users with their own
banks, Llama-3-70B-style KV with 8 queries, a 1M-fact bf16 bank with 256
queries); there a step is one batch of nq requests and `value` is the step
time divided by nq.

Prints one JSON line with µs per request, the inject kernel's achieved HBM
bandwidth against the 8 TB/s peak, and (default workload) the CPU oracle
timed on the host cores for a bounded sample of the same requests.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PCIE_PEAK_GBPS = 64.0     # PCIe 5.0 x16, one direction
HBM_PEAK_GBPS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama8b",
                    choices=["llama8b", "tiny", "concurrency", "llama70b", "retrieval1m"])
    ap.add_argument("--k", type=int, default=None, help="override k (llama8b sweep)")
    ap.add_argument("--streams", type=int, default=1,
                    help="HIP streams the requests are spread over (round robin)")
    ap.add_argument("--detail", action="store_true",
                    help="also time one stream (latency) and each call separately")
    ap.add_argument("--graph", action="store_true", help="also time the request as a HIP graph")
    ap.add_argument("--library-gemm", action="store_true",
                    help="also time the vendor GEMM (torch.matmul, bf16) on the same shared bank "
                         "and one step's queries, as a yardstick for the matrix-core scan")
    ap.add_argument("--no-two-streams", action="store_true",
                    help="skip the two-stream throughput figure (its kernels overlap, which "
                         "per-kernel profiles should not average in)")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip timing each step alone after evicting the caches (1 GiB of writes)")
    ap.add_argument("--store", default="device", choices=["device", "host"],
                    help="where the pre-RoPE K/V store lives: HBM, or pinned host memory "
                         "that the inject kernel reads over PCIe")
    ap.add_argument("--payloads", type=int, default=2048,
                    help="distinct fact payloads of a host store (facts alias onto them)")
    ap.add_argument("--rope", default="default", choices=["default", "llama3.1", "interleaved"],
                    help="rotary table / pair layout of the inject: theta^(-2j/D) half-split "
                         "(is_inject), Llama 3.1's scaled table, or interleaved pairs "
                         "(is_inject_rotary)")
    ap.add_argument("--consumer", action="store_true",
                    help="also time is_paged_scores (attention logits of a query after the "
                         "memory, 4 query heads per KV head) over every layer of each request")
    ap.add_argument("--retriever", default="exact", choices=["exact", "ann"],
                    help="exact top-k (is_retrieve), or the graph-ANN backend (is_ann_build "
                         "once, untimed; is_ann_search per step)")
    ap.add_argument("--beam", type=int, default=None,
                    help="ANN beam width (default: the smallest of 64/128/256 that holds k)")
    ap.add_argument("--width", type=int, default=4, help="ANN beam entries expanded per iteration")
    ap.add_argument("--degree", type=int, default=64, help="ANN graph out-degree")
    ap.add_argument("--seeds", type=int, default=1024, help="ANN search entry points")
    ap.add_argument("--max-iters", type=int, default=512)
    ap.add_argument("--path", default="fused", choices=["fused", "separate"],
                    help="fused: retrieve, then one place + inject launch; separate: retrieve, "
                         "slot map, inject (the other path is timed too and reported beside)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU time budget of each of the oracle baseline's two modes")
    ap.add_argument("--profile-pass", action="store_true",
                    help="for hardware-counter runs: the warm-up and timed steps once each "
                         "(one dispatch of the timed path per step) and a 1 GiB calibration "
                         "copy, nothing else; prints those steps' algorithmic bytes")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the HBM-traffic summary of two rocprofv3 --pmc runs of "
                         "--profile-pass (FETCH_SIZE, then WRITE_SIZE); each directory holds "
                         "the counter CSV and the run's JSON line as bench.json")
    ap.add_argument("--summarize-stats", metavar="DIR",
                    help="print the kernel-duration summary of a rocprofv3 --kernel-trace "
                         "--stats run whose JSON line is DIR/bench.json")
    ap.add_argument("--kernel", default=None,
                    help="kernel name fragment the summary is about (default: the inject "
                         "kernel of the run's path)")
    ap.add_argument("--title", default="", help="title line of the summary")
    ap.add_argument("--include", action="append", default=[],
                    help="kernel name fragment to list besides the library's own kernels "
                         "(repeatable), e.g. the vendor GEMM of --library-gemm")
    ap.add_argument("--cmd", action="append", default=[],
                    help="command that produced the profile (repeatable), quoted in the summary")
    return ap.parse_args()


def main():
    args = parse()
    if args.summarize_traffic:
        print(summarize_traffic(args))
        return
    if args.summarize_stats:
        print(summarize_stats(args))
        return
    if args.profile_pass:
        args.no_two_streams = True
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads
    from paper_2607_27090_amd import (IS_ROPE_HALF_SPLIT, IS_ROPE_INTERLEAVED, is_inject,
                                      is_inject_rotary, is_paged_scores, is_place_inject,
                                      is_slot_map, is_stream_copy)
    from paper_2607_27090_amd.pipeline import AnnIndex, RequestBuffers

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda"
    w = {"llama8b": workloads.LLAMA8B, "tiny": workloads.TINY,
         "concurrency": workloads.CONCURRENCY, "llama70b": workloads.LLAMA70B,
         "retrieval1m": workloads.RETRIEVAL1M}[args.workload]
    default_k = w.k
    if args.k is not None:
        w = w.with_(k=args.k)
    host_store = args.store == "host"
    if host_store and w.payloads is None:
        w = w.with_(payloads=args.payloads)
    nsteps = args.warmup + args.steps
    # requests per slot-map/inject call: the whole batch, except the 1M-fact
    # case whose 256 requests' pages would not fit at once
    wave = 64 if w.nq > 64 else w.nq
    nwaves = w.nq // wave

    t0 = time.time()
    # the paged cache is allocated first, as an engine allocates its KV cache
    # at start-up before a memory store fills up
    region_bytes = 2 * int(1.1 * wave * w.max_blocks) * w.page_size * w.L * w.H * w.D * 2
    R = max(1, min(8, int(60e9 // region_bytes)))
    bts, num_blocks = workloads.make_block_tables(w.with_(nq=R * wave), dev, variant=0)
    bts = bts.view(R, wave, -1)
    pk, pv, num_slots = workloads.make_pages(w, num_blocks, dev)
    bank = workloads.make_bank(w, dev)
    store = workloads.make_store(w, dev, host=host_store)
    queries = torch.stack([workloads.make_queries(w, dev, variant=i) for i in range(nsteps)])
    S = max(1, args.streams)
    # a second buffer set and stream for the two-stream throughput figure
    S_pool = max(S, 2) if (nwaves == 1 and R % 2 == 0 and not args.no_two_streams) else S
    bufs = [RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=bank.dtype,
                           max_tokens=w.max_tokens, device=dev) for _ in range(S_pool)]
    buf = bufs[0]
    ann = None
    if args.retriever == "ann":
        assert w.shared_bank, "the graph-ANN backend indexes one shared bank"
        beam = args.beam or next(b for b in (64, 128, 256) if b >= w.k)
        tb = time.time()
        index = AnnIndex(bank, degree=args.degree, n_seeds=args.seeds)
        torch.cuda.synchronize()
        ann = {"degree": args.degree, "beam": beam, "width": args.width,
               "n_seeds": index.n_seeds, "max_iters": args.max_iters,
               "build_s": round(time.time() - tb, 2)}
        log(f"ANN index: degree {args.degree}, {index.n_seeds} seeds, built in "
            f"{ann['build_s']} s")
        for b in bufs:
            b.ann_iters = torch.zeros(w.nq, dtype=torch.int32, device=dev)
            b.ann_scored = torch.zeros(w.nq, dtype=torch.int32, device=dev)

    def retrieve(q, b):
        if ann is None:
            b.retrieve(q, bank, bank_stride=0 if w.shared_bank else w.n * w.d_e)
        else:
            index.search(q, b.ids, nq=w.nq, k=w.k, beam=ann["beam"], width=ann["width"],
                         max_iters=ann["max_iters"], out_scores=b.scores, out_iters=b.ann_iters,
                         out_scored=b.ann_scored)

    lens, offs = store["fact_lens"], store["fact_offsets"]
    lens_stride = 0 if lens.shape[0] == 1 else w.n
    L, T, H, D = store["preK"].shape
    torch.cuda.synchronize()
    log(f"setup {time.time() - t0:.1f}s: {w.name}, store T={T} rows "
        f"({2 * store['preK'].numel() * 2 / 1e9:.1f} GB), pages {num_slots} slots, {R} regions")
    # requests that reuse a page region are always on the same stream
    assert S == 1 or (nwaves == 1 and R % S == 0), "concurrent requests would share page regions"

    def place(i, j, b=None):
        b = buf if b is None else b
        sl = slice(j * wave, (j + 1) * wave)
        ls = lens if lens_stride == 0 else lens[sl]
        is_slot_map(b.ids[sl], ls, w.start_pos, bts[(i * nwaves + j) % R], w.page_size,
                    b.slots[sl], b.positions[sl], b.m[sl], k=w.k, nq=wave, n=w.n,
                    lens_stride=lens_stride, max_blocks=bts.shape[-1], max_tokens=w.max_tokens,
                    status=b.status)

    rope_table = None
    if args.rope == "llama3.1":
        rope_table = torch.from_numpy(workloads.llama31_inv_freq(w.D, w.theta)).to(dev)
    pairing = IS_ROPE_INTERLEAVED if args.rope == "interleaved" else IS_ROPE_HALF_SPLIT
    fused = args.path == "fused"

    def inject(j, b=None):
        b = buf if b is None else b
        sl = slice(j * wave, (j + 1) * wave)
        ls = lens if lens_stride == 0 else lens[sl]
        os_ = offs if lens_stride == 0 else offs[sl]
        kw = dict(fact_offsets=os_, fact_lens=ls, m=b.m[sl], k=w.k, nq=wave, n=w.n,
                  lens_stride=lens_stride, max_tokens=w.max_tokens, L=L, H=H, D=D,
                  T_store=T, num_slots=num_slots, status=b.status)
        if args.rope == "default":
            is_inject(b.ids[sl], store["preK"], store["V"], b.slots[sl], b.positions[sl],
                      w.theta, pk, pv, **kw)
        else:
            is_inject_rotary(b.ids[sl], store["preK"], store["V"], b.slots[sl], b.positions[sl],
                             w.theta, pk, pv, inv_freq=rope_table, pairing=pairing, **kw)

    def place_inject(i, j, b=None):
        b = buf if b is None else b
        sl = slice(j * wave, (j + 1) * wave)
        ls = lens if lens_stride == 0 else lens[sl]
        os_ = offs if lens_stride == 0 else offs[sl]
        is_place_inject(b.ids[sl], store["preK"], store["V"], w.theta, pk, pv, b.slots[sl],
                        b.positions[sl], b.m[sl], fact_offsets=os_, fact_lens=ls,
                        start_pos=w.start_pos, block_table=bts[(i * nwaves + j) % R],
                        page_size=w.page_size, max_blocks=bts.shape[-1], k=w.k, nq=wave, n=w.n,
                        lens_stride=lens_stride, max_tokens=w.max_tokens, L=L, H=H, D=D,
                        T_store=T, num_slots=num_slots, inv_freq=rope_table, pairing=pairing,
                        status=b.status)

    def after_retrieve(i, b=None, use_fused=None):
        """Placement and injection of step i's requests."""
        for j in range(nwaves):
            if fused if use_fused is None else use_fused:
                place_inject(i, j, b)
            else:
                place(i, j, b)
                inject(j, b)

    def step(i, b=None, use_fused=None):
        b = buf if b is None else b
        retrieve(queries[i], b)
        after_retrieve(i, b, use_fused)

    main_stream = torch.cuda.current_stream()
    streams = [main_stream] + [torch.cuda.Stream() for _ in range(S_pool - 1)]

    def timed(nstreams, use_fused=None):
        """K steps spread round robin over nstreams streams, bracketed by
        events on the main stream that every other stream waits on and is
        waited for."""
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(main_stream)
        for s_ in streams[1:nstreams]:
            s_.wait_event(ev0)
        for i in range(args.warmup, nsteps):
            si = (i - args.warmup) % nstreams
            with torch.cuda.stream(streams[si]):
                step(i, bufs[si], use_fused)
        for s_ in streams[1:nstreams]:
            main_stream.wait_stream(s_)
        ev1.record(main_stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1)

    # ---- official timed region: K steps -----------------------------------------
    for i in range(args.warmup):
        with torch.cuda.stream(streams[i % S]):
            step(i, bufs[i % S])
    # the extra stream and buffer set of the two-stream figure are warmed up
    # too (a stream's first launches carry one-time queue set-up)
    for si in range(S, S_pool):
        for i in range(2):
            with torch.cuda.stream(streams[si]):
                step(i, bufs[si])
    torch.cuda.synchronize()
    # ---- warm steady state: the K steps back to back ----------------------------
    # (the bank and the placement arrays stay in the 256 MB Infinity Cache
    # from one request to the next)
    t_host = time.perf_counter()
    total_ms = timed(S)
    wall = time.perf_counter() - t_host
    warm_ms_per_step = total_ms / args.steps
    log(f"warm: {args.steps} steps over {S} stream(s): {total_ms:.3f} ms GPU "
        f"({wall * 1e3:.3f} ms host wall), {warm_ms_per_step * 1e3 / w.nq:.2f} us/request")

    if args.profile_pass:
        profile_pass_report(args, w, nsteps, nwaves, fused, queries, retrieve, place, bank,
                            buf, dev, torch, RequestBuffers, is_stream_copy)
        return

    # ---- official timed region: the same K steps, each from cold caches --------
    # Before each step (untimed) 1 GiB of writes evicts the bank, the
    # placement arrays and any page lines from the Infinity Cache and the
    # L2s, as the model's own layers would between two requests of a serving
    # engine. The flushes and steps are enqueued back to back (the host runs
    # ahead of the GPU, as an engine's does, so no launch waits for Python);
    # an event pair brackets each step and one synchronize ends the region.
    # `value` is the median step. A second pass of the same cold steps puts a
    # third event between the retrieval and the inject, for the retrieval's
    # share; it is kept out of the first pass because an event recorded
    # between two kernels holds the second one back by a few microseconds
    # (cold_split_pass_us_per_step_median shows by how much).
    cold, cold_ret, cold_split = [], [], []
    if not args.no_cold:
        flush = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        for split in (False, True):
            evs = []
            torch.cuda.synchronize()
            for i in range(args.warmup, nsteps):
                flush.fill_(i & 0xFF)
                a, m_, b = (torch.cuda.Event(enable_timing=True) for _ in range(3))
                a.record()
                retrieve(queries[i], buf)
                if split:
                    m_.record()
                after_retrieve(i, buf)
                b.record()
                evs.append((a, m_, b))
            torch.cuda.synchronize()
            for a, m_, b in evs:
                if split:
                    cold_ret.append(a.elapsed_time(m_))
                    cold_split.append(a.elapsed_time(b))
                else:
                    cold.append(a.elapsed_time(b))
        del flush
        log(f"cold: median {statistics.median(cold) * 1e3 / w.nq:.2f} us/request over "
            f"{len(cold)} steps (with an event after the retrieval: "
            f"{statistics.median(cold_split) * 1e3 / w.nq:.2f}, retrieval "
            f"{statistics.median(cold_ret) * 1e3:.2f} us/step)")
    ms_per_step = statistics.median(cold) if cold else warm_ms_per_step

    def pcts(xs):
        xs = sorted(xs)

        def at(p_):
            return xs[min(len(xs) - 1, int(round(p_ * (len(xs) - 1))))]
        return {"p10": round(at(0.1), 2), "p50": round(at(0.5), 2), "p90": round(at(0.9), 2),
                "mean": round(statistics.fmean(xs), 2)}
    # throughput with two requests in flight (requests alternate between two
    # streams, each with its own buffers and page regions)
    two_ms = None
    if S == 1 and S_pool >= 2:
        two_ms = timed(2) / args.steps
        log(f"two streams: {two_ms * 1e3 / w.nq:.1f} us per request")
    # the other path (separate slot map + inject, or the fused launch), same
    # steps, one stream, after its own warm-up
    for i in range(2):
        step(i, buf, not fused)
    other_ms = timed(S, not fused) / args.steps
    log(f"{'separate calls' if fused else 'fused place + inject'}: "
        f"{other_ms * 1e3 / w.nq:.1f} us per request")

    # ---- inject kernel alone: the same K requests' injects back to back -------
    # (their retrieval -- and, on the separate path, slot maps -- are
    # recomputed untimed into one buffer set per step, so only inject (or
    # place + inject) launches sit between the two events)
    sets = [RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=bank.dtype,
                           max_tokens=w.max_tokens, device=dev, workspace=buf.workspace)
            for _ in range(args.steps)]
    for si, i in enumerate(range(args.warmup, nsteps)):
        if ann is not None:
            sets[si].ann_iters = torch.zeros(w.nq, dtype=torch.int32, device=dev)
            sets[si].ann_scored = torch.zeros(w.nq, dtype=torch.int32, device=dev)
        retrieve(queries[i], sets[si])
        if not fused:
            for j in range(nwaves):
                place(i, j, sets[si])
    torch.cuda.synchronize()
    ei0, ei1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ei0.record()
    for si, i in enumerate(range(args.warmup, nsteps)):
        for j in range(nwaves):
            if fused:
                place_inject(i, j, sets[si])
            else:
                inject(j, sets[si])
    ei1.record()
    torch.cuda.synchronize()
    inj_launch_ms = ei0.elapsed_time(ei1) / (args.steps * nwaves)
    log(f"inject alone: {inj_launch_ms * 1e3:.1f} us per launch")

    # ---- the same launches with each request's blocks in a small pool ----------
    # (a side figure for how the pages' spread over the pool sets the inject's
    # rate: the timed steps draw each request's blocks at random from one of R
    # regions of a pool of 1.1 x R x max_blocks blocks; here they come from a
    # pool of 1.1 x max_blocks, as in the tests)
    dense_pool = None
    if fused and w.nq == 1 and not host_store and args.rope == "default":
        dbt, dnb = workloads.make_block_tables(w, dev, variant=1)
        dpk, dpv, dns = workloads.make_pages(w, dnb, dev)
        # own placement outputs: the timed steps' ones stay for the parity check
        d_slots = torch.empty(1, w.max_tokens, dtype=torch.int64, device=dev)
        d_pos = torch.empty(1, w.max_tokens, dtype=torch.int32, device=dev)
        d_m = torch.empty(len(sets), dtype=torch.int32, device=dev)
        d_status = torch.zeros(1, dtype=torch.int32, device=dev)

        def dense_launch(si):
            is_place_inject(sets[si].ids, store["preK"], store["V"], w.theta, dpk, dpv, d_slots,
                            d_pos, d_m[si:si + 1], fact_offsets=offs, fact_lens=lens,
                            start_pos=w.start_pos, block_table=dbt, page_size=w.page_size,
                            max_blocks=dbt.shape[-1], k=w.k, nq=1, n=w.n, lens_stride=lens_stride,
                            max_tokens=w.max_tokens, L=L, H=H, D=D, T_store=T, num_slots=dns,
                            status=d_status)
        for si in range(min(2, len(sets))):
            dense_launch(si)
        ed0, ed1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ed0.record()
        for si in range(len(sets)):
            dense_launch(si)
        ed1.record()
        torch.cuda.synchronize()
        assert int(d_status.item()) == 0, "device status flags raised"
        d_ms = ed0.elapsed_time(ed1) / args.steps
        dm = d_m.cpu().tolist()
        d_bytes = statistics.fmean(
            workloads.inject_algorithmic_bytes(w, m) + 12 * m for m in dm)
        d_gbps = d_bytes / (d_ms * 1e-3) / 1e9
        dense_pool = {"pool_GB": round(2 * dpk.numel() * 2 / 1e9, 2),
                      "timed_steps_pool_GB": round(2 * pk.numel() * 2 / 1e9, 2),
                      "inject_launch_us": round(d_ms * 1e3, 2), "GBps": round(d_gbps, 1),
                      "frac_of_peak": round(d_gbps / HBM_PEAK_GBPS, 4)}
        del dpk, dpv, d_slots, d_pos
        log(f"inject with the blocks in a {dense_pool['pool_GB']} GB pool: "
            f"{dense_pool['inject_launch_us']} us per launch, {dense_pool['frac_of_peak']} of peak")

    # ---- ANN: the search alone, the exact retrieval alone, recall ------------
    if ann is not None:
        ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ea.record()
        for si, i in enumerate(range(args.warmup, nsteps)):
            retrieve(queries[i], sets[si])
        eb.record()
        torch.cuda.synchronize()
        search_ms = ea.elapsed_time(eb) / args.steps
        exact = RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=bank.dtype,
                               max_tokens=1, device=dev)
        hits, ex_ms = 0, []
        for si, i in enumerate(range(args.warmup, nsteps)):
            xa, xb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            xa.record()
            exact.retrieve(queries[i], bank)
            xb.record()
            torch.cuda.synchronize()
            ex_ms.append(xa.elapsed_time(xb))
            got, want = sets[si].ids.cpu().tolist(), exact.ids.cpu().tolist()
            hits += sum(len(set(a) & set(b)) for a, b in zip(got, want))
        row_bytes = w.d_e * bank.element_size()
        scored = statistics.fmean(float(b.ann_scored.double().mean()) for b in sets)
        iters = statistics.fmean(float(b.ann_iters.double().mean()) for b in sets)
        # rows read by the search + neighbour lists + the seed scan, per launch
        ann_bytes = w.nq * (scored * row_bytes + iters * ann["width"] * args.degree * 4) \
            + ann["n_seeds"] * row_bytes
        ann.update({
            "recall_at_k": round(hits / (args.steps * w.nq * w.k), 4),
            "iters_mean": round(iters, 1), "rows_read_per_query": round(scored, 1),
            "search_us": round(search_ms * 1e3, 1),
            "exact_retrieve_us": round(statistics.median(ex_ms) * 1e3, 1),
            "search_bytes_per_launch": round(ann_bytes),
            "search_GBps": round(ann_bytes / (search_ms * 1e-3) / 1e9, 1),
        })
        log(f"ANN: recall@{w.k} {ann['recall_at_k']}, {iters:.1f} iterations, {scored:.0f} rows "
            f"per query; search {ann['search_us']} us vs exact {ann['exact_retrieve_us']} us "
            f"per launch; {ann['search_GBps']} GB/s")
        if not args.no_cpu_baseline:
            ann["cpu_baseline"] = ann_cpu_baseline(w, bank, index, queries[args.warmup], ann,
                                                   args, torch)

    # ---- optional: the consumer of the pages, every layer of every request ---
    consumer = None
    if args.consumer and nwaves == 1:
        Hq = 4 * w.H
        gq = torch.Generator(device=dev).manual_seed(99)
        qc = torch.randn(w.nq, Hq, w.D, generator=gq, device=dev).to(torch.bfloat16)
        sc = torch.empty(w.nq, Hq, w.max_tokens, device=dev)
        qpos = [(sets[si].m + w.start_pos).to(torch.int32) for si in range(args.steps)]
        ec0, ec1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ec0.record()
        for si, i in enumerate(range(args.warmup, nsteps)):
            for layer in range(w.L):
                is_paged_scores(qc, qpos[si], pk, layer, bts[(i * nwaves) % R], w.page_size,
                                w.start_pos, sets[si].m, sc, nq=w.nq, Hq=Hq, H=H, D=D, L=L,
                                num_slots=num_slots, max_blocks=bts.shape[-1],
                                max_tokens=w.max_tokens, rope_theta=w.theta,
                                status=sets[si].status)
        ec1.record()
        torch.cuda.synchronize()
        cons_ms = ec0.elapsed_time(ec1) / (args.steps * w.L)
        cons_bytes = statistics.fmean(int(b.m.sum()) for b in sets) * (H * D * 2 + Hq * 4)
        consumer = {"us_per_layer": round(cons_ms * 1e3, 2), "query_heads": Hq,
                    "GBps": round(cons_bytes / (cons_ms * 1e-3) / 1e9, 1)}
        log(f"consumer: {cons_ms * 1e3:.1f} us per layer, {consumer['GBps']} GB/s")
    latency_ms = None
    if args.detail and S > 1:
        latency_ms = timed(1) / args.steps
        log(f"one stream: {latency_ms * 1e3:.1f} us/step")

    # ---- per-request latency spread: the same K steps back to back with one
    # event at each step boundary (the steps still queue behind each other)
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    bounds[0].record()
    for si, i in enumerate(range(args.warmup, nsteps)):
        step(i)
        bounds[si + 1].record()
    torch.cuda.synchronize()
    latency_pct = pcts(bounds[j].elapsed_time(bounds[j + 1]) * 1e3 / w.nq
                       for j in range(args.steps))
    log(f"warm per-request latency: p10 {latency_pct['p10']} p50 {latency_pct['p50']} "
        f"p90 {latency_pct['p90']} us")
    cold_pct = pcts(c * 1e3 / w.nq for c in cold) if cold else None

    # ---- instrumented pass (--detail): per-call events, one stream --------------
    per = {"retrieve": [], "slot_map": [], "inject": [], "step": []}
    if fused:
        per = {"retrieve": [], "place_inject": [], "step": []}
    recs = []
    for i in (range(args.warmup, nsteps) if args.detail else ()):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2 + 2 * nwaves)]
        e[0].record()
        retrieve(queries[i], buf)
        e[1].record()
        for j in range(nwaves):
            if fused:
                e[2 + 2 * j].record()
                place_inject(i, j)
            else:
                place(i, j)
                e[2 + 2 * j].record()
                inject(j)
            e[3 + 2 * j].record()
        recs.append(e)
    torch.cuda.synchronize()
    for e in recs:
        per["retrieve"].append(e[0].elapsed_time(e[1]))
        prev, sm, inj = e[1], 0.0, 0.0
        for j in range(nwaves):
            sm += prev.elapsed_time(e[2 + 2 * j])
            inj += e[2 + 2 * j].elapsed_time(e[3 + 2 * j])
            prev = e[3 + 2 * j]
        if fused:
            per["place_inject"].append(inj)
        else:
            per["slot_map"].append(sm)
            per["inject"].append(inj)
        per["step"].append(e[0].elapsed_time(e[-1]))
    # placed tokens per step
    m_steps = [int(b.m.sum()) for b in sets]
    assert all(int(b.status.item()) == 0 for b in sets + bufs), "device status flags raised"
    inj_bytes = [workloads.inject_algorithmic_bytes(w, m) for m in m_steps]
    if fused:
        # the fused launch also writes each placed token's slot and position
        inj_bytes = [b_ + 12 * m for b_, m in zip(inj_bytes, m_steps)]
    # algorithmic bytes per inject launch / mean launch duration (timed region)
    achieved = statistics.fmean(inj_bytes) / nwaves / (inj_launch_ms * 1e-3) / 1e9
    ret_ms = statistics.fmean(per["retrieve"]) if per["retrieve"] else None
    scan_bytes = workloads.scan_algorithmic_bytes(w)
    scan_flop = 2.0 * w.n * w.d_e * w.nq
    if args.detail:
        log("per-call mean us: " + ", ".join(f"{k} {statistics.fmean(v) * 1e3:.1f}"
                                           for k, v in per.items()))
    log(f"inject: mean m={statistics.fmean(m_steps):.0f} tokens/step, "
        f"{statistics.fmean(inj_bytes) / 1e6:.1f} MB/step, {achieved:.0f} GB/s per launch")

    # ---- optional: the vendor GEMM on the same bank and queries -----------------
    # (dense scores [n][nq] in bf16, no top-k: a yardstick for the scan alone)
    library_gemm = None
    if args.library_gemm and w.shared_bank and bank.dtype == torch.bfloat16:
        qt = queries[args.warmup].reshape(w.nq, w.d_e).t().contiguous()
        bank2 = bank.reshape(w.n, w.d_e)
        gout = torch.empty(w.n, w.nq, dtype=torch.bfloat16, device=dev)
        for _ in range(3):
            torch.matmul(bank2, qt, out=gout)
        ge = [torch.cuda.Event(enable_timing=True) for _ in range(2 * args.steps)]
        for j in range(args.steps):
            ge[2 * j].record()
            torch.matmul(bank2, qt, out=gout)
            ge[2 * j + 1].record()
        torch.cuda.synchronize()
        g_ms = statistics.median(ge[2 * j].elapsed_time(ge[2 * j + 1]) for j in range(args.steps))
        library_gemm = {"what": "torch.matmul(bank [n][d], queries^T [d][nq]) -> bf16 [n][nq]",
                        "us_median": round(g_ms * 1e3, 1),
                        "TFLOPs": round(scan_flop / (g_ms * 1e-3) / 1e12, 1),
                        "bank_GBps": round(scan_bytes / (g_ms * 1e-3) / 1e9, 1)}
        del gout
        log(f"library GEMM on the same bank: {library_gemm['us_median']} us, "
            f"{library_gemm['TFLOPs']} TFLOP/s")

    # ---- optional: the same request captured as a HIP graph --------------------
    graph_us = None
    if args.graph and nwaves == 1:
        qbuf = queries[0].clone()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            retrieve(qbuf, buf)
            after_retrieve(0, buf)
        torch.cuda.current_stream().wait_stream(s)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            retrieve(qbuf, buf)
            after_retrieve(0, buf)
        torch.cuda.synchronize()
        times = []
        for i in range(args.warmup, nsteps):
            qbuf.copy_(queries[i])
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            g.replay()
            b.record()
            times.append((a, b))
        torch.cuda.synchronize()
        graph_us = statistics.median(a.elapsed_time(b) for a, b in times) * 1e3
        log(f"graph replay median {graph_us:.1f} us/step")

    # ---- copy ceiling: the library's streaming copy (C0) -----------------------
    # at the size of one inject launch (half its bytes read, half written)
    # and at 1 GiB, each timed as the mean of back-to-back launches; torch's
    # own copy of 1 GiB beside them
    def copy_rate(nbytes, reps, fn):
        nbytes = max(16, nbytes // 16 * 16)
        src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        fn(dst, src)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn(dst, src)
        b.record()
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / reps
        del src, dst
        return 2 * nbytes / (us * 1e-6) / 1e9, us

    half_inject = int(statistics.fmean(inj_bytes) / nwaves / 2)
    c0_gbps, c0_us = copy_rate(half_inject, 20, lambda d_, s_: is_stream_copy(d_, s_))
    c0_1g_gbps, _ = copy_rate(1 << 30, 5, lambda d_, s_: is_stream_copy(d_, s_))
    torch_gbps, _ = copy_rate(1 << 30, 5, lambda d_, s_: d_.copy_(s_))
    copy_gbps = c0_gbps
    log(f"C0 copy of {2 * half_inject / 1e6:.1f} MB: {c0_gbps:.0f} GB/s ({c0_us:.1f} us); "
        f"1 GiB: C0 {c0_1g_gbps:.0f} GB/s, torch {torch_gbps:.0f} GB/s")
    # with the store in host memory: a plain pinned-host -> device copy of
    # 1 GiB, the practical ceiling of the host link in this process
    pcie_gbps = None
    if host_store:
        hsrc = torch.empty(1 << 30, dtype=torch.uint8, pin_memory=True)
        ddst = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        ddst.copy_(hsrc, non_blocking=True)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(3):
            ddst.copy_(hsrc, non_blocking=True)
        b.record()
        torch.cuda.synchronize()
        pcie_gbps = 3 * (1 << 30) / (a.elapsed_time(b) * 1e-3) / 1e9
        del hsrc, ddst

    # ---- CPU baseline: the oracle on the host for a bounded sample ------------
    cpu = None
    if not args.no_cpu_baseline and not host_store and ann is None:
        cpu = cpu_baseline(w, bank, store, queries, bts, args, torch,
                           gpu={"sets": sets, "pk": pk, "pv": pv, "graph": args.graph})

    # HBM traffic of the timed kernel from the counter runs of the same bench
    # command (profiles/), with that run's own algorithmic bytes and ratio
    traffic = (measured_traffic(args.workload, fused)
               if w.k == default_k and args.rope == "default" and not host_store else None)

    out = {
        "metric": "µs per request (retrieve+RoPE-inject) at k=50; inject HBM GB/s vs peak",
        "value": round(ms_per_step * 1e3 / w.nq, 3),
        "unit": "us/request",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded N(0,1) bf16 pre-RoPE K/V, unit-norm embeddings)",
        "config": {
            "workload": (f"{w.name}: KV L={w.L} H={w.H} D={w.D} bf16; {w.n} facts per bank "
                         f"({'shared' if w.shared_bank else 'one per request'}) of "
                         f"U[{w.len_lo},{w.len_hi}] tokens; d_e={w.d_e} {w.emb_dtype}"
                         f"{' clustered' if w.clustered else ''}; {w.nq} request(s) per step; "
                         f"k={w.k}; page {w.page_size}; theta {w.theta:g}; "
                         f"start_pos {w.start_pos}"),
            "k": w.k, "n": w.n, "nq": w.nq, "kv_dtype": "bf16", "emb_dtype": w.emb_dtype,
            "mean_m_tokens_per_step": round(statistics.fmean(m_steps), 1),
            "rope": {"default": f"theta^(-2j/D), pairs (j, j+D/2)",
                     "llama3.1": "Llama 3.1 scaled table, pairs (j, j+D/2)",
                     "interleaved": "theta^(-2j/D), pairs (2j, 2j+1)"}[args.rope],
            "retriever": ("exact" if ann is None else
                          f"graph ANN (degree {ann['degree']}, beam {ann['beam']}, "
                          f"width {ann['width']}, {ann['n_seeds']} seeds)"),
            "store": ("pinned host memory, read over PCIe "
                      f"({w.payloads} payloads, {2 * store['preK'].numel() * 2 / 1e9:.1f} GB)"
                      if host_store else "HBM"),
        },
        "path": ("retrieve, then placement + slot map + inject in one launch" if fused
                 else "retrieve, slot map, inject (three calls)"),
        ("separate_calls_us_per_request" if fused else "fused_us_per_request"):
            round(other_ms * 1e3 / w.nq, 3),
        "streams": S,
        "throughput_2_streams_us_per_request": (None if two_ms is None
                                                else round(two_ms * 1e3 / w.nq, 3)),
        "inject_launch_us": round(inj_launch_ms * 1e3, 2),
        "inject_small_pool": dense_pool,
        "per_call_us": ({k: round(statistics.fmean(v) * 1e3, 2) for k, v in per.items()}
                        if args.detail else None),
        "latency_us_per_step": None if latency_ms is None else round(latency_ms * 1e3, 3),
        "timing": ("value and ms_per_step: median of the K steps, each from cold caches "
                   "(1 GiB of writes enqueued before it, untimed)" if cold else
                   "value and ms_per_step: K steps back to back (warm caches)"),
        "cold_us_per_request": cold_pct,
        "cold_retrieve_us_per_step_median": (round(statistics.median(cold_ret) * 1e3, 2)
                                             if cold else None),
        "cold_split_pass_us_per_step_median": (round(statistics.median(cold_split) * 1e3, 2)
                                               if cold else None),
        "warm_us_per_request": round(warm_ms_per_step * 1e3 / w.nq, 3),
        "warm_us_per_request_percentiles": latency_pct,
        "graph_step_us_median": None if graph_us is None else round(graph_us, 2),
        "inject_GBps": round(achieved, 1),
        "retrieve": None if ret_ms is None or ann is not None else {
            "us": round(ret_ms * 1e3, 2), "bank_bytes": scan_bytes,
            "GBps": round(scan_bytes / (ret_ms * 1e-3) / 1e9, 1),
            "TFLOPs": round(scan_flop / (ret_ms * 1e-3) / 1e12, 2)},
        "library_gemm": library_gemm,
        "copy_ceiling_GBps": round(copy_gbps, 1),
        "copy_ceiling": {
            "kernel": "is_stream_copy (non-temporal 16-byte grid-stride copy)",
            "bytes_moved": 2 * (half_inject // 16 * 16), "GBps": round(c0_gbps, 1),
            "us": round(c0_us, 2), "GBps_1GiB": round(c0_1g_gbps, 1),
            "torch_copy_GBps_1GiB": round(torch_gbps, 1),
            "inject_frac_of_ceiling": round(achieved / c0_gbps, 4)},
        "pcie_copy_ceiling_GBps": None if pcie_gbps is None else round(pcie_gbps, 1),
        "consumer": consumer,
        "ann": ann,
        "roofline": {
            "bound": "hbm",
            "kernel": "inject_kernel (place + inject)" if fused else "inject_kernel",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": None if traffic is None else traffic["traffic"],
            "traffic_unit": "HBM bytes per launch (scaled FETCH_SIZE + WRITE_SIZE)",
            "traffic_run_algorithmic_bytes_per_launch": (None if traffic is None
                                                         else traffic["algorithmic"]),
            "traffic_ratio": None if traffic is None else traffic["ratio"],
            "traffic_profile": None if traffic is None else traffic["profile"],
            "algorithmic_bytes_per_launch": round(statistics.fmean(inj_bytes) / nwaves),
        } if not host_store else {
            # the store half of the inject traffic crosses the host link
            "bound": "pcie",
            "kernel": "inject_kernel (place + inject)" if fused else "inject_kernel",
            "achieved": round(achieved / 2, 1),
            "peak": PCIE_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / 2 / PCIE_PEAK_GBPS, 4),
            "traffic": None,
            "algorithmic_bytes_per_launch": round(statistics.fmean(inj_bytes) / nwaves / 2),
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def profile_pass_report(args, w, nsteps, nwaves, fused, queries, retrieve, place, bank, buf,
                        dev, torch, RequestBuffers, is_stream_copy):
    """End of a --profile-pass run: every step so far (W warm-up + K timed)
    dispatched the timed path once per request wave. Their placed tokens are
    recomputed untimed with the retrieval and the slot map (no inject
    dispatch), so the counter means per inject dispatch pair with the mean
    algorithmic bytes of exactly those dispatches. Then a 1 GiB copy by the
    library's streaming copy calibrates the byte counters."""
    import workloads
    probe = RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=bank.dtype,
                           max_tokens=w.max_tokens, device=dev, workspace=buf.workspace)
    per_launch = []
    for i in range(nsteps):
        retrieve(queries[i], probe)
        for j in range(nwaves):
            place(i, j, probe)
        torch.cuda.synchronize()
        for j in range(nwaves):
            m = int(probe.m[j * (w.nq // nwaves):(j + 1) * (w.nq // nwaves)].sum())
            # the fused launch also writes each placed token's slot and position
            per_launch.append(workloads.inject_algorithmic_bytes(w, m) + (12 * m if fused else 0))
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        is_stream_copy(dst, src)
    torch.cuda.synchronize()
    print(json.dumps({
        "profile_pass": True, "workload": w.name, "k": w.k, "nq": w.nq,
        "path": "fused" if fused else "separate",
        "kernel": "inject_kernel<false, true>" if fused else "inject_kernel<false, false>",
        "inject_dispatches": len(per_launch),
        "algorithmic_bytes_per_launch": round(statistics.fmean(per_launch)),
        "calibration": {"kernel": "stream_copy_kernel", "dispatches": 3,
                        "bytes_each_way": 1 << 30},
    }), flush=True)


def _read_csvs(d, suffix):
    import csv
    import glob
    rows = []
    for path in sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)):
        with open(path) as f:
            rows.extend(csv.DictReader(f))
    if not rows:
        raise SystemExit(f"no *{suffix} under {d}")
    return rows


def _short_kernel(name):
    return name.split("(")[0].replace("void ", "").strip()


def _source_hashes():
    """Digests of the sources the inject launch is built from (its kernel,
    the shared device helpers, the launcher declarations and the ABI layer):
    a summary stops applying once any of them changes."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2607_27090_amd", "csrc")
    out = []
    for name in ("abi.hip", "common.hpp", "inject.hip", "launch.hpp"):
        with open(os.path.join(csrc, name), "rb") as f:
            out.append(f"{name} {hashlib.sha256(f.read()).hexdigest()}")
    return " ".join(out)


def summarize_traffic(args):
    """Markdown summary of two --pmc runs of --profile-pass: per-dispatch
    FETCH_SIZE and WRITE_SIZE (KiB) of the library's kernels, each scaled by
    what the same counter reads for the 1 GiB calibration copy, and the
    timed kernel's traffic against the run's algorithmic bytes."""
    import collections
    fdir, wdir = args.summarize_traffic
    runs = {}
    for counter, d in (("FETCH_SIZE", fdir), ("WRITE_SIZE", wdir)):
        by = collections.defaultdict(list)
        for r in _read_csvs(d, "counter_collection.csv"):
            if r["Counter_Name"] == counter:
                by[_short_kernel(r["Kernel_Name"])].append(float(r["Counter_Value"]))
        with open(os.path.join(d, "bench.json")) as f:
            meta = json.loads(f.read().strip().splitlines()[-1])
        runs[counter] = (by, meta)
    metas = [runs[c][1] for c in runs]
    assert metas[0]["algorithmic_bytes_per_launch"] == metas[1]["algorithmic_bytes_per_launch"], \
        "the two counter runs placed different tokens"
    meta = metas[0]
    frag = args.kernel or meta["kernel"]
    lines = [f"# {args.title or 'HBM traffic: ' + meta['workload']}", "",
             "Two counter runs of the bench's profile pass (one counter each), MI355X:", "",
             "```", *args.cmd, "```", ""]
    scaled = {}
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        by, _ = runs[counter]
        cal = [v for k, v in by.items() if "stream_copy_kernel" in k]
        cal = max(cal[0]) if cal else None
        if not cal:
            raise SystemExit(f"no calibration copy among the {counter} dispatches")
        factor = (1 << 30) / 1024 / cal
        lines += [f"{counter} (KiB per dispatch):", "",
                  "| kernel | dispatches | mean | min | max |", "|---|---:|---:|---:|---:|"]
        for k, v in sorted(by.items(), key=lambda kv: -statistics.fmean(kv[1])):
            if k.startswith("is::"):
                lines.append(f"| `{k}` | {len(v)} | {statistics.fmean(v):.1f} | {min(v):.1f} | "
                             f"{max(v):.1f} |")
        lines += ["", f"Calibration: the 1 GiB streaming copy reads back as {cal:.1f} KiB "
                  f"(factor {factor:.5f}).", ""]
        hits = [k for k in by if frag in k]
        if len(hits) != 1:
            raise SystemExit(f"kernel fragment {frag!r} matches {hits}")
        v = by[hits[0]]
        if len(v) != meta["inject_dispatches"]:
            raise SystemExit(f"{hits[0]}: {len(v)} dispatches, the run made "
                             f"{meta['inject_dispatches']}")
        scaled[counter] = statistics.fmean(v) * 1024 * factor
    total = scaled["FETCH_SIZE"] + scaled["WRITE_SIZE"]
    alg = meta["algorithmic_bytes_per_launch"]
    lines += [f"Timed kernel `{frag}`, mean over its {meta['inject_dispatches']} dispatches "
              f"(every warm-up and timed step once):", "",
              f"* read: {scaled['FETCH_SIZE'] / 1e6:.2f} MB",
              f"* write: {scaled['WRITE_SIZE'] / 1e6:.2f} MB",
              f"* total: {total / 1e6:.2f} MB against {alg / 1e6:.2f} MB algorithmic "
              f"(the same dispatches): ratio {total / alg:.4f}", "",
              f"traffic_bytes_per_launch: {round(total)}",
              f"algorithmic_bytes_per_launch: {alg}",
              f"source_sha256: {_source_hashes()}"]
    return "\n".join(lines)


def summarize_stats(args):
    """Markdown summary of a --kernel-trace --stats run: the library's kernels
    with calls and mean / min / max durations, beside the run's own
    event-timed launch figure."""
    rows = _read_csvs(args.summarize_stats, "kernel_stats.csv")
    with open(os.path.join(args.summarize_stats, "bench.json")) as f:
        meta = json.loads(f.read().strip().splitlines()[-1])
    lines = [f"# {args.title or 'Kernel durations'}", "", "MI355X, ROCm 7.2:", "", "```",
             *args.cmd, "```", "",
             "| kernel | calls | mean us | min us | max us | share of GPU time |",
             "|---|---:|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = _short_kernel(r["Name"])
        if not name.startswith("is::") and not any(f in r["Name"] for f in args.include):
            continue
        if len(name) > 90:
            name = name[:87] + "..."
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.1f}% |")
    roof = meta.get("roofline", {})
    lines += ["", f"The same run's bench line: value {meta.get('value')} {meta.get('unit')} "
              f"({meta.get('timing', '')}), warm {meta.get('warm_us_per_request')} us/request, "
              f"inject launch {meta.get('inject_launch_us')} us event-timed, "
              f"{roof.get('achieved')} GB/s = {roof.get('frac')} of {roof.get('peak')} GB/s."]
    if meta.get("library_gemm"):
        g = meta["library_gemm"]
        lines += ["", f"Vendor GEMM on the same bank and queries ({g['what']}): "
                  f"{g['us_median']} us event-timed median, {g['TFLOPs']} TFLOP/s, "
                  f"bank read at {g['bank_GBps']} GB/s."]
    return "\n".join(lines)


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


# committed counter summaries per (workload at its default k, fused path):
# file and the key of its per-launch figure
TRAFFIC_PROFILES = {
    ("llama8b", True): ("place_inject_llama8b_k50_traffic.md", "traffic_bytes_per_launch"),
    ("llama8b", False): ("inject_kernel_llama8b_k50_traffic.md", "traffic_bytes_per_launch"),
    ("concurrency", True): ("place_inject_concurrency64_k50_traffic.md",
                            "traffic_bytes_per_launch"),
    ("llama70b", True): ("place_inject_llama70b_k100_traffic.md", "traffic_bytes_per_launch"),
    ("retrieval1m", True): ("place_inject_retrieval1m_k100_traffic.md",
                            "traffic_bytes_per_launch"),
}


def measured_traffic(workload, fused):
    """HBM traffic per inject launch from the committed counter summary of the
    workload and path timed: {traffic, algorithmic, ratio, profile}, where
    algorithmic is the profiled run's own algorithmic bytes per launch. None
    when there is no summary or the kernel sources changed since the counters
    were taken."""
    import hashlib
    import re
    if (workload, fused) not in TRAFFIC_PROFILES:
        return None
    fname, key = TRAFFIC_PROFILES[(workload, fused)]
    path = os.path.join(ROOT, "profiles", fname)
    csrc = os.path.join(ROOT, "paper_2607_27090_amd", "csrc")
    try:
        text = open(path).read()
        tb = int(re.search(rf"^{key}: (\d+)", text, re.M).group(1))
        ab = int(re.search(rf"^{key.replace('traffic_', 'algorithmic_')}: (\d+)", text,
                           re.M).group(1))
        want = dict(re.findall(r"(\S+\.h\w*) ([0-9a-f]{64})", text))
    except (OSError, AttributeError):
        return None
    if not want:
        return None
    for name, digest in want.items():
        with open(os.path.join(csrc, name), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != digest:
                return None
    return {"traffic": tb, "algorithmic": ab, "ratio": round(tb / ab, 4),
            "profile": f"profiles/{fname}"}


def ann_cpu_baseline(w, bank, index, query, ann, args, torch):
    """The oracle's beam search (oracle/ann.c, one thread) over the same graph
    and seeds, one query at a time, for about half of --cpu-seconds."""
    import numpy as np
    import oracle

    def host(t):
        if t.dtype == torch.float32:
            return t.contiguous().cpu().numpy(), oracle.F32
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16), oracle.BF16

    bh, odt = host(bank)
    qh, _ = host(query)
    G = index.graph.cpu().numpy()
    seeds = index.seed_ids.cpu().numpy()
    t0, done = time.perf_counter(), 0
    while done < w.nq and time.perf_counter() - t0 < args.cpu_seconds / 2:
        oracle.ann_search(qh[done:done + 1], bh, w.n, w.d_e, G, seeds, ann["beam"], w.k,
                          ann["max_iters"], width=ann["width"], dtype=odt)
        done += 1
    el = time.perf_counter() - t0
    log(f"cpu oracle (graph search): {done} queries, {el:.1f}s")
    return {"value": round(el / done * 1e6, 1), "unit": "us/query", "cores": 1,
            "cpu_model": _cpu_model(), "kind": "oracle",
            "sample": f"{done} of the {w.nq} queries of one step, the same graph and seeds"}


def _lscpu_model():
    """The host CPU's model name as lscpu prints it (else /proc/cpuinfo's)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.strip().lower().startswith("model name"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    return _cpu_model()


def cpu_baseline(w, bank, store, queries, bts, args, torch, gpu=None):
    """The oracle timed on whole requests of the workload on the host, in two
    modes: one thread (the plain serial program) and every core this process
    may run on (its OpenMP loops over scores, queries and (layer, head) of the
    inject). A request is: exact binary64 scores over its whole bank, a full
    sort, the slot map, and the fp64 RoPE inject of all its placed tokens in
    every layer. Requests are taken from the last timed step backwards
    (every request of a step in turn); the one-thread mode runs until its
    budget (--cpu-seconds) is spent, at least one request, and the all-core
    mode then runs the same requests. For one-request workloads, up to 4 of
    them whose page region no later step rewrote are compared with what the
    GPU wrote (`gpu`: the per-step buffers and the page pools)."""
    import numpy as np
    import oracle

    def u16(t):
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

    def host_emb(t):
        if t.dtype == torch.float32:
            return t.contiguous().cpu().numpy(), oracle.F32
        return u16(t), oracle.BF16

    def bf16_f64(x):
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)

    def ordered(x):  # bf16 bit patterns as integers in value order
        x = x.astype(np.int64)
        return np.where(x & 0x8000, -(x & 0x7FFF), x & 0x7FFF)

    cores = len(os.sched_getaffinity(0))
    lens_all = store["fact_lens"].cpu().numpy()
    offs_all = store["fact_offsets"].cpu().numpy()
    L, T, H, D = store["preK"].shape
    R = bts.shape[0]
    wave = bts.shape[1]
    nwaves = w.nq // wave
    last = args.warmup + args.steps - 1
    shared = None
    if w.shared_bank:
        shared = host_emb(bank)

    def prepare(i, r):
        """Host inputs of request r of step i (untimed): its query, bank,
        tables, block table and a compact copy of the stored rows of the
        facts it will choose."""
        q, dt = host_emb(queries[i][r:r + 1])
        bh = shared[0] if shared is not None else host_emb(bank[r])[0]
        ti = 0 if lens_all.shape[0] == 1 else r
        lens, offs = lens_all[ti:ti + 1], offs_all[ti:ti + 1]
        bt = bts[(i * nwaves + r // wave) % R][r % wave:r % wave + 1].cpu().numpy()
        with oracle.using_threads(cores):
            ids_peek, _, _ = oracle.retrieve(q, bh, w.n, w.d_e, w.k, 1, 0, dt)
        coffs = np.zeros_like(offs)
        pieces, cur = [], 0
        for c in ids_peek[0]:
            pieces.append((int(offs[0, c]), int(lens[0, c])))
            coffs[0, c] = cur
            cur += int(lens[0, c])
        Kc = np.empty((L, cur, H, D), dtype=np.uint16)
        Vc = np.empty_like(Kc)
        at = 0
        for off, ln in pieces:
            Kc[:, at:at + ln] = u16(store["preK"][:, off:off + ln]).reshape(L, ln, H, D)
            Vc[:, at:at + ln] = u16(store["V"][:, off:off + ln]).reshape(L, ln, H, D)
            at += ln
        sm = oracle.slot_map(ids_peek, lens, w.start_pos, bt, w.page_size, w.k, 1, w.n, 0,
                             bt.shape[1], w.max_tokens, 1)
        return dict(i=i, r=r, q=q, dt=dt, bank=bh, lens=lens, coffs=coffs, bt=bt, Kc=Kc, Vc=Vc,
                    cur=cur, num_slots=(int(bt.max()) + 1) * w.page_size,
                    slots=sm["slots"][0, :int(sm["m"][0])])

    def run(req):
        """One request through the oracle; returns (seconds, results). The
        host page pools are allocated and the pages the request writes are
        touched before the clock starts (first-touch page faults belong to
        the harness, not to the oracle)."""
        hk = np.zeros((L, req["num_slots"], H, D), dtype=np.uint16)
        hv = np.zeros_like(hk)
        hk[:, req["slots"]] = 1
        hv[:, req["slots"]] = 1
        t0 = time.perf_counter()
        ids, _, _ = oracle.retrieve(req["q"], req["bank"], w.n, w.d_e, w.k, 1, 0, req["dt"])
        sm = oracle.slot_map(ids, req["lens"], w.start_pos, req["bt"], w.page_size, w.k, 1,
                             w.n, 0, req["bt"].shape[1], w.max_tokens, 1)
        oracle.inject(ids, req["Kc"], req["Vc"], sm["slots"], sm["positions"], w.theta, hk, hv,
                      req["coffs"], req["lens"], sm["m"], w.k, 1, w.n, 0, 1, w.max_tokens, L, H,
                      D, req["cur"], req["num_slots"])
        return time.perf_counter() - t0, (ids, sm, hk, hv)

    # one thread: requests from the last timed step backwards within budget
    order, single, tokens = [], [], 0
    results = []  # outputs of the first requests the parity check may use
    while (not single or sum(single) < args.cpu_seconds) and len(order) < args.steps * w.nq:
        n_ = len(order)
        req = prepare(last - n_ // w.nq, n_ % w.nq)
        with oracle.using_threads(1):
            sec, res = run(req)
        single.append(sec)
        tokens += int(res[1]["m"][0])
        order.append((req["i"], req["r"]))
        if w.nq == 1 and len(results) < R:
            results.append((req, res))
        del req, res
    # every core: the same requests, within the same budget
    multi = []
    for i, r in order:
        if multi and sum(multi) >= args.cpu_seconds:
            break
        req = prepare(i, r)
        with oracle.using_threads(cores):
            multi.append(run(req)[0])
        del req
    us1 = statistics.fmean(single) * 1e6
    usn = statistics.fmean(multi) * 1e6
    log(f"cpu oracle: {len(single)} requests at 1 thread {us1:.0f} us/request; "
        f"{len(multi)} at {cores} threads {usn:.0f} us/request")

    par = None
    if gpu is not None and w.nq == 1:
        par = {"requests": 0, "ids_equal": 0, "placement_equal": True, "v_bit_exact": True,
               "k_in_tolerance": True, "k_elements": 0, "k_not_bit_exact": 0, "k_max_ulp": 0,
               "k_floor_rescued": 0}
        for req, (ids, sm, hk, hv) in results:
            i = req["i"]
            # the GPU's results of this request, while its pages are still in
            # place (the last R steps; region 0 is reused by --graph)
            if par["requests"] >= 4 or i <= last - R or (gpu["graph"] and i % R == 0):
                continue
            g = gpu["sets"][i - args.warmup]
            par["requests"] += 1
            if not np.array_equal(g.ids[0].cpu().numpy(), ids[0]):
                continue  # a near-tie swap: the pages then hold other facts
            par["ids_equal"] += 1
            m = int(sm["m"][0])
            slots = sm["slots"][0, :m]
            par["placement_equal"] &= bool(
                int(g.m[0]) == m and np.array_equal(g.slots[0, :m].cpu().numpy(), slots)
                and np.array_equal(g.positions[0, :m].cpu().numpy(), sm["positions"][0, :m]))
            sl = torch.from_numpy(slots).to(gpu["pk"].device)
            gk, gv = u16(gpu["pk"][:, sl]), u16(gpu["pv"][:, sl])
            ok_, ov_ = hk[:, slots], hv[:, slots]
            par["v_bit_exact"] &= bool(np.array_equal(gv, ov_))
            src = req["coffs"][0, sm["fact"][0, :m]] + sm["tok"][0, :m]
            for layer in range(L):  # one layer at a time keeps the temporaries small
                gk2, ok2 = gk[layer].reshape(-1, D), ok_[layer].reshape(-1, D)
                if np.array_equal(gk2, ok2):
                    par["k_elements"] += int(gk2.size)
                    continue
                x = bf16_f64(req["Kc"][layer, src].reshape(-1, D))
                pair = np.hypot(x[:, :D // 2], x[:, D // 2:])
                pair = np.concatenate([pair, pair], axis=1)
                ulp = np.abs(ordered(gk2) - ordered(ok2))
                err = np.abs(bf16_f64(gk2) - bf16_f64(ok2))
                rel_ok = err <= 2.0 ** -7 * np.abs(bf16_f64(ok2))
                floor_ok = err <= 2.0 ** -20 * pair
                par["k_in_tolerance"] &= bool(((ulp <= 1) | rel_ok | floor_ok).all())
                par["k_elements"] += int(gk2.size)
                par["k_not_bit_exact"] += int((gk2 != ok2).sum())
                par["k_max_ulp"] = max(par["k_max_ulp"], int(ulp.max()))
                par["k_floor_rescued"] += int(((ulp > 1) & ~rel_ok & floor_ok).sum())
        log(f"cpu oracle parity of {par['requests']} timed requests: {par}")
    what = (f"scores over all {w.n} facts of its bank, full sort, slot map, fp64 RoPE inject of "
            f"its placed tokens x {L} layers")
    return {
        "value": round(usn, 1),
        "unit": "us/request",
        "cores": cores,
        "cpu_model": _lscpu_model(),
        "affinity_cpus": cores,
        "kind": "oracle",
        "sample": (f"{len(multi)} whole requests ({what}) on {cores} threads; "
                   f"{tokens} placed tokens over the {len(single)} requests of the one-thread "
                   f"mode"),
        "single_thread": {"value": round(us1, 1), "unit": "us/request", "cores": 1,
                          "requests": len(single)},
        "parity": par,
    }


if __name__ == "__main__":
    main()
