"""Shared GPU-test plumbing: build a seeded workload instance on the device,
run one pass of the HIP path through the C ABI, and check it against the
oracle (full or sampled)."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import workloads
from paper_2607_27090_amd.pipeline import RequestBuffers, run_request
from tests import parity


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def u16(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def host_emb(t: torch.Tensor):
    """(array, oracle dtype) of an embedding tensor."""
    if t.dtype == torch.float32:
        return t.contiguous().cpu().numpy(), oracle.F32
    return u16(t), oracle.BF16


class Instance:
    def __init__(self, w: workloads.Workload, device="cuda", variant=0, store=None, bank=None,
                 max_tokens=None):
        self.w = w
        self.bank = workloads.make_bank(w, device) if bank is None else bank
        self.query = workloads.make_queries(w, device, variant)
        self.store = workloads.make_store(w, device) if store is None else store
        self.max_tokens = w.max_tokens if max_tokens is None else max_tokens
        mb = -(-(w.start_pos + self.max_tokens) // w.page_size)
        self.bt, self.num_blocks = workloads.make_block_tables(w, device, variant, max_blocks=mb)
        self.pk, self.pv, self.num_slots = workloads.make_pages(w, self.num_blocks, device)
        self.buf = RequestBuffers(n=w.n, d=w.d_e, k=w.k, nq=w.nq, emb_dtype=self.bank.dtype,
                                  max_tokens=self.max_tokens, device=device)

    def run(self, reverse_rank=1, inv_freq=None, interleaved=False, stream=None, sync=True,
            fused=False):
        """One pass; inv_freq (float64 numpy [D/2]) and interleaved select the
        rotary table and pair layout (kept for the checks). ``stream`` (a
        torch stream, default the current one) takes the calls; with
        ``sync=False`` the pass is left in flight; ``fused`` replaces the slot
        map and inject calls by the one place + inject call."""
        from paper_2607_27090_amd import IS_ROPE_HALF_SPLIT, IS_ROPE_INTERLEAVED
        w = self.w
        self.inv_freq, self.interleaved = inv_freq, bool(interleaved)
        tf = None if inv_freq is None else torch.from_numpy(np.ascontiguousarray(
            inv_freq, dtype=np.float64)).cuda()
        run_request(self.buf, self.query, self.bank, self.store, self.bt, self.pk, self.pv,
                    start_pos=w.start_pos, page_size=w.page_size, rope_theta=w.theta,
                    shared_bank=w.shared_bank, reverse_rank=reverse_rank, inv_freq=tf,
                    pairing=IS_ROPE_INTERLEAVED if interleaved else IS_ROPE_HALF_SPLIT,
                    fused=fused, stream=stream)
        if sync:
            torch.cuda.synchronize()

    # ---- checks --------------------------------------------------------------

    def check_retrieve(self, queries=None):
        """Oracle scores + full sort for the given queries (default: all)."""
        w = self.w
        qs = range(w.nq) if queries is None else queries
        gids = self.buf.ids.cpu().numpy()
        gsc = self.buf.scores.cpu().numpy()
        near = 0
        for r in qs:
            qh, dt = host_emb(self.query[r:r + 1])
            bank_r = self.bank if w.shared_bank else self.bank[r]
            bh, _ = host_emb(bank_r)
            ids_o, _, s_all = oracle.retrieve(qh, bh, w.n, w.d_e, w.k, 1, 0, dt)
            s = s_all[0]
            near += parity.check_ids(gids[r], ids_o[0], s, w.n)
            qd = oracle.bf16_to_f64(qh) if dt == oracle.BF16 else qh.astype(np.float64)
            rows = bh[gids[r]]
            rd = oracle.bf16_to_f64(rows) if dt == oracle.BF16 else rows.astype(np.float64)
            mag = np.abs(rd * qd).sum(axis=1)
            parity.check_scores(gsc[r], s[gids[r]], mag)
        return near

    def check_slot_map(self):
        w = self.w
        gids = self.buf.ids.cpu().numpy()
        lens = self.store["fact_lens"].cpu().numpy()
        lens_stride = 0 if lens.shape[0] == 1 else w.n
        bt = self.bt.cpu().numpy()
        o = oracle.slot_map(gids, lens, w.start_pos, bt, w.page_size, w.k, w.nq, w.n, lens_stride,
                            bt.shape[1], self.max_tokens, 1)
        gm = self.buf.m.cpu().numpy()
        assert int(self.buf.status.item()) == o["status"] == 0
        assert np.array_equal(gm, o["m"])
        gs = self.buf.slots.cpu().numpy()
        gp = self.buf.positions.cpu().numpy()
        for r in range(w.nq):
            m = gm[r]
            assert np.array_equal(gs[r, :m], o["slots"][r, :m])
            assert np.array_equal(gp[r, :m], o["positions"][r, :m])
        self._place = o
        return o

    def check_inject_full(self, foreign_slots=None):
        """Oracle inject into host pools of the same size; compare everything.
        ``foreign_slots`` are slots of the same pool that other requests wrote
        (left out of the check that nothing outside the placement changed)."""
        w = self.w
        o = self._place
        L, T, H, D = self.store["preK"].shape
        gids = self.buf.ids.cpu().numpy()
        lens = self.store["fact_lens"].cpu().numpy()
        offs = self.store["fact_offsets"].cpu().numpy()
        lens_stride = 0 if lens.shape[0] == 1 else w.n
        # a compact host copy of just the stored rows the chosen facts use
        pieces, coffs = [], np.zeros_like(offs)
        cur = 0
        for r in range(w.nq):
            b = 0 if lens_stride == 0 else r
            for c in gids[r]:
                pieces.append((int(offs[b, c]), int(lens[b, c])))
                coffs[b, c] = cur
                cur += int(lens[b, c])
        Kc = np.empty((L, cur, H, D), dtype=np.uint16)
        Vc = np.empty((L, cur, H, D), dtype=np.uint16)
        at = 0
        for (off, ln) in pieces:
            Kc[:, at:at + ln] = u16(self.store["preK"][:, off:off + ln])
            Vc[:, at:at + ln] = u16(self.store["V"][:, off:off + ln])
            at += ln
        hk = np.full((L, self.num_slots, H, D), parity.SENTINEL, dtype=np.uint16)
        hv = hk.copy()
        st = oracle.inject(gids, Kc, Vc, o["slots"], o["positions"], w.theta, hk, hv, coffs,
                           lens, o["m"], w.k, w.nq, w.n, lens_stride, 1, self.max_tokens, L, H, D,
                           cur, self.num_slots, inv_freq=getattr(self, "inv_freq", None),
                           interleaved=getattr(self, "interleaved", False))
        assert st == 0
        gk, gv = u16(self.pk), u16(self.pv)
        own = np.ones(self.num_slots, dtype=bool)
        if foreign_slots is not None:
            own[np.asarray(foreign_slots, dtype=np.int64)] = False
        assert np.array_equal(gv[:, own], hv[:, own]), "V pages differ"
        same = gk == hk
        touched = np.zeros(self.num_slots, dtype=bool)
        for r in range(w.nq):
            touched[o["slots"][r, :o["m"][r]]] = True
        assert not (touched & ~own).any(), "own and foreign slots overlap"
        untouched = ~touched & own
        assert same[:, untouched].all(), "a slot outside the placement was written"
        pre = np.empty((L, self.num_slots, H, D), dtype=np.uint16)
        # unrotated inputs at each target slot, for the pair-norm floor
        for r in range(w.nq):
            m = o["m"][r]
            src = coffs_rows(o, r, coffs, lens_stride)
            pre[:, o["slots"][r, :m]] = Kc[:, src]
        floor = parity.check_k_rows(gk[:, touched], hk[:, touched], pre[:, touched], D,
                                    getattr(self, "interleaved", False))
        return floor

    def check_inject_sampled(self, frac=0.01, seed=0, max_rows=20000):
        """Sampled (request, token, layer) rows + every fact's first and last
        token, rotated by the oracle from the stored rows; V bit-exact;
        a sample of untouched slots must still hold the sentinel."""
        w = self.w
        o = self._place
        L, T, H, D = self.store["preK"].shape
        rng = np.random.default_rng(seed)
        lens = self.store["fact_lens"].cpu().numpy()
        offs = self.store["fact_offsets"].cpu().numpy()
        per_bank = lens.shape[0] != 1
        rr, tt, ll = [], [], []
        for r in range(w.nq):
            m = int(o["m"][r])
            if m == 0:
                continue
            fact, tok = o["fact"][r, :m], o["tok"][r, :m]
            edge = np.nonzero((tok == 0) | (np.r_[fact[1:] != fact[:-1], True]))[0]
            cnt = max(1, int(frac * m * L))
            pick_t = rng.integers(0, m, cnt)
            pick_l = rng.integers(0, L, cnt)
            rr += [r] * (cnt + edge.size)
            tt += list(pick_t) + list(edge)
            ll += list(pick_l) + list(rng.integers(0, L, edge.size))
        rr, tt, ll = np.array(rr), np.array(tt), np.array(ll)
        if rr.size > max_rows:
            sel = rng.choice(rr.size, max_rows, replace=False)
            rr, tt, ll = rr[sel], tt[sel], ll[sel]
        facts = o["fact"][rr, tt]
        toks = o["tok"][rr, tt]
        b = rr if per_bank else np.zeros_like(rr)
        src = offs[b, facts] + toks
        slots = o["slots"][rr, tt]
        pos = o["positions"][rr, tt]
        li = torch.from_numpy(ll).cuda()
        si = torch.from_numpy(src).cuda()
        di = torch.from_numpy(slots).cuda()
        # (a host-resident store is indexed on the host)
        sd = self.store["preK"].device
        kin = u16(self.store["preK"][li.to(sd), si.to(sd)]).reshape(-1, H * D)
        vin = u16(self.store["V"][li.to(sd), si.to(sd)]).reshape(-1, H * D)
        gk = u16(self.pk[li, di]).reshape(-1, H * D)
        gv = u16(self.pv[li, di]).reshape(-1, H * D)
        assert np.array_equal(gv, vin), "V rows differ"
        want = oracle.rope_rows_bf16(kin, pos, w.theta, H, D)
        floor = parity.check_k_rows(gk, want, kin, D)
        # untouched slots keep the sentinel
        placed = np.concatenate([o["slots"][r, :o["m"][r]] for r in range(w.nq)])
        touched = np.zeros(self.num_slots, dtype=bool)
        touched[placed] = True
        free = np.nonzero(~touched)[0]
        if free.size:
            probe = rng.choice(free, min(2000, free.size), replace=False)
            pl = rng.integers(0, L, probe.size)
            pk = u16(self.pk[torch.from_numpy(pl).cuda(), torch.from_numpy(probe).cuda()])
            pvv = u16(self.pv[torch.from_numpy(pl).cuda(), torch.from_numpy(probe).cuda()])
            assert (pk == parity.SENTINEL).all() and (pvv == parity.SENTINEL).all()
        return rr.size, floor


def coffs_rows(o, r, coffs, lens_stride):
    m = int(o["m"][r])
    fact, tok = o["fact"][r, :m], o["tok"][r, :m]
    b = 0 if lens_stride == 0 else r
    return coffs[b, fact] + tok
