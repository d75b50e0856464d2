"""The consumer of the injected pages on the GPU (is_paged_scores): attention
logits of a query placed right after the memory against the injected keys,
read back through the block table. Checked against the oracle on the GPU's
own pages, and against Theorem "Chunked RoPE Injection" (§5.1): each logit
equals the stored pre-RoPE key's logit at relative position p - N, up to the
bf16 rounding of the injected key."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2607_27090_amd import (IS_DEV_BT_SHORT, IS_ROPE_HALF_SPLIT, IS_ROPE_INTERLEAVED,
                                  is_paged_scores)
from tests.gpu_harness import Instance, log, u16

pytestmark = pytest.mark.gpu

W = workloads.LLAMA8B.with_(n=1500, k=12, L=3, index=61)


def _query(w, Hq, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return torch.randn(w.nq, Hq, w.D, generator=g, device="cuda").to(torch.bfloat16)


def _gpu_scores(inst, q, qpos, layer, f, interleaved, max_blocks=None, status=None):
    w = inst.w
    Hq = q.shape[1]
    sc = torch.full((w.nq, Hq, inst.max_tokens), float("nan"), device="cuda")
    tf = None if f is None else torch.from_numpy(np.ascontiguousarray(f)).cuda()
    mb = inst.bt.shape[1] if max_blocks is None else max_blocks
    is_paged_scores(q, qpos, inst.pk, layer, inst.bt, w.page_size, w.start_pos, inst.buf.m, sc,
                    nq=w.nq, Hq=Hq, H=w.H, D=w.D, L=w.L, num_slots=inst.num_slots,
                    max_blocks=mb, max_tokens=inst.max_tokens, rope_theta=w.theta,
                    inv_freq=tf, pairing=IS_ROPE_INTERLEAVED if interleaved else IS_ROPE_HALF_SPLIT,
                    status=status)
    torch.cuda.synchronize()
    return sc.cpu().numpy()


@pytest.mark.parametrize("G,table,interleaved", [(4, None, False), (1, None, False),
                                                  (8, "llama3.1", True)])
def test_paged_scores_match_oracle_and_the_theorem(G, table, interleaved):
    w = W
    f = workloads.llama31_inv_freq(w.D, w.theta) if table else None
    inst = Instance(w)
    inst.run(inv_freq=f, interleaved=interleaved)
    o = inst.check_slot_map()
    Hq = G * w.H
    q = _query(w, Hq, 70 + G)
    m = int(inst.buf.m[0])
    N = w.start_pos + m
    qpos = torch.tensor([N], dtype=torch.int32, device="cuda")
    fr = oracle.default_inv_freq(w.theta, w.D) if f is None else f
    qh = u16(q)
    pages = u16(inst.pk)
    D, half = w.D, w.D // 2
    for layer in (0, w.L - 1):
        gs = _gpu_scores(inst, q, qpos, layer, f, interleaved)
        os_, st = oracle.paged_scores(qh, np.array([N], dtype=np.int32), pages, layer,
                                      inst.bt.cpu().numpy(), w.page_size, w.start_pos,
                                      inst.buf.m.cpu().numpy(), w.theta, 1, Hq, w.H, D,
                                      inst.num_slots, inst.bt.shape[1], inst.max_tokens,
                                      inv_freq=f, interleaved=interleaved)
        assert st == 0
        assert np.isnan(gs[0, :, m:]).all() and not np.isnan(gs[0, :, :m]).any()
        # magnitude sum_j |(R q)_j k_j| <= |q| |k| per (head, token)
        qd = oracle.bf16_to_f64(qh[0])                                   # [Hq][D]
        kp = oracle.bf16_to_f64(pages[layer][o["slots"][0, :m]])         # [m][H][D]
        mag = np.linalg.norm(qd, axis=1)[:, None] * np.linalg.norm(kp, axis=2).T.repeat(G, 0)
        err = np.abs(gs[0, :, :m] - os_[0, :, :m])
        assert (err <= 2.0 ** -16 * mag).all(), f"worst {np.max(err / mag):.3e}"
        # the theorem: the pre-RoPE key's logit at relative position p - N
        src = inst.store["fact_offsets"].cpu().numpy()[0][o["fact"][0, :m]] + o["tok"][0, :m]
        kpre = oracle.bf16_to_f64(u16(inst.store["preK"][layer][torch.from_numpy(src).cuda()]))
        rel = (w.start_pos + np.arange(m)) - N
        for hq in range(Hq):
            kk = kpre[:, hq // G, :]
            if interleaved:
                zq, zk = qd[hq, 0::2] + 1j * qd[hq, 1::2], kk[:, 0::2] + 1j * kk[:, 1::2]
            else:
                zq, zk = qd[hq, :half] + 1j * qd[hq, half:], kk[:, :half] + 1j * kk[:, half:]
            want = np.real(np.sum(np.conj(zq)[None, :] * zk * np.exp(1j * rel[:, None] * fr[None, :]),
                                  axis=1))
            assert np.all(np.abs(gs[0, hq, :m] - want) <= 2.0 ** -8 * mag[hq]), hq
    log(f"consumer G={G} table={table} interleaved={interleaved}: m={m}, {Hq} query heads, "
        f"oracle and theorem hold on layers 0 and {w.L - 1}")


def test_paged_scores_flags_a_short_table():
    inst = Instance(W)
    inst.run()
    q = _query(W, 4 * W.H, 80)
    m = int(inst.buf.m[0])
    qpos = torch.tensor([W.start_pos + m], dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    short = (W.start_pos + m // 2) // W.page_size
    gs = _gpu_scores(inst, q, qpos, 0, None, False, max_blocks=short, status=status)
    assert int(status.item()) & IS_DEV_BT_SHORT
    ok = short * W.page_size - W.start_pos
    assert not np.isnan(gs[0, :, :ok]).any() and np.isnan(gs[0, :, ok:]).all()
