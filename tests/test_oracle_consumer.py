"""Pins for the oracle's consumer of the injected pages (Theorem "Chunked
RoPE Injection", §5.1; the query follows the memory, §3.3): the logits of a
query at position N against keys injected at positions p equal, up to the
bf16 rounding of the injected keys, the logits of the stored pre-RoPE keys at
relative position p - N (an independent complex form); they do not change
when placement and query are shifted together or when the pages are
permuted; grouped-query heads read their own KV head; table errors flag."""
import numpy as np
import pytest

import oracle
import workloads

THETA = 500000.0


def _case(seed, H=2, Hq=4, D=32, L=2, P=4, start=40, k=3, perm=True, table=None):
    rng = np.random.default_rng(seed)
    n, T = 5, 60
    lens = np.array([[5, 7, 3, 9, 4]], dtype=np.int32)
    offs = np.array([[0, 5, 12, 15, 24]], dtype=np.int64)
    ids = np.array([[3, 0, 1]], dtype=np.int32)
    K = oracle.f64_to_bf16(rng.standard_normal((L, T, H, D)))
    V = oracle.f64_to_bf16(rng.standard_normal((L, T, H, D)))
    q = oracle.f64_to_bf16(rng.standard_normal((1, Hq, D)))
    max_tokens = 32
    mb = -(-(start + max_tokens) // P)
    nblk = mb + 3
    bt = (rng.permutation(nblk)[:mb] if perm else np.arange(mb)).astype(np.int32)[None, :]
    o = oracle.slot_map(ids, lens, start, bt, P, k, 1, n, 0, mb, max_tokens, 1)
    pk = np.zeros((L, nblk * P, H, D), dtype=np.uint16)
    pv = np.zeros_like(pk)
    st = oracle.inject(ids, K, V, o["slots"], o["positions"], THETA, pk, pv, offs, lens, o["m"],
                       k, 1, n, 0, 1, max_tokens, L, H, D, T, nblk * P, inv_freq=table)
    assert st == 0
    return dict(K=K, q=q, o=o, pk=pk, bt=bt, ids=ids, lens=lens, offs=offs, H=H, Hq=Hq, D=D,
                L=L, P=P, start=start, mb=mb, nblk=nblk, max_tokens=max_tokens, table=table)


def _scores(c, qpos, layer=0, bt=None, start=None):
    return oracle.paged_scores(c["q"], np.array([qpos], dtype=np.int32), c["pk"], layer,
                               c["bt"] if bt is None else bt, c["P"],
                               c["start"] if start is None else start, c["o"]["m"], THETA, 1,
                               c["Hq"], c["H"], c["D"], c["nblk"] * c["P"], c["mb"],
                               c["max_tokens"], inv_freq=c["table"])


@pytest.mark.parametrize("table", [None, "llama3.1"])
def test_logits_equal_relative_position_form(table):
    D = 32
    f = None if table is None else workloads.llama31_inv_freq(D, THETA)
    c = _case(400, D=D, table=f)
    m = int(c["o"]["m"][0])
    N = c["start"] + m  # the query right after the memory
    for layer in range(c["L"]):
        s, st = _scores(c, N, layer)
        assert st == 0
        fr = oracle.default_inv_freq(THETA, D) if f is None else f
        for hq in range(c["Hq"]):
            qd = oracle.bf16_to_f64(c["q"][0, hq])
            zq = qd[: D // 2] + 1j * qd[D // 2:]
            for idx in range(m):
                fact, tok = c["o"]["fact"][0, idx], c["o"]["tok"][0, idx]
                kd = oracle.bf16_to_f64(c["K"][layer, c["offs"][0, fact] + tok, hq // 2])
                zk = kd[: D // 2] + 1j * kd[D // 2:]
                p = c["start"] + idx
                want = np.real(np.sum(np.conj(zq) * zk * np.exp(1j * (p - N) * fr)))
                mag = np.sum(np.abs(qd) * np.abs(kd))
                assert abs(s[0, hq, idx] - want) <= 2.0 ** -8 * mag
        assert np.isnan(s[0, :, m:]).all()


def test_shifting_memory_and_query_together_keeps_the_logits():
    a = _case(401, start=40)
    b = _case(401, start=40 + 37)
    m = int(a["o"]["m"][0])
    sa, _ = _scores(a, 40 + m)
    sb, _ = _scores(b, 77 + m)
    mag = np.abs(sa[0, :, :m]).max()
    assert np.max(np.abs(sa[0, :, :m] - sb[0, :, :m])) <= 2.0 ** -7 * mag


def test_block_table_permutation_does_not_change_the_logits():
    a = _case(402, perm=True)
    b = _case(402, perm=False)
    m = int(a["o"]["m"][0])
    sa, _ = _scores(a, 40 + m)
    sb, _ = _scores(b, 40 + m)
    assert np.array_equal(sa[0, :, :m], sb[0, :, :m])


def test_query_heads_read_their_own_kv_head():
    c = _case(403, H=2, Hq=4)
    c["pk"][:, :, 1, :] = 0  # kv head 1 serves query heads 2 and 3
    m = int(c["o"]["m"][0])
    s, _ = _scores(c, 40 + m)
    assert (s[0, 2:, :m] == 0).all() and (s[0, :2, :m] != 0).any()


def test_short_block_table_is_flagged_and_skipped():
    c = _case(404)
    m = int(c["o"]["m"][0])
    short = c["bt"][:, :(c["start"] + 5) // c["P"]]
    s, st = oracle.paged_scores(c["q"], np.array([40 + m], dtype=np.int32), c["pk"], 0, short,
                                c["P"], c["start"], c["o"]["m"], THETA, 1, c["Hq"], c["H"],
                                c["D"], c["nblk"] * c["P"], short.shape[1], c["max_tokens"])
    assert st & oracle.BT_SHORT
    last_ok = short.shape[1] * c["P"] - c["start"]
    assert np.isnan(s[0, :, last_ok:m]).all() and not np.isnan(s[0, :, :last_ok]).any()
