"""CPU-only checks of the C ABI: the library loads, exports every entry point
declared in include/inferscale.h, and rejects misuse on the host before
anything is enqueued (no call here reaches a kernel launch)."""
import ctypes
import os
import re

import pytest

import paper_2607_27090_amd as isl

HDR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                   "inferscale.h")
A = 1 << 20  # a 256-byte aligned fake device address (never dereferenced)


def declared():
    src = open(HDR).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(is_[a-z_]+)\s*\(", src)))


def test_header_declares_the_exported_set():
    assert declared() == sorted(isl.EXPORTED)


def test_every_declared_symbol_is_exported():
    lib = isl.load_library()
    for name in declared():
        assert hasattr(lib, name), name
    assert isl.is_version().startswith("inferscale-gfx950")


def _retrieve(**kw):
    a = dict(q=A, bank=A, n=1000, d=64, k=10, ids=A, scores=A, nq=1, stride=0, dt=0, ws=A,
             wsb=1 << 30, stream=None)
    a.update(kw)
    lib = isl.load_library()
    return lib.is_retrieve(a["q"], a["bank"], a["n"], a["d"], a["k"], a["ids"], a["scores"],
                           a["nq"], a["stride"], a["dt"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), isl.IS_ERR_INVALID),
    (dict(bank=None), isl.IS_ERR_INVALID),
    (dict(ids=None), isl.IS_ERR_INVALID),
    (dict(k=0), isl.IS_ERR_INVALID),
    (dict(k=1001), isl.IS_ERR_INVALID),
    (dict(n=5000, k=1025), isl.IS_ERR_INVALID),
    (dict(d=60), isl.IS_ERR_INVALID),
    (dict(d=0), isl.IS_ERR_INVALID),
    (dict(n=0), isl.IS_ERR_INVALID),
    (dict(nq=0), isl.IS_ERR_INVALID),
    (dict(dt=7), isl.IS_ERR_UNSUPPORTED),
    (dict(stride=-8), isl.IS_ERR_INVALID),
    (dict(stride=12), isl.IS_ERR_INVALID),
    (dict(q=A + 4), isl.IS_ERR_INVALID),
    (dict(bank=A + 8), isl.IS_ERR_INVALID),
    (dict(ws=None), isl.IS_ERR_WORKSPACE),
    (dict(wsb=16), isl.IS_ERR_WORKSPACE),
    (dict(ws=A + 16), isl.IS_ERR_INVALID),
])
def test_retrieve_rejects(kw, code):
    assert _retrieve(**kw) == code
    assert isl.load_library().is_last_error().decode()


def test_workspace_size_is_pure_host():
    assert isl.is_retrieve_workspace_size(10000, 768, 50, 1) >= 10000 * 4
    big = isl.is_retrieve_workspace_size(300000, 16, 1024, 1)
    assert big >= 300000 * 4 + 2 * 19 * 1024 * 8
    with pytest.raises(isl.InferScaleError):
        isl.is_retrieve_workspace_size(10, 8, 11, 1)


def _slot_map(**kw):
    a = dict(ids=A, lens=A, start=0, bt=A, P=16, slots=A, pos=A, m=A, k=5, nq=1, n=100, ls=0,
             mb=10, mt=100, rev=1, status=A)
    a.update(kw)
    return isl.load_library().is_slot_map(a["ids"], a["lens"], a["start"], a["bt"], a["P"],
                                          a["slots"], a["pos"], a["m"], a["k"], a["nq"], a["n"],
                                          a["ls"], a["mb"], a["mt"], a["rev"], a["status"], None)


@pytest.mark.parametrize("kw", [
    dict(ids=None), dict(lens=None), dict(bt=None), dict(slots=None), dict(pos=None),
    dict(m=None), dict(k=0), dict(k=1025), dict(nq=0), dict(n=0), dict(P=0), dict(start=-1),
    dict(mb=-1), dict(mt=-1), dict(start=2 ** 31 - 10), dict(ls=-1), dict(slots=A + 4),
    dict(ids=A + 2), dict(status=A + 1),
])
def test_slot_map_rejects(kw):
    assert _slot_map(**kw) == isl.IS_ERR_INVALID


def _inject(**kw):
    a = dict(ids=A, K=A, V=A, slots=A, pos=A, theta=500000.0, pk=A, pv=A, offs=A, lens=A, m=A,
             k=5, nq=1, n=100, ls=0, rev=1, mt=100, L=2, H=8, D=128, T=1000, ns=1000, status=A)
    a.update(kw)
    return isl.load_library().is_inject(a["ids"], a["K"], a["V"], a["slots"], a["pos"],
                                        a["theta"], a["pk"], a["pv"], a["offs"], a["lens"],
                                        a["m"], a["k"], a["nq"], a["n"], a["ls"], a["rev"],
                                        a["mt"], a["L"], a["H"], a["D"], a["T"], a["ns"],
                                        a["status"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(ids=None), isl.IS_ERR_INVALID), (dict(K=None), isl.IS_ERR_INVALID),
    (dict(V=None), isl.IS_ERR_INVALID), (dict(pk=None), isl.IS_ERR_INVALID),
    (dict(m=None), isl.IS_ERR_INVALID), (dict(k=0), isl.IS_ERR_INVALID),
    (dict(nq=0), isl.IS_ERR_INVALID), (dict(nq=70000), isl.IS_ERR_INVALID),
    (dict(L=0), isl.IS_ERR_INVALID), (dict(H=0), isl.IS_ERR_INVALID),
    (dict(D=15), isl.IS_ERR_UNSUPPORTED), (dict(D=24), isl.IS_ERR_UNSUPPORTED),
    (dict(D=528), isl.IS_ERR_UNSUPPORTED), (dict(T=-1), isl.IS_ERR_INVALID),
    (dict(theta=0.0), isl.IS_ERR_INVALID), (dict(theta=float("inf")), isl.IS_ERR_INVALID),
    (dict(theta=float("nan")), isl.IS_ERR_INVALID), (dict(K=A + 8), isl.IS_ERR_INVALID),
    (dict(pv=A + 4), isl.IS_ERR_INVALID), (dict(slots=A + 4), isl.IS_ERR_INVALID),
])
def test_inject_rejects(kw, code):
    assert _inject(**kw) == code


def test_binding_refuses_host_tensors():
    import torch
    t = torch.zeros(4, 8)
    with pytest.raises(ValueError):
        isl.is_retrieve(t, t, 4, 8, 1, torch.zeros(1, 1, dtype=torch.int32),
                        workspace=torch.zeros(256, dtype=torch.uint8))


def _rotary(**kw):
    a = dict(ids=A, K=A, V=A, slots=A, pos=A, theta=500000.0, pk=A, pv=A, offs=A, lens=A, m=A,
             k=5, nq=1, n=100, ls=0, rev=1, mt=100, L=2, H=8, D=128, T=1000, ns=1000, f=None,
             pairing=0, status=A)
    a.update(kw)
    return isl.load_library().is_inject_rotary(
        a["ids"], a["K"], a["V"], a["slots"], a["pos"], a["theta"], a["pk"], a["pv"], a["offs"],
        a["lens"], a["m"], a["k"], a["nq"], a["n"], a["ls"], a["rev"], a["mt"], a["L"], a["H"],
        a["D"], a["T"], a["ns"], a["f"], a["pairing"], a["status"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(pairing=2), isl.IS_ERR_INVALID), (dict(pairing=-1), isl.IS_ERR_INVALID),
    (dict(f=A + 4), isl.IS_ERR_INVALID), (dict(theta=0.0), isl.IS_ERR_INVALID),
    (dict(ids=None), isl.IS_ERR_INVALID), (dict(D=24), isl.IS_ERR_UNSUPPORTED),
    # no table: theta must be valid; the pointer check refuses a fake store
    (dict(theta=float("nan")), isl.IS_ERR_INVALID), (dict(), isl.IS_ERR_INVALID),
])
def test_inject_rotary_rejects(kw, code):
    assert _rotary(**kw) == code


def _place_inject(**kw):
    a = dict(ids=A, K=A, V=A, offs=A, lens=A, start=0, bt=A, P=16, mb=10, theta=500000.0,
             f=None, pairing=0, pk=A, pv=A, slots=A, pos=A, m=A, k=5, nq=1, n=100, ls=0, rev=1,
             mt=100, L=2, H=8, D=128, T=1000, ns=1000, status=A)
    a.update(kw)
    return isl.load_library().is_place_inject(
        a["ids"], a["K"], a["V"], a["offs"], a["lens"], a["start"], a["bt"], a["P"], a["mb"],
        a["theta"], a["f"], a["pairing"], a["pk"], a["pv"], a["slots"], a["pos"], a["m"], a["k"],
        a["nq"], a["n"], a["ls"], a["rev"], a["mt"], a["L"], a["H"], a["D"], a["T"], a["ns"],
        a["status"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(ids=None), isl.IS_ERR_INVALID), (dict(K=None), isl.IS_ERR_INVALID),
    (dict(bt=None), isl.IS_ERR_INVALID), (dict(slots=None), isl.IS_ERR_INVALID),
    (dict(pos=None), isl.IS_ERR_INVALID), (dict(m=None), isl.IS_ERR_INVALID),
    (dict(pk=None), isl.IS_ERR_INVALID), (dict(k=0), isl.IS_ERR_INVALID),
    (dict(k=1025), isl.IS_ERR_INVALID), (dict(nq=0), isl.IS_ERR_INVALID),
    (dict(nq=70000), isl.IS_ERR_INVALID), (dict(n=0), isl.IS_ERR_INVALID),
    (dict(P=0), isl.IS_ERR_INVALID), (dict(start=-1), isl.IS_ERR_INVALID),
    (dict(mb=-1), isl.IS_ERR_INVALID), (dict(mt=-1), isl.IS_ERR_INVALID),
    (dict(start=2 ** 31 - 10), isl.IS_ERR_INVALID), (dict(ls=-1), isl.IS_ERR_INVALID),
    (dict(L=0), isl.IS_ERR_INVALID), (dict(D=24), isl.IS_ERR_UNSUPPORTED),
    (dict(D=528), isl.IS_ERR_UNSUPPORTED), (dict(T=-1), isl.IS_ERR_INVALID),
    (dict(ns=-1), isl.IS_ERR_INVALID), (dict(theta=0.0), isl.IS_ERR_INVALID),
    (dict(theta=float("nan")), isl.IS_ERR_INVALID), (dict(pairing=2), isl.IS_ERR_INVALID),
    (dict(f=A + 4), isl.IS_ERR_INVALID), (dict(K=A + 8), isl.IS_ERR_INVALID),
    (dict(slots=A + 4), isl.IS_ERR_INVALID), (dict(bt=A + 2), isl.IS_ERR_INVALID),
    (dict(m=A + 2), isl.IS_ERR_INVALID), (dict(status=A + 1), isl.IS_ERR_INVALID),
    # every argument valid: the pointer check refuses a fake store
    (dict(), isl.IS_ERR_INVALID),
])
def test_place_inject_rejects(kw, code):
    assert _place_inject(**kw) == code
    assert isl.load_library().is_last_error().decode()


def _scores(**kw):
    a = dict(q=A, qpos=A, pk=A, layer=0, bt=A, P=16, start=0, m=A, sc=A, nq=1, Hq=32, H=8,
             D=128, L=2, ns=1000, mb=10, mt=100, theta=500000.0, f=None, pairing=0, status=A)
    a.update(kw)
    return isl.load_library().is_paged_scores(
        a["q"], a["qpos"], a["pk"], a["layer"], a["bt"], a["P"], a["start"], a["m"], a["sc"],
        a["nq"], a["Hq"], a["H"], a["D"], a["L"], a["ns"], a["mb"], a["mt"], a["theta"], a["f"],
        a["pairing"], a["status"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), isl.IS_ERR_INVALID), (dict(sc=None), isl.IS_ERR_INVALID),
    (dict(nq=0), isl.IS_ERR_INVALID), (dict(Hq=12), isl.IS_ERR_UNSUPPORTED),
    (dict(Hq=8 * 9), isl.IS_ERR_UNSUPPORTED), (dict(D=96), isl.IS_ERR_UNSUPPORTED),
    (dict(D=8), isl.IS_ERR_UNSUPPORTED), (dict(Hq=64, D=256), isl.IS_ERR_UNSUPPORTED),
    (dict(layer=2), isl.IS_ERR_INVALID), (dict(layer=-1), isl.IS_ERR_INVALID),
    (dict(P=0), isl.IS_ERR_INVALID), (dict(mb=0), isl.IS_ERR_INVALID),
    (dict(theta=0.0), isl.IS_ERR_INVALID), (dict(pairing=3), isl.IS_ERR_INVALID),
    (dict(pk=A + 8), isl.IS_ERR_INVALID), (dict(f=A + 4), isl.IS_ERR_INVALID),
])
def test_paged_scores_rejects(kw, code):
    assert _scores(**kw) == code


def _ann_build(**kw):
    a = dict(bank=A, n=1000, d=64, R=16, dt=1, ns=8, G=A, F=None, sid=A, sb=A, ws=A,
             wsb=1 << 34)
    a.update(kw)
    return isl.load_library().is_ann_build(a["bank"], a["n"], a["d"], a["R"], a["dt"], a["ns"],
                                           a["G"], a["F"], a["sid"], a["sb"], a["ws"], a["wsb"],
                                           None)


@pytest.mark.parametrize("kw,code", [
    (dict(bank=None), isl.IS_ERR_INVALID), (dict(G=None), isl.IS_ERR_INVALID),
    (dict(n=1), isl.IS_ERR_INVALID), (dict(d=12), isl.IS_ERR_INVALID),
    (dict(d=8200), isl.IS_ERR_INVALID), (dict(dt=3), isl.IS_ERR_UNSUPPORTED),
    (dict(R=0), isl.IS_ERR_INVALID), (dict(R=129), isl.IS_ERR_INVALID),
    (dict(n=10, R=10), isl.IS_ERR_INVALID), (dict(ns=-1), isl.IS_ERR_INVALID),
    (dict(ns=1001), isl.IS_ERR_INVALID), (dict(sid=None), isl.IS_ERR_INVALID),
    (dict(sb=None), isl.IS_ERR_INVALID), (dict(bank=A + 8), isl.IS_ERR_INVALID),
    (dict(G=A + 2), isl.IS_ERR_INVALID), (dict(ws=None), isl.IS_ERR_WORKSPACE),
    (dict(wsb=1024), isl.IS_ERR_WORKSPACE), (dict(ws=A + 64), isl.IS_ERR_INVALID),
])
def test_ann_build_rejects(kw, code):
    assert _ann_build(**kw) == code
    assert isl.load_library().is_last_error().decode()


def _ann_search(**kw):
    a = dict(q=A, nq=4, bank=A, n=1000, d=64, dt=1, G=A, R=16, sid=A, sb=A, ns=8, B=64, P=1,
             k=10, T=100, ids=A, sc=None, it=None, ev=None, st=None, ws=A, wsb=1 << 34)
    a.update(kw)
    return isl.load_library().is_ann_search(
        a["q"], a["nq"], a["bank"], a["n"], a["d"], a["dt"], a["G"], a["R"], a["sid"], a["sb"],
        a["ns"], a["B"], a["P"], a["k"], a["T"], a["ids"], a["sc"], a["it"], a["ev"], a["st"],
        a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), isl.IS_ERR_INVALID), (dict(G=None), isl.IS_ERR_INVALID),
    (dict(sid=None), isl.IS_ERR_INVALID), (dict(sb=None), isl.IS_ERR_INVALID),
    (dict(ids=None), isl.IS_ERR_INVALID), (dict(nq=0), isl.IS_ERR_INVALID),
    (dict(nq=65536), isl.IS_ERR_INVALID), (dict(d=4104), isl.IS_ERR_UNSUPPORTED),
    (dict(dt=0, d=2056), isl.IS_ERR_UNSUPPORTED), (dict(R=129), isl.IS_ERR_INVALID),
    (dict(ns=0), isl.IS_ERR_INVALID), (dict(ns=1001), isl.IS_ERR_INVALID),
    (dict(B=0), isl.IS_ERR_INVALID), (dict(B=257), isl.IS_ERR_INVALID),
    (dict(P=0), isl.IS_ERR_INVALID), (dict(P=5), isl.IS_ERR_INVALID),
    (dict(P=3, R=100), isl.IS_ERR_INVALID), (dict(k=0), isl.IS_ERR_INVALID),
    (dict(k=65), isl.IS_ERR_INVALID), (dict(T=-1), isl.IS_ERR_INVALID),
    (dict(q=A + 4), isl.IS_ERR_INVALID), (dict(sb=A + 8), isl.IS_ERR_INVALID),
    (dict(it=A + 2), isl.IS_ERR_INVALID), (dict(ev=A + 2), isl.IS_ERR_INVALID),
    (dict(ws=None), isl.IS_ERR_WORKSPACE),
    (dict(wsb=512), isl.IS_ERR_WORKSPACE),
])
def test_ann_search_rejects(kw, code):
    assert _ann_search(**kw) == code
    assert isl.load_library().is_last_error().decode()


def test_ann_workspace_sizes_are_pure_host():
    assert isl.is_ann_build_workspace_size(1000000, 1024, 64, isl.IS_DTYPE_BF16) > 1000000 * 64 * 4
    assert isl.is_ann_search_workspace_size(1024, 1024, 64, 256, isl.IS_DTYPE_BF16) >= 256 * 64 * 8
    with pytest.raises(isl.InferScaleError):
        isl.is_ann_build_workspace_size(10, 64, 10, isl.IS_DTYPE_F32)


def _noalloc(**kw):
    a = dict(q=A, bank=A, n=1000, d=64, k=10, ids=A, scores=A, nq=1, stride=0, dt=0,
             stream=None)
    a.update(kw)
    lib = isl.load_library()
    return lib.is_retrieve_noalloc(a["q"], a["bank"], a["n"], a["d"], a["k"], a["ids"],
                                   a["scores"], a["nq"], a["stride"], a["dt"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), isl.IS_ERR_INVALID),
    (dict(ids=None), isl.IS_ERR_INVALID),
    (dict(k=0), isl.IS_ERR_INVALID),
    (dict(d=60), isl.IS_ERR_INVALID),
    (dict(dt=7), isl.IS_ERR_UNSUPPORTED),
    (dict(stride=12), isl.IS_ERR_INVALID),
    (dict(bank=A + 8), isl.IS_ERR_INVALID),
    # scores alone need nq * n * 4 bytes: beyond the fixed 16 MiB array
    (dict(n=5_000_000), isl.IS_ERR_WORKSPACE),
    (dict(n=100_000, nq=64), isl.IS_ERR_WORKSPACE),
])
def test_retrieve_noalloc_rejects_on_host(kw, code):
    assert _noalloc(**kw) == code
    assert isl.load_library().is_last_error()


def test_retrieve_noalloc_limit_message_names_the_sizes():
    assert _noalloc(n=5_000_000) == isl.IS_ERR_WORKSPACE
    msg = isl.load_library().is_last_error().decode()
    assert "is_retrieve_noalloc" in msg and str(isl.IS_RETRIEVE_NOALLOC_MAX_BYTES) in msg
    # the workspace is_retrieve would need is the figure it reports
    need = isl.is_retrieve_workspace_size(5_000_000, 64, 10, 1, 0)
    assert str(need) in msg


@pytest.mark.parametrize("dst,src,nbytes", [
    (None, A, 64), (A, None, 64), (A + 8, 2 * A, 64), (A, 2 * A + 4, 64), (A, 2 * A, 65),
    (A, A + 32, 64),  # overlapping
])
def test_stream_copy_rejects(dst, src, nbytes):
    lib = isl.load_library()
    assert lib.is_stream_copy(dst, src, nbytes, None) == isl.IS_ERR_INVALID
    assert lib.is_last_error()


def test_stream_copy_of_nothing_enqueues_nothing():
    assert isl.load_library().is_stream_copy(None, None, 0, None) == isl.IS_OK
