"""Plain CPU oracle for the retrieve + Chunked-RoPE inject path (binary64).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product library. The arithmetic is
in ``oracle.c`` (plain C, compiled with gcc); this module only marshals numpy
arrays into it. It shares no code with the HIP library.

Paper passages followed (InferScale):
  * scores / top-k: §3.2 "Persistent memory store and retrieval" (top-k
    search by inner product over fact embeddings), exact brute force;
  * placement: §5.2 "Position policy" (contiguous facts, cumulative offsets,
    most relevant fact adjacent to the query);
  * slots: §2.2 paged KV cache (fixed-size blocks through a block table);
  * rotation: §2.4 and Theorem "Chunked RoPE Injection" (§5.1); with the
    model's own rotary table and pair layout, §3.3 and §6.1;
  * composition and scatter: §3.3 and §3.4;
  * the consumer of the pages (attention logits of the query that follows
    the memory): Theorem "Chunked RoPE Injection", §5.1;
  * the graph-ANN backend (proximity graph and beam search, §2.6 and §6.1)
    in ``ann.c``, with the readings stated at its top.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_SRCS = [_SRC, os.path.join(_HERE, "ann.c")]
_LIB = os.path.join(_HERE, "liboracle.so")

F32 = 0
BF16 = 1

ID_RANGE = 1
BT_SHORT = 2
CAPACITY = 4
BAD_LEN = 8
BAD_BLOCK = 16
SLOT_RANGE = 32
SRC_RANGE = 64

_lib = None


def build() -> str:
    """Compile oracle.c and ann.c into liboracle.so with gcc (strict IEEE, no
    fast-math; OpenMP for the loops over independent outputs)."""
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fno-fast-math", "-ffp-contract=off",
           "-fopenmp", "-std=c11", "-Wall", "-Wno-maybe-uninitialized", "-o", _LIB, *_SRCS,
           "-lm"]
    subprocess.run(cmd, check=True)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < max(map(os.path.getmtime, _SRCS)):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32, i64, f64, u16 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_uint16
    lib.oracle_set_threads.argtypes = [i32]
    lib.oracle_set_threads.restype = None
    lib.oracle_threads.argtypes = []
    lib.oracle_threads.restype = i32
    lib.oracle_bf16_to_double.argtypes = [u16]
    lib.oracle_bf16_to_double.restype = f64
    lib.oracle_double_to_bf16.argtypes = [f64]
    lib.oracle_double_to_bf16.restype = u16
    lib.oracle_double_to_bf16_n.argtypes = [P, i64, P]
    lib.oracle_double_to_bf16_n.restype = None
    lib.oracle_scores.argtypes = [P, P, i64, i32, i32, i64, i32, P]
    lib.oracle_scores.restype = ctypes.c_int
    lib.oracle_topk.argtypes = [P, i64, i32, i32, P, P]
    lib.oracle_topk.restype = ctypes.c_int
    lib.oracle_slot_map.argtypes = [P, P, i32, P, i32, i32, i32, i64, i64, i32, i32, i32,
                                    P, P, P, P, P, P]
    lib.oracle_slot_map.restype = ctypes.c_int
    lib.oracle_rope_f64.argtypes = [P, f64, f64, i32, P]
    lib.oracle_rope_f64.restype = None
    lib.oracle_rope_bf16.argtypes = [P, i64, f64, i32, P]
    lib.oracle_rope_bf16.restype = None
    lib.oracle_inject.argtypes = [P, P, P, P, P, f64, P, P, P, P, P, i32, i32, i64, i64, i32,
                                  i32, i32, i32, i32, i64, i64, P]
    lib.oracle_inject.restype = ctypes.c_int
    lib.oracle_rope_table_f64.argtypes = [P, f64, P, i32, i32, P]
    lib.oracle_rope_table_f64.restype = None
    lib.oracle_rope_table_bf16.argtypes = [P, i64, P, i32, i32, P]
    lib.oracle_rope_table_bf16.restype = None
    lib.oracle_default_inv_freq.argtypes = [f64, i32, P]
    lib.oracle_default_inv_freq.restype = None
    lib.oracle_inject_rotary.argtypes = [P, P, P, P, P, f64, P, P, P, P, P, i32, i32, i64, i64,
                                         i32, i32, i32, i32, i32, i64, i64, P, i32, P]
    lib.oracle_inject_rotary.restype = ctypes.c_int
    lib.oracle_paged_scores.argtypes = [P, P, P, i32, P, i32, i32, P, f64, P, i32, i32, i32,
                                        i32, i32, i64, i32, i32, P, P]
    lib.oracle_paged_scores.restype = ctypes.c_int
    lib.oracle_ann_knn.argtypes = [P, i64, i32, i32, i32, P]
    lib.oracle_ann_knn.restype = ctypes.c_int
    lib.oracle_ann_merge.argtypes = [P, i64, i32, P]
    lib.oracle_ann_merge.restype = ctypes.c_int
    lib.oracle_ann_build.argtypes = [P, i64, i32, i32, i32, P, P]
    lib.oracle_ann_build.restype = ctypes.c_int
    lib.oracle_ann_search.argtypes = [P, i32, P, i64, i32, i32, P, i32, P, i32, i32, i32, i32,
                                      i32, P, P, P, P]
    lib.oracle_ann_search.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ---- threads ------------------------------------------------------------------

_threads_setting = 0  # 0: the OpenMP default (OMP_NUM_THREADS, else every core)


def set_threads(n: int) -> None:
    """Threads of the scores, top-k and inject loops (0: the OpenMP default).
    Results do not depend on it: every output is computed by one thread."""
    global _threads_setting
    _threads_setting = max(0, int(n))
    _load().oracle_set_threads(_threads_setting)


def threads() -> int:
    """Threads the next scores / top-k / inject call will use."""
    return int(_load().oracle_threads())


class using_threads:
    """Context manager: run the oracle on ``n`` threads inside the block."""

    def __init__(self, n: int):
        self.n = int(n)

    def __enter__(self):
        self._old = _threads_setting
        set_threads(self.n)
        return self

    def __exit__(self, *exc):
        set_threads(self._old)
        return False


# ---- number formats -------------------------------------------------------

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact decode of bf16 bit patterns (uint16) to float64."""
    b = _c(bits, np.uint16)
    with np.errstate(invalid="ignore"):
        return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16(x) -> np.ndarray:
    """Round float64 values to bf16 (nearest, ties to even), as uint16 bits."""
    lib = _load()
    xs = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(xs.shape, dtype=np.uint16)
    lib.oracle_double_to_bf16_n(_ptr(xs), xs.size, _ptr(out))
    return out


# ---- the path ---------------------------------------------------------------

def scores(query: np.ndarray, bank: np.ndarray, n: int, d: int, nq: int,
           bank_stride: int = 0, dtype: int = F32) -> np.ndarray:
    """float64 [nq][n] inner products. query/bank: float32 arrays or bf16
    bit patterns (uint16) matching ``dtype``."""
    lib = _load()
    et = np.float32 if dtype == F32 else np.uint16
    q = _c(query, et)
    b = _c(bank, et)
    out = np.empty((nq, n), dtype=np.float64)
    rc = lib.oracle_scores(_ptr(q), _ptr(b), n, d, nq, bank_stride, dtype, _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_scores rejected its arguments (rc={rc})")
    return out


def topk(sc: np.ndarray, k: int):
    """Full-sort top-k: (ids int32 [nq][k], scores float64 [nq][k])."""
    lib = _load()
    s = _c(sc, np.float64)
    nq, n = s.shape
    ids = np.empty((nq, k), dtype=np.int32)
    vals = np.empty((nq, k), dtype=np.float64)
    rc = lib.oracle_topk(_ptr(s), n, k, nq, _ptr(ids), _ptr(vals))
    if rc != 0:
        raise ValueError(f"oracle_topk rejected its arguments (rc={rc})")
    return ids, vals


def retrieve(query, bank, n, d, k, nq=1, bank_stride=0, dtype=F32):
    """Scores then full-sort top-k; returns (ids, scores_f64, all_scores_f64)."""
    sc = scores(query, bank, n, d, nq, bank_stride, dtype)
    ids, vals = topk(sc, k)
    return ids, vals, sc


def slot_map(ids, fact_lens, start_pos, block_table, page_size, k, nq, n,
             lens_stride, max_blocks, max_tokens, reverse_rank=1):
    """Returns dict(slots, positions, m, fact, tok, status); rows of max_tokens
    beyond m are left at -1."""
    lib = _load()
    ids_ = _c(ids, np.int32)
    lens_ = _c(fact_lens, np.int32)
    bt_ = _c(block_table, np.int32)
    slots = np.full((nq, max_tokens), -1, dtype=np.int64)
    pos = np.full((nq, max_tokens), -1, dtype=np.int32)
    fact = np.full((nq, max_tokens), -1, dtype=np.int32)
    tok = np.full((nq, max_tokens), -1, dtype=np.int32)
    m = np.zeros((nq,), dtype=np.int32)
    status = np.zeros((1,), dtype=np.uint32)
    rc = lib.oracle_slot_map(_ptr(ids_), _ptr(lens_), start_pos, _ptr(bt_), page_size, k, nq, n,
                             lens_stride, max_blocks, max_tokens, reverse_rank,
                             _ptr(slots), _ptr(pos), _ptr(m), _ptr(fact), _ptr(tok), _ptr(status))
    if rc != 0:
        raise ValueError(f"oracle_slot_map rejected its arguments (rc={rc})")
    return dict(slots=slots, positions=pos, m=m, fact=fact, tok=tok, status=int(status[0]))


def rope_f64(x, p, theta, D):
    """R_p x for one head vector x (float64 [D]) in binary64."""
    lib = _load()
    xs = _c(x, np.float64)
    y = np.empty_like(xs)
    lib.oracle_rope_f64(_ptr(xs), float(p), float(theta), D, _ptr(y))
    return y


def rope_bf16(x_bits, p, theta, D):
    """bf16 head vector in, bf16 head vector out (uint16 bit patterns)."""
    lib = _load()
    xs = _c(x_bits, np.uint16)
    y = np.empty_like(xs)
    lib.oracle_rope_bf16(_ptr(xs), int(p), float(theta), D, _ptr(y))
    return y


def rope_rows_bf16(rows, positions, theta, H, D):
    """Rotate a batch of (token) rows [R][H*D] bf16 bits, row i at positions[i]."""
    rows = _c(rows, np.uint16).reshape(-1, H, D)
    out = np.empty_like(rows)
    for i in range(rows.shape[0]):
        for h in range(H):
            out[i, h] = rope_bf16(rows[i, h], int(positions[i]), theta, D)
    return out.reshape(-1, H * D)


def default_inv_freq(theta, D):
    """inv_freq[j] = theta^(-2j/D), j < D/2 (binary64)."""
    lib = _load()
    out = np.empty(D // 2, dtype=np.float64)
    lib.oracle_default_inv_freq(float(theta), D, _ptr(out))
    return out


def rope_table_f64(x, p, inv_freq, D, interleaved=False):
    """R_p x with a given frequency table and pair layout (binary64)."""
    lib = _load()
    xs = _c(x, np.float64)
    f = _c(inv_freq, np.float64)
    y = np.empty_like(xs)
    lib.oracle_rope_table_f64(_ptr(xs), float(p), _ptr(f), D, int(bool(interleaved)), _ptr(y))
    return y


def rope_table_bf16(x_bits, p, inv_freq, D, interleaved=False):
    """bf16 head vector in, bf16 out, with a given table and pair layout."""
    lib = _load()
    xs = _c(x_bits, np.uint16)
    f = _c(inv_freq, np.float64)
    y = np.empty_like(xs)
    lib.oracle_rope_table_bf16(_ptr(xs), int(p), _ptr(f), D, int(bool(interleaved)), _ptr(y))
    return y


def inject(ids, preK, V, slots, positions, rope_theta, paged_k, paged_v, fact_offsets,
           fact_lens, m, k, nq, n, lens_stride, reverse_rank, max_tokens, L, H, D,
           T_store, num_slots, inv_freq=None, interleaved=False):
    """Writes paged_k / paged_v (uint16 arrays, modified in place); returns status.
    inv_freq [D/2] (None: rope_theta's default table) and interleaved select
    the model's rotary table and pair layout."""
    lib = _load()
    ids_ = _c(ids, np.int32)
    pk = _c(preK, np.uint16)
    vv = _c(V, np.uint16)
    sl = _c(slots, np.int64)
    po = _c(positions, np.int32)
    fo = _c(fact_offsets, np.int64)
    fl = _c(fact_lens, np.int32)
    mm = _c(m, np.int32)
    for a in (paged_k, paged_v):
        assert a.dtype == np.uint16 and a.flags["C_CONTIGUOUS"]
    status = np.zeros((1,), dtype=np.uint32)
    f = None if inv_freq is None else _c(inv_freq, np.float64)
    rc = lib.oracle_inject_rotary(_ptr(ids_), _ptr(pk), _ptr(vv), _ptr(sl), _ptr(po),
                                  float(rope_theta), _ptr(paged_k), _ptr(paged_v), _ptr(fo),
                                  _ptr(fl), _ptr(mm), k, nq, n, lens_stride, reverse_rank,
                                  max_tokens, L, H, D, T_store, num_slots, _ptr(f),
                                  int(bool(interleaved)), _ptr(status))
    if rc != 0:
        raise ValueError(f"oracle_inject rejected its arguments (rc={rc})")
    return int(status[0])


def paged_scores(q, qpos, paged_k, layer, block_table, page_size, start_pos, m, rope_theta,
                 nq, Hq, H, D, num_slots, max_blocks, max_tokens, inv_freq=None,
                 interleaved=False):
    """Attention logits of each request's query (rotated to qpos[r]) against
    its placed tokens' keys read through the block table; float64
    [nq][Hq][max_tokens], NaN beyond m. Returns (scores, status)."""
    lib = _load()
    q_ = _c(q, np.uint16)
    qp = _c(qpos, np.int32)
    pk = _c(paged_k, np.uint16)
    bt = _c(block_table, np.int32)
    mm = _c(m, np.int32)
    f = None if inv_freq is None else _c(inv_freq, np.float64)
    out = np.full((nq, Hq, max_tokens), np.nan)
    status = np.zeros((1,), dtype=np.uint32)
    rc = lib.oracle_paged_scores(_ptr(q_), _ptr(qp), _ptr(pk), layer, _ptr(bt), page_size,
                                 start_pos, _ptr(mm), float(rope_theta), _ptr(f),
                                 int(bool(interleaved)), nq, Hq, H, D, num_slots, max_blocks,
                                 max_tokens, _ptr(out), _ptr(status))
    if rc != 0:
        raise ValueError(f"oracle_paged_scores rejected its arguments (rc={rc})")
    return out, int(status[0])



# ---- graph-ANN backend (ann.c) ---------------------------------------------

def _emb(a, dtype):
    return _c(a, np.float32 if dtype == F32 else np.uint16)


def ann_knn(bank, n, d, R, dtype=F32) -> np.ndarray:
    """Forward lists F [n][R]: the R best j != i by inner product, best first,
    equal scores to the lower id."""
    lib = _load()
    b = _emb(bank, dtype)
    F = np.empty((n, R), dtype=np.int32)
    rc = lib.oracle_ann_knn(_ptr(b), n, d, dtype, R, _ptr(F))
    if rc != 0:
        raise ValueError(f"oracle_ann_knn rejected its arguments (rc={rc})")
    return F


def ann_merge(F) -> np.ndarray:
    """Final lists G [n][R] from forward lists F (forward half, reverse edges,
    forward fill)."""
    lib = _load()
    F_ = _c(F, np.int32)
    n, R = F_.shape
    G = np.empty((n, R), dtype=np.int32)
    rc = lib.oracle_ann_merge(_ptr(F_), n, R, _ptr(G))
    if rc != 0:
        raise ValueError(f"oracle_ann_merge rejected its arguments (rc={rc})")
    return G


def ann_build(bank, n, d, R, dtype=F32):
    """(F, G): forward lists and final graph."""
    lib = _load()
    b = _emb(bank, dtype)
    F = np.empty((n, R), dtype=np.int32)
    G = np.empty((n, R), dtype=np.int32)
    rc = lib.oracle_ann_build(_ptr(b), n, d, dtype, R, _ptr(F), _ptr(G))
    if rc != 0:
        raise ValueError(f"oracle_ann_build rejected its arguments (rc={rc})")
    return F, G


def ann_search(query, bank, n, d, graph, seeds, beam, k, max_iters, width=1, dtype=F32):
    """Beam search: returns dict(ids int32 [nq][k], scores float64 [nq][k],
    iters int32 [nq], status)."""
    lib = _load()
    q = _emb(query, dtype)
    nq = q.size // d
    b = _emb(bank, dtype)
    g = _c(graph, np.int32)
    R = g.shape[1]
    s = _c(seeds, np.int32)
    ids = np.empty((nq, k), dtype=np.int32)
    vals = np.empty((nq, k), dtype=np.float64)
    iters = np.empty((nq,), dtype=np.int32)
    status = np.zeros((1,), dtype=np.uint32)
    rc = lib.oracle_ann_search(_ptr(q), nq, _ptr(b), n, d, dtype, _ptr(g), R, _ptr(s), s.size,
                               beam, width, k, max_iters, _ptr(ids), _ptr(vals), _ptr(iters),
                               _ptr(status))
    if rc != 0:
        raise ValueError(f"oracle_ann_search rejected its arguments (rc={rc})")
    return dict(ids=ids, scores=vals, iters=iters, status=int(status[0]))
