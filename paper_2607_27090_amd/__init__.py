"""Python binding of libinferscale (MI355X / gfx950).

Argument marshalling only: every step of the retrieve + Chunked-RoPE inject
path runs in the library's HIP kernels. Tensors are torch device tensors;
their data pointers and torch's current HIP stream are handed to the C ABI
declared in include/inferscale.h. If the library is not built, importing the
functions raises: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch  # loaded first so the library binds to torch's HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libinferscale.so")

IS_OK = 0
IS_ERR_INVALID = -1
IS_ERR_UNSUPPORTED = -2
IS_ERR_WORKSPACE = -3
IS_ERR_HIP = -4

IS_DTYPE_F32 = 0
IS_DTYPE_BF16 = 1

IS_DEV_ID_RANGE = 1
IS_DEV_BT_SHORT = 2
IS_DEV_CAPACITY = 4
IS_DEV_BAD_LEN = 8
IS_DEV_BAD_BLOCK = 16
IS_DEV_SLOT_RANGE = 32
IS_DEV_SRC_RANGE = 64

IS_MAX_K = 1024
IS_MAX_HEAD_DIM = 512
IS_RETRIEVE_NOALLOC_MAX_BYTES = 16 << 20

IS_ROPE_HALF_SPLIT = 0
IS_ROPE_INTERLEAVED = 1

IS_ANN_MAX_DEGREE = 128
IS_ANN_MAX_BEAM = 256
IS_ANN_MAX_WIDTH = 4
IS_ANN_MAX_EXPAND = 256

EXPORTED = ("is_version", "is_last_error", "is_retrieve_workspace_size", "is_retrieve",
            "is_retrieve_noalloc", "is_slot_map", "is_stream_copy", "is_inject", "is_inject_rotary", "is_place_inject", "is_paged_scores",
            "is_ann_build_workspace_size", "is_ann_build", "is_ann_search_workspace_size",
            "is_ann_search")


class InferScaleError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn} returned {code}: {msg}")
        self.code = code


_lib = None


def load_library() -> ctypes.CDLL:
    """Load libinferscale.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(LIB_PATH, mode=os.RTLD_NOW | os.RTLD_LOCAL)
    P = ctypes.c_void_p
    i32, i64, sz, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
    lib.is_version.argtypes = []
    lib.is_version.restype = ctypes.c_char_p
    lib.is_last_error.argtypes = []
    lib.is_last_error.restype = ctypes.c_char_p
    lib.is_retrieve_workspace_size.argtypes = [i64, i32, i32, i32, i32, ctypes.POINTER(sz)]
    lib.is_retrieve_workspace_size.restype = ctypes.c_int
    lib.is_retrieve.argtypes = [P, P, i64, i32, i32, P, P, i32, i64, i32, P, sz, P]
    lib.is_retrieve.restype = ctypes.c_int
    lib.is_retrieve_noalloc.argtypes = [P, P, i64, i32, i32, P, P, i32, i64, i32, P]
    lib.is_retrieve_noalloc.restype = ctypes.c_int
    lib.is_stream_copy.argtypes = [P, P, sz, P]
    lib.is_stream_copy.restype = ctypes.c_int
    lib.is_slot_map.argtypes = [P, P, i32, P, i32, P, P, P, i32, i32, i64, i64, i32, i32, i32, P, P]
    lib.is_slot_map.restype = ctypes.c_int
    lib.is_inject.argtypes = [P, P, P, P, P, f32, P, P, P, P, P, i32, i32, i64, i64, i32, i32,
                              i32, i32, i32, i64, i64, P, P]
    lib.is_inject.restype = ctypes.c_int
    lib.is_inject_rotary.argtypes = [P, P, P, P, P, f32, P, P, P, P, P, i32, i32, i64, i64, i32,
                                     i32, i32, i32, i32, i64, i64, P, i32, P, P]
    lib.is_inject_rotary.restype = ctypes.c_int
    lib.is_place_inject.argtypes = [P, P, P, P, P, i32, P, i32, i32, f32, P, i32, P, P, P, P, P,
                                    i32, i32, i64, i64, i32, i32, i32, i32, i32, i64, i64, P, P]
    lib.is_place_inject.restype = ctypes.c_int
    lib.is_paged_scores.argtypes = [P, P, P, i32, P, i32, i32, P, P, i32, i32, i32, i32, i32,
                                    i64, i32, i32, f32, P, i32, P, P]
    lib.is_paged_scores.restype = ctypes.c_int
    lib.is_ann_build_workspace_size.argtypes = [i64, i32, i32, i32, ctypes.POINTER(sz)]
    lib.is_ann_build_workspace_size.restype = ctypes.c_int
    lib.is_ann_build.argtypes = [P, i64, i32, i32, i32, i32, P, P, P, P, P, sz, P]
    lib.is_ann_build.restype = ctypes.c_int
    lib.is_ann_search_workspace_size.argtypes = [i32, i32, i32, i32, i32, ctypes.POINTER(sz)]
    lib.is_ann_search_workspace_size.restype = ctypes.c_int
    lib.is_ann_search.argtypes = [P, i32, P, i64, i32, i32, P, i32, P, P, i32, i32, i32, i32,
                                  i32, P, P, P, P, P, P, sz, P]
    lib.is_ann_search.restype = ctypes.c_int
    _lib = lib
    return lib


def _store_ptr(x):
    """Pointer of a pre-RoPE store tensor: device memory, or pinned host memory
    that the inject kernel reads over the host link (the library checks that
    it is mapped for the device)."""
    if isinstance(x, torch.Tensor) and not x.is_cuda:
        if not x.is_pinned():
            raise ValueError("a host-resident store must be pinned (pin_memory=True)")
        if not x.is_contiguous():
            raise ValueError("libinferscale takes contiguous tensors")
        return x.data_ptr()
    return _ptr(x)


def _check(fn: str, rc: int) -> None:
    if rc != IS_OK:
        msg = load_library().is_last_error().decode(errors="replace")
        raise InferScaleError(fn, rc, msg)


def _ptr(x):
    """Device pointer of a contiguous device tensor (None -> NULL)."""
    if x is None:
        return None
    if not isinstance(x, torch.Tensor):
        raise TypeError(f"expected a torch tensor, got {type(x)}")
    if not x.is_cuda:
        raise ValueError("libinferscale takes device tensors")
    if not x.is_contiguous():
        raise ValueError("libinferscale takes contiguous tensors")
    return x.data_ptr()


_I32 = (torch.int32,)
_I64 = (torch.int64,)
_F32 = (torch.float32,)
_BF16 = (torch.bfloat16,)
_F64 = (torch.float64,)
_FLAGS = (torch.int32, getattr(torch, "uint32", torch.int32))


class _Ptr:
    """A checked tensor argument; becomes its pointer when the call is made."""
    __slots__ = ("x", "store")

    def __init__(self, x, store):
        self.x, self.store = x, store


def _arg(x, name: str, dtypes, numel: int, *, optional: bool = False, store: bool = False):
    """Checks one tensor argument against the C ABI's element type and the
    element count the call's shape arguments imply, so that a wrong dtype or
    a short buffer is refused on the host instead of being read or written
    past its end on the device. Every argument of a call is checked before
    any of them is turned into a pointer (see _call)."""
    if x is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(x, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor, got {type(x).__name__}")
    if x.dtype not in dtypes:
        raise ValueError(f"{name} must be {' or '.join(str(d) for d in dtypes)}, got {x.dtype}")
    if x.numel() < numel:
        raise ValueError(f"{name} holds {x.numel()} elements; the call needs at least {numel}")
    return _Ptr(x, store)


class _Stream:
    """The stream argument of a call, looked up when the call is made."""
    __slots__ = ("s",)

    def __init__(self, s):
        self.s = s


def _call(fn: str, *args) -> None:
    """Calls the C entry point `fn` with checked tensor arguments turned into
    device (or pinned-host store) pointers and the stream looked up, and
    raises on an error code."""
    raw = [(_store_ptr(a.x) if a.store else _ptr(a.x)) if isinstance(a, _Ptr) else a
           for a in args]
    raw = [_resolve_stream(a.s) if isinstance(a, _Stream) else a for a in raw]
    _check(fn, getattr(load_library(), fn)(*raw))


def _table(n: int, nq: int, stride: int) -> int:
    """Entries a per-request table with `stride` elements between requests
    spans (stride 0: one shared table of n entries)."""
    return n if stride == 0 else (nq - 1) * stride + n


# torch's current raw stream without building a Stream object (the public
# torch.cuda.current_stream() costs ~2.6 us of host time per call)
_current_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_current_device = getattr(torch._C, "_cuda_getDevice", None)


def _stream(stream):
    return _Stream(stream)


def _resolve_stream(stream):
    if stream is None:
        if _current_raw_stream is not None and _current_device is not None:
            return _current_raw_stream(_current_device())
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _emb_dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return IS_DTYPE_F32
    if t.dtype == torch.bfloat16:
        return IS_DTYPE_BF16
    raise ValueError(f"embeddings must be float32 or bfloat16, got {t.dtype}")


def is_version() -> str:
    return load_library().is_version().decode()


def is_retrieve_workspace_size(n: int, d: int, k: int, nq: int = 1,
                               dtype: int = IS_DTYPE_F32) -> int:
    out = ctypes.c_size_t(0)
    _check("is_retrieve_workspace_size",
           load_library().is_retrieve_workspace_size(n, d, k, nq, dtype, ctypes.byref(out)))
    return out.value


def is_retrieve(query_emb, bank, n, d, k, out_ids, out_scores=None, *, nq=1, bank_stride=0,
                workspace=None, stream=None) -> None:
    """Exact top-k by inner product (see include/inferscale.h)."""
    dt = _emb_dtype(query_emb)
    if workspace is None:
        raise ValueError("is_retrieve needs a workspace tensor "
                         "(is_retrieve_workspace_size bytes of device memory)")
    ws_bytes = workspace.numel() * workspace.element_size()
    _call("is_retrieve",
        _arg(query_emb, "query_emb", (query_emb.dtype,), nq * d),
        _arg(bank, "bank", (query_emb.dtype,), _table(n * d, nq, bank_stride)), n, d, k,
        _arg(out_ids, "out_ids", _I32, nq * k),
        _arg(out_scores, "out_scores", _F32, nq * k, optional=True), nq, bank_stride,
        dt, _Ptr(workspace, False), ws_bytes, _stream(stream))


def is_retrieve_noalloc(query_emb, bank, n, d, k, out_ids, out_scores=None, *, nq=1,
                        bank_stride=0, stream=None) -> None:
    """is_retrieve with the library's fixed scratch array instead of a
    workspace, for callers that cannot allocate (see include/inferscale.h)."""
    dt = _emb_dtype(query_emb)
    _call("is_retrieve_noalloc",
        _arg(query_emb, "query_emb", (query_emb.dtype,), nq * d),
        _arg(bank, "bank", (query_emb.dtype,), _table(n * d, nq, bank_stride)), n, d, k,
        _arg(out_ids, "out_ids", _I32, nq * k),
        _arg(out_scores, "out_scores", _F32, nq * k, optional=True), nq, bank_stride,
        dt, _stream(stream))


def is_stream_copy(dst, src, stream=None) -> None:
    """dst[:] = src[:] by the library's streaming copy (equal byte sizes; see
    include/inferscale.h)."""
    nb = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nb:
        raise ValueError("dst and src must hold the same number of bytes")
    _call("is_stream_copy", _Ptr(dst, False), _Ptr(src, False), nb, _stream(stream))


def is_slot_map(ids, fact_lens, start_pos, block_table, page_size, out_slots, out_positions,
                out_m, *, k, nq, n, lens_stride, max_blocks, max_tokens, reverse_rank=1,
                status=None, stream=None) -> None:
    """Placement + slot map (see include/inferscale.h)."""
    _call("is_slot_map",
        _arg(ids, "ids", _I32, nq * k), _arg(fact_lens, "fact_lens", _I32,
                                             _table(n, nq, lens_stride)),
        start_pos, _arg(block_table, "block_table", _I32, nq * max_blocks), page_size,
        _arg(out_slots, "out_slots", _I64, nq * max_tokens),
        _arg(out_positions, "out_positions", _I32, nq * max_tokens),
        _arg(out_m, "out_m", _I32, nq), k, nq, n, lens_stride, max_blocks, max_tokens,
        reverse_rank, _arg(status, "status", _FLAGS, 1, optional=True), _stream(stream))


def is_inject(ids, preK, V, slots, positions, rope_theta, paged_k, paged_v, *, fact_offsets,
              fact_lens, m, k, nq, n, lens_stride, reverse_rank=1, max_tokens, L, H, D,
              T_store, num_slots, status=None, stream=None) -> None:
    """Fused gather + RoPE + scatter (see include/inferscale.h)."""
    a = _inject_args(ids, preK, V, slots, positions, paged_k, paged_v, fact_offsets, fact_lens,
                     m, k, nq, n, lens_stride, max_tokens, L, H, D, T_store, num_slots)
    _call("is_inject",
        a["ids"], a["preK"], a["V"], a["slots"], a["positions"], float(rope_theta), a["paged_k"],
        a["paged_v"], a["fact_offsets"], a["fact_lens"], a["m"], k, nq, n, lens_stride,
        reverse_rank, max_tokens, L, H, D, T_store, num_slots,
        _arg(status, "status", _FLAGS, 1, optional=True), _stream(stream))


def _inject_args(ids, preK, V, slots, positions, paged_k, paged_v, fact_offsets, fact_lens, m,
                 k, nq, n, lens_stride, max_tokens, L, H, D, T_store, num_slots):
    """Checked pointers of the arguments is_inject and its variants share
    (for is_place_inject, slots, positions and m are its outputs)."""
    store = L * T_store * H * D
    pages = L * num_slots * H * D
    table = _table(n, nq, lens_stride)
    return {
        "ids": _arg(ids, "ids", _I32, nq * k),
        "preK": _arg(preK, "preK", _BF16, store, store=True),
        "V": _arg(V, "V", _BF16, store, store=True),
        "slots": _arg(slots, "slots", _I64, nq * max_tokens),
        "positions": _arg(positions, "positions", _I32, nq * max_tokens),
        "paged_k": _arg(paged_k, "paged_k", _BF16, pages),
        "paged_v": _arg(paged_v, "paged_v", _BF16, pages),
        "fact_offsets": _arg(fact_offsets, "fact_offsets", _I64, table),
        "fact_lens": _arg(fact_lens, "fact_lens", _I32, table),
        "m": _arg(m, "m", _I32, nq),
    }


def is_inject_rotary(ids, preK, V, slots, positions, rope_theta, paged_k, paged_v, *,
                     fact_offsets, fact_lens, m, k, nq, n, lens_stride, reverse_rank=1,
                     max_tokens, L, H, D, T_store, num_slots, inv_freq=None,
                     pairing=IS_ROPE_HALF_SPLIT, status=None, stream=None) -> None:
    """is_inject with the model's rotary table (float64 device tensor [D/2],
    None: rope_theta's default table) and pair layout (see include/inferscale.h)."""
    a = _inject_args(ids, preK, V, slots, positions, paged_k, paged_v, fact_offsets, fact_lens,
                     m, k, nq, n, lens_stride, max_tokens, L, H, D, T_store, num_slots)
    _call("is_inject_rotary",
        a["ids"], a["preK"], a["V"], a["slots"], a["positions"], float(rope_theta), a["paged_k"],
        a["paged_v"], a["fact_offsets"], a["fact_lens"], a["m"], k, nq, n, lens_stride,
        reverse_rank, max_tokens, L, H, D, T_store, num_slots,
        _arg(inv_freq, "inv_freq", _F64, D // 2, optional=True), int(pairing),
        _arg(status, "status", _FLAGS, 1, optional=True), _stream(stream))


def is_place_inject(ids, preK, V, rope_theta, paged_k, paged_v, out_slots, out_positions, out_m,
                    *, fact_offsets, fact_lens, start_pos, block_table, page_size, max_blocks, k,
                    nq, n, lens_stride, reverse_rank=1, max_tokens, L, H, D, T_store, num_slots,
                    inv_freq=None, pairing=IS_ROPE_HALF_SPLIT, status=None, stream=None) -> None:
    """Slot map + inject in one launch (see include/inferscale.h)."""
    a = _inject_args(ids, preK, V, out_slots, out_positions, paged_k, paged_v, fact_offsets,
                     fact_lens, out_m, k, nq, n, lens_stride, max_tokens, L, H, D, T_store,
                     num_slots)
    _call("is_place_inject",
        a["ids"], a["preK"], a["V"], a["fact_offsets"], a["fact_lens"], start_pos,
        _arg(block_table, "block_table", _I32, nq * max_blocks), page_size, max_blocks,
        float(rope_theta), _arg(inv_freq, "inv_freq", _F64, D // 2, optional=True),
        int(pairing), a["paged_k"], a["paged_v"], a["slots"], a["positions"], a["m"], k, nq, n,
        lens_stride, reverse_rank, max_tokens, L, H, D, T_store, num_slots,
        _arg(status, "status", _FLAGS, 1, optional=True), _stream(stream))


def is_paged_scores(q, qpos, paged_k, layer, block_table, page_size, start_pos, m, scores, *,
                    nq, Hq, H, D, L, num_slots, max_blocks, max_tokens, rope_theta,
                    inv_freq=None, pairing=IS_ROPE_HALF_SPLIT, status=None, stream=None) -> None:
    """Attention logits of each request's query against its injected keys
    read through the block table (see include/inferscale.h)."""
    _call("is_paged_scores",
        _arg(q, "q", _BF16, nq * Hq * D), _arg(qpos, "qpos", _I32, nq),
        _arg(paged_k, "paged_k", _BF16, L * num_slots * H * D), layer,
        _arg(block_table, "block_table", _I32, nq * max_blocks), page_size, start_pos,
        _arg(m, "m", _I32, nq), _arg(scores, "scores", _F32, nq * Hq * max_tokens), nq, Hq, H,
        D, L, num_slots, max_blocks, max_tokens, float(rope_theta),
        _arg(inv_freq, "inv_freq", _F64, D // 2, optional=True), int(pairing),
        _arg(status, "status", _FLAGS, 1, optional=True), _stream(stream))



def is_ann_build_workspace_size(n: int, d: int, degree: int, dtype: int = IS_DTYPE_F32) -> int:
    out = ctypes.c_size_t(0)
    _check("is_ann_build_workspace_size",
           load_library().is_ann_build_workspace_size(n, d, degree, dtype, ctypes.byref(out)))
    return out.value


def is_ann_build(bank, n, d, degree, graph, *, n_seeds=0, fwd=None, seed_ids=None,
                 seed_bank=None, workspace=None, stream=None) -> None:
    """Proximity graph over the bank, plus the search's seeds (see
    include/inferscale.h)."""
    dt = _emb_dtype(bank)
    if workspace is None:
        raise ValueError("is_ann_build needs a workspace tensor "
                         "(is_ann_build_workspace_size bytes of device memory)")
    ws_bytes = workspace.numel() * workspace.element_size()
    _call("is_ann_build",
        _arg(bank, "bank", (bank.dtype,), n * d), n, d, degree, dt, n_seeds,
        _arg(graph, "graph", _I32, n * degree), _arg(fwd, "fwd", _I32, n * degree, optional=True),
        _arg(seed_ids, "seed_ids", _I32, n_seeds, optional=n_seeds == 0),
        _arg(seed_bank, "seed_bank", (bank.dtype,), n_seeds * d, optional=n_seeds == 0),
        _Ptr(workspace, False), ws_bytes, _stream(stream))


def is_ann_search_workspace_size(n_seeds: int, d: int, beam: int, nq: int = 1,
                                 dtype: int = IS_DTYPE_F32) -> int:
    out = ctypes.c_size_t(0)
    _check("is_ann_search_workspace_size",
           load_library().is_ann_search_workspace_size(n_seeds, d, beam, nq, dtype,
                                                       ctypes.byref(out)))
    return out.value


def is_ann_search(query_emb, bank, n, d, graph, degree, seed_ids, seed_bank, out_ids, *,
                  nq=1, n_seeds, beam=64, width=1, k, max_iters, out_scores=None, out_iters=None,
                  out_scored=None, status=None, workspace=None, stream=None) -> None:
    """Beam search over the proximity graph (see include/inferscale.h)."""
    dt = _emb_dtype(query_emb)
    if workspace is None:
        raise ValueError("is_ann_search needs a workspace tensor "
                         "(is_ann_search_workspace_size bytes of device memory)")
    ws_bytes = workspace.numel() * workspace.element_size()
    et = (query_emb.dtype,)
    _call("is_ann_search",
        _arg(query_emb, "query_emb", et, nq * d), nq, _arg(bank, "bank", et, n * d), n, d, dt,
        _arg(graph, "graph", _I32, n * degree), degree, _arg(seed_ids, "seed_ids", _I32, n_seeds),
        _arg(seed_bank, "seed_bank", et, n_seeds * d), n_seeds, beam, width, k, max_iters,
        _arg(out_ids, "out_ids", _I32, nq * k),
        _arg(out_scores, "out_scores", _F32, nq * k, optional=True),
        _arg(out_iters, "out_iters", _I32, nq, optional=True),
        _arg(out_scored, "out_scored", _I32, nq, optional=True),
        _arg(status, "status", _FLAGS, 1, optional=True), _Ptr(workspace, False), ws_bytes,
        _stream(stream))
