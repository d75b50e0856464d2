"""Seeded synthetic inputs shaped like the paper's serving workloads.

This module only draws inputs and sizes buffers; it holds none of the
retrieve / placement / rotation arithmetic, so both the HIP path and the
oracle can be fed from it without sharing any of the method.

Shapes follow the paper's setting (§3.5 storage formula: per-token KV of
2*L*H*D*b bytes; §2.2 16-token pages; short facts a few dozen tokens long;
top-k up to 50 per request, §6.2) with synthetic values:

* fact embeddings: N(0, I) rows L2-normalised in fp32 (then rounded to bf16
  for the bf16 configurations); the clustered bank uses
  x = normalize(c + sigma * g / sqrt(d)) around 256 unit centroids;
* queries: drawn the same way, independently of the bank;
* fact lengths: integers uniform in [lo, hi], both ends inclusive;
* pre-RoPE keys and values: N(0, 1) rounded to bf16;
* block tables: disjoint slices of a random permutation of the page pool;
* page pools: filled with a sentinel bit pattern so untouched slots are
  detectable.

When the full per-fact KV store would not fit in one GPU's memory, facts are
aliased onto a pool of distinct payloads: fact_offsets[id] points at a
payload, fact_lens[id] is that payload's length.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import torch

SENTINEL_BITS = 0x7FA5  # a bf16 NaN pattern the path never produces
BASE_SEED = 20260727


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    L: int
    H: int
    D: int
    n: int                 # facts per bank
    len_lo: int
    len_hi: int
    d_e: int               # embedding dimension
    emb_dtype: str         # "f32" or "bf16"
    nq: int                # concurrent queries
    shared_bank: bool      # one bank for every query, or one bank per query
    k: int
    page_size: int
    theta: float
    start_pos: int
    clustered: bool = False
    centroids: int = 256
    sigma: float = 0.1
    payloads: Optional[int] = None   # distinct KV payloads (None: one per fact)
    index: int = 0

    @property
    def max_tokens(self) -> int:
        return self.k * self.len_hi

    @property
    def max_blocks(self) -> int:
        return -(-(self.start_pos + self.max_tokens) // self.page_size)

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


TINY = Workload("tiny", L=4, H=8, D=128, n=256, len_lo=16, len_hi=48, d_e=384, emb_dtype="f32",
                nq=1, shared_bank=True, k=5, page_size=16, theta=500000.0, start_pos=64, index=0)
LLAMA8B = Workload("llama3.1-8b", L=32, H=8, D=128, n=10000, len_lo=16, len_hi=64, d_e=768,
                   emb_dtype="f32", nq=1, shared_bank=True, k=50, page_size=16, theta=500000.0,
                   start_pos=128, index=1)
CONCURRENCY = Workload("concurrency-64users", L=32, H=8, D=128, n=2000, len_lo=16, len_hi=64,
                       d_e=768, emb_dtype="f32", nq=64, shared_bank=False, k=50, page_size=16,
                       theta=500000.0, start_pos=128, payloads=8192, index=2)
LLAMA70B = Workload("llama3-70b", L=80, H=8, D=128, n=100000, len_lo=16, len_hi=96, d_e=1024,
                    emb_dtype="bf16", nq=8, shared_bank=True, k=100, page_size=16,
                    theta=500000.0, start_pos=128, payloads=2048, index=3)
RETRIEVAL1M = Workload("retrieval-1m", L=32, H=8, D=128, n=1000000, len_lo=16, len_hi=64,
                       d_e=1024, emb_dtype="bf16", nq=256, shared_bank=True, k=100, page_size=32,
                       theta=500000.0, start_pos=128, clustered=True, payloads=2048, index=4)

ALL = [TINY, LLAMA8B, CONCURRENCY, LLAMA70B, RETRIEVAL1M]


def llama31_inv_freq(D: int, theta: float = 500000.0, factor: float = 8.0,
                     low_freq_factor: float = 1.0, high_freq_factor: float = 4.0,
                     original_context: int = 8192):
    """A model's own rotary table: Llama 3.1's published RoPE frequency
    scaling applied to theta^(-2j/D) (binary64, [D/2]). Wavelengths below
    original_context / high_freq_factor keep their frequency, those above
    original_context / low_freq_factor are divided by `factor`, and the band
    in between interpolates linearly in original_context / wavelength."""
    import numpy as np
    base = theta ** (-np.arange(0, D, 2, dtype=np.float64) / D)
    out = base.copy()
    lo_wl = original_context / low_freq_factor
    hi_wl = original_context / high_freq_factor
    for j, f in enumerate(base):
        wl = 2.0 * math.pi / f
        if wl < hi_wl:
            continue
        if wl > lo_wl:
            out[j] = f / factor
        else:
            smooth = (original_context / wl - low_freq_factor) / (high_freq_factor - low_freq_factor)
            out[j] = (1.0 - smooth) * f / factor + smooth * f
    return out


def kv_bytes_per_token(w: Workload) -> int:
    """Stored KV bytes of one fact token across all layers (K and V, bf16):
    2 * L * H * D * 2 (§3.5 with c = 1, b = 2)."""
    return 2 * w.L * w.H * w.D * 2


def inject_algorithmic_bytes(w: Workload, m_total: int) -> int:
    """Bytes the inject step must move for m_total placed tokens: every token's
    K and V rows are read once and written once."""
    return 2 * m_total * kv_bytes_per_token(w)


def scan_algorithmic_bytes(w: Workload) -> int:
    """Embedding bytes one retrieve call must read (each bank once)."""
    esz = 4 if w.emb_dtype == "f32" else 2
    banks = 1 if w.shared_bank else w.nq
    return banks * w.n * w.d_e * esz


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _seed(w: Workload, stream: int, extra: int = 0) -> int:
    return BASE_SEED + w.index + 1000 * stream + 1_000_003 * extra


def _unit_rows(rows: int, d: int, g: torch.Generator, device) -> torch.Tensor:
    x = torch.randn(rows, d, generator=g, device=device, dtype=torch.float32)
    return x / x.norm(dim=1, keepdim=True)


def _to_emb(x: torch.Tensor, w: Workload) -> torch.Tensor:
    return x if w.emb_dtype == "f32" else x.to(torch.bfloat16)


def make_bank(w: Workload, device, chunk_rows: int = 1 << 16) -> torch.Tensor:
    """Embedding bank(s): [n][d_e] when shared, else [nq][n][d_e]."""
    banks = 1 if w.shared_bank else w.nq
    total = banks * w.n
    dt = torch.float32 if w.emb_dtype == "f32" else torch.bfloat16
    out = torch.empty(total, w.d_e, dtype=dt, device=device)
    g = _gen(_seed(w, 1), device)
    cent = _centroids(w, device) if w.clustered else None
    for s in range(0, total, chunk_rows):
        e = min(total, s + chunk_rows)
        if cent is None:
            out[s:e] = _to_emb(_unit_rows(e - s, w.d_e, g, device), w)
        else:
            out[s:e] = _to_emb(_clustered_rows(e - s, w, cent, g, device), w)
    return out if w.shared_bank else out.view(w.nq, w.n, w.d_e)


def _centroids(w: Workload, device) -> torch.Tensor:
    return _unit_rows(w.centroids, w.d_e, _gen(_seed(w, 7), device), device)


def _clustered_rows(rows, w, cent, g, device):
    a = torch.randint(0, w.centroids, (rows,), generator=g, device=device)
    noise = torch.randn(rows, w.d_e, generator=g, device=device) * (w.sigma / math.sqrt(w.d_e))
    x = cent[a] + noise
    return x / x.norm(dim=1, keepdim=True)


def make_queries(w: Workload, device, variant: int = 0) -> torch.Tensor:
    """[nq][d_e] query embeddings; ``variant`` selects an independent draw."""
    g = _gen(_seed(w, 2, variant), device)
    if w.clustered:
        x = _clustered_rows(w.nq, w, _centroids(w, device), g, device)
    else:
        x = _unit_rows(w.nq, w.d_e, g, device)
    return _to_emb(x, w)


def make_store(w: Workload, device, chunk_tokens: int = 1 << 14, host: bool = False):
    """Pre-RoPE K and V stores plus per-fact lengths and row offsets.

    Returns dict(preK, V: bf16 [L][T_store][H][D]; fact_lens: int32 [banks][n];
    fact_offsets: int64 [banks][n]; T_store). With host=True, preK and V live
    in pinned host memory (the values are generated on `device` exactly as for
    a device store and copied over chunk by chunk); lengths and offsets stay
    on `device`."""
    banks = 1 if w.shared_bank else w.nq
    g = _gen(_seed(w, 3), "cpu")
    if w.payloads is None:
        lens = torch.randint(w.len_lo, w.len_hi + 1, (banks * w.n,), generator=g, dtype=torch.int64)
        offs = torch.cumsum(lens, 0) - lens
        T_store = int(lens.sum())
    else:
        plen = torch.randint(w.len_lo, w.len_hi + 1, (w.payloads,), generator=g, dtype=torch.int64)
        poff = torch.cumsum(plen, 0) - plen
        which = torch.randint(0, w.payloads, (banks * w.n,), generator=g)
        lens = plen[which]
        offs = poff[which]
        T_store = int(plen.sum())
    row = w.H * w.D
    where = dict(device="cpu", pin_memory=True) if host else dict(device=device)
    preK = torch.empty(w.L, T_store, row, dtype=torch.bfloat16, **where)
    V = torch.empty(w.L, T_store, row, dtype=torch.bfloat16, **where)
    gk = _gen(_seed(w, 4), device)
    gv = _gen(_seed(w, 5), device)
    for l in range(w.L):
        for s in range(0, T_store, chunk_tokens):
            e = min(T_store, s + chunk_tokens)
            preK[l, s:e] = torch.randn(e - s, row, generator=gk, device=device).to(torch.bfloat16)
            V[l, s:e] = torch.randn(e - s, row, generator=gv, device=device).to(torch.bfloat16)
    return dict(preK=preK.view(w.L, T_store, w.H, w.D), V=V.view(w.L, T_store, w.H, w.D),
                fact_lens=lens.to(torch.int32).view(banks, w.n).to(device),
                fact_offsets=offs.view(banks, w.n).to(device), T_store=T_store)


def make_block_tables(w: Workload, device, variant: int = 0, pool_factor: float = 1.1,
                      max_blocks: Optional[int] = None):
    """Disjoint random block tables over one shared page pool.

    Returns (block_table int32 [nq][max_blocks], num_blocks)."""
    mb = w.max_blocks if max_blocks is None else max_blocks
    num_blocks = int(math.ceil(pool_factor * w.nq * mb))
    g = _gen(_seed(w, 6, variant), "cpu")
    perm = torch.randperm(num_blocks, generator=g)[: w.nq * mb].to(torch.int32)
    return perm.view(w.nq, mb).to(device), num_blocks


def make_pages(w: Workload, num_blocks: int, device):
    """Sentinel-filled K and V page pools, bf16 [L][num_blocks*page_size][H][D]."""
    num_slots = num_blocks * w.page_size
    pk = torch.empty(w.L, num_slots, w.H, w.D, dtype=torch.bfloat16, device=device)
    pv = torch.empty_like(pk)
    fill_sentinel(pk)
    fill_sentinel(pv)
    return pk, pv, num_slots


def fill_sentinel(t: torch.Tensor) -> None:
    t.view(torch.int16).fill_(SENTINEL_BITS)
