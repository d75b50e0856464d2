"""Device buffers and call sequencing for one retrieve -> slot map -> inject
pass (plumbing around the three C-ABI calls; no arithmetic of the path lives
here)."""
from __future__ import annotations

import torch

from . import (IS_DTYPE_BF16, IS_DTYPE_F32, IS_ROPE_HALF_SPLIT, is_ann_build,
               is_ann_build_workspace_size, is_ann_search, is_ann_search_workspace_size,
               is_inject, is_inject_rotary, is_place_inject, is_retrieve,
               is_retrieve_workspace_size, is_slot_map)


class RequestBuffers:
    """Outputs and scratch of a batch of nq requests, allocated once.

    ids/scores [nq][k], slots/positions [nq][max_tokens], m [nq], status [1]
    and the retrieval workspace, all on ``device``."""

    def __init__(self, *, n: int, d: int, k: int, nq: int, emb_dtype: torch.dtype,
                 max_tokens: int, device="cuda", workspace=None):
        dt = IS_DTYPE_F32 if emb_dtype == torch.float32 else IS_DTYPE_BF16
        self.n, self.d, self.k, self.nq, self.max_tokens = n, d, k, nq, max_tokens
        ws = is_retrieve_workspace_size(n, d, k, nq, dt)
        if workspace is not None:
            # shared scratch: callers on one stream may reuse it in turn
            assert workspace.numel() * workspace.element_size() >= ws
            self.workspace = workspace
        else:
            self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=device)
        self.ids = torch.empty(nq, k, dtype=torch.int32, device=device)
        self.scores = torch.empty(nq, k, dtype=torch.float32, device=device)
        self.slots = torch.full((nq, max(max_tokens, 1)), -1, dtype=torch.int64, device=device)
        self.positions = torch.full((nq, max(max_tokens, 1)), -1, dtype=torch.int32, device=device)
        self.m = torch.zeros(nq, dtype=torch.int32, device=device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)

    def retrieve(self, query, bank, *, bank_stride=0, stream=None):
        is_retrieve(query, bank, self.n, self.d, self.k, self.ids, self.scores, nq=self.nq,
                    bank_stride=bank_stride, workspace=self.workspace, stream=stream)

    def slot_map(self, fact_lens, start_pos, block_table, page_size, *, lens_stride,
                 reverse_rank=1, stream=None):
        is_slot_map(self.ids, fact_lens, start_pos, block_table, page_size, self.slots,
                    self.positions, self.m, k=self.k, nq=self.nq, n=self.n,
                    lens_stride=lens_stride, max_blocks=block_table.shape[-1],
                    max_tokens=self.max_tokens, reverse_rank=reverse_rank, status=self.status,
                    stream=stream)

    def inject(self, preK, V, rope_theta, paged_k, paged_v, *, fact_offsets, fact_lens,
               lens_stride, reverse_rank=1, inv_freq=None, pairing=IS_ROPE_HALF_SPLIT,
               stream=None):
        L, T_store, H, D = preK.shape
        kw = dict(fact_offsets=fact_offsets, fact_lens=fact_lens, m=self.m, k=self.k,
                  nq=self.nq, n=self.n, lens_stride=lens_stride, reverse_rank=reverse_rank,
                  max_tokens=self.max_tokens, L=L, H=H, D=D, T_store=T_store,
                  num_slots=paged_k.shape[1], status=self.status, stream=stream)
        if inv_freq is None and pairing == IS_ROPE_HALF_SPLIT:
            is_inject(self.ids, preK, V, self.slots, self.positions, rope_theta, paged_k,
                      paged_v, **kw)
        else:
            is_inject_rotary(self.ids, preK, V, self.slots, self.positions, rope_theta, paged_k,
                             paged_v, inv_freq=inv_freq, pairing=pairing, **kw)


    def place_inject(self, preK, V, rope_theta, paged_k, paged_v, *, fact_offsets, fact_lens,
                     lens_stride, start_pos, block_table, page_size, reverse_rank=1,
                     inv_freq=None, pairing=IS_ROPE_HALF_SPLIT, stream=None):
        L, T_store, H, D = preK.shape
        is_place_inject(self.ids, preK, V, rope_theta, paged_k, paged_v, self.slots,
                        self.positions, self.m, fact_offsets=fact_offsets, fact_lens=fact_lens,
                        start_pos=start_pos, block_table=block_table, page_size=page_size,
                        max_blocks=block_table.shape[-1], k=self.k, nq=self.nq, n=self.n,
                        lens_stride=lens_stride, reverse_rank=reverse_rank,
                        max_tokens=self.max_tokens, L=L, H=H, D=D, T_store=T_store,
                        num_slots=paged_k.shape[1], inv_freq=inv_freq, pairing=pairing,
                        status=self.status, stream=stream)


def run_request(buf: RequestBuffers, query, bank, store, block_table, paged_k, paged_v, *,
                start_pos, page_size, rope_theta, shared_bank=True, reverse_rank=1,
                inv_freq=None, pairing=IS_ROPE_HALF_SPLIT, fused=False, stream=None):
    """Enqueue retrieve -> slot map -> inject for every request of ``buf``
    (``fused``: retrieve -> one place + inject launch, same results).

    ``store`` is a dict with preK, V ([L][T_store][H][D] bf16), fact_lens
    ([banks][n] int32) and fact_offsets ([banks][n] int64)."""
    n, d = buf.n, buf.d
    bank_stride = 0 if shared_bank else n * d
    lens_stride = 0 if store["fact_lens"].shape[0] == 1 else n
    buf.retrieve(query, bank, bank_stride=bank_stride, stream=stream)
    if fused:
        buf.place_inject(store["preK"], store["V"], rope_theta, paged_k, paged_v,
                         fact_offsets=store["fact_offsets"], fact_lens=store["fact_lens"],
                         lens_stride=lens_stride, start_pos=start_pos, block_table=block_table,
                         page_size=page_size, reverse_rank=reverse_rank, inv_freq=inv_freq,
                         pairing=pairing, stream=stream)
        return
    buf.slot_map(store["fact_lens"], start_pos, block_table, page_size, lens_stride=lens_stride,
                 reverse_rank=reverse_rank, stream=stream)
    buf.inject(store["preK"], store["V"], rope_theta, paged_k, paged_v,
               fact_offsets=store["fact_offsets"], fact_lens=store["fact_lens"],
               lens_stride=lens_stride, reverse_rank=reverse_rank, inv_freq=inv_freq,
               pairing=pairing, stream=stream)


class AnnIndex:
    """Proximity graph of one bank with the search's seeds (built on the
    device by is_ann_build), and cached search workspaces."""

    def __init__(self, bank: torch.Tensor, *, degree: int = 64, n_seeds: int = 1024,
                 keep_forward: bool = False, stream=None):
        n, d = bank.shape
        dev = bank.device
        self.bank, self.n, self.d, self.degree = bank, n, d, degree
        self.dtype = IS_DTYPE_F32 if bank.dtype == torch.float32 else IS_DTYPE_BF16
        self.n_seeds = min(n_seeds, n)
        self.graph = torch.empty(n, degree, dtype=torch.int32, device=dev)
        self.fwd = torch.empty(n, degree, dtype=torch.int32, device=dev) if keep_forward else None
        self.seed_ids = torch.empty(self.n_seeds, dtype=torch.int32, device=dev)
        self.seed_bank = torch.empty(self.n_seeds, d, dtype=bank.dtype, device=dev)
        ws = torch.empty(is_ann_build_workspace_size(n, d, degree, self.dtype), dtype=torch.uint8,
                         device=dev)
        is_ann_build(bank, n, d, degree, self.graph, n_seeds=self.n_seeds, fwd=self.fwd,
                     seed_ids=self.seed_ids, seed_bank=self.seed_bank, workspace=ws,
                     stream=stream)
        self._ws = {}

    def workspace(self, nq: int, beam: int) -> torch.Tensor:
        key = (nq, beam)
        if key not in self._ws:
            size = is_ann_search_workspace_size(self.n_seeds, self.d, beam, nq, self.dtype)
            self._ws[key] = torch.empty(max(size, 256), dtype=torch.uint8, device=self.bank.device)
        return self._ws[key]

    def search(self, query, out_ids, *, nq: int, k: int, beam: int = 64, width: int = 1,
               max_iters: int = 256, out_scores=None, out_iters=None, out_scored=None, status=None,
               stream=None):
        is_ann_search(query, self.bank, self.n, self.d, self.graph, self.degree, self.seed_ids,
                      self.seed_bank, out_ids, nq=nq, n_seeds=self.n_seeds, beam=beam,
                      width=width, k=k, max_iters=max_iters, out_scores=out_scores,
                      out_iters=out_iters, out_scored=out_scored, status=status,
                      workspace=self.workspace(nq, beam),
                      stream=stream)
