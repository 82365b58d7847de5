"""One layer's sparse decode step on the GPU: owns the summaries, the selection buffers and
the workspaces, and calls the three libvx entry points in order.

Stage order per decode step (Sec. 3.1: the cache stage is query-independent, then the
indexer stage, then attention over the selected pages):
  summarize (only the page that received the new token) -> score + top-K -> sparse decode.
"""
from __future__ import annotations

from typing import Optional

import torch

from . import vx


class SparseDecoder:
    def __init__(self, kv: vx.PagedKV, batch: vx.BatchSpec, num_q_heads: int, kind: int, n_sink: int,
                 n_local: int, max_sel: int, sm_scale: float, two_pass: bool = True):
        self.kv, self.batch = kv, batch
        self.num_q_heads, self.kind = num_q_heads, kind
        self.n_sink, self.n_local, self.max_sel, self.sm_scale = n_sink, n_local, max_sel, sm_scale
        P, H, ps, Dqk = kv.k.shape
        Dv = kv.v.shape[3] if kv.v is not None else kv.head_dim_v
        dev = kv.k.device
        B = batch.seq_lens.numel()
        self.mean = torch.empty((P, H, Dqk), dtype=torch.float32, device=dev) if kind == vx.MEAN_DOT else None
        # bf16 copy of the means: the first, half-size pass of the exact two-pass selection
        use_bf = kind == vx.MEAN_DOT and two_pass and batch.max_pages_per_seq <= vx.TWO_PASS_MAX_PAGES
        self.mean_bf16 = torch.empty((P, H, Dqk), dtype=torch.bfloat16, device=dev) if use_bf else None
        need_max = kind in (vx.MAX_DOT, vx.QUEST)
        self.max = torch.empty((P, H, Dqk), dtype=torch.bfloat16, device=dev) if need_max else None
        self.min = torch.empty((P, H, Dqk), dtype=torch.bfloat16, device=dev) if kind == vx.QUEST else None
        self.sel_pages = torch.empty((B, H, max_sel), dtype=torch.int32, device=dev)
        self.sel_count = torch.empty((B,), dtype=torch.int32, device=dev)
        self.out = torch.empty((B, num_q_heads, Dv), dtype=torch.bfloat16, device=dev)
        ws_s = vx.workspace_size(vx.STAGE_SCORE_TOPK, kv, batch, num_q_heads, max_sel)
        ws_d = vx.workspace_size(vx.STAGE_DECODE, kv, batch, num_q_heads, max_sel)
        self.ws_score = torch.empty((ws_s,), dtype=torch.uint8, device=dev)
        self.ws_decode = torch.empty((ws_d,), dtype=torch.uint8, device=dev)

    def summarize(self, first_page: Optional[torch.Tensor] = None, stream=None):
        vx.page_summarize(self.kv, self.batch, first_page, self.mean, self.max, self.min, stream,
                          mean_bf16=self.mean_bf16)

    def select(self, q: torch.Tensor, pages_budget: torch.Tensor, stream=None):
        vx.page_score_topk(q, self.kv, self.batch, self.kind, self.mean, self.max, self.min, pages_budget,
                           self.n_sink, self.n_local, self.max_sel, self.sel_pages, self.sel_count,
                           self.ws_score, stream, mean_bf16=self.mean_bf16)

    def decode(self, q: torch.Tensor, sel_pages: Optional[torch.Tensor] = None,
               sel_count: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        sp = self.sel_pages if sel_pages is None else sel_pages
        sc = self.sel_count if sel_count is None else sel_count
        vx.sparse_paged_decode(q, self.kv, self.batch, sp, sc, sp.shape[-1], self.sm_scale, self.out,
                               self.ws_decode, stream)
        return self.out

    def step(self, q: torch.Tensor, pages_budget: torch.Tensor, first_page: Optional[torch.Tensor],
             stream=None) -> torch.Tensor:
        """One decode step: refresh the newest page's summary, select, attend."""
        self.summarize(first_page, stream)
        self.select(q, pages_budget, stream)
        return self.decode(q, stream=stream)
