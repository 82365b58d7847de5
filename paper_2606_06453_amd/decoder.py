"""One layer's sparse decode step on the GPU: owns the summaries, the selection buffers and
the workspaces, and calls the three libvx entry points in order.

Stage order per decode step (Sec. 3.1: the cache stage is query-independent, then the
indexer stage, then attention over the selected pages):
  summarize (only the page that received the new token) -> score + top-K -> sparse decode.
"""
from __future__ import annotations

import ctypes
from typing import Optional

import torch

from . import vx


class SparseDecoder:
    def __init__(self, kv: vx.PagedKV, batch: vx.BatchSpec, num_q_heads: int, kind: int, n_sink: int,
                 n_local: int, max_sel: int, sm_scale: float, two_pass: Optional[bool] = None, topk_options=None):
        """topk_options: vx.topk_options(...) for the approximate radix top-k in the indexer step
        (Sec. 5.2), or None for the exact selection.  two_pass (block-mean kinds): score a bf16
        copy of the Mean with an error bound and re-score the undecided pages (True), score the
        fp32 Mean in one pass (False), or choose by the batch's size (None).  Both give the same
        selection."""
        self.kv, self.batch = kv, batch
        self.topk_options = topk_options
        approx = topk_options is not None and (topk_options.tolerate_ratio > 0 or topk_options.remap != 0)
        self.num_q_heads, self.kind = num_q_heads, kind
        self.n_sink, self.n_local, self.max_sel, self.sm_scale = n_sink, n_local, max_sel, sm_scale
        P, H, ps, Dqk = kv.k.shape
        Dv = kv.v.shape[3] if kv.v is not None else kv.head_dim_v
        dev = kv.k.device
        B = batch.seq_lens.numel()
        r = ps // kv.block_size if kv.block_size else 1      # summaries per page (one per block)
        P *= r
        self.mean = torch.empty((P, H, Dqk), dtype=torch.float32, device=dev) if kind in vx.NEEDS_MEAN else None
        # bf16 copy of the means: the first, half-size pass of the exact two-pass selection
        if two_pass is None:
            two_pass = B * batch.max_pages_per_seq * r * H >= vx.TWO_PASS_MIN_ROWS
        use_bf = (kind in vx.TWO_PASS_KINDS and two_pass and not approx
                  and batch.max_pages_per_seq * r <= vx.TWO_PASS_MAX_PAGES)
        self.mean_bf16 = torch.empty((P, H, Dqk), dtype=torch.bfloat16, device=dev) if use_bf else None
        need_max = kind in vx.NEEDS_MAX
        self.max = torch.empty((P, H, Dqk), dtype=torch.bfloat16, device=dev) if need_max else None
        self.min = torch.empty((P, H, Dqk), dtype=torch.bfloat16, device=dev) if kind in vx.NEEDS_MIN else None
        self.sel_pages = torch.empty((B, H, max_sel), dtype=torch.int32, device=dev)
        self.sel_count = torch.empty((B,), dtype=torch.int32, device=dev)
        self.out = torch.empty((B, num_q_heads, Dv), dtype=torch.bfloat16, device=dev)
        ws_s = vx.workspace_size(vx.STAGE_SCORE_TOPK, kv, batch, num_q_heads, max_sel)
        ws_d = vx.workspace_size(vx.STAGE_DECODE, kv, batch, num_q_heads, max_sel)
        self.ws_score = torch.empty((ws_s,), dtype=torch.uint8, device=dev)
        # zero-filled once: its split counters must start at zero (every call leaves them zero)
        self.ws_decode = torch.zeros((ws_d,), dtype=torch.uint8, device=dev)

        self._bound = {}

    def _bound_call(self, key, make):
        """The step's calls with their arguments marshalled once, keyed by the tensors that vary."""
        c = self._bound.get(key)
        if c is None:
            if len(self._bound) >= 32:
                self._bound.clear()
            c = make()
            self._bound[key] = c
        return c

    def summarize(self, first_page: Optional[torch.Tensor] = None, stream=None):
        if first_page is None:           # prefill: every page (not a per-step call)
            vx.page_summarize(self.kv, self.batch, None, self.mean, self.max, self.min, stream,
                              mean_bf16=self.mean_bf16)
            return
        self._bound_call(("summarize", first_page.data_ptr()), lambda: vx.BoundCall(
            vx.lib().vx_page_summarize,
            (self.kv.ref(), self.batch.ref(), first_page.data_ptr(), vx._ptr(self.mean), vx._ptr(self.mean_bf16),
             vx._ptr(self.max), vx._ptr(self.min), None), 7))(stream)

    def append(self, k_new: torch.Tensor, v_new: Optional[torch.Tensor], stream=None):
        """The step's cache stage in one launch: new K/V rows at token seq_lens[i]-1, then that
        page's summaries."""
        assert k_new.is_contiguous() and (v_new is None or v_new.is_contiguous())
        self._bound_call(("append", k_new.data_ptr(), None if v_new is None else v_new.data_ptr()),
                         lambda: vx.BoundCall(
            vx.lib().vx_kv_append_summarize,
            (self.kv.ref(), self.batch.ref(), k_new.data_ptr(), vx._ptr(v_new), vx._ptr(self.mean),
             vx._ptr(self.mean_bf16), vx._ptr(self.max), vx._ptr(self.min), None), 8))(stream)

    def select(self, q: torch.Tensor, pages_budget: torch.Tensor, stream=None):
        assert q.is_contiguous() and pages_budget.is_contiguous()
        self._bound_call(("select", q.data_ptr(), pages_budget.data_ptr()), lambda: vx.BoundCall(
            vx.lib().vx_page_score_topk,
            (q.data_ptr(), q.shape[1], self.kv.ref(), self.batch.ref(), self.kind, vx._ptr(self.mean),
             vx._ptr(self.mean_bf16), vx._ptr(self.max), vx._ptr(self.min), pages_budget.data_ptr(), self.n_sink,
             self.n_local, self.max_sel, self.sel_pages.data_ptr(), self.sel_count.data_ptr(),
             self.ws_score.data_ptr(), self.ws_score.numel(),
             None if self.topk_options is None else ctypes.byref(self.topk_options), None), 18))(stream)

    def append_select(self, k_new: torch.Tensor, v_new: Optional[torch.Tensor], q: torch.Tensor,
                      pages_budget: torch.Tensor, stream=None):
        """append() then select(), with the append inside the top-K launch when that is exact
        (vx_append_score_topk)."""
        assert k_new.is_contiguous() and (v_new is None or v_new.is_contiguous())
        assert q.is_contiguous() and pages_budget.is_contiguous()
        key = ("append_select", k_new.data_ptr(), None if v_new is None else v_new.data_ptr(), q.data_ptr(),
               pages_budget.data_ptr())
        self._bound_call(key, lambda: vx.BoundCall(
            vx.lib().vx_append_score_topk,
            (self.kv.ref(), self.batch.ref(), k_new.data_ptr(), vx._ptr(v_new), vx._ptr(self.mean),
             vx._ptr(self.mean_bf16), vx._ptr(self.max), vx._ptr(self.min), q.data_ptr(), q.shape[1], self.kind,
             pages_budget.data_ptr(), self.n_sink, self.n_local, self.max_sel, self.sel_pages.data_ptr(),
             self.sel_count.data_ptr(), self.ws_score.data_ptr(), self.ws_score.numel(),
             None if self.topk_options is None else ctypes.byref(self.topk_options), None), 20))(stream)

    def decode(self, q: torch.Tensor, sel_pages: Optional[torch.Tensor] = None,
               sel_count: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        sp = self.sel_pages if sel_pages is None else sel_pages
        sc = self.sel_count if sel_count is None else sel_count
        assert q.is_contiguous() and sp.is_contiguous() and sc.is_contiguous()
        self._bound_call(("decode", q.data_ptr(), sp.data_ptr(), sc.data_ptr(), sp.shape[-1]), lambda: vx.BoundCall(
            vx.lib().vx_sparse_paged_decode,
            (q.data_ptr(), q.shape[1], self.kv.ref(), self.batch.ref(), sp.data_ptr(), sc.data_ptr(), sp.shape[-1],
             float(self.sm_scale), self.out.data_ptr(), self.ws_decode.data_ptr(), self.ws_decode.numel(), None),
            11))(stream)
        return self.out

    def step(self, q: torch.Tensor, pages_budget: torch.Tensor, first_page: Optional[torch.Tensor],
             stream=None, kv_new=None) -> torch.Tensor:
        """One decode step: refresh the newest page's summary (with kv_new = (k_new, v_new): append
        the new rows and refresh them inside the selection's launches), select, attend."""
        if kv_new is not None:
            self.append_select(kv_new[0], kv_new[1], q, pages_budget, stream)
        else:
            self.summarize(first_page, stream)
            self.select(q, pages_budget, stream)
        return self.decode(q, stream=stream)
