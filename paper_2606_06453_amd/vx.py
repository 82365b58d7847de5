"""Thin ctypes binding of ``libvx.so`` (declared in ``include/vx.h``).

Argument marshalling only: every step of the decode path runs in the library's HIP
kernels.  torch supplies device memory and the current stream.  If the library is
missing the binding raises; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvx.so")

MEAN_DOT, QUEST, MAX_DOT = 0, 1, 2
QUEST_CONSENSUS, ENVELOPE_LOWER, QUEST_RECTIFIED = 3, 4, 5     # Appendix G envelope flows
MEAN_DOT_CONTENT, NSA, MEAN_DOT_SMOOTH = 6, 7, 8                 # rope-unaware, NSA, smoothing
NEEDS_MEAN = (MEAN_DOT, MEAN_DOT_CONTENT, NSA, MEAN_DOT_SMOOTH)
TWO_PASS_KINDS = (MEAN_DOT, MEAN_DOT_CONTENT)                    # may pass the bf16 Mean copy
NEEDS_MAX = (MAX_DOT, QUEST, QUEST_CONSENSUS, ENVELOPE_LOWER, QUEST_RECTIFIED)
NEEDS_MIN = (QUEST, QUEST_CONSENSUS, ENVELOPE_LOWER)
STAGE_SCORE_TOPK, STAGE_DECODE = 0, 1
KV_BF16, KV_FP8_E4M3, KV_FP8_E5M2 = 0, 1, 2


def kv_dtype_code(t: torch.Tensor) -> int:
    """vx_kv_dtype of a cache tensor: bfloat16, float8_e4m3fn (OCP E4M3) or float8_e5m2."""
    codes = {torch.bfloat16: KV_BF16, torch.float8_e4m3fn: KV_FP8_E4M3, torch.float8_e5m2: KV_FP8_E5M2}
    if t.dtype not in codes:
        raise TypeError(f"KV cache dtype {t.dtype} is not bfloat16, float8_e4m3fn or float8_e5m2")
    return codes[t.dtype]
TWO_PASS_MAX_PAGES = 4096     # block-mean two-pass selection: max_pages_per_seq bound
# Below this many summary rows (batch x blocks per request x KV heads) the decoder scores the
# block mean in one pass: the bound pass saves half the summary bytes, but its re-scoring of the
# undecided pages adds a dependent round trip to the top-K kernel, which a short score stream does
# not pay back (MLA geometry, 16384 rows: score + top-K 22.9 us in one pass against 25.1 us in
# two; Llama-3-8B-shaped layer, 10^6 rows: 54.5 us in two passes against 72.8 us in one).
TWO_PASS_MIN_ROWS = 65536

_STATUS = {0: "VX_OK", 1: "VX_ERR_INVALID_ARG", 2: "VX_ERR_UNSUPPORTED", 3: "VX_ERR_WORKSPACE", 4: "VX_ERR_HIP"}


class VxError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class _Cache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("num_phys_pages", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("head_dim_qk", ctypes.c_int32), ("head_dim_v", ctypes.c_int32), ("kv_dtype", ctypes.c_int32),
                ("k_scale", ctypes.c_float), ("v_scale", ctypes.c_float), ("block_size", ctypes.c_int32)]


class _Batch(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
                ("page_indptr", ctypes.c_void_p), ("page_indices", ctypes.c_void_p),
                ("seq_lens", ctypes.c_void_p)]


_lib = None


def lib():
    """Load libvx.so from the package directory (never a fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               f"or python paper_2606_06453_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.vx_version.restype = ctypes.c_uint32
        L.vx_last_error.restype = ctypes.c_char_p
        L.vx_workspace_size.argtypes = [i32, P, P, i32, i32, ctypes.POINTER(sz)]
        L.vx_page_summarize.argtypes = [P, P, P, P, P, P, P, P]
        L.vx_page_score_topk.argtypes = [P, i32, P, P, i32, P, P, P, P, P, i32, i32, i32, P, P, P, sz, P, P]
        L.vx_sparse_paged_decode.argtypes = [P, i32, P, P, P, P, i32, ctypes.c_float, P, P, sz, P]
        L.vx_page_score.argtypes = [P, i32, P, P, i32, P, P, P, P, i32, P]
        L.vx_topk_select.argtypes = [P, i32, i32, i32, P, P, i32, i32, i32, P, P, P, P]
        L.vx_score_flow.argtypes = [i32, P, P, i32, i32, i32, i32, P, P]
        L.vx_stream_read.argtypes = [P, sz, P, i32, P]
        L.vx_kv_append_summarize.argtypes = [P, P, P, P, P, P, P, P, P]
        L.vx_sparse_paged_decode_noalloc.argtypes = [P, i32, P, P, P, P, i32, ctypes.c_float, P, P]
        L.vx_append_score_topk.argtypes = [P, P, P, P, P, P, P, P, P, i32, i32, P, i32, i32, i32, P, P, P, sz, P, P]
        for f in (L.vx_workspace_size, L.vx_page_summarize, L.vx_page_score_topk, L.vx_sparse_paged_decode,
                  L.vx_page_score, L.vx_topk_select, L.vx_score_flow, L.vx_kv_append_summarize,
                  L.vx_stream_read, L.vx_sparse_paged_decode_noalloc, L.vx_append_score_topk):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def version() -> int:
    return int(lib().vx_version())


def _check(status: int):
    if status != 0:
        raise VxError(status, lib().vx_last_error().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    assert t.is_contiguous(), "tensors passed to libvx must be contiguous"
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


@dataclass
class PagedKV:
    """Paged KV cache: k [P][H][ps][Dqk], v [P][H][ps][Dv] or None (V = K[..., :Dv]); bf16, or
    fp8 (float8_e4m3fn / float8_e5m2) codes whose values are k_scale * code and v_scale * code."""
    k: torch.Tensor
    v: Optional[torch.Tensor]
    head_dim_v: Optional[int] = None
    k_scale: float = 1.0
    v_scale: float = 1.0
    block_size: int = 0      # 0: one block per page; else 16 or 32 dividing the page size

    def struct(self) -> _Cache:
        P, H, ps, Dqk = self.k.shape
        Dv = self.v.shape[3] if self.v is not None else (self.head_dim_v or Dqk)
        dt = kv_dtype_code(self.k)
        if self.v is not None and kv_dtype_code(self.v) != dt:
            raise TypeError("K and V caches must have the same dtype")
        return _Cache(_ptr(self.k), _ptr(self.v), P, H, ps, Dqk, Dv, dt, float(self.k_scale), float(self.v_scale),
                      int(self.block_size))

    def ref(self):
        """A by-reference argument holding this geometry, built once (the tensors must not be
        replaced afterwards)."""
        if getattr(self, "_ref", None) is None:
            self._st = self.struct()
            self._ref = ctypes.byref(self._st)
        return self._ref


@dataclass
class BatchSpec:
    """Ragged batch over the paged cache: int32 device tensors plus a host bound on P_i."""
    page_indptr: torch.Tensor
    page_indices: torch.Tensor
    seq_lens: torch.Tensor
    max_pages_per_seq: int

    def struct(self) -> _Batch:
        return _Batch(self.seq_lens.numel(), int(self.max_pages_per_seq), _ptr(self.page_indptr),
                      _ptr(self.page_indices), _ptr(self.seq_lens))

    def ref(self):
        """A by-reference argument holding this batch, built once (see PagedKV.ref)."""
        if getattr(self, "_ref", None) is None:
            self._st = self.struct()
            self._ref = ctypes.byref(self._st)
        return self._ref


def workspace_size(stage: int, kv: PagedKV, batch: BatchSpec, num_q_heads: int, max_sel: int) -> int:
    out = ctypes.c_size_t(0)
    c, b = kv.struct(), batch.struct()
    _check(lib().vx_workspace_size(stage, ctypes.byref(c), ctypes.byref(b), num_q_heads, max_sel,
                                   ctypes.byref(out)))
    return int(out.value)


def page_summarize(kv: PagedKV, batch: BatchSpec, first_page: Optional[torch.Tensor] = None,
                   mean: Optional[torch.Tensor] = None, max: Optional[torch.Tensor] = None,
                   min: Optional[torch.Tensor] = None, stream=None,
                   mean_bf16: Optional[torch.Tensor] = None) -> None:
    c, b = kv.struct(), batch.struct()
    _check(lib().vx_page_summarize(ctypes.byref(c), ctypes.byref(b), _ptr(first_page), _ptr(mean),
                                   _ptr(mean_bf16), _ptr(max), _ptr(min), _stream(stream)))


def kv_append_summarize(kv: PagedKV, batch: BatchSpec, k_new: torch.Tensor, v_new: Optional[torch.Tensor],
                        mean: Optional[torch.Tensor] = None, max: Optional[torch.Tensor] = None,
                        min: Optional[torch.Tensor] = None, stream=None,
                        mean_bf16: Optional[torch.Tensor] = None) -> None:
    """Writes k_new [B][H][Dqk] / v_new [B][H][Dv] (the cache's dtype) at token seq_lens[i]-1 and
    refreshes that page's summaries, in one launch."""
    for t in (k_new, v_new):
        if t is not None and t.dtype != kv.k.dtype:
            raise TypeError(f"new rows must have the cache's dtype {kv.k.dtype} (got {t.dtype})")
    c, b = kv.struct(), batch.struct()
    _check(lib().vx_kv_append_summarize(ctypes.byref(c), ctypes.byref(b), _ptr(k_new), _ptr(v_new), _ptr(mean),
                                        _ptr(mean_bf16), _ptr(max), _ptr(min), _stream(stream)))


class _TopkOptions(ctypes.Structure):
    _fields_ = [("tolerate_ratio", ctypes.c_float), ("seed", ctypes.c_uint32), ("remap", ctypes.c_int32)]


REMAP_NONE, REMAP_AFFINE = 0, 1


def topk_options(tolerate_ratio: float = 0.0, seed: int = 0, remap: int = REMAP_NONE) -> _TopkOptions:
    return _TopkOptions(float(tolerate_ratio), int(seed) & 0xFFFFFFFF, int(remap))


def page_score_topk(q: torch.Tensor, kv: PagedKV, batch: BatchSpec, kind: int,
                    mean: Optional[torch.Tensor], max: Optional[torch.Tensor], min: Optional[torch.Tensor],
                    pages_budget: torch.Tensor, n_sink: int, n_local: int, max_sel: int,
                    sel_pages: torch.Tensor, sel_count: torch.Tensor, workspace: torch.Tensor,
                    stream=None, mean_bf16: Optional[torch.Tensor] = None,
                    options: Optional[_TopkOptions] = None) -> None:
    c, b = kv.struct(), batch.struct()
    _check(lib().vx_page_score_topk(_ptr(q), q.shape[1], ctypes.byref(c), ctypes.byref(b), kind, _ptr(mean),
                                    _ptr(mean_bf16), _ptr(max), _ptr(min), _ptr(pages_budget), n_sink, n_local,
                                    max_sel,
                                    _ptr(sel_pages), _ptr(sel_count), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(),
                                    None if options is None else ctypes.byref(options), _stream(stream)))


def append_score_topk(kv: PagedKV, batch: BatchSpec, k_new: torch.Tensor, v_new: Optional[torch.Tensor],
                      mean: Optional[torch.Tensor], max: Optional[torch.Tensor], min: Optional[torch.Tensor],
                      q: torch.Tensor, kind: int, pages_budget: torch.Tensor, n_sink: int, n_local: int,
                      max_sel: int, sel_pages: torch.Tensor, sel_count: torch.Tensor, workspace: torch.Tensor,
                      stream=None, mean_bf16: Optional[torch.Tensor] = None,
                      options: Optional[_TopkOptions] = None) -> None:
    """kv_append_summarize followed by page_score_topk, the append inside the top-K launch."""
    for t in (k_new, v_new):
        if t is not None and t.dtype != kv.k.dtype:
            raise TypeError(f"new rows must have the cache's dtype {kv.k.dtype} (got {t.dtype})")
    c, b = kv.struct(), batch.struct()
    _check(lib().vx_append_score_topk(ctypes.byref(c), ctypes.byref(b), _ptr(k_new), _ptr(v_new), _ptr(mean),
                                      _ptr(mean_bf16), _ptr(max), _ptr(min), _ptr(q), q.shape[1], kind,
                                      _ptr(pages_budget), n_sink, n_local, max_sel, _ptr(sel_pages),
                                      _ptr(sel_count), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                      None if options is None else ctypes.byref(options), _stream(stream)))


def page_score(q: torch.Tensor, kv: PagedKV, batch: BatchSpec, kind: int, mean: Optional[torch.Tensor],
               max: Optional[torch.Tensor], min: Optional[torch.Tensor], scores: torch.Tensor, stream=None) -> None:
    """One-pass fp32 scores into scores [H][B][stride] (float32, contiguous)."""
    assert scores.dtype == torch.float32 and scores.dim() == 3
    c, b = kv.struct(), batch.struct()
    _check(lib().vx_page_score(_ptr(q), q.shape[1], ctypes.byref(c), ctypes.byref(b), kind, _ptr(mean), _ptr(max),
                               _ptr(min), _ptr(scores), scores.shape[2], _stream(stream)))


def score_flow(kind: int, scores_in: torch.Tensor, scores_out: torch.Tensor, num_kv_heads: int,
               num_items: torch.Tensor, stream=None) -> None:
    """Last steps of the NSA / smoothing flows: scores_in [rows][B][stride] (NSA: a row per query
    head) -> scores_out [H][B][stride] (float32)."""
    assert scores_in.dtype == torch.float32 and scores_out.dtype == torch.float32 and scores_out.dim() == 3
    H, B, stride = scores_out.shape
    assert H == num_kv_heads and scores_in.shape[1:] == (B, stride)
    rows = scores_in.shape[0]
    _check(lib().vx_score_flow(kind, _ptr(scores_in), _ptr(scores_out), stride, num_kv_heads,
                               rows if kind == NSA else num_kv_heads, B, _ptr(num_items), _stream(stream)))


def stream_read(buf: torch.Tensor, sink: torch.Tensor, stream=None) -> None:
    """The streaming-read measurement kernel over the bytes of buf (contiguous, 16-byte
    multiple); sink: int32 device tensor with one entry per workgroup."""
    _check(lib().vx_stream_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), sink.numel(),
                                _stream(stream)))


def topk_select(scores: torch.Tensor, num_items: torch.Tensor, pages_budget: torch.Tensor, n_sink: int,
                n_local: int, max_sel: int, sel_pages: torch.Tensor, sel_count: torch.Tensor,
                tolerate_ratio: float = 0.0, seed: int = 0, remap: int = REMAP_NONE, stream=None) -> None:
    """Exact or approximate radix selection from scores [H][B][stride] (float32)."""
    assert scores.dtype == torch.float32 and scores.dim() == 3
    H, B, stride = scores.shape
    opt = topk_options(tolerate_ratio, seed, remap)
    _check(lib().vx_topk_select(_ptr(scores), stride, H, B, _ptr(num_items), _ptr(pages_budget), n_sink, n_local,
                                max_sel, ctypes.byref(opt), _ptr(sel_pages), _ptr(sel_count), _stream(stream)))


def sparse_paged_decode(q: torch.Tensor, kv: PagedKV, batch: BatchSpec, sel_pages: torch.Tensor,
                        sel_count: torch.Tensor, max_sel: int, sm_scale: float, out: torch.Tensor,
                        workspace: torch.Tensor, stream=None) -> None:
    c, b = kv.struct(), batch.struct()
    _check(lib().vx_sparse_paged_decode(_ptr(q), q.shape[1], ctypes.byref(c), ctypes.byref(b), _ptr(sel_pages),
                                        _ptr(sel_count), max_sel, float(sm_scale), _ptr(out), _ptr(workspace),
                                        workspace.numel() * workspace.element_size(), _stream(stream)))


def sparse_paged_decode_noalloc(q: torch.Tensor, kv: PagedKV, batch: BatchSpec, sel_pages: torch.Tensor,
                                sel_count: torch.Tensor, max_sel: int, sm_scale: float, out: torch.Tensor,
                                stream=None) -> None:
    """vx_sparse_paged_decode on the library's static per-GPU scratch (no workspace)."""
    c, b = kv.struct(), batch.struct()
    _check(lib().vx_sparse_paged_decode_noalloc(_ptr(q), q.shape[1], ctypes.byref(c), ctypes.byref(b),
                                                _ptr(sel_pages), _ptr(sel_count), max_sel, float(sm_scale),
                                                _ptr(out), _stream(stream)))


class BoundCall:
    """One entry point with every argument marshalled once; calling it only swaps in the
    stream.  For per-step loops whose buffers stay fixed (argument marshalling only, like the
    functions above)."""

    def __init__(self, fn, args: tuple, stream_index: int):
        self.fn, self.args, self.si = fn, list(args), stream_index

    def __call__(self, stream=None):
        self.args[self.si] = _stream(stream)
        _check(self.fn(*self.args))
