"""ctypes front end of the plain fp64 CPU oracle (``oracle/vxo.c``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU-baseline leg
use it; the product path never does.  It imports nothing from the HIP package.

Arrays are numpy; bf16 tensors are accepted as torch bfloat16 tensors or uint16 arrays of
their bit patterns.  An 8-bit floating-point KV cache is a torch float8_e4m3fn or float8_e5m2
tensor (OCP E4M3 / E5M2 codes), passed with its per-tensor scale.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "vxo.c")
LIB = os.path.join(HERE, "libvxo.so")
# Test hook: run the pins against another build of the oracle (the mutation test uses it).
_LIB_OVERRIDE = os.environ.get("VXO_LIB")

MEAN_DOT, QUEST, MAX_DOT = 0, 1, 2
QUEST_CONSENSUS, ENVELOPE_LOWER, QUEST_RECTIFIED = 3, 4, 5     # Appendix G envelope flows
MEAN_DOT_CONTENT = 6     # Eq. 2 over the content channels (rope-unaware MLA flow, Sec. 6.2)
NSA = 7                  # NSA block top-k flow: per-head softmax of the Mean logits, conv, head sum
MEAN_DOT_SMOOTH = 8      # positional smoothing (Appendix G): Conv of the Eq. 2 scores
# Conv1d kernel of the NSA and smoothing flows along the page axis (zero padding): the
# [0.25, 0.5, 0.25] kernel of Appendix G's positional smoothing; the NSA listing gives none.
CONV_TAPS = (0.25, 0.5, 0.25)
KV_BF16, KV_FP8_E4M3, KV_FP8_E5M2 = 0, 1, 2

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, IEEE semantics, OpenMP over independent units)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-o", tmp, SRC, "-lm"])
        os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            L = ctypes.CDLL(_LIB_OVERRIDE)
        else:
            build(force=False)
            L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
        L.vxo_error.restype = ctypes.c_char_p
        L.vxo_num_threads.restype = i32
        L.vxo_set_num_threads.argtypes = [i32]
        L.vxo_set_num_threads.restype = None
        f32 = ctypes.c_float
        L.vxo_summarize.argtypes = [P, i32, f32, i64, i32, i32, i32, i32, P, P, P, P, P, P, P]
        L.vxo_score.argtypes = [i32, P, i32, i32, i32, i32, i32, i32, P, P, P, P, P, P]
        L.vxo_kv_append.argtypes = [P, P, i32, i64, i32, i32, i32, i32, i32, P, P, P, P, P]
        L.vxo_head_logits.argtypes = [P, i32, i32, i32, i32, i32, P, P, P, P, P]
        L.vxo_nsa_scores.argtypes = [P, i32, i32, i32, i32, P, P, P, P]
        L.vxo_smooth_scores.argtypes = [P, i32, i32, i32, P, P, P, P]
        L.vxo_select.argtypes = [P, i32, i32, i32, P, P, P, i32, i32, i32, P, P, P, P]
        L.vxo_attend.argtypes = [P, i32, P, P, i32, f32, f32, i32, i32, i32, i32, i32, P, P, P, P, P, i32, f64, P]
        L.vxo_fp8_dequantize.argtypes = [P, i64, i32, f32, P]
        L.vxo_topk_select.argtypes = [P, i32, i32, i32, P, P, i32, i32, i32, ctypes.c_float, ctypes.c_uint32, i32,
                                      P, P]
        for f in (L.vxo_summarize, L.vxo_score, L.vxo_select, L.vxo_attend, L.vxo_topk_select,
                  L.vxo_fp8_dequantize):
            f.restype = i32
        _lib = L
    return _lib


def num_threads() -> int:
    return int(lib().vxo_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the following oracle calls (independent units only; results are unchanged)."""
    lib().vxo_set_num_threads(int(n))


def _bits(x) -> np.ndarray:
    """uint16 bit patterns of a bf16 tensor (or pass-through for uint16 arrays)."""
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        assert x.dtype == np.uint16
        return np.ascontiguousarray(x)
    import torch
    assert x.dtype == torch.bfloat16
    return x.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _cache(x):
    """(contiguous host array, kv format) of a KV cache tensor: bf16 bits or fp8 codes."""
    if x is None:
        return None, None
    if isinstance(x, np.ndarray):
        return _bits(x), KV_BF16
    import torch
    if x.dtype == torch.bfloat16:
        return _bits(x), KV_BF16
    fmt = {torch.float8_e4m3fn: KV_FP8_E4M3, torch.float8_e5m2: KV_FP8_E5M2}[x.dtype]
    return x.detach().cpu().contiguous().view(torch.uint8).numpy(), fmt


def fp8_dequantize(codes, fmt, scale) -> np.ndarray:
    """fp32 cache values of fp8 codes (uint8 array) of format fmt with a per-tensor scale."""
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    out = np.empty(c.shape, np.float32)
    _check(lib().vxo_fp8_dequantize(_p(c), c.size, int(fmt), float(scale), _p(out)))
    return out


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _p(a) -> Optional[int]:
    return None if a is None else a.ctypes.data


def _check(rc: int):
    if rc != 0:
        raise ValueError("oracle: " + lib().vxo_error().decode())


def summarize(k, page_size, page_indptr, page_indices, seq_lens, first_page=None, k_scale=1.0):
    """Returns (mean, max, min), each fp64 [P_phys][H][D]; rows never referenced are NaN."""
    kb, fmt = _cache(k)
    P, H, ps, D = kb.shape
    assert ps == page_size
    mean = np.full((P, H, D), np.nan)
    mx = np.full((P, H, D), np.nan)
    mn = np.full((P, H, D), np.nan)
    ind, idx, lens = _i32(page_indptr), _i32(page_indices), _i32(seq_lens)
    fp = None if first_page is None else _i32(first_page)
    _check(lib().vxo_summarize(_p(kb), fmt, float(k_scale), P, H, ps, D, len(lens), _p(ind), _p(idx), _p(lens),
                               _p(fp), _p(mean), _p(mx), _p(mn)))
    return mean, mx, mn


def reblock(k, v, page_size, block_size, page_indptr, page_indices, seq_lens):
    """Blocks smaller than pages (Appendix E template: block_size below page_size) as pages of
    their own: with r = page_size / block_size, block b of physical page p is the virtual
    physical page p * r + b of block_size tokens,
        k'[p * r + b][h][t] = k[p][h][b * block_size + t],
    and logical block jb of request i (jb < ceil(L_i / block_size)) is virtual page
    page_indices[page_indptr[i] + jb // r] * r + jb % r.  Every oracle function applied to the
    returned problem with page_size = block_size computes the block-granular step: summaries
    per block (indexed by virtual page), scores, sink / local / budget counts and selected ids
    in blocks, attention over the selected blocks' tokens.
    Returns (k', v', page_indptr', page_indices')."""
    import torch
    assert page_size % block_size == 0
    r = page_size // block_size
    def split(x):
        if x is None:
            return None
        P, H, ps, D = x.shape
        return x.reshape(P, H, r, block_size, D).permute(0, 2, 1, 3, 4).reshape(P * r, H, block_size, D).contiguous()
    ind, idx, lens = _i32(page_indptr), _i32(page_indices), _i32(seq_lens)
    nb = (lens.astype(np.int64) + block_size - 1) // block_size
    ind2 = np.zeros(len(lens) + 1, np.int32)
    ind2[1:] = np.cumsum(nb)
    idx2 = np.empty(int(ind2[-1]), np.int32)
    for i in range(len(lens)):
        jb = np.arange(nb[i])
        idx2[ind2[i]:ind2[i + 1]] = idx[ind[i] + jb // r] * r + jb % r
    return split(k), split(v), ind2, idx2


def kv_append(k, v, page_size, page_indptr, page_indices, seq_lens, k_new, v_new=None, head_dim_v=None,
              k_scale=1.0):
    """The decode step's cache stage: copies of k / v (torch bf16 or fp8, v None = aliased) with
    each request's new rows k_new [B][H][Dqk] (v_new [B][H][Dv]) written at token seq_lens[i]-1,
    followed by the summaries of the pages from the last one on.
    Returns (k, v, (mean, max, min), first_page)."""
    import torch
    kb, fmt = _cache(k)
    vb, _ = _cache(v)
    kb, vb = kb.copy(), (None if vb is None else vb.copy())
    kn, _ = _cache(k_new)
    vn = None if v_new is None else _cache(v_new)[0]
    kn = np.ascontiguousarray(kn)
    vn = None if vn is None else np.ascontiguousarray(vn)
    Pp, H, ps, Dqk = kb.shape
    Dv = vb.shape[3] if vb is not None else (head_dim_v or Dqk)
    ind, idx, lens = _i32(page_indptr), _i32(page_indices), _i32(seq_lens)
    _check(lib().vxo_kv_append(_p(kb), _p(vb), fmt, Pp, H, ps, Dqk, Dv, len(lens), _p(ind), _p(idx), _p(lens),
                               _p(kn), _p(vn)))
    def back(a, like):
        if a is None:
            return None
        t = torch.from_numpy(a)
        return t.view(torch.bfloat16) if like.dtype == torch.bfloat16 else t.view(like.dtype)
    k2, v2 = back(kb, k), back(vb, v if v is not None else k)
    first = ((lens - 1) // ps).astype(np.int32)
    return k2, v2, summarize(k2, ps, page_indptr, page_indices, seq_lens, first_page=first, k_scale=k_scale), first


def score(kind, q, num_kv_heads, page_size, page_indptr, page_indices, seq_lens, sa, sb=None, content_dims=None):
    """fp64 ragged scores [page_indptr[-1]][H].  content_dims: channels scored by
    MEAN_DOT_CONTENT (the first head_dim_v channels of an MLA latent)."""
    qb = _bits(q)
    B, Hq, D = qb.shape
    ind, idx, lens = _i32(page_indptr), _i32(page_indices), _i32(seq_lens)
    sa = np.ascontiguousarray(sa, dtype=np.float64)
    sb = None if sb is None else np.ascontiguousarray(sb, dtype=np.float64)
    out = np.full((int(ind[-1]), num_kv_heads), np.nan)
    Dc = D if content_dims is None else int(content_dims)
    _check(lib().vxo_score(kind, _p(qb), Hq, num_kv_heads, D, Dc, page_size, B, _p(ind), _p(idx), _p(lens),
                           _p(sa), _p(sb), _p(out)))
    return out


def head_logits(q, num_kv_heads, page_size, page_indptr, page_indices, seq_lens, mean):
    """Per-query-head logits fp32(q_r . Mean_j) as fp64, ragged [page_indptr[-1]][Hq]."""
    qb = _bits(q)
    B, Hq, D = qb.shape
    ind, idx, lens = _i32(page_indptr), _i32(page_indices), _i32(seq_lens)
    mean = np.ascontiguousarray(mean, dtype=np.float64)
    out = np.full((int(ind[-1]), Hq), np.nan)
    _check(lib().vxo_head_logits(_p(qb), Hq, num_kv_heads, D, page_size, B, _p(ind), _p(idx), _p(lens),
                                 _p(mean), _p(out)))
    return out


def nsa_scores(logits, num_kv_heads, page_size, page_indptr, seq_lens, taps=CONV_TAPS):
    """NSA block scores from ragged logits [..][Hq]: ragged [..][H]."""
    z = np.ascontiguousarray(logits, dtype=np.float64)
    Hq = z.shape[1]
    ind, lens = _i32(page_indptr), _i32(seq_lens)
    w = np.ascontiguousarray(taps, dtype=np.float64)
    out = np.full((int(ind[-1]), num_kv_heads), np.nan)
    _check(lib().vxo_nsa_scores(_p(z), Hq, num_kv_heads, page_size, len(lens), _p(ind), _p(lens), _p(w), _p(out)))
    return out


def smooth_scores(scores, page_size, page_indptr, seq_lens, taps=CONV_TAPS):
    """Conv1d along the page axis of a ragged [..][H] score table."""
    x = np.ascontiguousarray(scores, dtype=np.float64)
    H = x.shape[1]
    ind, lens = _i32(page_indptr), _i32(seq_lens)
    w = np.ascontiguousarray(taps, dtype=np.float64)
    out = np.full_like(x, np.nan)
    _check(lib().vxo_smooth_scores(_p(x), H, page_size, len(lens), _p(ind), _p(lens), _p(w), _p(out)))
    return out


def flow_scores(kind, q, num_kv_heads, page_size, page_indptr, page_indices, seq_lens, mean, mx, mn,
                head_dim_v=None):
    """The block scores of a score flow (kinds 0..8) from the summaries it reads."""
    if kind == MEAN_DOT:
        return score(MEAN_DOT, q, num_kv_heads, page_size, page_indptr, page_indices, seq_lens, mean)
    if kind == MEAN_DOT_CONTENT:
        return score(MEAN_DOT_CONTENT, q, num_kv_heads, page_size, page_indptr, page_indices, seq_lens, mean,
                     content_dims=head_dim_v)
    if kind == NSA:
        z = head_logits(q, num_kv_heads, page_size, page_indptr, page_indices, seq_lens, mean)
        return nsa_scores(z, num_kv_heads, page_size, page_indptr, seq_lens)
    if kind == MEAN_DOT_SMOOTH:
        s = score(MEAN_DOT, q, num_kv_heads, page_size, page_indptr, page_indices, seq_lens, mean)
        return smooth_scores(s, page_size, page_indptr, seq_lens)
    if kind in (MAX_DOT, QUEST_RECTIFIED):
        return score(kind, q, num_kv_heads, page_size, page_indptr, page_indices, seq_lens, mx)
    return score(kind, q, num_kv_heads, page_size, page_indptr, page_indices, seq_lens, mx, mn)


def select(scores, num_kv_heads, page_size, page_indptr, seq_lens, pages_budget, n_sink, n_local, max_sel):
    """Returns (sel_pages [B][H][max_sel], sel_count [B], s_kth [B][H], s_next [B][H])."""
    ind, lens, bud = _i32(page_indptr), _i32(seq_lens), _i32(pages_budget)
    B = len(lens)
    scores = np.ascontiguousarray(scores, dtype=np.float64)
    sel = np.empty((B, num_kv_heads, max_sel), np.int32)
    cnt = np.empty(B, np.int32)
    kth = np.empty((B, num_kv_heads))
    nxt = np.empty((B, num_kv_heads))
    _check(lib().vxo_select(_p(scores), num_kv_heads, page_size, B, _p(ind), _p(lens), _p(bud),
                            n_sink, n_local, max_sel, _p(sel), _p(cnt), _p(kth), _p(nxt)))
    return sel, cnt, kth, nxt


def topk_select(scores, num_items, pages_budget, n_sink, n_local, max_sel, tau=0.0, seed=0, remap=0):
    """Approximate radix top-k over fp32 scores [H][B][stride] (num_items[i] pages of request
    i).  Returns (sel_pages [B][H][max_sel], sel_count [B])."""
    sc = np.ascontiguousarray(scores, dtype=np.float32)
    H, B, stride = sc.shape
    n, bud = _i32(num_items), _i32(pages_budget)
    sel = np.empty((B, H, max_sel), np.int32)
    cnt = np.empty(B, np.int32)
    _check(lib().vxo_topk_select(_p(sc), stride, H, B, _p(n), _p(bud), n_sink, n_local, max_sel, float(np.float32(tau)),
                                 int(seed) & 0xFFFFFFFF, int(remap), _p(sel), _p(cnt)))
    return sel, cnt


def attend(q, k, v, page_size, page_indptr, page_indices, seq_lens, sel_pages, sel_count, sm_scale,
           head_dim_v=None, k_scale=1.0, v_scale=1.0):
    """fp64 output [B][Hq][Dv].  v=None means V = K[..., :head_dim_v] (MLA)."""
    qb = _bits(q)
    kb, fmt = _cache(k)
    vb, vfmt = _cache(v)
    assert vb is None or vfmt == fmt, "K and V caches must have the same dtype"
    B, Hq, Dqk = qb.shape
    _, H, ps, _ = kb.shape
    Dv = vb.shape[3] if vb is not None else head_dim_v
    ind, idx, lens = _i32(page_indptr), _i32(page_indices), _i32(seq_lens)
    sel, cnt = _i32(sel_pages), _i32(sel_count)
    max_sel = sel.shape[-1]
    out = np.empty((B, Hq, Dv))
    _check(lib().vxo_attend(_p(qb), Hq, _p(kb), _p(vb), fmt, float(k_scale), float(v_scale), H, ps, Dqk, Dv, B,
                            _p(ind), _p(idx), _p(lens), _p(sel), _p(cnt), max_sel, float(sm_scale), _p(out)))
    return out


def pipeline(q, k, v, cfg_kind, page_size, page_indptr, page_indices, seq_lens, pages_budget,
             n_sink, n_local, max_sel, sm_scale, head_dim_v=None, k_scale=1.0, v_scale=1.0):
    """The whole decode step: summaries -> scores -> selection -> attention."""
    mean, mx, mn = summarize(k, page_size, page_indptr, page_indices, seq_lens, k_scale=k_scale)
    H = _cache(k)[0].shape[1]
    Dv = head_dim_v if v is None else _cache(v)[0].shape[3]
    sc = flow_scores(cfg_kind, q, H, page_size, page_indptr, page_indices, seq_lens, mean, mx, mn, head_dim_v=Dv)
    sel, cnt, kth, nxt = select(sc, H, page_size, page_indptr, seq_lens, pages_budget, n_sink, n_local, max_sel)
    out = attend(q, k, v, page_size, page_indptr, page_indices, seq_lens, sel, cnt, sm_scale, head_dim_v,
                 k_scale=k_scale, v_scale=v_scale)
    return dict(mean=mean, max=mx, min=mn, scores=sc, sel=sel, cnt=cnt, kth=kth, next=nxt, out=out)
