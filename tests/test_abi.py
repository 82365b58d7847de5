"""The C-ABI library loads and exports every entry point include/vx.h declares, and its
host-side argument checks reject bad calls before any GPU work.  No GPU needed: every call
here returns before a kernel launch."""
import ctypes
import os
import re

import pytest
import torch

from paper_2606_06453_amd import vx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vx.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(vx_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert {"vx_version", "vx_last_error", "vx_workspace_size", "vx_page_summarize", "vx_page_score_topk",
            "vx_sparse_paged_decode", "vx_page_score", "vx_topk_select", "vx_score_flow",
            "vx_kv_append_summarize", "vx_append_score_topk"} <= set(names)
    lib = ctypes.CDLL(vx.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_version():
    assert vx.version() == (0 << 16) | 3


def _kv(D=128, H=8, ps=16, P=10, v=True, Dv=None, dtype=torch.bfloat16, k_scale=1.0, v_scale=1.0):
    k = torch.zeros((P, H, ps, D), dtype=dtype)
    vv = torch.zeros((P, H, ps, Dv or D), dtype=dtype) if v else None
    return vx.PagedKV(k, vv, Dv or D, k_scale=k_scale, v_scale=v_scale)


def _batch(B=2, maxP=5):
    return vx.BatchSpec(torch.zeros(B + 1, dtype=torch.int32), torch.zeros(B * maxP, dtype=torch.int32),
                        torch.ones(B, dtype=torch.int32), maxP)


def test_workspace_sizes():
    kv, b = _kv(), _batch(B=4, maxP=100)
    s = vx.workspace_size(vx.STAGE_SCORE_TOPK, kv, b, 32, 16)
    # fp32 planes [B][max_pages rounded up to 4]: max(2 H, Hq + H) of them (bounds; NSA logits)
    assert s == (32 + 8) * 4 * 100 * 4
    assert vx.workspace_size(vx.STAGE_SCORE_TOPK, kv, b, 8, 16) == 2 * 8 * 4 * 100 * 4
    d = vx.workspace_size(vx.STAGE_DECODE, kv, b, 32, 16)
    assert d > 0 and d % 256 == 0


def _status(fn):
    with pytest.raises(vx.VxError) as e:
        fn()
    return e.value.status, str(e.value)


def test_rejects_bad_geometry():
    b = _batch()
    st, msg = _status(lambda: vx.workspace_size(vx.STAGE_DECODE, _kv(D=96), b, 32, 8))
    assert st == 2 and "head_dim_qk" in msg
    st, _ = _status(lambda: vx.workspace_size(vx.STAGE_DECODE, _kv(ps=8), b, 32, 8))
    assert st == 2
    st, _ = _status(lambda: vx.workspace_size(vx.STAGE_DECODE, _kv(), b, 30, 8))       # 30 % 8 != 0
    assert st == 1
    st, _ = _status(lambda: vx.workspace_size(vx.STAGE_DECODE, _kv(H=1), b, 32, 8))    # group 32 > 16
    assert st == 2
    st, _ = _status(lambda: vx.workspace_size(vx.STAGE_DECODE, _kv(H=6), b, 12, 8))    # H not a power of 2
    assert st == 2
    st, _ = _status(lambda: vx.workspace_size(vx.STAGE_DECODE, _kv(D=576, H=1, v=False, Dv=256), b, 16, 8))
    assert st == 2


def test_fp8_cache_checks():
    b = _batch()
    e4 = torch.float8_e4m3fn
    assert vx.workspace_size(vx.STAGE_DECODE, _kv(dtype=e4, k_scale=0.01, v_scale=0.02), b, 32, 8) > 0
    assert vx.workspace_size(vx.STAGE_DECODE, _kv(dtype=torch.float8_e5m2), b, 32, 8) > 0
    # an fp8 MLA latent (V aliased at the latent's scale)
    assert vx.workspace_size(vx.STAGE_DECODE, _kv(D=576, H=1, v=False, Dv=512, dtype=e4, k_scale=0.02), b, 16, 8) > 0
    for ks, vs in [(0.0, 1.0), (1.0, -2.0), (float("inf"), 1.0), (float("nan"), 1.0)]:
        st, msg = _status(lambda: vx.workspace_size(vx.STAGE_DECODE, _kv(dtype=e4, k_scale=ks, v_scale=vs), b,
                                                    32, 8))
        assert st == 1 and "scale" in msg
    kv = _kv()
    kv.v = torch.zeros(kv.v.shape, dtype=e4)
    with pytest.raises(TypeError):                   # K and V must share the element type
        kv.struct()
    with pytest.raises(TypeError):
        vx.PagedKV(torch.zeros((2, 1, 16, 64), dtype=torch.float16), None, 64).struct()


def test_rejects_bad_selection_arguments():
    kv, b = _kv(), _batch()
    q = torch.zeros((2, 32, 128), dtype=torch.bfloat16)
    mean = torch.zeros((10, 8, 128))
    bud = torch.zeros(2, dtype=torch.int32)
    sel = torch.zeros((2, 8, 8), dtype=torch.int32)
    cnt = torch.zeros(2, dtype=torch.int32)
    ws = torch.zeros(4 * 8 * 5 * 2, dtype=torch.uint8)
    call = lambda **kw: vx.page_score_topk(q, kv, b, kw.get("kind", vx.MEAN_DOT), kw.get("mean", mean), None, None,
                                           bud, kw.get("ns", 1), kw.get("nl", 4), kw.get("ms", 8), sel, cnt,
                                           kw.get("ws", ws), stream=0, options=kw.get("opt"))
    st, _ = _status(lambda: call(ns=5, nl=4))          # n_sink + n_local > max_sel
    assert st == 1
    st, _ = _status(lambda: call(mean=None))           # MEAN_DOT without Mean
    assert st == 1
    st, _ = _status(lambda: call(kind=vx.QUEST))       # Quest without Max/Min
    assert st == 1
    st, msg = _status(lambda: call(ws=torch.zeros(16, dtype=torch.uint8)))
    assert st == 3 and "workspace" in msg
    st, msg = _status(lambda: call(kind=9))
    assert st == 1 and "unknown" in msg
    for kind in (vx.MEAN_DOT_CONTENT, vx.NSA, vx.MEAN_DOT_SMOOTH):    # all read the Mean
        st, msg = _status(lambda: call(kind=kind, mean=None))
        assert st == 1 and "Mean" in msg
    st, _ = _status(lambda: call(kind=vx.QUEST_CONSENSUS))   # needs Max and Min
    assert st == 1
    st, _ = _status(lambda: call(kind=vx.ENVELOPE_LOWER))
    assert st == 1
    # approximate selection options on the fused call
    st, msg = _status(lambda: call(opt=vx.topk_options(tolerate_ratio=1.5)))
    assert st == 1 and "tolerate_ratio" in msg
    st, msg = _status(lambda: call(opt=vx.topk_options(tolerate_ratio=0.2, remap=3)))
    assert st == 1 and "remap" in msg


def test_rejects_bad_decode_arguments():
    kv, b = _kv(), _batch()
    q = torch.zeros((2, 32, 128), dtype=torch.bfloat16)
    sel = torch.zeros((2, 8, 8), dtype=torch.int32)
    cnt = torch.zeros(2, dtype=torch.int32)
    out = torch.zeros((2, 32, 128), dtype=torch.bfloat16)
    ws = torch.zeros(16, dtype=torch.uint8)
    st, _ = _status(lambda: vx.sparse_paged_decode(q, kv, b, sel, cnt, 8, 0.1, out, ws, stream=0))
    assert st == 3
    st, _ = _status(lambda: vx.sparse_paged_decode(q, kv, b, sel, cnt, 8, -1.0, out, ws, stream=0))
    assert st == 1
    st, _ = _status(lambda: vx.sparse_paged_decode(q, _kv(v=False), b, sel, cnt, 8, 0.1, out, ws, stream=0))
    assert st == 2      # GQA needs a separate V cache
    st, msg = _status(lambda: vx.sparse_paged_decode(q, kv, b, sel, cnt, (1 << 24) + 1, 0.1, out, ws, stream=0))
    assert st == 2 and "2^24" in msg      # slot indices are 32-bit in the kernels


def test_last_error_is_thread_local():
    import threading
    kv, b = _kv(D=96), _batch()
    msgs = []

    def worker():
        try:
            vx.workspace_size(vx.STAGE_DECODE, _kv(ps=8), b, 32, 8)
        except vx.VxError as e:
            msgs.append(str(e))

    try:
        vx.workspace_size(vx.STAGE_DECODE, kv, b, 32, 8)
    except vx.VxError:
        pass
    t = threading.Thread(target=worker)
    t.start()
    t.join()
    assert "head_dim_qk" in vx.lib().vx_last_error().decode()
    assert "page_size" in msgs[0]


def test_rejects_bad_topk_select_arguments():
    sc = torch.zeros((2, 3, 10), dtype=torch.float32)
    n, bud = torch.ones(3, dtype=torch.int32), torch.ones(3, dtype=torch.int32)
    sel, cnt = torch.zeros((3, 2, 8), dtype=torch.int32), torch.zeros(3, dtype=torch.int32)
    st, msg = _status(lambda: vx.topk_select(sc, n, bud, 1, 2, 8, sel, cnt, tolerate_ratio=1.5, stream=0))
    assert st == 1 and "tolerate_ratio" in msg
    st, msg = _status(lambda: vx.topk_select(sc, n, bud, 1, 2, 8, sel, cnt, remap=7, stream=0))
    assert st == 1 and "remap" in msg
    st, msg = _status(lambda: vx.topk_select(sc, n, bud, 5, 4, 8, sel, cnt, stream=0))
    assert st == 1 and "n_sink" in msg


def test_rejects_bad_page_score_arguments():
    kv, b = _kv(), _batch(B=2, maxP=5)
    q = torch.zeros((2, 32, 128), dtype=torch.bfloat16)
    mean = torch.zeros((10, 8, 128), dtype=torch.float32)
    st, msg = _status(lambda: vx.page_score(q, kv, b, vx.MEAN_DOT, mean, None, None,
                                            torch.zeros((8, 2, 4), dtype=torch.float32), stream=0))
    assert st == 1 and "score_stride" in msg
    st, msg = _status(lambda: vx.page_score(q, kv, b, vx.QUEST, None, None, None,
                                            torch.zeros((8, 2, 5), dtype=torch.float32), stream=0))
    assert st == 1 and "Max and Min" in msg


def test_flow_kinds_and_score_flow_checks():
    """NSA runs on the GQA geometry only; the content and smoothing flows also on MLA.
    vx_score_flow takes the two flow kinds, distinct buffers and groups of at most 16 heads."""
    b = _batch()
    mla = _kv(D=576, H=1, v=False, Dv=512)
    q = torch.zeros((2, 16, 576), dtype=torch.bfloat16)
    mean = torch.zeros((10, 1, 576))
    bud = torch.zeros(2, dtype=torch.int32)
    sel, cnt = torch.zeros((2, 1, 8), dtype=torch.int32), torch.zeros(2, dtype=torch.int32)
    ws = torch.zeros(16, dtype=torch.uint8)
    st, msg = _status(lambda: vx.page_score_topk(q, mla, b, vx.NSA, mean, None, None, bud, 1, 4, 8, sel, cnt, ws,
                                                 stream=0))
    assert st == 2 and "MLA" in msg
    for kind in (vx.MEAN_DOT_CONTENT, vx.MEAN_DOT_SMOOTH):             # past the kind check: workspace
        st, msg = _status(lambda: vx.page_score_topk(q, mla, b, kind, mean, None, None, bud, 1, 4, 8, sel, cnt, ws,
                                                     stream=0))
        assert st == 3
    sin = torch.zeros((8, 2, 12), dtype=torch.float32)
    sout = torch.zeros((2, 2, 12), dtype=torch.float32)
    n = torch.ones(2, dtype=torch.int32)
    st, msg = _status(lambda: vx.score_flow(vx.MEAN_DOT, sin, sout, 2, n, stream=0))
    assert st == 1 and "NSA" in msg
    st, msg = _status(lambda: vx._check(vx.lib().vx_score_flow(vx.NSA, sout.data_ptr(), sout.data_ptr(), 12, 2, 8,
                                                               2, n.data_ptr(), None)))
    assert st == 1 and "differ" in msg
    st, msg = _status(lambda: vx._check(vx.lib().vx_score_flow(vx.NSA, sin.data_ptr(), sout.data_ptr(), 12, 1, 17,
                                                               2, n.data_ptr(), None)))
    assert st == 1 and "16" in msg


def test_append_checks():
    """The fused append needs k_new, and v_new exactly when V is a separate cache."""
    b = _batch()
    kn = torch.zeros((2, 8, 128), dtype=torch.bfloat16)
    st, msg = _status(lambda: vx.kv_append_summarize(_kv(), b, kn, None, stream=0))
    assert st == 1 and "v_new" in msg
    mla = _kv(D=576, H=1, v=False, Dv=512)
    kn1 = torch.zeros((2, 1, 576), dtype=torch.bfloat16)
    st, msg = _status(lambda: vx.kv_append_summarize(mla, b, kn1, kn1[:, :, :512].contiguous(), stream=0))
    assert st == 1 and "aliased" in msg
    st, msg = _status(lambda: vx._check(vx.lib().vx_kv_append_summarize(
        __import__("ctypes").byref(mla.struct()), __import__("ctypes").byref(b.struct()), None, None, None, None,
        None, None, None)))
    assert st == 1 and "k_new" in msg
    with pytest.raises(TypeError):
        vx.kv_append_summarize(_kv(), b, kn.float(), kn, stream=0)


def test_append_score_topk_checks():
    """The append inside the selection call checks its new rows like vx_kv_append_summarize,
    before any selection argument."""
    b = _batch()
    kn = torch.zeros((2, 8, 128), dtype=torch.bfloat16)
    st, msg = _status(lambda: vx.append_score_topk(_kv(), b, kn, None, None, None, None, kn, vx.MEAN_DOT, kn,
                                                   0, 0, 1, kn, kn, kn, stream=0))
    assert st == 1 and "v_new" in msg
    mla = _kv(D=576, H=1, v=False, Dv=512)
    kn1 = torch.zeros((2, 1, 576), dtype=torch.bfloat16)
    st, msg = _status(lambda: vx.append_score_topk(mla, b, kn1, kn1[:, :, :512].contiguous(), None, None, None, kn1,
                                                   vx.MEAN_DOT, kn1, 0, 0, 1, kn1, kn1, kn1, stream=0))
    assert st == 1 and "aliased" in msg


def test_block_size_checks():
    """block_size: 0, the page size, or 16 / 32 dividing it; the score workspace counts blocks."""
    b = _batch(B=4, maxP=100)
    for ps, bs in [(32, 16), (64, 16), (64, 32), (16, 16), (32, 0)]:
        kv = _kv(ps=ps)
        kv.block_size = bs
        r = ps // bs if bs else 1
        assert vx.workspace_size(vx.STAGE_SCORE_TOPK, kv, b, 32, 16) == (32 + 8) * 4 * 100 * r * 4
    for ps, bs in [(16, 32), (32, 8), (64, 48), (16, 64)]:
        kv = _kv(ps=ps)
        kv.block_size = bs
        st, msg = _status(lambda: vx.workspace_size(vx.STAGE_DECODE, kv, b, 32, 8))
        assert st == 2 and "block_size" in msg


def test_stream_read_checks():
    """The streaming-read measurement utility rejects unaligned or empty ranges and bad grids."""
    buf = torch.zeros(64, dtype=torch.uint8)
    sink = torch.zeros(4, dtype=torch.int32)
    st, msg = _status(lambda: vx._check(vx.lib().vx_stream_read(buf.data_ptr(), 24, sink.data_ptr(), 4, None)))
    assert st == 1 and "multiple of 16" in msg
    st, msg = _status(lambda: vx._check(vx.lib().vx_stream_read(buf.data_ptr() + 8, 16, sink.data_ptr(), 4, None)))
    assert st == 1 and "aligned" in msg
    st, msg = _status(lambda: vx._check(vx.lib().vx_stream_read(buf.data_ptr(), 64, sink.data_ptr(), 0, None)))
    assert st == 1 and "workgroups" in msg
