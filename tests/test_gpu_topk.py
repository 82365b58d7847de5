"""The scoring and selection operators (vx_page_score, vx_topk_select) against the oracle, on
the GPU.  The approximate radix top-k (tolerate ratio, remapping, seeded window) must pick
exactly the oracle's pages from the same fp32 scores; the exact selection from scores must
equal the fused score + top-K entry point."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2606_06453_amd import vx, workloads as W
from paper_2606_06453_amd.workloads import synthetic_scores
from paper_2606_06453_amd.decoder import SparseDecoder
from tests._compare import GpuWorkload, last_page_index

pytestmark = pytest.mark.gpu


def _gpu_select(sc, n, bud, n_sink, n_local, max_sel, tau, seed, remap):
    H, B, _ = sc.shape
    sel = torch.full((B, H, max_sel), -7, dtype=torch.int32, device="cuda")
    cnt = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    vx.topk_select(torch.from_numpy(sc).cuda(), torch.from_numpy(np.asarray(n, np.int32)).cuda(),
                   torch.from_numpy(np.asarray(bud, np.int32)).cuda(), n_sink, n_local, max_sel, sel, cnt,
                   tolerate_ratio=tau, seed=seed, remap=remap)
    torch.cuda.synchronize()
    return sel.cpu().numpy(), cnt.cpu().numpy()


@pytest.mark.parametrize("dist", ["normal", "lognormal", "uniform", "bimodal", "ties"])
@pytest.mark.parametrize("tau", [0.0, 0.1, 0.3, 1.0])
@pytest.mark.parametrize("remap", [0, 1])
def test_topk_select_matches_oracle(dist, tau, remap):
    H, B, stride = 4, 6, 2100
    seed = 1000 * ["normal", "lognormal", "uniform", "bimodal", "ties"].index(dist) + int(tau * 100) * 2 + remap
    sc = synthetic_scores(dist, H, B, stride, seed=seed)
    n = [2100, 1, 37, 1024, 1500, 2099]
    bud = [130, 5, 40, 200, 0, 64]
    g_sel, g_cnt = _gpu_select(sc, n, bud, 1, 4, 256, tau, 12345, remap)
    o_sel, o_cnt = O.topk_select(sc, n, bud, 1, 4, 256, tau=tau, seed=12345, remap=remap)
    assert (g_cnt == o_cnt).all()
    assert (g_sel == o_sel).all()


@pytest.mark.parametrize("tau,remap", [(0.0, 0), (0.2, 0), (0.2, 1)])
@pytest.mark.parametrize("stride,n", [(8192, [8192, 4097]), (9000, [9000, 8500])])
def test_topk_select_long_rows(tau, remap, stride, n):
    """Up to 8192 candidates (32 per thread) keys stay in registers; longer rows recompute them
    from the scores."""
    H, B = 2, 2
    sc = synthetic_scores("normal", H, B, stride, seed=7)
    bud = [1000, 700]
    g_sel, g_cnt = _gpu_select(sc, n, bud, 1, 4, 1024, tau, 3, remap)
    o_sel, o_cnt = O.topk_select(sc, n, bud, 1, 4, 1024, tau=tau, seed=3, remap=remap)
    assert (g_cnt == o_cnt).all() and (g_sel == o_sel).all()


@pytest.mark.parametrize("name", ["llama3_8b_layer", "long_gen_quest", "large_gqa"])
def test_score_then_exact_select_equals_the_fused_call(name):
    wl = W.make(W.SMALL[name])
    c = wl.cfg
    gw = GpuWorkload(wl)
    dec = SparseDecoder(gw.kv, gw.batch, c.num_q_heads, c.kind, c.n_sink, c.n_local, wl.max_sel, c.sm_scale,
                        two_pass=False)
    dec.summarize()
    dec.select(gw.q, gw.budget)
    ref_sel, ref_cnt = dec.sel_pages.clone(), dec.sel_count.clone()
    H, B = c.num_kv_heads, c.batch
    stride = (wl.max_pages + 3) & ~3
    scores = torch.full((H, B, stride), float("nan"), dtype=torch.float32, device="cuda")
    vx.page_score(gw.q, gw.kv, gw.batch, c.kind, dec.mean, dec.max, dec.min, scores)
    n = torch.from_numpy(wl.pages.astype(np.int32)).cuda()
    sel = torch.empty_like(dec.sel_pages)
    cnt = torch.empty_like(dec.sel_count)
    vx.topk_select(scores, n, gw.budget, c.n_sink, c.n_local, wl.max_sel, sel, cnt)
    torch.cuda.synchronize()
    assert torch.equal(cnt, ref_cnt) and torch.equal(sel, ref_sel)
    # the scores themselves: the fp32 summaries (Mean rounded to fp32) and the final rounding
    # keep them within 2e-5 of the oracle's fp64 scores, far inside the 1e-4 comparison band
    k = wl.k_storage("cpu")
    mean, mx, mn = O.summarize(k, c.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens)
    sa, sb = {O.MEAN_DOT: (mean, None), O.MAX_DOT: (mx, None), O.QUEST: (mx, mn)}[c.kind]
    ref = O.score(c.kind, wl.q, H, c.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens, sa, sb)
    got = scores.cpu().numpy()
    for i in range(B):
        for h in range(H):
            r = ref[wl.page_indptr[i]: wl.page_indptr[i + 1], h]
            g = got[h, i, : len(r)]
            assert np.abs(g.astype(np.float64) - r).max() <= 2e-5, (i, h)


@pytest.mark.parametrize("name", ["llama3_8b_layer", "long_gen_quest", "large_gqa"])
@pytest.mark.parametrize("tau,remap", [(0.2, 0), (0.3, 1), (0.0, 1), (1.0, 0)])
def test_fused_approximate_selection(name, tau, remap):
    """vx_page_score_topk with approximate options (Sec. 5.2 in the indexer step): the same
    selection, bit for bit, as vx_page_score followed by vx_topk_select with those options, and as
    the oracle's approximate select run on the GPU's fp32 scores."""
    wl = W.make(W.SMALL[name])
    c = wl.cfg
    gw = GpuWorkload(wl)
    opt = vx.topk_options(tolerate_ratio=tau, seed=77, remap=remap)
    dec = SparseDecoder(gw.kv, gw.batch, c.num_q_heads, c.kind, c.n_sink, c.n_local, wl.max_sel, c.sm_scale,
                        topk_options=opt)
    dec.summarize()
    dec.select(gw.q, gw.budget)
    fused_sel, fused_cnt = dec.sel_pages.clone(), dec.sel_count.clone()
    H, B = c.num_kv_heads, c.batch
    stride = (wl.max_pages + 3) & ~3
    scores = torch.full((H, B, stride), float("nan"), dtype=torch.float32, device="cuda")
    vx.page_score(gw.q, gw.kv, gw.batch, c.kind, dec.mean, dec.max, dec.min, scores)
    n = torch.from_numpy(wl.pages.astype(np.int32)).cuda()
    sel = torch.empty_like(dec.sel_pages)
    cnt = torch.empty_like(dec.sel_count)
    vx.topk_select(scores, n, gw.budget, c.n_sink, c.n_local, wl.max_sel, sel, cnt, tolerate_ratio=tau, seed=77,
                   remap=remap)
    torch.cuda.synchronize()
    assert torch.equal(cnt, fused_cnt) and torch.equal(sel, fused_sel)
    o_sel, o_cnt = O.topk_select(scores.cpu().numpy(), wl.pages, wl.pages_budget, c.n_sink, c.n_local, wl.max_sel,
                                 tau=tau, seed=77, remap=remap)
    assert (o_cnt == fused_cnt.cpu().numpy()).all() and (o_sel == fused_sel.cpu().numpy()).all()


@pytest.mark.parametrize("kind", [O.QUEST, O.QUEST_CONSENSUS, O.ENVELOPE_LOWER, O.QUEST_RECTIFIED, O.MAX_DOT])
@pytest.mark.parametrize("D", [64, 128])
def test_envelope_scores_match_oracle(kind, D):
    """vx_page_score of every Max/Min kind against the oracle's fp64 scores: the GPU sums
    exact fp32 products in fp64 and rounds once, so the two agree to fp32 rounding."""
    from tests._problems import random_problem
    lens = [16 * 9 + 1, 16 * 4, 5, 16 * 30 + 8]
    pb = random_problem(70 + D + kind, lens, Hq=12, H=2, D=D, ps=16, extra_pages=5)
    kv = vx.PagedKV(pb.k.cuda(), pb.v.cuda(), D)
    P = (pb.seq_lens + 15) // 16
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    Pp = pb.k.shape[0]
    mx = torch.zeros((Pp, 2, D), dtype=torch.bfloat16, device="cuda")
    mn = torch.zeros((Pp, 2, D), dtype=torch.bfloat16, device="cuda")
    vx.page_summarize(kv, batch, None, None, mx, mn)
    stride = (int(P.max()) + 3) & ~3
    sc = torch.full((2, len(lens), stride), float("nan"), device="cuda")
    vx.page_score(pb.q.cuda(), kv, batch, kind, None, mx, None if kind in (O.MAX_DOT, O.QUEST_RECTIFIED) else mn, sc)
    torch.cuda.synchronize()
    _, omx, omn = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    ref = O.score(kind, pb.q, 2, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, omx,
                  None if kind in (O.MAX_DOT, O.QUEST_RECTIFIED) else omn)
    got = sc.cpu().numpy()
    for i in range(len(lens)):
        r = ref[pb.page_indptr[i]:pb.page_indptr[i + 1]].T        # [H][P_i]
        g = got[:, i, :P[i]].astype(np.float64)
        assert np.abs(g - r).max() <= 2.0 ** -23 * (1 + np.abs(r).max())


def _mean_problem(seed, D, Hq, H, Dv=None, alias=False):
    from tests._problems import random_problem
    lens = [16 * 9 + 1, 16 * 4, 5, 16 * 30 + 8]
    pb = random_problem(seed, lens, Hq=Hq, H=H, D=D, ps=16, Dv=Dv, alias_v=alias, extra_pages=5)
    kv = vx.PagedKV(pb.k.cuda(), None if pb.v is None else pb.v.cuda(), pb.head_dim_v)
    P = (pb.seq_lens + 15) // 16
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    mean = torch.zeros((pb.k.shape[0], H, D), dtype=torch.float32, device="cuda")
    vx.page_summarize(kv, batch, None, mean)
    omean, _, _ = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    return pb, kv, batch, P, mean, omean


def _rows(table, ragged, P, i):
    """GPU rows [rows][P_i] of request i and the oracle's ragged rows, transposed to match."""
    return table[:, i, :P[i]].astype(np.float64), ragged.T[:, :P[i]]


@pytest.mark.parametrize("D,Hq,H,Dv,alias", [(64, 12, 2, None, False), (128, 8, 1, None, False),
                                             (576, 16, 1, 512, True)])
def test_content_scores_match_oracle(D, Hq, H, Dv, alias):
    """Rope-unaware block score (Eq. 2 over the first head_dim_v channels): the MLA latent's 64
    rope channels are left out; on GQA it is the block-mean score."""
    pb, kv, batch, P, mean, omean = _mean_problem(80 + D, D, Hq, H, Dv, alias)
    stride = (int(P.max()) + 3) & ~3
    sc = torch.full((H, pb.batch, stride), float("nan"), device="cuda")
    vx.page_score(pb.q.cuda(), kv, batch, vx.MEAN_DOT_CONTENT, mean, None, None, sc)
    torch.cuda.synchronize()
    ref = O.score(O.MEAN_DOT_CONTENT, pb.q, H, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, omean,
                  content_dims=pb.head_dim_v)
    got = sc.cpu().numpy()
    for i in range(pb.batch):
        g, r = _rows(got, ref[pb.page_indptr[i]:pb.page_indptr[i + 1]], P, i)
        assert np.abs(g - r).max() <= 2e-5, i


@pytest.mark.parametrize("kind", [O.NSA, O.MEAN_DOT_SMOOTH])
@pytest.mark.parametrize("D,Hq,H", [(64, 12, 2), (128, 32, 8), (128, 16, 1), (128, 8, 4), (64, 4, 4)])
def test_flow_scores_match_oracle(kind, D, Hq, H):
    """The NSA and smoothing flows as operators: vx_page_score writes the first step (per-head
    logits; block-mean scores) within fp32 rounding of the oracle's; vx_score_flow's softmax,
    convolution and sum on those GPU values match the oracle's on the same values to fp32
    rounding."""
    pb, kv, batch, P, mean, omean = _mean_problem(90 + D + Hq + kind, D, Hq, H)
    stride = (int(P.max()) + 3) & ~3
    rows = Hq if kind == O.NSA else H
    first = torch.full((rows, pb.batch, stride), float("nan"), device="cuda")
    vx.page_score(pb.q.cuda(), kv, batch, kind, mean, None, None, first)
    out = torch.full((H, pb.batch, stride), float("nan"), device="cuda")
    n = torch.from_numpy(P.astype(np.int32)).cuda()
    vx.score_flow(kind, first, out, H, n)
    torch.cuda.synchronize()
    a = (pb.q, H, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, omean)
    ref1 = O.head_logits(*a) if kind == O.NSA else O.score(O.MEAN_DOT, a[0], *a[1:])
    f = first.cpu().numpy()
    ragged = np.concatenate([f[:, i, :P[i]].T for i in range(pb.batch)]).astype(np.float64)   # [T][rows]
    for i in range(pb.batch):
        g, r = _rows(f, ref1[pb.page_indptr[i]:pb.page_indptr[i + 1]], P, i)
        assert np.abs(g - r).max() <= 2e-5 * (1 + np.abs(r).max()), i
    if kind == O.NSA:
        ref2 = O.nsa_scores(ragged, H, 16, pb.page_indptr, pb.seq_lens)
    else:
        ref2 = O.smooth_scores(ragged, 16, pb.page_indptr, pb.seq_lens)
    o = out.cpu().numpy()
    for i in range(pb.batch):
        g, r = _rows(o, ref2[pb.page_indptr[i]:pb.page_indptr[i + 1]], P, i)
        assert (np.abs(g - r) <= 2.0 ** -23 * np.abs(r) + 1e-30).all(), i
