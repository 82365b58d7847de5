"""The envelope kinds' exact two-pass selection (Sec. 3.2 Quest; Appendix G envelope flows) on
the GPU: an fp32 bound pass, then an exact re-scoring of the pages whose intervals cannot be
placed.  The fused call must select exactly what the one-pass path selects (vx_page_score, then
the exact vx_topk_select), and every interval of the bound pass must hold the one-pass score.
Groups of up to 4 query heads per KV head take the two-pass path; larger groups stay one-pass
and are covered here too."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2606_06453_amd import vx
from paper_2606_06453_amd.decoder import SparseDecoder
from tests._compare import check_selection
from tests._problems import random_problem

pytestmark = pytest.mark.gpu

ENV = [O.QUEST, O.QUEST_CONSENSUS, O.ENVELOPE_LOWER, O.QUEST_RECTIFIED]


def _run(pb, kind, budget, n_sink, n_local, max_sel):
    """Fused selection, the one-pass scores and the one-pass selection."""
    kv = vx.PagedKV(pb.k.cuda(), None if pb.v is None else pb.v.cuda(), pb.head_dim_v)
    P = (pb.seq_lens + pb.page_size - 1) // pb.page_size
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    Hq, H, B = pb.q.shape[1], pb.k.shape[1], pb.batch
    dec = SparseDecoder(kv, batch, Hq, kind, n_sink, n_local, max_sel, 0.1)
    dec.summarize()
    q = pb.q.cuda()
    bud = torch.tensor(budget, dtype=torch.int32).cuda()
    dec.select(q, bud)
    stride = (int(P.max()) + 3) & ~3
    scores = torch.full((H, B, stride), float("nan"), dtype=torch.float32, device="cuda")
    vx.page_score(q, kv, batch, kind, dec.mean, dec.max, dec.min, scores)
    sel = torch.empty_like(dec.sel_pages)
    cnt = torch.empty_like(dec.sel_count)
    vx.topk_select(scores, torch.from_numpy(P.astype(np.int32)).cuda(), bud, n_sink, n_local, max_sel, sel, cnt)
    torch.cuda.synchronize()
    return dec, scores, sel, cnt, P


def _bound_planes(dec, H, B, stride):
    """The bound pass's lower and upper score planes, [H][B][stride] each, from the front of the
    fused call's workspace."""
    ws = dec.ws_score.view(torch.float32)
    n = H * B * stride
    return ws[:n].view(H, B, stride), ws[n:2 * n].view(H, B, stride)


@pytest.mark.parametrize("kind", ENV)
@pytest.mark.parametrize("ps,D,Hq,H", [(16, 64, 4, 1), (32, 128, 8, 2), (16, 128, 6, 2), (32, 64, 2, 2),
                                       (16, 128, 2, 1), (16, 64, 16, 2)])
def test_two_pass_equals_one_pass(kind, ps, D, Hq, H):
    lens = [ps * 300 + 3, ps * 41, 1, ps * 170 + ps // 2, ps * 9 - 1]
    pb = random_problem(2000 + 17 * kind + ps + D + Hq, lens, Hq=Hq, H=H, D=D, ps=ps, extra_pages=5)
    budget = [40, 17, 3, 90, 100]
    dec, scores, sel, cnt, P = _run(pb, kind, budget, 1, 4, 64)
    assert torch.equal(dec.sel_count, cnt)
    assert torch.equal(dec.sel_pages, sel)
    r = O.pipeline(pb.q, pb.k, pb.v, kind, ps, pb.page_indptr, pb.page_indices, pb.seq_lens, budget, 1, 4, 64, 0.1,
                   pb.head_dim_v)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], pb.page_indptr, P, 1, 4)


@pytest.mark.parametrize("kind", ENV)
@pytest.mark.parametrize("spread", [0.0, 20.0])
def test_bounds_hold_the_one_pass_scores(kind, spread):
    """Every page's interval from the bound pass holds its one-pass score; spread scales each
    key channel by 2^u with u uniform in [-spread, spread], so that the terms of a sum span many
    binades."""
    ps, D, Hq, H = 16, 128, 8, 2
    lens = [ps * 700 + 5, ps * 300, ps * 33 + 1]
    pb = random_problem(2100 + kind + int(spread), lens, Hq=Hq, H=H, D=D, ps=ps)
    if spread:
        g = torch.Generator().manual_seed(7 + kind)
        e = (torch.rand(1, 1, 1, D, generator=g) * 2 - 1) * spread
        pb.k = (pb.k.float() * torch.exp2(torch.round(e))).to(torch.bfloat16)
    dec, scores, sel, cnt, P = _run(pb, kind, [70, 50, 12], 1, 2, 80)
    assert torch.equal(dec.sel_pages, sel) and torch.equal(dec.sel_count, cnt)
    lo, up = _bound_planes(dec, H, pb.batch, scores.shape[2])
    for i in range(pb.batch):
        n = int(P[i])
        s, l, u = scores[:, i, :n], lo[:, i, :n], up[:, i, :n]
        assert torch.isfinite(l).all() and torch.isfinite(u).all()
        assert (l <= s).all() and (s <= u).all(), (i, float((l - s).max()), float((s - u).max()))
        # the intervals are narrow (2^-18 of the query's 1-norm times the largest summary value)
        width = (u - l) / s.abs().clamp_min(1e-30)
        assert float(width.median()) < 2.0 ** -6


@pytest.mark.parametrize("kind", [O.QUEST, O.QUEST_CONSENSUS])
@pytest.mark.parametrize("n_pages,noise", [(400, 2.0 ** -9), (1500, 0.0)])
def test_near_ties(kind, n_pages, noise):
    """Pages whose keys differ by about the bf16 resolution, or not at all: their intervals
    overlap, so the re-scoring decides (with noise 0 every full page ties, more pages are
    undecided than the compact list holds, and the lowest page indices must win)."""
    ps, D, Hq, H = 16, 128, 8, 2
    g = torch.Generator().manual_seed(91 + n_pages + kind)
    base = torch.randn(1, H, ps, D, generator=g)
    k = (base + noise * torch.randn(n_pages + 2, H, ps, D, generator=g)).to(torch.bfloat16)
    lens = np.array([n_pages * ps - 3], np.int32)
    indptr = np.array([0, n_pages], np.int32)
    idx = np.random.default_rng(6).permutation(n_pages + 2)[:n_pages].astype(np.int32)
    q = torch.randn(1, Hq, D, generator=g).to(torch.bfloat16)

    class _P:
        pass
    pb = _P()
    pb.q, pb.k, pb.v, pb.seq_lens, pb.page_indptr, pb.page_indices = q, k, k, lens, indptr, idx
    pb.page_size, pb.head_dim_v, pb.batch = ps, D, 1
    dec, scores, sel, cnt, P = _run(pb, kind, [60], 1, 2, 64)
    assert torch.equal(dec.sel_pages, sel) and torch.equal(dec.sel_count, cnt)
    if noise == 0.0:
        # the last page is partial, so its Max / Min differ; all full pages tie
        got = dec.sel_pages.cpu().numpy()[0]
        for h in range(H):
            chosen = [j for j in got[h].tolist() if j not in (-1, 0, n_pages - 2, n_pages - 1)]
            assert chosen == list(range(1, 58))
    r = O.pipeline(q, k, k, kind, ps, indptr, idx, lens, [60], 1, 2, 64, 0.1)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], indptr, np.array([n_pages]), 1, 2)
