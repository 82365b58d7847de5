"""Parity of the HIP path (through the C ABI) with the fp64 oracle, on the GPU.

Sizes are small enough for the oracle to finish in seconds.  They span several 16-token
tiles, ragged lengths and partial last pages, and use every page size, head geometry and
score kind of the five workloads.
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2606_06453_amd import workloads as W
from paper_2606_06453_amd import vx
from paper_2606_06453_amd.decoder import SparseDecoder
from tests._compare import OUT_ATOL, GpuWorkload, check_selection, last_page_index, max_abs_err, newest_rows

pytestmark = pytest.mark.gpu

GQA = ["tiny_gqa", "llama3_8b_layer", "long_gen_quest", "large_gqa"]
ALL = GQA + ["mla_absorbed"]


def _oracle(wl):
    c = wl.cfg
    k = wl.k_storage("cpu")
    v = wl.v_storage("cpu")
    r = O.pipeline(wl.q, k, v, c.kind, c.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens,
                   wl.pages_budget, c.n_sink, c.n_local, wl.max_sel, c.sm_scale, c.head_dim_v)
    r["k"], r["v"] = k, v
    return r


def _decoder(gw):
    c = gw.wl.cfg
    return SparseDecoder(gw.kv, gw.batch, c.num_q_heads, c.kind, c.n_sink, c.n_local, gw.wl.max_sel,
                         c.sm_scale)


def _referenced(wl):
    return np.unique(wl.page_indices)


@pytest.mark.parametrize("name", ["llama3_8b_layer", "mla_absorbed"])
def test_generator_is_identical_on_gpu(name):
    wl = W.make(W.SMALL[name])
    k = wl.k_storage("cuda")
    sub = [0, 3, wl.num_phys_pages - 1]
    assert torch.equal(k[sub].cpu().view(torch.int16), wl.k_pages(sub).view(torch.int16))


@pytest.mark.parametrize("name", ALL)
def test_summaries_match_oracle(name):
    wl = W.make(W.SMALL[name])
    gw = GpuWorkload(wl)
    P, H, _, D = gw.k.shape
    mean = torch.full((P, H, D), float("nan"), device="cuda")
    mx = torch.zeros((P, H, D), dtype=torch.bfloat16, device="cuda")
    mn = torch.zeros((P, H, D), dtype=torch.bfloat16, device="cuda")
    vx.page_summarize(gw.kv, gw.batch, None, mean, mx, mn)
    torch.cuda.synchronize()
    om, ox, on = O.summarize(wl.k_storage("cpu"), wl.cfg.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens)
    ref = _referenced(wl)
    gm = mean.cpu().numpy().astype(np.float64)[ref]
    # fp32 accumulation over <= 64 bf16 values, one rounding of the quotient
    kmax = np.abs(wl.k_storage("cpu").float().numpy()).max()
    assert np.abs(gm - om[ref]).max() <= 4 * 2.0 ** -24 * kmax * 2
    assert np.array_equal(mx.float().cpu().numpy().astype(np.float64)[ref], ox[ref])
    assert np.array_equal(mn.float().cpu().numpy().astype(np.float64)[ref], on[ref])


def test_incremental_summarize_touches_only_later_pages():
    wl = W.make(W.SMALL["llama3_8b_layer"])
    gw = GpuWorkload(wl)
    P, H, _, D = gw.k.shape
    mean = torch.full((P, H, D), -7.0, device="cuda")
    first = last_page_index(wl)
    vx.page_summarize(gw.kv, gw.batch, first, mean, None, None)
    torch.cuda.synchronize()
    om, _, _ = O.summarize(wl.k_storage("cpu"), wl.cfg.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens,
                           first_page=(wl.pages - 1))
    gm = mean.cpu().numpy().astype(np.float64)
    for i in range(wl.cfg.batch):
        for j in range(int(wl.pages[i])):
            p = int(wl.page_indices[wl.page_indptr[i] + j])
            if j == wl.pages[i] - 1:
                assert np.abs(gm[p] - om[p]).max() < 1e-5
            else:
                assert (gm[p] == -7.0).all()


@pytest.mark.parametrize("ps,D,H,alias,fp8", [(16, 128, 8, False, None), (32, 64, 2, False, None),
                                              (64, 576, 1, True, None), (16, 128, 4, False, torch.float8_e4m3fn),
                                              (32, 64, 2, False, torch.float8_e5m2),
                                              (64, 576, 1, True, torch.float8_e4m3fn)])
def test_append_summarize_matches_oracle(ps, D, H, alias, fp8):
    """The fused cache stage of a decode step: appending each request's newest token to a cache
    stripped of it restores the cache bit for bit, and the receiving pages' summaries equal the
    oracle's and, bit for bit, an unfused vx_page_summarize of the restored cache."""
    from tests._problems import fp8_problem, random_problem, strip_last_token
    lens = [ps * 5 + 3, ps * 2 + 1, ps, 7, ps * 9]
    pb = random_problem(500 + ps + D, lens, Hq=H * 2, H=H, D=D, ps=ps, Dv=512 if alias else None, alias_v=alias,
                        extra_pages=4)
    ks = 1.0
    if fp8 is not None:
        ks = 0.03
        pb = fp8_problem(pb, fp8, ks, 0.02)
    k, v, kn, vn = strip_last_token(pb, 501)
    kv = vx.PagedKV(k.cuda(), None if v is None else v.cuda(), pb.head_dim_v, k_scale=ks, v_scale=0.02)
    P = (pb.seq_lens + ps - 1) // ps
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    Pp = pb.k.shape[0]
    outs = [torch.full((Pp, H, D), float("nan"), device="cuda"),
            torch.zeros((Pp, H, D), dtype=torch.bfloat16, device="cuda"),
            torch.zeros((Pp, H, D), dtype=torch.bfloat16, device="cuda"),
            torch.zeros((Pp, H, D), dtype=torch.bfloat16, device="cuda")]
    vx.kv_append_summarize(kv, batch, kn.cuda(), None if vn is None else vn.cuda(), outs[0], outs[2], outs[3],
                           mean_bf16=outs[1])
    torch.cuda.synchronize()
    as_bytes = lambda t: t.cpu().contiguous().view(torch.uint8)
    assert torch.equal(as_bytes(kv.k), as_bytes(pb.k))
    if not alias:
        assert torch.equal(as_bytes(kv.v), as_bytes(pb.v))
    # unfused: vx_page_summarize of the restored cache from the receiving pages on
    ref = [torch.full_like(o, float("nan")) if o.dtype == torch.float32 else torch.zeros_like(o) for o in outs]
    first = torch.from_numpy(((pb.seq_lens - 1) // ps).astype(np.int32)).cuda()
    vx.page_summarize(kv, batch, first, ref[0], ref[2], ref[3], mean_bf16=ref[1])
    torch.cuda.synchronize()
    pages = [int(pb.page_indices[pb.page_indptr[i] + (int(pb.seq_lens[i]) - 1) // ps]) for i in range(pb.batch)]
    for o, r in zip(outs, ref):
        assert torch.equal(as_bytes(o[pages]), as_bytes(r[pages]))
    _, _, (om, ox, on), _ = O.kv_append(k, v, ps, pb.page_indptr, pb.page_indices, pb.seq_lens, kn, vn,
                                        head_dim_v=pb.head_dim_v, k_scale=ks)
    kmax = max(np.abs(ox[pages]).max(), np.abs(on[pages]).max())     # bounds |k| on these pages
    assert np.abs(outs[0].cpu().numpy().astype(np.float64)[pages] - om[pages]).max() <= 4 * 2.0 ** -24 * kmax * 2
    assert np.array_equal(outs[2].float().cpu().numpy().astype(np.float64)[pages], ox[pages])
    assert np.array_equal(outs[3].float().cpu().numpy().astype(np.float64)[pages], on[pages])


@pytest.mark.parametrize("name", ALL)
def test_selection_matches_oracle(name):
    wl = W.make(W.SMALL[name])
    c = wl.cfg
    gw = GpuWorkload(wl)
    dec = _decoder(gw)
    dec.summarize()
    dec.select(gw.q, gw.budget)
    torch.cuda.synchronize()
    r = _oracle(wl)
    exempt = check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"],
                             r["scores"], r["kth"], r["next"], wl.page_indptr, wl.pages, c.n_sink, c.n_local)
    assert exempt <= max(1, wl.cfg.batch * wl.cfg.num_kv_heads // 20)


@pytest.mark.parametrize("name", ALL)
def test_decode_on_oracle_selection(name):
    wl = W.make(W.SMALL[name])
    gw = GpuWorkload(wl)
    dec = _decoder(gw)
    r = _oracle(wl)
    sel = torch.from_numpy(r["sel"]).cuda()
    cnt = torch.from_numpy(r["cnt"]).cuda()
    out = dec.decode(gw.q, sel, cnt)
    torch.cuda.synchronize()
    assert np.abs(r["out"]).max() < 4
    err = max_abs_err(out, r["out"])
    assert err <= OUT_ATOL, err


@pytest.mark.parametrize("name", ALL)
def test_end_to_end_step(name):
    """Full step on the GPU; the attention output is checked against the oracle's attention on
    the GPU's (validated) selection."""
    wl = W.make(W.SMALL[name])
    c = wl.cfg
    gw = GpuWorkload(wl)
    dec = _decoder(gw)
    dec.summarize()
    out = dec.step(gw.q, gw.budget, last_page_index(wl))
    torch.cuda.synchronize()
    r = _oracle(wl)
    gsel, gcnt = dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy()
    check_selection(gsel, gcnt, r["sel"], r["cnt"], r["scores"], r["kth"], r["next"], wl.page_indptr, wl.pages,
                    c.n_sink, c.n_local)
    ref = O.attend(wl.q, r["k"], r["v"], c.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens, gsel, gcnt,
                   c.sm_scale, c.head_dim_v)
    assert max_abs_err(out, ref) <= OUT_ATOL


def test_run_twice_is_bitwise_identical():
    wl = W.make(W.SMALL["large_gqa"])
    gw = GpuWorkload(wl)
    dec = _decoder(gw)
    dec.summarize()
    a = dec.step(gw.q, gw.budget, last_page_index(wl)).clone()
    sa = dec.sel_pages.clone()
    b = dec.step(gw.q, gw.budget, last_page_index(wl))
    torch.cuda.synchronize()
    assert torch.equal(sa, dec.sel_pages)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("name,fused", [("llama3_8b_layer", False), ("long_gen_quest", False), ("mla_absorbed", False),
                                        ("llama3_8b_layer", True), ("mla_absorbed", True)])
def test_hip_graph_replays_match_eager(name, fused):
    """A decode step captured in a HIP graph and replayed several times, with eager work and
    synchronisations between the replays, gives the eager selection and output bit for bit.
    fused: the step appends each request's newest rows inside the top-K launch (the selection
    workgroups for the block mean; append workgroups of their own beside the one-wave selection
    for the MLA latent), re-writing the same rows on every replay."""
    wl = W.make(W.SMALL[name])
    gw = GpuWorkload(wl)
    dec = _decoder(gw)
    dec.summarize()
    first = None if fused else last_page_index(wl)
    kw = dict(kv_new=newest_rows(wl, gw)) if fused else {}
    ref = dec.step(gw.q, gw.budget, first, **kw).clone()
    ref_sel, ref_cnt = dec.sel_pages.clone(), dec.sel_count.clone()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dec.step(gw.q, gw.budget, first, **kw)
    for r in range(3):
        dec.out.zero_()
        dec.sel_pages.fill_(-7)
        dec.sel_count.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(dec.sel_pages, ref_sel), f"replay {r}: selection differs"
        assert torch.equal(dec.sel_count, ref_cnt), f"replay {r}: counts differ"
        assert torch.equal(dec.out.view(torch.int16), ref.view(torch.int16)), f"replay {r}: output differs"


# ------------------------------------------------------------------------------------------
# edge cases on hand-built problems
# ------------------------------------------------------------------------------------------
def _problem_on_gpu(pb, kind, budget, n_sink, n_local, max_sel, sm_scale):
    from tests._problems import Problem  # noqa: F401
    kv = vx.PagedKV(pb.k.cuda(), None if pb.v is None else pb.v.cuda(), pb.head_dim_v)
    P = (pb.seq_lens + pb.page_size - 1) // pb.page_size
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    dec = SparseDecoder(kv, batch, pb.q.shape[1], kind, n_sink, n_local, max_sel, sm_scale)
    return dec, torch.tensor(budget, dtype=torch.int32).cuda(), P


@pytest.mark.parametrize("ps,D,Hq,H", [(16, 64, 4, 1), (32, 128, 8, 1), (64, 128, 16, 2), (16, 128, 12, 2),
                                       (32, 64, 16, 1), (64, 64, 3, 3 // 3)])
@pytest.mark.parametrize("kind", [O.MEAN_DOT, O.QUEST, O.MAX_DOT, O.QUEST_CONSENSUS, O.ENVELOPE_LOWER,
                                  O.QUEST_RECTIFIED, O.MEAN_DOT_CONTENT, O.NSA, O.MEAN_DOT_SMOOTH])
def test_geometries_and_kinds(ps, D, Hq, H, kind):
    from tests._problems import random_problem
    lens = [ps * 9 + 1, ps * 4, 5, ps * 13 + ps // 2, 1, ps * 2 - 1]
    pb = random_problem(100 + ps + D + Hq, lens, Hq=Hq, H=H, D=D, ps=ps, extra_pages=7)
    budget = [5, 3, 1, 6, 2, 9]
    max_sel, n_sink, n_local = 8, 1, 2
    sm = 1.0 / math.sqrt(D)
    dec, bud, P = _problem_on_gpu(pb, kind, budget, n_sink, n_local, max_sel, sm)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    out = dec.decode(q)
    torch.cuda.synchronize()
    r = O.pipeline(pb.q, pb.k, pb.v, kind, ps, pb.page_indptr, pb.page_indices, pb.seq_lens, budget, n_sink,
                   n_local, max_sel, sm, pb.head_dim_v)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], pb.page_indptr, P, n_sink, n_local)
    ref = O.attend(pb.q, pb.k, pb.v, ps, pb.page_indptr, pb.page_indices, pb.seq_lens,
                   dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), sm, pb.head_dim_v)
    assert max_abs_err(out, ref) <= OUT_ATOL


def _random_selection(rng, P, cnt, H, max_sel):
    """Ascending random subsets of cnt[i] of request i's P[i] pages, per KV head, -1 padded."""
    sel = np.full((len(P), H, max_sel), -1, np.int32)
    for i in range(len(P)):
        for h in range(H):
            sel[i, h, : cnt[i]] = np.sort(rng.choice(int(P[i]), size=int(cnt[i]), replace=False))
    return sel


def _decode_on(dec, pb, sel, cnt, sm):
    """vx_sparse_paged_decode on a given selection, and the oracle's attention on it."""
    out = dec.decode(pb.q.cuda(), torch.from_numpy(sel).cuda(), torch.from_numpy(np.asarray(cnt, np.int32)).cuda())
    torch.cuda.synchronize()
    ref = O.attend(pb.q, pb.k, pb.v, pb.page_size, pb.page_indptr, pb.page_indices, pb.seq_lens, sel,
                   np.asarray(cnt, np.int32), sm, pb.head_dim_v)
    return out.clone(), ref


@pytest.mark.parametrize("H,Hq,long_pages,short_pages,n_short", [
    (1, 4, 64, 2, 100),       # 101 pairs: the long pair is split over six workgroups
    (4, 16, 300, 3, 129),     # 520 pairs: one workgroup per pair, however long
])
def test_decode_plan_with_skewed_counts(H, Hq, long_pages, short_pages, n_short):
    """The decode plan cuts a pair with many selected pages into splits of bounded size and
    merges them in the split kernel, while the many short pairs stay whole (some select nothing).
    Two calls in a row with different selections: the split counters are back at zero after the
    first."""
    from tests._problems import random_problem
    rng = np.random.default_rng(long_pages)
    B = 1 + n_short
    lens = [16 * (long_pages + 9) + 3] + [int(x) for x in rng.integers(16 * short_pages + 1, 16 * 9, size=n_short)]
    pb = random_problem(31 + long_pages, lens, Hq=Hq, H=H, D=128, ps=16, extra_pages=2)
    P = (np.asarray(lens) + 15) // 16
    sm = 1.0 / math.sqrt(128)
    dec, _, _ = _problem_on_gpu(pb, O.MEAN_DOT, [1] * B, 0, 0, long_pages, sm)
    for call in range(2):
        cnt = np.array([long_pages - 7 * call] + [int(x) for x in rng.integers(0, short_pages + 1, size=n_short)],
                       np.int32)
        sel = _random_selection(rng, P, cnt, H, long_pages)
        out, ref = _decode_on(dec, pb, sel, cnt, sm)
        assert max_abs_err(out, ref) <= OUT_ATOL, call
        zero = np.flatnonzero(cnt == 0)
        assert (out[torch.from_numpy(zero).cuda()].float() == 0).all()


@pytest.mark.parametrize("D", [64, 128])
def test_many_pairs_three_wave_workgroups(D):
    """880 (request, KV head) pairs: more than four waves per pair can keep resident on 256 CUs,
    so the split kernel runs three-wave workgroups (one per pair)."""
    from tests._problems import random_problem
    rng = np.random.default_rng(D)
    lens = [int(x) for x in rng.integers(1, 16 * 24, size=110)]
    pb = random_problem(900 + D, lens, Hq=16, H=8, D=D, ps=16, extra_pages=3)
    budget = [int(x) for x in rng.integers(0, 14, size=110)]
    max_sel, n_sink, n_local = 12, 1, 2
    sm = 1.0 / math.sqrt(D)
    dec, bud, P = _problem_on_gpu(pb, O.MAX_DOT, budget, n_sink, n_local, max_sel, sm)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    out = dec.decode(q)
    torch.cuda.synchronize()
    ref = O.attend(pb.q, pb.k, pb.v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens,
                   dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), sm, pb.head_dim_v)
    assert max_abs_err(out, ref) <= OUT_ATOL


@pytest.mark.parametrize("D,dtype,B,H", [(64, "bf16", 517, 2), (128, "bf16", 517, 2), (128, "fp8_e4m3", 517, 2),
                                         (64, "bf16", 1024, 1)])
def test_many_pairs_with_skewed_counts(D, dtype, B, H):
    """1034 (request, KV head) pairs (or 1024 requests of one KV head), one split each, with
    skewed selection counts (0 to 40 pages, some requests with none): more pairs than four-wave
    workgroups can keep resident, in bf16 and fp8, so the workgroups serve the requests in the
    count-balanced order (blocks of 128 and 256 positions, the last one partial at 517).  Two
    calls in a row with different selections."""
    from tests._problems import random_problem
    rng = np.random.default_rng(D + len(dtype) + B)
    Hq = 4
    lens = [int(x) for x in np.clip(np.exp(rng.normal(math.log(300), 0.9, size=B)), 1, 16 * 48)]
    pb = random_problem(1300 + D, lens, Hq=Hq, H=H, D=D, ps=16, extra_pages=3)
    P = (np.asarray(lens) + 15) // 16
    sm = 1.0 / math.sqrt(D)
    max_sel = 40
    kw = {}
    if dtype == "bf16":
        dec, _, _ = _problem_on_gpu(pb, O.MEAN_DOT, [1] * B, 0, 0, max_sel, sm)
    else:
        from tests._problems import fp8_problem
        kw = dict(k_scale=0.021, v_scale=0.0377)
        pb = fp8_problem(pb, torch.float8_e4m3fn, kw["k_scale"], kw["v_scale"])
        kv = vx.PagedKV(pb.k.cuda(), pb.v.cuda(), D, **kw)
        batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                             torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
        dec = SparseDecoder(kv, batch, Hq, O.MEAN_DOT, 0, 0, max_sel, sm)
    for call in range(2):
        cnt = np.minimum(P, rng.integers(0, max_sel + 1, size=B)).astype(np.int32)
        cnt[rng.integers(0, B, size=5)] = 0
        sel = _random_selection(rng, P, cnt, H, max_sel)
        out = dec.decode(pb.q.cuda(), torch.from_numpy(sel).cuda(), torch.from_numpy(cnt).cuda())
        torch.cuda.synchronize()
        ref = O.attend(pb.q, pb.k, pb.v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, sel, cnt, sm, D, **kw)
        assert max_abs_err(out, ref) <= OUT_ATOL, call
        zero = np.flatnonzero(cnt == 0)
        assert (out[torch.from_numpy(zero).cuda()].float() == 0).all()


def test_empty_selection_and_all_pages():
    from tests._problems import random_problem
    pb = random_problem(7, [40, 16 * 6 + 3, 16 * 20], Hq=8, H=2, D=128, ps=16)
    budget = [0, 100, 3]          # nothing / every page / top-K
    dec, bud, P = _problem_on_gpu(pb, O.MEAN_DOT, budget, 0, 0, 16, 0.088)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    out = dec.decode(q)
    torch.cuda.synchronize()
    cnt = dec.sel_count.cpu().numpy()
    assert cnt.tolist() == [0, 7, 3]
    assert (out[0].float() == 0).all()
    r = O.pipeline(pb.q, pb.k, pb.v, O.MEAN_DOT, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, budget, 0, 0,
                   16, 0.088)
    assert max_abs_err(out, r["out"]) <= OUT_ATOL


def test_prefix_shared_pages():
    from tests._problems import random_problem
    pb = random_problem(8, [16 * 10, 16 * 12 + 5], Hq=8, H=2, D=128, ps=16, extra_pages=2)
    idx = pb.page_indices.copy()
    idx[pb.page_indptr[1]:pb.page_indptr[1] + 6] = idx[:6]     # request 1 shares request 0's prefix
    pb.page_indices = idx
    budget = [6, 6]
    dec, bud, P = _problem_on_gpu(pb, O.QUEST, budget, 1, 1, 8, 0.088)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    out = dec.decode(q)
    torch.cuda.synchronize()
    r = O.pipeline(pb.q, pb.k, pb.v, O.QUEST, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, budget, 1, 1, 8,
                   0.088)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], pb.page_indptr, P, 1, 1)
    ref = O.attend(pb.q, pb.k, pb.v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens,
                   dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), 0.088)
    assert max_abs_err(out, ref) <= OUT_ATOL


def test_ties_go_to_the_lower_page_index():
    """Identical pages give identical scores: the lowest indices must win, as in the oracle."""
    from tests._problems import random_problem
    pb = random_problem(9, [16 * 12], Hq=4, H=1, D=64, ps=16)
    k = pb.k.clone()
    for j in range(12):           # every logical page holds the same keys
        k[int(pb.page_indices[j])] = pb.k[int(pb.page_indices[0])]
    pb.k = k
    dec, bud, P = _problem_on_gpu(pb, O.MEAN_DOT, [4], 0, 0, 4, 0.125)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    torch.cuda.synchronize()
    assert dec.sel_pages.cpu().numpy()[0, 0].tolist() == [0, 1, 2, 3]


@pytest.mark.parametrize("ps", [16, 32, 64])
@pytest.mark.parametrize("kind", [O.MEAN_DOT, O.MEAN_DOT_CONTENT, O.MEAN_DOT_SMOOTH])
def test_mla_geometry(ps, kind):
    """Absorbed-weight MLA: 16 heads share a 576-channel latent, V = latent[:512]; ragged
    lengths with partial pages, a one-token request, and several splits per request.  Scored
    on the full latent (rope-aware), on its 512 content channels (rope-unaware) and smoothed."""
    from tests._problems import random_problem
    lens = [ps * 30 + 5, 7, ps * 3, ps * 17 + ps // 2 + 1, 1]
    pb = random_problem(300 + ps, lens, Hq=16, H=1, D=576, ps=ps, Dv=512, alias_v=True, extra_pages=3)
    budget = [20, 4, 2, 9, 1]
    max_sel, n_sink, n_local = 24, 1, 4
    sm = 1.0 / math.sqrt(576)
    dec, bud, P = _problem_on_gpu(pb, kind, budget, n_sink, n_local, max_sel, sm)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    out = dec.decode(q)
    torch.cuda.synchronize()
    r = O.pipeline(pb.q, pb.k, None, kind, ps, pb.page_indptr, pb.page_indices, pb.seq_lens, budget,
                   n_sink, n_local, max_sel, sm, 512)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], pb.page_indptr, P, n_sink, n_local)
    ref = O.attend(pb.q, pb.k, None, ps, pb.page_indptr, pb.page_indices, pb.seq_lens,
                   dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), sm, 512)
    assert max_abs_err(out, ref) <= OUT_ATOL


def test_mla_one_split():
    """MLA with one selected page per request (max_sel = 1): a request never has more splits
    than selection slots, so the split kernel writes the bf16 output itself instead of
    partials for the merge."""
    from tests._problems import random_problem
    ps = 64
    lens = [ps * 6 + 9, 40, ps * 2, 1]
    pb = random_problem(377, lens, Hq=16, H=1, D=576, ps=ps, Dv=512, alias_v=True, extra_pages=2)
    budget = [1, 1, 1, 1]
    sm = 1.0 / math.sqrt(576)
    dec, bud, P = _problem_on_gpu(pb, O.MEAN_DOT, budget, 0, 0, 1, sm)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    out = dec.decode(q)
    torch.cuda.synchronize()
    r = O.pipeline(pb.q, pb.k, None, O.MEAN_DOT, ps, pb.page_indptr, pb.page_indices, pb.seq_lens, budget,
                   0, 0, 1, sm, 512)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], pb.page_indptr, P, 0, 0)
    ref = O.attend(pb.q, pb.k, None, ps, pb.page_indptr, pb.page_indices, pb.seq_lens,
                   dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), sm, 512)
    assert max_abs_err(out, ref) <= OUT_ATOL


# ------------------------------------------------------------------------------------------
# exact two-pass block-mean selection: a bf16 first pass with a rigorous score interval, then
# fp32 re-scoring of the undecided pages; the selection must equal the one-pass selection bit
# for bit (and so pass the oracle's band rule like it)
# ------------------------------------------------------------------------------------------
def _one_and_two_pass(kv, batch, Hq, n_sink, n_local, max_sel, q, bud, sm=0.1):
    d1 = SparseDecoder(kv, batch, Hq, vx.MEAN_DOT, n_sink, n_local, max_sel, sm, two_pass=False)
    d2 = SparseDecoder(kv, batch, Hq, vx.MEAN_DOT, n_sink, n_local, max_sel, sm, two_pass=True)
    assert d1.mean_bf16 is None and d2.mean_bf16 is not None
    for d in (d1, d2):
        d.summarize()
        d.select(q, bud)
    torch.cuda.synchronize()
    return d1, d2


def _assert_same_selection(d1, d2):
    assert torch.equal(d1.sel_count, d2.sel_count)
    assert torch.equal(d1.sel_pages, d2.sel_pages)


def test_bf16_mean_copy_is_rne_of_fp32_mean():
    wl = W.make(W.SMALL["llama3_8b_layer"])
    gw = GpuWorkload(wl)
    P, H, _, D = gw.k.shape
    mean = torch.zeros((P, H, D), device="cuda")
    mbf = torch.zeros((P, H, D), dtype=torch.bfloat16, device="cuda")
    vx.page_summarize(gw.kv, gw.batch, None, mean, None, None, mean_bf16=mbf)
    torch.cuda.synchronize()
    ref = _referenced(wl)
    assert torch.equal(mbf[ref].view(torch.int16).cpu(), mean[ref].cpu().to(torch.bfloat16).view(torch.int16))


@pytest.mark.parametrize("name", ["tiny_gqa", "llama3_8b_layer", "mla_absorbed"])
def test_two_pass_equals_one_pass_on_workloads(name):
    wl = W.make(W.SMALL[name])
    c = wl.cfg
    gw = GpuWorkload(wl)
    d1, d2 = _one_and_two_pass(gw.kv, gw.batch, c.num_q_heads, c.n_sink, c.n_local, wl.max_sel, gw.q, gw.budget)
    _assert_same_selection(d1, d2)
    r = _oracle(wl)
    check_selection(d2.sel_pages.cpu().numpy(), d2.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], wl.page_indptr, wl.pages, c.n_sink, c.n_local)


@pytest.mark.parametrize("ps,D,Hq,H", [(16, 64, 4, 1), (32, 128, 8, 2), (64, 128, 16, 4), (16, 128, 12, 2),
                                       (16, 576, 16, 1), (64, 576, 16, 1)])
def test_two_pass_equals_one_pass_on_geometries(ps, D, Hq, H):
    from tests._problems import random_problem
    lens = [ps * 300 + 3, ps * 41, 1, ps * 170 + ps // 2, ps * 9 - 1]
    mla = D == 576
    pb = random_problem(500 + ps + D + Hq, lens, Hq=Hq, H=H, D=D, ps=ps, extra_pages=5,
                        Dv=512 if mla else None, alias_v=mla)
    budget = [40, 17, 3, 90, 100]
    max_sel, n_sink, n_local = 64, 1, 4
    kv = vx.PagedKV(pb.k.cuda(), None if pb.v is None else pb.v.cuda(), pb.head_dim_v)
    P = (pb.seq_lens + ps - 1) // ps
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    q = pb.q.cuda()
    d1, d2 = _one_and_two_pass(kv, batch, Hq, n_sink, n_local, max_sel, q,
                               torch.tensor(budget, dtype=torch.int32).cuda())
    _assert_same_selection(d1, d2)


@pytest.mark.parametrize("n_pages,noise", [(400, 2.0 ** -12), (1500, 0.0)])
def test_two_pass_near_ties(n_pages, noise):
    """Pages that differ by far less than the bf16 resolution of their means: the bounds overlap
    for most pages, so they go through the exact re-scoring.  With noise 0 every page ties and
    more pages are undecided than the compact list holds (the re-score-all fallback); the lowest
    page indices must win."""
    ps, D, Hq, H = 16, 128, 8, 2
    g = torch.Generator().manual_seed(77 + n_pages)
    base = torch.randn(1, H, ps, D, generator=g)
    k = (base + noise * torch.randn(n_pages + 2, H, ps, D, generator=g)).to(torch.bfloat16)
    lens = np.array([n_pages * ps - 3], np.int32)
    indptr = np.array([0, n_pages], np.int32)
    idx = np.random.default_rng(5).permutation(n_pages + 2)[:n_pages].astype(np.int32)
    q = torch.randn(1, Hq, D, generator=g).to(torch.bfloat16)
    kv = vx.PagedKV(k.cuda(), k.cuda(), D)
    batch = vx.BatchSpec(torch.from_numpy(indptr).cuda(), torch.from_numpy(idx).cuda(),
                         torch.from_numpy(lens).cuda(), n_pages)
    d1, d2 = _one_and_two_pass(kv, batch, Hq, 1, 2, 64, q.cuda(), torch.tensor([60], dtype=torch.int32).cuda())
    _assert_same_selection(d1, d2)
    if noise == 0.0:
        # the last page is partial, so its mean differs; all full pages tie
        sel = d2.sel_pages.cpu().numpy()[0]
        for h in range(H):
            chosen = [j for j in sel[h].tolist() if j not in (-1, 0, n_pages - 2, n_pages - 1)]
            assert chosen == list(range(1, 58))
    r = O.pipeline(q, k, k, O.MEAN_DOT, ps, indptr, idx, lens, [60], 1, 2, 64, 0.1)
    check_selection(d2.sel_pages.cpu().numpy(), d2.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], indptr, np.array([n_pages]), 1, 2)


@pytest.mark.parametrize("kind", [O.MEAN_DOT, O.QUEST, O.MAX_DOT, O.NSA, O.MEAN_DOT_SMOOTH, O.MEAN_DOT_CONTENT])
def test_requests_longer_than_4096_pages(kind):
    """Past 4096 pages per request the selection runs the general radix kernel (and MEAN_DOT
    ignores the bf16 copy); a second, short request keeps the batch ragged."""
    from tests._problems import random_problem
    lens = [16 * 4500 + 7, 16 * 37]
    pb = random_problem(900 + kind, lens, Hq=4, H=2, D=64, ps=16)
    budget = [70, 9]
    max_sel, n_sink, n_local = 80, 1, 3
    dec, bud, P = _problem_on_gpu(pb, kind, budget, n_sink, n_local, max_sel, 0.125)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    torch.cuda.synchronize()
    r = O.pipeline(pb.q, pb.k, pb.v, kind, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, budget, n_sink,
                   n_local, max_sel, 0.125, pb.head_dim_v)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], pb.page_indptr, P, n_sink, n_local)



# ------------------------------------------------------------------------------------------
# blocks below the page size: summaries, scores, selection and attention per block of
# block_size tokens inside the paged layout, against the oracle on the re-blocked problem
# ------------------------------------------------------------------------------------------
_BLOCK_GQA = [(32, 16, 128, 8, 2), (64, 16, 64, 12, 4), (64, 32, 128, 16, 1)]


# the MLA geometry scores with the block mean only
@pytest.mark.parametrize("ps,bs,D,Hq,H,kind", [g + (k,) for g in _BLOCK_GQA for k in (O.MEAN_DOT, O.QUEST, O.NSA)]
                         + [(32, 16, 576, 16, 1, O.MEAN_DOT)])
def test_blocks_below_page_size(ps, bs, D, Hq, H, kind):
    from tests._problems import random_problem
    mla = D == 576
    lens = [ps * 9 + bs + 1, ps * 4, 5, ps * 13 + ps // 2, 1, ps * 2 - 1]
    pb = random_problem(700 + ps + bs + D + kind, lens, Hq=Hq, H=H, D=D, ps=ps, Dv=512 if mla else None,
                        alias_v=mla, extra_pages=5)
    r = ps // bs
    budget = [9, 5, 1, 12, 2, 4]
    max_sel, n_sink, n_local = 16, 1, 2
    sm = 1.0 / math.sqrt(D)
    kv = vx.PagedKV(pb.k.cuda(), None if mla else pb.v.cuda(), pb.head_dim_v, block_size=bs)
    P = (pb.seq_lens + ps - 1) // ps
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    dec = SparseDecoder(kv, batch, Hq, kind, n_sink, n_local, max_sel, sm)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, torch.tensor(budget, dtype=torch.int32).cuda())
    out = dec.decode(q)
    torch.cuda.synchronize()
    k2, v2, ind2, idx2 = O.reblock(pb.k, pb.v, ps, bs, pb.page_indptr, pb.page_indices, pb.seq_lens)
    res = O.pipeline(pb.q, k2, v2, kind, bs, ind2, idx2, pb.seq_lens, budget, n_sink, n_local, max_sel, sm,
                     pb.head_dim_v)
    # summaries per physical block (virtual page p * r + b)
    used = np.unique(idx2)
    if dec.mean is not None:
        gm = dec.mean.cpu().numpy().astype(np.float64)
        assert np.abs(gm[used] - res["mean"][used]).max() <= 4 * 2.0 ** -24 * 8 * 2
    if dec.max is not None:
        assert np.array_equal(dec.max.float().cpu().numpy().astype(np.float64)[used], res["max"][used])
    nblk = (pb.seq_lens + bs - 1) // bs
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), res["sel"], res["cnt"],
                    res["scores"], res["kth"], res["next"], ind2, nblk, n_sink, n_local)
    ref = O.attend(pb.q, k2, v2, bs, ind2, idx2, pb.seq_lens, dec.sel_pages.cpu().numpy(),
                   dec.sel_count.cpu().numpy(), sm, pb.head_dim_v)
    assert max_abs_err(out, ref) <= OUT_ATOL
    assert r > 1


def test_blocks_append_refreshes_the_last_block():
    """The fused append with blocks below the page size refreshes only the block holding the new
    token (first_page counts blocks), bit-identical to the unfused refresh."""
    from tests._problems import random_problem, strip_last_token
    ps, bs = 64, 16
    lens = [ps * 3 + 40, ps + 17, 16, 5]
    pb = random_problem(777, lens, Hq=8, H=2, D=128, ps=ps, extra_pages=2)
    k, v, kn, vn = strip_last_token(pb, 778)
    kv = vx.PagedKV(k.cuda(), v.cuda(), 128, block_size=bs)
    P = (pb.seq_lens + ps - 1) // ps
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    rows = pb.k.shape[0] * (ps // bs)
    mean = torch.full((rows, 2, 128), -7.0, device="cuda")
    mx = torch.zeros((rows, 2, 128), dtype=torch.bfloat16, device="cuda")
    vx.kv_append_summarize(kv, batch, kn.cuda(), vn.cuda(), mean, mx, None)
    torch.cuda.synchronize()
    assert torch.equal(kv.k.cpu().view(torch.int16), pb.k.view(torch.int16))
    k2, _, ind2, idx2 = O.reblock(pb.k, pb.v, ps, bs, pb.page_indptr, pb.page_indices, pb.seq_lens)
    first = ((pb.seq_lens - 1) // bs).astype(np.int32)
    om, ox, _ = O.summarize(k2, bs, ind2, idx2, pb.seq_lens, first_page=first)
    gm = mean.cpu().numpy().astype(np.float64)
    gx = mx.float().cpu().numpy().astype(np.float64)
    for i in range(pb.batch):
        for jb in range(int(ind2[i + 1] - ind2[i])):
            vb = int(idx2[ind2[i] + jb])
            if jb == first[i]:
                assert np.abs(gm[vb] - om[vb]).max() <= 1e-5 and np.array_equal(gx[vb], ox[vb])
            else:
                assert (gm[vb] == -7.0).all()


@pytest.mark.parametrize("n_pages,tied", [(600, True), (3000, False), (512, True), (511, False), (513, True)])
def test_many_pages_in_the_threshold_buckets(n_pages, tied):
    """One-pass scores whose threshold buckets hold more than a wave of candidates (all pages
    tied; NSA's skewed softmax scores) go through an exact radix select over those pages.  At
    most 512 pages per request run the one-wave selection instead (512 and 511 here; 513 is
    the first size past it)."""
    from tests._problems import random_problem
    ps, D, Hq, H = 16, 64, 4, 2
    lens = [n_pages * ps - 5]
    pb = random_problem(990 + n_pages, lens, Hq=Hq, H=H, D=D, ps=ps)
    kind = O.MAX_DOT if tied else O.NSA
    if tied:
        pb.k[:] = pb.k[:1]                      # every physical page the same: every score ties
        pb.k[int(pb.page_indices[n_pages - 1])] = pb.k[0]
    budget, max_sel, n_sink, n_local = [200], 256, 1, 4
    dec, bud, P = _problem_on_gpu(pb, kind, budget, n_sink, n_local, max_sel, 0.125)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    torch.cuda.synchronize()
    r = O.pipeline(pb.q, pb.k, pb.v, kind, ps, pb.page_indptr, pb.page_indices, pb.seq_lens, budget, n_sink,
                   n_local, max_sel, 0.125, pb.head_dim_v)
    sel, cnt = dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy()
    check_selection(sel, cnt, r["sel"], r["cnt"], r["scores"], r["kth"], r["next"], pb.page_indptr, P, n_sink,
                    n_local, band=1e-4 if tied else 1e-7)
    if tied:
        # the last page is partial (its Max differs); the 195 free slots go to pages 1..195
        for h in range(H):
            chosen = [j for j in sel[0, h].tolist() if j not in (-1, 0) and j < n_pages - 4]
            assert chosen == list(range(1, 196))
