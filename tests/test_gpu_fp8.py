"""fp8 KV caches (Sec. 5.3; Appendix E: fp8_e4m3 / fp8_e5m2) on the GPU against the oracle.

The cache holds OCP E4M3 or E5M2 codes with one scale for K and one for V (an MLA latent: one
scale, V being its first 512 channels); every step uses the values scale * code.  Same
comparison rules as the bf16 parity tests.
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2606_06453_amd import vx, workloads as W
from paper_2606_06453_amd.decoder import SparseDecoder
from tests._compare import OUT_ATOL, GpuWorkload, check_selection, max_abs_err
from tests._problems import fp8_problem, random_problem

pytestmark = pytest.mark.gpu

NAMES = ["tiny_gqa", "llama3_8b_layer", "long_gen_quest", "mla_absorbed", "large_gqa"]
KV = ["fp8_e4m3", "fp8_e5m2"]


def _small(name, kv):
    return W.make(W.SMALL[name].with_kv_dtype(kv))


@pytest.mark.parametrize("kv", KV)
def test_fp8_generator_is_identical_on_gpu(kv):
    wl = _small("llama3_8b_layer", kv)
    g = wl.k_storage("cuda").cpu().view(torch.uint8)
    c = wl.k_storage("cpu").view(torch.uint8)
    assert torch.equal(g, c)
    assert torch.equal(wl.v_storage("cuda").cpu().view(torch.uint8), wl.v_storage("cpu").view(torch.uint8))


@pytest.mark.parametrize("kv", KV)
@pytest.mark.parametrize("name", NAMES)
def test_fp8_summaries_match_oracle(name, kv):
    wl = _small(name, kv)
    c = wl.cfg
    gw = GpuWorkload(wl)
    P, H, _, D = gw.k.shape
    mean = torch.full((P, H, D), float("nan"), device="cuda")
    mx = torch.zeros((P, H, D), dtype=torch.bfloat16, device="cuda")
    mn = torch.zeros((P, H, D), dtype=torch.bfloat16, device="cuda")
    vx.page_summarize(gw.kv, gw.batch, None, mean, mx, mn)
    torch.cuda.synchronize()
    kc = wl.k_storage("cpu")
    om, ox, on = O.summarize(kc, c.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens, k_scale=c.k_scale)
    ref = np.unique(wl.page_indices)
    kmax = float(np.abs(O.fp8_dequantize(kc.view(torch.uint8).numpy(),
                                         O.KV_FP8_E4M3 if kv == "fp8_e4m3" else O.KV_FP8_E5M2,
                                         c.k_scale)).max())
    # fp32 accumulation over <= 64 values, one rounding of the quotient
    assert np.abs(mean.cpu().numpy().astype(np.float64)[ref] - om[ref]).max() <= 4 * 2.0 ** -24 * kmax * 2
    assert np.array_equal(mx.float().cpu().numpy().astype(np.float64)[ref], ox[ref])
    assert np.array_equal(mn.float().cpu().numpy().astype(np.float64)[ref], on[ref])


@pytest.mark.parametrize("kv", KV)
@pytest.mark.parametrize("name", NAMES)
def test_fp8_end_to_end_step(name, kv):
    wl = _small(name, kv)
    c = wl.cfg
    gw = GpuWorkload(wl)
    dec = SparseDecoder(gw.kv, gw.batch, c.num_q_heads, c.kind, c.n_sink, c.n_local, wl.max_sel, c.sm_scale)
    dec.summarize()
    dec.select(gw.q, gw.budget)
    out = dec.decode(gw.q)
    torch.cuda.synchronize()
    kc, vc = wl.k_storage("cpu"), wl.v_storage("cpu")
    r = O.pipeline(wl.q, kc, vc, c.kind, c.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens,
                   wl.pages_budget, c.n_sink, c.n_local, wl.max_sel, c.sm_scale, c.head_dim_v,
                   k_scale=c.k_scale, v_scale=c.v_scale)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], wl.page_indptr, wl.pages, c.n_sink, c.n_local)
    ref = O.attend(wl.q, kc, vc, c.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens,
                   dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), c.sm_scale, c.head_dim_v,
                   k_scale=c.k_scale, v_scale=c.v_scale)
    assert max_abs_err(out, ref) <= OUT_ATOL


def _gpu_problem(pb, kind, budget, n_sink, n_local, max_sel, sm, ks, vs):
    kv = vx.PagedKV(pb.k.cuda(), pb.v.cuda(), pb.head_dim_v, k_scale=ks, v_scale=vs)
    P = (pb.seq_lens + pb.page_size - 1) // pb.page_size
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    dec = SparseDecoder(kv, batch, pb.q.shape[1], kind, n_sink, n_local, max_sel, sm)
    return dec, torch.tensor(budget, dtype=torch.int32).cuda(), P


@pytest.mark.parametrize("dtype", [torch.float8_e4m3fn, torch.float8_e5m2])
@pytest.mark.parametrize("ps,D,Hq,H", [(16, 64, 4, 1), (32, 128, 8, 1), (64, 128, 16, 2), (16, 128, 12, 2)])
@pytest.mark.parametrize("kind", [O.MEAN_DOT, O.QUEST, O.MAX_DOT])
def test_fp8_geometries_and_kinds(dtype, ps, D, Hq, H, kind):
    ks, vs = 0.021, 0.0377
    lens = [ps * 9 + 1, ps * 4, 5, ps * 13 + ps // 2, 1, ps * 2 - 1]
    pb = fp8_problem(random_problem(300 + ps + D + Hq, lens, Hq=Hq, H=H, D=D, ps=ps, extra_pages=7), dtype, ks, vs)
    budget = [5, 3, 1, 6, 2, 9]
    max_sel, n_sink, n_local = 8, 1, 2
    sm = 1.0 / math.sqrt(D)
    dec, bud, P = _gpu_problem(pb, kind, budget, n_sink, n_local, max_sel, sm, ks, vs)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    out = dec.decode(q)
    torch.cuda.synchronize()
    r = O.pipeline(pb.q, pb.k, pb.v, kind, ps, pb.page_indptr, pb.page_indices, pb.seq_lens, budget, n_sink,
                   n_local, max_sel, sm, pb.head_dim_v, k_scale=ks, v_scale=vs)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], pb.page_indptr, P, n_sink, n_local)
    ref = O.attend(pb.q, pb.k, pb.v, ps, pb.page_indptr, pb.page_indices, pb.seq_lens,
                   dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), sm, pb.head_dim_v,
                   k_scale=ks, v_scale=vs)
    assert max_abs_err(out, ref) <= OUT_ATOL


@pytest.mark.parametrize("dtype", [torch.float8_e4m3fn, torch.float8_e5m2])
def test_fp8_many_pairs_three_wave_workgroups(dtype):
    """880 pairs: the three-wave split kernel on an fp8 cache."""
    rng = np.random.default_rng(5)
    lens = [int(x) for x in rng.integers(1, 16 * 24, size=110)]
    ks, vs = 0.015, 0.015       # randn reaches ~5.7 here: codes stay below 448
    pb = fp8_problem(random_problem(950, lens, Hq=16, H=8, D=128, ps=16, extra_pages=3), dtype, ks, vs)
    budget = [int(x) for x in rng.integers(0, 14, size=110)]
    dec, bud, P = _gpu_problem(pb, O.MAX_DOT, budget, 1, 2, 12, 1 / math.sqrt(128), ks, vs)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, bud)
    out = dec.decode(q)
    torch.cuda.synchronize()
    ref = O.attend(pb.q, pb.k, pb.v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens,
                   dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), 1 / math.sqrt(128), pb.head_dim_v,
                   k_scale=ks, v_scale=vs)
    assert max_abs_err(out, ref) <= OUT_ATOL


@pytest.mark.parametrize("dtype", [torch.float8_e4m3fn, torch.float8_e5m2])
@pytest.mark.parametrize("kind", [O.MEAN_DOT, O.MEAN_DOT_CONTENT])
@pytest.mark.parametrize("B", [3, 40])
def test_fp8_mla_latent(dtype, kind, B):
    """An fp8 MLA latent (16 query heads share one 576-channel latent, V its first 512 channels
    at the latent's scale): 3 requests split over many workgroups (the merge launch) and 40 over
    few, ragged lengths and partial last pages."""
    ks = 0.0155                  # randn reaches ~5.5 here: E4M3 codes stay below 448
    rng = np.random.default_rng(B)
    lens = [int(x) for x in rng.integers(1, 64 * 12, size=B)]
    pb = fp8_problem(random_problem(600 + B + kind, lens, Hq=16, H=1, D=576, ps=64, Dv=512, alias_v=True,
                                    extra_pages=3), dtype, ks, 1.0)
    budget = [int(x) for x in rng.integers(0, 9, size=B)]
    max_sel, n_sink, n_local = 8, 1, 1
    sm = 1.0 / 24
    kv = vx.PagedKV(pb.k.cuda(), None, 512, k_scale=ks, v_scale=1.0)
    P = (pb.seq_lens + 63) // 64
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    dec = SparseDecoder(kv, batch, 16, kind, n_sink, n_local, max_sel, sm)
    q = pb.q.cuda()
    dec.summarize()
    dec.select(q, torch.tensor(budget, dtype=torch.int32).cuda())
    out = dec.decode(q)
    torch.cuda.synchronize()
    r = O.pipeline(pb.q, pb.k, None, kind, 64, pb.page_indptr, pb.page_indices, pb.seq_lens, budget, n_sink,
                   n_local, max_sel, sm, 512, k_scale=ks)
    check_selection(dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), r["sel"], r["cnt"], r["scores"],
                    r["kth"], r["next"], pb.page_indptr, P, n_sink, n_local)
    ref = O.attend(pb.q, pb.k, None, 64, pb.page_indptr, pb.page_indices, pb.seq_lens,
                   dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy(), sm, 512, k_scale=ks)
    assert max_abs_err(out, ref) <= OUT_ATOL
