"""vx_append_score_topk (the decode step's append inside the top-K launch) against the two calls
it stands for, vx_kv_append_summarize then vx_page_score_topk, on the GPU: the caches, every
summary buffer and the selection must come out bit for bit the same.  Covered: the bucketed
selection paths that carry the append (two-pass block mean, one-pass block mean and Max,
two-pass Quest), the MLA latent (its 64 x 576 and 32 x 576 blocks refreshed by workgroups of
their own in the one-pass selection launch, also with an fp8 latent), an fp8 cache, blocks below
the page size, and the cases that append first instead (n_local = 0, NSA, an approximate
selection, a 64 x 576 block on the two-pass path)."""
import pytest
import torch

from oracle import oracle as O
from paper_2606_06453_amd import vx
from tests._problems import fp8_problem, random_problem, strip_last_token

pytestmark = pytest.mark.gpu

CASES = [
    # name, ps, bs, D, Hq, H, kind, two_pass, fp8, n_local, tau
    ("mean_two_pass", 16, 0, 128, 8, 2, O.MEAN_DOT, True, None, 2, 0.0),
    ("mean_one_pass", 16, 0, 64, 4, 1, O.MEAN_DOT, False, None, 3, 0.0),
    ("max_one_pass", 32, 0, 128, 8, 2, O.MAX_DOT, False, None, 1, 0.0),
    ("quest_two_pass", 16, 0, 128, 8, 2, O.QUEST, False, None, 2, 0.0),
    ("rectified", 32, 0, 64, 8, 2, O.QUEST_RECTIFIED, False, None, 2, 0.0),
    ("mla_latent", 64, 0, 576, 16, 1, O.MEAN_DOT, True, None, 2, 0.0),   # appends first (64 x 576, two passes)
    ("mla_latent_one_pass", 64, 0, 576, 16, 1, O.MEAN_DOT, False, None, 2, 0.0),   # append workgroups
    ("mla_latent_fp8", 64, 0, 576, 16, 1, O.MEAN_DOT, False, torch.float8_e5m2, 1, 0.0),
    ("mla_latent_pages_of_32", 32, 0, 576, 16, 1, O.MEAN_DOT, False, None, 2, 0.0),
    ("pages_of_64", 64, 0, 128, 8, 2, O.MEAN_DOT, True, None, 2, 0.0),   # 64 x 128: still fused
    ("fp8_e4m3", 16, 0, 128, 8, 2, O.MEAN_DOT, True, torch.float8_e4m3fn, 2, 0.0),
    ("blocks_of_16", 32, 16, 128, 8, 2, O.QUEST, False, None, 2, 0.0),
    ("no_local_window", 16, 0, 128, 8, 2, O.MEAN_DOT, True, None, 0, 0.0),
    ("nsa_flow", 16, 0, 64, 8, 2, O.NSA, False, None, 2, 0.0),
    ("approximate", 16, 0, 128, 8, 2, O.MEAN_DOT, False, None, 2, 0.25),
]


def _state(pb, k, v, ks, vs, bs, H, D):
    """A cache (copies of k, v) and its summary buffers, summarised over the stripped cache."""
    kv = vx.PagedKV(k.clone().cuda(), None if v is None else v.clone().cuda(), pb.head_dim_v, k_scale=ks,
                    v_scale=vs, block_size=bs)
    r = pb.page_size // bs if bs else 1
    P = (pb.seq_lens + pb.page_size - 1) // pb.page_size
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).cuda(), torch.from_numpy(pb.page_indices).cuda(),
                         torch.from_numpy(pb.seq_lens).cuda(), int(P.max()))
    rows = k.shape[0] * r
    mean = torch.zeros((rows, H, D), device="cuda")
    mbf = torch.zeros((rows, H, D), dtype=torch.bfloat16, device="cuda")
    mx = torch.zeros((rows, H, D), dtype=torch.bfloat16, device="cuda")
    mn = torch.zeros((rows, H, D), dtype=torch.bfloat16, device="cuda")
    vx.page_summarize(kv, batch, None, mean, mx, mn, mean_bf16=mbf)
    return kv, batch, [mean, mbf, mx, mn]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_append_inside_selection_equals_separate_calls(case):
    name, ps, bs, D, Hq, H, kind, two_pass, fp8, n_local, tau = case
    mla = D == 576
    r = ps // bs if bs else 1
    lens = [ps * 40 + 3, ps * 9 + 1, ps * 3, 7, ps * 25 + ps // 2, ps * 14]
    pb = random_problem(2200 + ps + D + Hq + n_local, lens, Hq=Hq, H=H, D=D, ps=ps, Dv=512 if mla else None,
                        alias_v=mla, extra_pages=4)
    ks, vs = 1.0, 1.0
    if fp8 is not None:
        ks, vs = 0.021, 0.0377
        pb = fp8_problem(pb, fp8, ks, vs)
    k, v, kn, vn = strip_last_token(pb, 2201)
    budget = torch.tensor([12 * r, 5 * r, 4 * r, 1, 20 * r, 9 * r], dtype=torch.int32).cuda()
    max_sel, n_sink = 24 * r, 1 * r
    nl = n_local * r
    q = pb.q.cuda()
    opt = vx.topk_options(tolerate_ratio=tau, seed=5) if tau else None
    outs = []
    for fused in (False, True):
        kv, batch, (mean, mbf, mx, mn) = _state(pb, k, v, ks, vs, bs, H, D)
        ws = torch.zeros(vx.workspace_size(vx.STAGE_SCORE_TOPK, kv, batch, Hq, max_sel), dtype=torch.uint8,
                         device="cuda")
        sel = torch.full((pb.batch, H, max_sel), -7, dtype=torch.int32, device="cuda")
        cnt = torch.full((pb.batch,), -7, dtype=torch.int32, device="cuda")
        knc, vnc = kn.cuda(), None if vn is None else vn.cuda()
        bf = mbf if two_pass else None           # the bf16 Mean copy is maintained and read, or neither
        if fused:
            vx.append_score_topk(kv, batch, knc, vnc, mean, mx, mn, q, kind, budget, n_sink, nl, max_sel, sel, cnt,
                                 ws, mean_bf16=bf, options=opt)
        else:
            vx.kv_append_summarize(kv, batch, knc, vnc, mean, mx, mn, mean_bf16=bf)
            vx.page_score_topk(q, kv, batch, kind, mean, mx, mn, budget, n_sink, nl, max_sel, sel, cnt, ws,
                               mean_bf16=bf, options=opt)
        torch.cuda.synchronize()
        outs.append([kv.k, kv.v, mean, mbf, mx, mn, sel, cnt])
    as_bytes = lambda t: None if t is None else t.cpu().contiguous().view(torch.uint8)
    for a, b, what in zip(outs[0], outs[1], ["k", "v", "mean", "mean_bf16", "max", "min", "sel_pages", "sel_count"]):
        if a is None:
            assert b is None
            continue
        assert torch.equal(as_bytes(a), as_bytes(b)), what
    # the appended rows are the stripped token's
    assert torch.equal(as_bytes(outs[1][0]), as_bytes(pb.k))
