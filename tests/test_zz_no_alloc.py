"""The allocation-free decode entry point (vx_sparse_paged_decode_noalloc) against the
workspace entry point (vx_sparse_paged_decode) and the oracle, through the C ABI: two calls in
a row on the library's static scratch, the second with a smaller batch."""
import math

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2606_06453_amd import vx
from tests._compare import OUT_ATOL, max_abs_err
from tests._problems import random_problem

pytestmark = pytest.mark.gpu


def _case(seed, lens, Hq, H, D, ps, cnt, alias_v=False):
    pb = random_problem(seed, lens, Hq=Hq, H=H, D=D, ps=ps, Dv=512 if alias_v else None, alias_v=alias_v,
                        extra_pages=3)
    rng = np.random.default_rng(seed)
    P = (np.asarray(lens) + ps - 1) // ps
    max_sel = int(max(cnt))
    sel = np.full((len(lens), H, max_sel), -1, np.int32)
    for i in range(len(lens)):
        for h in range(H):
            sel[i, h, : cnt[i]] = np.sort(rng.choice(int(P[i]), size=int(cnt[i]), replace=False))
    return pb, P, sel, np.asarray(cnt, np.int32), max_sel


def _run_both(pb, P, sel, cnt, max_sel):
    dev = "cuda"
    kv = vx.PagedKV(pb.k.to(dev), None if pb.v is None else pb.v.to(dev), pb.head_dim_v)
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).to(dev), torch.from_numpy(pb.page_indices).to(dev),
                         torch.from_numpy(pb.seq_lens).to(dev), int(P.max()))
    q = pb.q.to(dev)
    Hq = pb.q.shape[1]
    sm = 1.0 / math.sqrt(pb.k.shape[-1])
    sel_d, cnt_d = torch.from_numpy(sel).to(dev), torch.from_numpy(cnt).to(dev)
    ws = torch.zeros(vx.workspace_size(vx.STAGE_DECODE, kv, batch, Hq, max_sel), dtype=torch.uint8, device=dev)
    out_ws = torch.full((pb.batch, Hq, pb.head_dim_v), float("nan"), dtype=torch.bfloat16, device=dev)
    out_na = torch.full_like(out_ws, float("nan"))
    vx.sparse_paged_decode(q, kv, batch, sel_d, cnt_d, max_sel, sm, out_ws, ws)
    vx.sparse_paged_decode_noalloc(q, kv, batch, sel_d, cnt_d, max_sel, sm, out_na)
    torch.cuda.synchronize()
    ref = O.attend(pb.q, pb.k, pb.v, pb.page_size, pb.page_indptr, pb.page_indices, pb.seq_lens, sel, cnt, sm,
                   pb.head_dim_v)
    return out_ws, out_na, ref


@pytest.mark.parametrize("geom", ["gqa", "mla"])
def test_noalloc_decode_matches_the_workspace_entry_point(geom):
    print(f"[no_alloc] {geom}", flush=True)
    if geom == "gqa":
        # 101 pairs with one long pair split over several workgroups (counters and partials in
        # the scratch), then a smaller batch
        big = _case(5, [16 * 70 + 3] + [16 * 4 + 1] * 100, 4, 1, 128, 16, [64] + [2] * 100)
        small = _case(6, [16 * 40 + 7, 16 * 3, 50], 4, 1, 128, 16, [33, 3, 4])
    else:
        big = _case(7, [64 * 40] * 6, 16, 1, 576, 64, [32] * 6, alias_v=True)
        small = _case(8, [64 * 9 + 5, 64 * 20], 16, 1, 576, 64, [8, 5], alias_v=True)
    for name, c in (("first", big), ("second, smaller", small)):
        out_ws, out_na, ref = _run_both(*c)
        assert torch.equal(out_na.view(torch.int16), out_ws.view(torch.int16)), name
        assert max_abs_err(out_na, ref) <= OUT_ATOL, name


def test_noalloc_rejects_a_batch_beyond_its_scratch():
    # 255 MLA requests run two splits each: 510 partial rows of 16 x 512 fp32, above 12 MiB
    pb, P, sel, cnt, max_sel = _case(9, [64 * 3] * 255, 16, 1, 576, 64, [2] * 255, alias_v=True)
    dev = "cuda"
    kv = vx.PagedKV(pb.k.to(dev), None, pb.head_dim_v)
    batch = vx.BatchSpec(torch.from_numpy(pb.page_indptr).to(dev), torch.from_numpy(pb.page_indices).to(dev),
                         torch.from_numpy(pb.seq_lens).to(dev), int(P.max()))
    need = vx.workspace_size(vx.STAGE_DECODE, kv, batch, 16, max_sel)
    assert need > 12 << 20
    out = torch.empty((pb.batch, 16, 512), dtype=torch.bfloat16, device=dev)
    with pytest.raises(vx.VxError) as e:
        vx.sparse_paged_decode_noalloc(pb.q.to(dev), kv, batch, torch.from_numpy(sel).to(dev),
                                       torch.from_numpy(cnt).to(dev), max_sel, 0.04, out)
    assert e.value.status == 3 and "static buffer" in str(e.value)
