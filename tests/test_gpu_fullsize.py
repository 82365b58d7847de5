"""Full-size workloads on the GPU, checked on sampled (request, KV head) units.

Each of the five workloads runs at its stated size in the launch configuration the bench
times: a full summarize (prefill), then one decode step (the fused KV append + summary refresh
of the newest page, appending each request's own newest rows; score + top-K; split-K decode +
merge).  The oracle then recomputes, for a few sampled requests and
KV heads, everything from the same seeded inputs: the summaries of every page, the scores,
the selection and the attention output.  Inputs are regenerated on the host from the
counter-based generator, one KV head at a time.  Requests and heads are independent, so a
sampled unit's oracle result is exact for that unit.  The indexer variants (NSA, positional
smoothing, the envelope flows, the rope-unaware MLA score) run the same check on the workload
whose shape the bench times them on.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2606_06453_amd import workloads as W
from paper_2606_06453_amd.decoder import SparseDecoder
from tests._compare import OUT_ATOL, GpuWorkload, check_selection, newest_rows

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _samples(wl, n_req=3, n_heads=2):
    rng = np.random.default_rng(1234)
    B, H = wl.cfg.batch, wl.cfg.num_kv_heads
    reqs = sorted({0, B - 1, int(np.argmax(wl.seq_lens)), int(np.argmin(wl.seq_lens))})[:n_req + 1]
    heads = sorted(set([0, H - 1] + rng.integers(0, H, size=n_heads).tolist()))[:n_heads]
    return reqs, heads


CASES = [(n, "bf16", None) for n in W.CONFIG_ORDER] + [(n, "fp8_e4m3", None) for n in
                                                         ("llama3_8b_layer", "long_gen_quest", "mla_absorbed",
                                                          "large_gqa")]
# the indexer variants at the shapes `bench.py --config <workload> --kind <kind>` times
CASES += [("llama3_8b_layer", "bf16", "nsa"), ("llama3_8b_layer", "bf16", "mean_dot_smooth"),
          ("long_gen_quest", "bf16", "quest_consensus"), ("long_gen_quest", "bf16", "envelope_lower"),
          ("long_gen_quest", "bf16", "quest_rectified"), ("mla_absorbed", "bf16", "mean_dot_content")]


@pytest.mark.parametrize("name,kv_dtype,kind", CASES)
def test_full_size_sampled_units(name, kv_dtype, kind):
    cfg = W.CONFIGS[name].with_kv_dtype(kv_dtype)
    if kind is not None:
        cfg = cfg.replace(kind={v: k for k, v in W.KIND_NAMES.items()}[kind])
    wl = W.make(cfg)
    c = wl.cfg
    print(f"[fullsize] {name} ({kv_dtype}, {kind or 'own flow'}): generating {wl.num_phys_pages} pages", flush=True)
    gw = GpuWorkload(wl)
    dec = SparseDecoder(gw.kv, gw.batch, c.num_q_heads, c.kind, c.n_sink, c.n_local, wl.max_sel, c.sm_scale)
    dec.summarize()
    k_before = gw.k.view(torch.uint8).sum(dtype=torch.int64)
    out = dec.step(gw.q, gw.budget, None, kv_new=newest_rows(wl, gw))
    torch.cuda.synchronize()
    assert gw.k.view(torch.uint8).sum(dtype=torch.int64) == k_before       # the same rows written back
    gsel, gcnt = dec.sel_pages.cpu().numpy(), dec.sel_count.cpu().numpy()
    gout = out.float().cpu().numpy()
    S = {"mean": dec.mean, "max": dec.max, "min": dec.min}
    del gw
    reqs, heads = _samples(wl)
    g = c.group
    exempt = 0
    for i in reqs:
        b0, b1 = int(wl.page_indptr[i]), int(wl.page_indptr[i + 1])
        phys = wl.page_indices[b0:b1]
        for h in heads:
            print(f"[fullsize] {name}: oracle for request {i} (L={wl.seq_lens[i]}), KV head {h}", flush=True)
            k = wl.head_pages(phys, h, "k")
            v = None if c.v_alias else wl.head_pages(phys, h, "v")
            q = wl.q[i:i + 1, h * g:(h + 1) * g].contiguous()
            ind = np.array([0, b1 - b0], np.int32)
            idx = np.arange(b1 - b0, dtype=np.int32)
            lens = wl.seq_lens[i:i + 1]
            r = O.pipeline(q, k, v, c.kind, c.page_size, ind, idx, lens, wl.pages_budget[i:i + 1], c.n_sink,
                           c.n_local, wl.max_sel, c.sm_scale, c.head_dim_v, k_scale=c.k_scale, v_scale=c.v_scale)
            # summaries of a sample of this request's pages (GPU rows are indexed by physical page)
            pick = np.unique(np.linspace(0, b1 - b0 - 1, 16).astype(int))
            for key, ref in (("mean", r["mean"]), ("max", r["max"]), ("min", r["min"])):
                if S[key] is None:
                    continue
                got = S[key][torch.from_numpy(phys[pick].astype(np.int64)).cuda(), h].float().cpu().numpy()
                want = ref[pick, 0]
                if key == "mean":
                    # fp32 running sum over <= page_size cache values (|x| < 4.4 for bf16, at most the
                    # 6.6 the fp8 K scale maps the largest code to), one rounded division
                    kabs = 4.4 if kv_dtype == "bf16" else 6.6
                    assert np.abs(got - want).max() <= c.page_size * 2.0 ** -23 * kabs
                else:
                    assert np.array_equal(got.astype(np.float64), want)
            sel_u = gsel[i:i + 1, h:h + 1]
            exempt += check_selection(sel_u, gcnt[i:i + 1], r["sel"], r["cnt"], r["scores"], r["kth"], r["next"],
                                      ind, wl.pages[i:i + 1], c.n_sink, c.n_local)
            ref = O.attend(q, k, v, c.page_size, ind, idx, lens, sel_u, gcnt[i:i + 1], c.sm_scale, c.head_dim_v,
                           k_scale=c.k_scale, v_scale=c.v_scale)
            err = float(np.abs(gout[i, h * g:(h + 1) * g] - ref[0]).max())
            assert err <= OUT_ATOL, (i, h, err)
    print(f"[fullsize] {name}: {len(reqs) * len(heads)} sampled units match the oracle ({exempt} near-tie exempt)",
          flush=True)
    if c.planted[0] != "none" and kind is None:      # planted for the workload's own flow
        for i in reqs:
            for h in heads:
                chosen = set(gsel[i, h, : gcnt[i]].tolist())
                assert set(wl.planted[(i, h)].tolist()) <= chosen, (i, h)
