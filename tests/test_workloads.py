"""The seeded input generator: determinism, slice regeneration, and the planted-page recipe."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2606_06453_amd import workloads as W


def test_lowbias32_is_a_bijection_on_a_sample():
    x = torch.arange(0, 1 << 18, dtype=torch.int64) * 16411 + 7
    h = W.lowbias32(x & 0xFFFFFFFF)
    assert torch.unique(h).numel() == x.numel()
    assert int(h.min()) >= 0 and int(h.max()) < (1 << 32)


def test_counter_normals_shape_and_moments():
    x = W.counter_normals(1234, 0, 1 << 20, "cpu").double()
    assert abs(x.mean().item()) < 5e-3 and abs(x.std().item() - 1) < 5e-3
    assert x.abs().max().item() < 4.4


def test_slices_regenerate_bit_identically():
    cfg = W.SMALL["llama3_8b_layer"]
    wl = W.make(cfg)
    full = wl.k_storage()
    vfull = wl.v_storage()
    sub = [5, 0, int(wl.num_phys_pages) - 1, 17]
    assert torch.equal(wl.k_pages(sub).view(torch.int16), full[sub].view(torch.int16))
    assert torch.equal(wl.v_pages(sub).view(torch.int16), vfull[sub].view(torch.int16))
    wl2 = W.make(cfg)
    assert torch.equal(wl2.q.view(torch.int16), wl.q.view(torch.int16))
    assert np.array_equal(wl2.page_indices, wl.page_indices)


def test_planted_keys_follow_the_recipe():
    """Planted pages hold bf16(fp32(k) + fp32(qbar/2)) on every token."""
    wl = W.make(W.CONFIGS["tiny_gqa"])
    (i, h), js = next(iter(wl.planted.items()))
    p = int(wl.page_indices[wl.page_indptr[i] + js[0]])
    ps, D = wl.cfg.page_size, wl.cfg.head_dim_qk
    per_page = wl.cfg.num_kv_heads * ps * D
    ctr = torch.arange(p * per_page, (p + 1) * per_page, dtype=torch.int64)
    raw = W.counter_normals_at(wl.key_k, ctr).view(wl.cfg.num_kv_heads, ps, D)[h]
    want = (raw + torch.from_numpy(wl.qbar32()[i, h]) * 0.5).to(torch.bfloat16)
    assert torch.equal(wl.k_pages([p])[0, h].view(torch.int16), want.view(torch.int16))


def test_full_configs_have_the_stated_shapes():
    c = W.CONFIGS
    wl = W.make(c["llama3_8b_layer"])
    assert wl.seq_lens.min() >= 8192 and wl.seq_lens.max() <= 32768 and len(wl.seq_lens) == 64
    assert wl.max_sel == 128
    n_planted = [len(v) for v in wl.planted.values()]
    assert len(wl.planted) == 64 * 8 and min(n_planted) >= 10
    wl5 = W.make(c["large_gqa"])
    assert wl5.seq_lens.min() >= 4096 and wl5.seq_lens.max() <= 65536
    assert 8000 < np.median(wl5.seq_lens) < 32000
    assert np.array_equal(wl5.pages_budget, np.ceil(0.01 * wl5.pages) + 5)
    wl3 = W.make(c["long_gen_quest"])
    assert (wl3.pages == 4096).all()
    wl4 = W.make(c["mla_absorbed"])
    assert (wl4.pages == 512).all() and wl4.cfg.v_alias


def test_tiny_config_oracle_recovers_planted_pages():
    """Block top-k finds the pages whose keys lean towards the query (Sec. 3.1 motivation):
    with the full tiny workload, the oracle's top-8 contains all 4 planted pages."""
    wl = W.make(W.CONFIGS["tiny_gqa"])
    c = wl.cfg
    k = wl.k_storage()
    v = wl.v_storage()
    r = O.pipeline(wl.q, k, v, O.MEAN_DOT, c.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens,
                   wl.pages_budget, c.n_sink, c.n_local, wl.max_sel, c.sm_scale)
    sel = set(r["sel"][0, 0, : r["cnt"][0]].tolist())
    assert r["cnt"][0] == 8
    assert set(wl.planted[(0, 0)].tolist()) <= sel
    assert np.abs(r["out"]).max() < 4


@pytest.mark.parametrize("name", ["llama3_8b_layer", "long_gen_quest", "mla_absorbed", "large_gqa"])
def test_small_variants_run_through_the_oracle(name):
    wl = W.make(W.SMALL[name])
    c = wl.cfg
    k = wl.k_storage()
    v = wl.v_storage()
    r = O.pipeline(wl.q, k, v, c.kind, c.page_size, wl.page_indptr, wl.page_indices, wl.seq_lens,
                   wl.pages_budget, c.n_sink, c.n_local, wl.max_sel, c.sm_scale, c.head_dim_v)
    assert (r["cnt"] == np.minimum(wl.pages_budget, wl.pages)).all()
    assert np.abs(r["out"]).max() < 4
    if c.planted[0] == "frac":
        for (i, h), js in wl.planted.items():
            chosen = set(r["sel"][i, h, : r["cnt"][i]].tolist())
            assert set(js.tolist()) <= chosen
