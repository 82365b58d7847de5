"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU).

Each test checks the oracle against something other than itself: a hand-worked example, a
library routine, a different route to the same quantity, an invariant, or brute force.
"""
import itertools
import math
import os

import numpy as np
import pytest
import torch

from oracle import oracle as O
from tests._problems import fp8_problem, random_problem, request_kv, strip_last_token, valid_keys

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.txt")


def _golden():
    sec, out = None, {}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if line.startswith("["):
            sec = line.strip("[]")
            out[sec] = {}
            continue
        key, *vals = line.split()
        out[sec][key] = [float(v) for v in vals]
    return out


def _bf16(vals, shape):
    return torch.tensor(vals, dtype=torch.float64).reshape(shape).to(torch.bfloat16)


# --------------------------------------------------------------------------------------
# hand-worked examples (tests/golden/hand_examples.txt)
# --------------------------------------------------------------------------------------
def test_golden_block_topk():
    """Sec. 3.1 Eqs. 1-4 on a hand-worked example with a partial last page and a tie."""
    G = _golden()["block_topk"]
    ps, L = int(G["page_size"][0]), int(G["seq_len"][0])
    # the unused slot of the partial last page holds junk that must never be read
    k = _bf16(G["keys"] + [100, -100], (3, 1, ps, 2))
    v = _bf16(G["values"] + [50, 50], (3, 1, ps, 2))
    q = _bf16(G["q"], (1, 2, 2))
    ind, idx, lens = [0, 3], [0, 1, 2], [L]
    mean, _, _ = O.summarize(k, ps, ind, idx, lens)
    assert np.array_equal(mean.reshape(-1), np.array(G["mean"]))
    sc = O.score(O.MEAN_DOT, q, 1, ps, ind, idx, lens, mean)
    assert np.array_equal(sc[:, 0], np.array(G["scores"]))
    sel, cnt, kth, nxt = O.select(sc, 1, ps, ind, lens, [1], 0, 0, 1)
    assert cnt[0] == 1 and sel[0, 0, 0] == int(G["top1"][0])
    out = O.attend(q, k, v, ps, ind, idx, lens, sel, cnt, 1.0)
    np.testing.assert_allclose(out[0, 0], G["o0"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(out[0, 1], G["o1"], rtol=0, atol=1e-15)


def test_golden_quest():
    """Sec. 3.2 Quest on a hand-worked example (sign handling of q against Max/Min)."""
    G = _golden()["quest"]
    ps, L = int(G["page_size"][0]), int(G["seq_len"][0])
    k = _bf16(G["keys"], (2, 1, ps, 2))
    q = _bf16(G["q"], (1, 2, 2))
    ind, idx, lens = [0, 2], [0, 1], [L]
    _, mx, mn = O.summarize(k, ps, ind, idx, lens)
    assert np.array_equal(mx.reshape(-1), np.array(G["max"]))
    assert np.array_equal(mn.reshape(-1), np.array(G["min"]))
    sc = O.score(O.QUEST, q, 1, ps, ind, idx, lens, mx, mn)
    assert np.array_equal(sc[:, 0], np.array(G["scores"]))


# --------------------------------------------------------------------------------------
# summaries: closed form against numpy's reductions
# --------------------------------------------------------------------------------------
@pytest.mark.parametrize("ps", [16, 32])
def test_summaries_match_numpy(ps):
    pb = random_problem(1, [5 * ps + 3, 2 * ps, 1, ps - 1], Hq=8, H=2, D=64, ps=ps, extra_pages=3)
    mean, mx, mn = O.summarize(pb.k, ps, pb.page_indptr, pb.page_indices, pb.seq_lens)
    for i in range(pb.batch):
        P = int(pb.page_indptr[i + 1] - pb.page_indptr[i])
        for j in range(P):
            p = int(pb.page_indices[pb.page_indptr[i] + j])
            for h in range(pb.num_kv_heads):
                x = valid_keys(pb, i, h, j).numpy()
                np.testing.assert_allclose(mean[p, h], np.mean(x, axis=0), rtol=1e-15, atol=1e-15)
                assert np.array_equal(mx[p, h], np.max(x, axis=0))
                assert np.array_equal(mn[p, h], np.min(x, axis=0))
    used = set(pb.page_indices.tolist())
    for p in range(pb.k.shape[0]):
        if p not in used:
            assert np.isnan(mean[p]).all()


def test_summaries_first_page_only_touches_later_pages():
    pb = random_problem(2, [70, 33], Hq=4, H=1, D=64, ps=16)
    first = [3, 1]
    mean, mx, mn = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, first_page=first)
    full, _, _ = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    for i in range(2):
        P = int(pb.page_indptr[i + 1] - pb.page_indptr[i])
        for j in range(P):
            p = int(pb.page_indices[pb.page_indptr[i] + j])
            if j >= first[i]:
                assert np.array_equal(mean[p], full[p])
            else:
                assert np.isnan(mean[p]).all()


@pytest.mark.parametrize("alias", [False, True])
def test_append_restores_the_cache_and_its_summaries(alias):
    """Removing each request's newest token and appending it again gives back the cache bit for
    bit; the refreshed summaries of the receiving pages equal numpy's mean / max / min of their
    valid tokens, including a token that opens a new page (one valid token)."""
    lens = [16 * 5 + 3, 16 * 2 + 1, 16, 7]     # request 1's token opens page 2; request 2 fills page 0
    pb = random_problem(71, lens, Hq=4, H=2, D=64, ps=16, Dv=48 if alias else None, alias_v=alias, extra_pages=2)
    k, v, kn, vn = strip_last_token(pb, 72)
    assert not torch.equal(k, pb.k)
    k2, v2, (mean, mx, mn), first = O.kv_append(k, v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, kn, vn,
                                                head_dim_v=pb.head_dim_v)
    assert torch.equal(k2, pb.k)
    assert (v2 is None) == alias and (alias or torch.equal(v2, pb.v))
    assert list(first) == [5, 2, 0, 0]
    for i in range(pb.batch):
        j = int(first[i])
        p = int(pb.page_indices[pb.page_indptr[i] + j])
        for h in range(2):
            kt = valid_keys(pb, i, h, j).numpy()
            assert np.allclose(mean[p, h], kt.mean(0), rtol=0, atol=1e-15)
            assert np.array_equal(mx[p, h], kt.max(0)) and np.array_equal(mn[p, h], kt.min(0))


def test_append_writes_only_the_new_slots():
    """Every other element of the caches is left as it was (fp8 codes are copied as codes)."""
    pb = random_problem(73, [16 * 3 + 9, 40], Hq=2, H=2, D=64, ps=16, extra_pages=3)
    f8 = fp8_problem(pb, torch.float8_e4m3fn, 0.02, 0.03)
    kn = torch.randn(2, 2, 64).to(torch.float8_e4m3fn)
    vn = torch.randn(2, 2, 64).to(torch.float8_e4m3fn)
    k2, v2, _, _ = O.kv_append(f8.k, f8.v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, kn, vn, k_scale=0.02)
    changed_k = (k2.view(torch.uint8) != f8.k.view(torch.uint8)).nonzero().tolist()
    changed_v = (v2.view(torch.uint8) != f8.v.view(torch.uint8)).nonzero().tolist()
    slots = {(int(pb.page_indices[pb.page_indptr[i] + (int(pb.seq_lens[i]) - 1) // 16]), (int(pb.seq_lens[i]) - 1) % 16)
             for i in range(2)}
    assert {(a, c) for a, _, c, _ in changed_k} <= slots and {(a, c) for a, _, c, _ in changed_v} <= slots
    for i in range(2):
        p, t = int(pb.page_indices[pb.page_indptr[i] + (int(pb.seq_lens[i]) - 1) // 16]), (int(pb.seq_lens[i]) - 1) % 16
        assert torch.equal(k2[p, :, t].view(torch.uint8), kn[i].view(torch.uint8))
        assert torch.equal(v2[p, :, t].view(torch.uint8), vn[i].view(torch.uint8))


@pytest.mark.parametrize("ps,bs", [(32, 16), (64, 16), (64, 32)])
def test_reblocked_summaries_are_per_block(ps, bs):
    """Blocks below the page size: the summary of block b of logical page j is numpy's mean / max /
    min over that block's valid tokens in the original page layout."""
    lens = [ps * 3 + bs + 3, ps + 1, bs - 5, ps * 2]
    pb = random_problem(75 + ps + bs, lens, Hq=4, H=2, D=64, ps=ps, extra_pages=2)
    k2, _, ind2, idx2 = O.reblock(pb.k, pb.v, ps, bs, pb.page_indptr, pb.page_indices, pb.seq_lens)
    mean, mx, mn = O.summarize(k2, bs, ind2, idx2, pb.seq_lens)
    r = ps // bs
    for i in range(pb.batch):
        L = int(pb.seq_lens[i])
        assert ind2[i + 1] - ind2[i] == -(-L // bs)
        for jb in range(-(-L // bs)):
            p = int(pb.page_indices[pb.page_indptr[i] + jb // r])
            t0 = (jb % r) * bs
            n = min(bs, L - jb * bs)
            kt = pb.k[p, :, t0:t0 + n].to(torch.float64).numpy()          # [H][n][D]
            v = int(idx2[ind2[i] + jb])
            assert v == p * r + jb % r
            assert np.allclose(mean[v], kt.mean(1), rtol=0, atol=1e-15)
            assert np.array_equal(mx[v], kt.max(1)) and np.array_equal(mn[v], kt.min(1))


def test_reblocking_keeps_every_valid_token():
    """Attending every block equals attending every page, and both equal torch's SDPA; with
    block_size = page_size reblocking is the identity."""
    ps, bs = 32, 16
    lens = [ps * 4 + 7, 17, ps]
    pb = random_problem(77, lens, Hq=4, H=2, D=64, ps=ps, extra_pages=1)
    k2, v2, ind2, idx2 = O.reblock(pb.k, pb.v, ps, bs, pb.page_indptr, pb.page_indices, pb.seq_lens)
    sel_p, cnt_p = _all_pages(pb, 8)
    nb = (pb.seq_lens + bs - 1) // bs
    sel_b = np.full((pb.batch, 2, 16), -1, np.int32)
    for i in range(pb.batch):
        sel_b[i, :, :nb[i]] = np.arange(nb[i])
    o_pages = O.attend(pb.q, pb.k, pb.v, ps, pb.page_indptr, pb.page_indices, pb.seq_lens, sel_p, cnt_p, 0.125)
    o_blocks = O.attend(pb.q, k2, v2, bs, ind2, idx2, pb.seq_lens, sel_b, nb.astype(np.int32), 0.125)
    assert np.allclose(o_blocks, o_pages, rtol=0, atol=1e-13)
    for i in range(pb.batch):
        for h in range(2):
            K, V = request_kv(pb, i, h)
            q = pb.q[i, 2 * h:2 * h + 2].to(torch.float64)
            ref = torch.nn.functional.scaled_dot_product_attention(q[None, :, None], K[None, None].expand(1, 2, -1, -1),
                                                                 V[None, None].expand(1, 2, -1, -1), scale=0.125)
            assert np.allclose(o_blocks[i, 2 * h:2 * h + 2], ref[0, :, 0].numpy(), rtol=0, atol=1e-12)
    same = O.reblock(pb.k, pb.v, ps, ps, pb.page_indptr, pb.page_indices, pb.seq_lens)
    assert torch.equal(same[0], pb.k) and torch.equal(same[1], pb.v)
    assert np.array_equal(same[2], pb.page_indptr) and np.array_equal(same[3], pb.page_indices)


# --------------------------------------------------------------------------------------
# scores
# --------------------------------------------------------------------------------------
def test_mean_score_equals_tokenwise_route():
    """Eq. 2 is linear in the keys: mean_r q_r . mean_t k_t == mean over (r, t) of q_r . k_t."""
    pb = random_problem(3, [16 * 9 + 5, 16 * 3, 7], Hq=12, H=3, D=64, ps=16)
    g = 4
    mean, _, _ = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    sc = O.score(O.MEAN_DOT, pb.q, 3, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, mean)
    for i in range(pb.batch):
        P = int(pb.page_indptr[i + 1] - pb.page_indptr[i])
        for h in range(3):
            qg = pb.q[i, h * g:(h + 1) * g].to(torch.float64)
            for j in range(P):
                kt = valid_keys(pb, i, h, j)
                ref = (qg @ kt.T).mean().item()          # every (head, token) pair, then the mean
                assert abs(sc[pb.page_indptr[i] + j, h] - ref) <= 1e-12 * (1 + abs(ref))


def test_max_dot_score_equals_group_mean_query():
    """Max-summary scoring: mean over heads of q_r . Max equals (mean of q_r) . Max."""
    pb = random_problem(4, [16 * 6 + 1, 40], Hq=6, H=1, D=64, ps=16)
    _, mx, _ = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    sc = O.score(O.MAX_DOT, pb.q, 1, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, mx)
    for i in range(pb.batch):
        qbar = pb.q[i].to(torch.float64).mean(0)
        P = int(pb.page_indptr[i + 1] - pb.page_indptr[i])
        for j in range(P):
            kmax = valid_keys(pb, i, 0, j).max(0).values
            ref = float(qbar @ kmax)
            assert abs(sc[pb.page_indptr[i] + j, 0] - ref) <= 1e-12 * (1 + abs(ref))


def test_quest_is_an_upper_bound_and_tight_on_single_tokens():
    """Quest bounds every token's dot product from above; with one valid token it is exact."""
    lens = [16 * 5 + 1, 33]   # request 0 ends in a one-token page
    pb = random_problem(5, lens, Hq=8, H=2, D=64, ps=16)
    _, mx, mn = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    sc = O.score(O.QUEST, pb.q, 2, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, mx, mn)
    g = 4
    for i in range(pb.batch):
        P = int(pb.page_indptr[i + 1] - pb.page_indptr[i])
        for h in range(2):
            qg = pb.q[i, h * g:(h + 1) * g].to(torch.float64)
            for j in range(P):
                kt = valid_keys(pb, i, h, j)
                best = float((qg @ kt.T).max())
                s = sc[pb.page_indptr[i] + j, h]
                assert s >= best - 1e-12
                if kt.shape[0] == 1:
                    assert abs(s - best) <= 1e-12 * (1 + abs(best))


def _envelope_case(seed, nonneg=False):
    lens = [16 * 5 + 1, 33, 16 * 2]   # request 0 ends in a one-token page
    pb = random_problem(seed, lens, Hq=8, H=2, D=64, ps=16)
    if nonneg:
        pb.q = pb.q.abs()
        pb.k = pb.k.abs()
    _, mx, mn = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    return pb, mx, mn


def _token_dots(pb, i, h, j, g=4):
    """[g][n] fp64 dot products of the group's query heads with the page's valid keys."""
    qg = pb.q[i, h * g:(h + 1) * g].to(torch.float64)
    return (qg @ valid_keys(pb, i, h, j).T).numpy()


def _pages(pb):
    for i in range(pb.batch):
        for j in range(int(pb.page_indptr[i + 1] - pb.page_indptr[i])):
            yield i, j


def test_head_consensus_quest_bounds_and_special_cases():
    """Appendix G head-consensus Quest: each head's envelope sum bounds that head's token dots
    from above, so the minimum over heads is >= min_h max_t q_h.k_t; with one token it is exactly
    min_h q_h.k; it never exceeds Quest; with one query head per KV head it is Quest."""
    pb, mx, mn = _envelope_case(51)
    args = (2, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, mx, mn)
    con = O.score(O.QUEST_CONSENSUS, pb.q, *args)
    qst = O.score(O.QUEST, pb.q, *args)
    assert (con <= qst + 1e-12).all()
    for i, j in _pages(pb):
        for h in range(2):
            d = _token_dots(pb, i, h, j)
            s = con[pb.page_indptr[i] + j, h]
            assert s >= d.max(axis=1).min() - 1e-12
            if d.shape[1] == 1:
                assert abs(s - d.min()) <= 1e-12 * (1 + abs(s))
    q1 = pb.q[:, ::4].contiguous()                      # g = 1: one head per KV head
    a1 = (2, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, mx, mn)
    assert np.array_equal(O.score(O.QUEST_CONSENSUS, q1, *a1), O.score(O.QUEST, q1, *a1))


def test_pessimistic_envelope_is_a_lower_bound():
    """Appendix G pessimistic envelope: each head's sum of min(q Max, q Min) bounds every token's
    dot product from below, so the score is <= max_h min_t q_h.k_t, with equality on one token."""
    pb, mx, mn = _envelope_case(53)
    low = O.score(O.ENVELOPE_LOWER, pb.q, 2, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, mx, mn)
    for i, j in _pages(pb):
        for h in range(2):
            d = _token_dots(pb, i, h, j)
            s = low[pb.page_indptr[i] + j, h]
            assert s <= d.min(axis=1).max() + 1e-12
            if d.shape[1] == 1:
                assert abs(s - d.max()) <= 1e-12 * (1 + abs(s))


def test_rectified_quest_special_cases():
    """Appendix G rectified Quest: with non-negative queries and keys it equals Quest; on a
    one-token page it is max_h sum_c ReLU(q_hc k_c) computed from the key itself; it never
    reads the Min summary."""
    pb, mx, mn = _envelope_case(55, nonneg=True)
    args = (2, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    rec = O.score(O.QUEST_RECTIFIED, pb.q, *args, mx)
    assert np.array_equal(rec, O.score(O.QUEST, pb.q, *args, mx, mn))
    pb, mx, mn = _envelope_case(57)
    args = (2, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    rec = O.score(O.QUEST_RECTIFIED, pb.q, *args, mx)
    for i, j in _pages(pb):
        for h in range(2):
            kt = valid_keys(pb, i, h, j)
            if kt.shape[0] == 1:
                qg = pb.q[i, h * 4:(h + 1) * 4].to(torch.float64)
                ref = torch.clamp(qg * kt, min=0).sum(dim=1).max().item()
                assert abs(rec[pb.page_indptr[i] + j, h] - ref) <= 1e-12 * (1 + abs(ref))
            assert rec[pb.page_indptr[i] + j, h] >= 0.0          # a sum of ReLUs


def test_content_score_equals_tokenwise_route_on_content_channels():
    """Rope-unaware MLA score (Sec. 6.2 ablation): Eq. 2 over the first Dc channels equals the
    mean over (head, token) pairs of q_r[:Dc] . k_t[:Dc]; the rope channels do not enter it."""
    pb = random_problem(61, [16 * 4 + 3, 16 * 2], Hq=4, H=1, D=72, ps=16, Dv=64, alias_v=True)
    mean, _, _ = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    args = (1, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, mean)
    sc = O.score(O.MEAN_DOT_CONTENT, pb.q, *args, content_dims=64)
    full = O.score(O.MEAN_DOT, pb.q, *args)
    for i, j in _pages(pb):
        qg = pb.q[i, :, :64].to(torch.float64)
        kt = valid_keys(pb, i, 0, j)[:, :64]
        ref = (qg @ kt.T).mean().item()
        assert abs(sc[pb.page_indptr[i] + j, 0] - ref) <= 1e-12 * (1 + abs(ref))
    assert not np.allclose(sc, full)                     # the rope channels did matter
    q0 = pb.q.clone()
    q0[:, :, 64:] = 0                                    # a query with no rope part: the full score
    assert np.allclose(O.score(O.MEAN_DOT_CONTENT, q0, *args, content_dims=64), O.score(O.MEAN_DOT, q0, *args),
                       rtol=0, atol=1e-13)


def _conv_torch(x, taps):
    """[rows][P] fp64 rows convolved along P by torch's conv1d with zero padding 1."""
    w = torch.tensor(taps, dtype=torch.float64).view(1, 1, 3)
    return torch.nn.functional.conv1d(torch.as_tensor(x, dtype=torch.float64).unsqueeze(1), w, padding=1).squeeze(1)


def test_head_logits_match_torch():
    """NSA logits (each query head against the Mean summaries): q_r . Mean_j with the GQA head
    mapping, rounded to fp32."""
    pb = random_problem(63, [16 * 5 + 7, 16 * 3], Hq=6, H=2, D=64, ps=16)
    mean, _, _ = O.summarize(pb.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens)
    z = O.head_logits(pb.q, 2, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, mean)
    for i, j in _pages(pb):
        for r in range(6):
            c = valid_keys(pb, i, r // 3, j).mean(0)
            ref = float(pb.q[i, r].to(torch.float64) @ c)
            got = z[pb.page_indptr[i] + j, r]
            assert got == float(np.float32(got))                 # stored at fp32 precision
            assert abs(got - ref) <= 2.0 ** -23 * abs(ref) + 1e-300


@pytest.mark.parametrize("taps", [(0.25, 0.5, 0.25), (0.1, 0.3, 0.6)])
def test_nsa_scores_match_torch_softmax_conv_sum(taps):
    """NSA block top-k flow: softmax over pages per query head, conv1d along pages (zero padding,
    asymmetric taps catch a reversed kernel), sum over the group's heads; against torch."""
    rng = np.random.default_rng(65)
    lens = np.array([16 * 9 + 2, 16, 40], np.int32)
    P = (lens + 15) // 16
    ind = np.concatenate([[0], np.cumsum(P)]).astype(np.int32)
    Hq, H = 6, 2
    z = rng.normal(0, 3, size=(int(ind[-1]), Hq)).astype(np.float32).astype(np.float64)
    sc = O.nsa_scores(z, H, 16, ind, lens, taps=taps)
    for i in range(len(lens)):
        zi = torch.tensor(z[ind[i]:ind[i + 1]].T)                   # [Hq][P_i]
        p = torch.softmax(zi, dim=1)
        y = _conv_torch(p, taps)
        ref = y.view(H, Hq // H, -1).sum(1).T.numpy()                # [P_i][H]
        assert np.allclose(sc[ind[i]:ind[i + 1]], ref, rtol=1e-13, atol=1e-16)


def test_nsa_scores_invariants():
    """Softmax rows sum to one: with the identity kernel the scores of a request sum to g; with
    [1/4, 1/2, 1/4] and zero padding the two end pages each lose a quarter of their mass.  Adding
    a constant to a head's logits changes nothing; a one-page request scores w1 * g."""
    rng = np.random.default_rng(67)
    lens = np.array([16 * 12, 5, 16 * 3 + 1], np.int32)
    P = (lens + 15) // 16
    ind = np.concatenate([[0], np.cumsum(P)]).astype(np.int32)
    Hq, H, g = 8, 2, 4
    z = rng.normal(0, 2, size=(int(ind[-1]), Hq))
    ident = O.nsa_scores(z, H, 16, ind, lens, taps=(0.0, 1.0, 0.0))
    tri = O.nsa_scores(z, H, 16, ind, lens)
    shifted = O.nsa_scores(z + rng.normal(0, 5, size=(1, Hq)), H, 16, ind, lens)
    assert np.allclose(shifted, tri, rtol=1e-12, atol=1e-15)
    for i in range(len(lens)):
        rows = slice(ind[i], ind[i + 1])
        assert np.allclose(ident[rows].sum(0), g, rtol=1e-13)
        lost = 0.25 * (ident[ind[i]] + ident[ind[i + 1] - 1]) if P[i] > 1 else 0.5 * ident[ind[i]]
        assert np.allclose(tri[rows].sum(0), g - lost, rtol=1e-13)
    assert np.allclose(tri[ind[1]], 0.5 * g, rtol=1e-15)              # request 1 has one page


def test_smooth_scores_match_torch_conv1d():
    """Positional smoothing (Appendix G): a 3-tap conv1d along each request's pages."""
    rng = np.random.default_rng(69)
    lens = np.array([16 * 7 + 3, 16, 33], np.int32)
    P = (lens + 15) // 16
    ind = np.concatenate([[0], np.cumsum(P)]).astype(np.int32)
    x = rng.normal(size=(int(ind[-1]), 3))
    for taps in [(0.25, 0.5, 0.25), (0.1, 0.3, 0.6)]:
        y = O.smooth_scores(x, 16, ind, lens, taps=taps)
        for i in range(len(lens)):
            ref = _conv_torch(x[ind[i]:ind[i + 1]].T, taps).T.numpy()
            assert np.allclose(y[ind[i]:ind[i + 1]], ref, rtol=1e-14, atol=1e-16)


# --------------------------------------------------------------------------------------
# selection: brute force over subsets
# --------------------------------------------------------------------------------------
def _brute_force(scores, P, Ktot, n_sink, n_local):
    forced = set(range(min(n_sink, P))) | set(range(max(0, P - n_local), P))
    if Ktot >= P:
        return list(range(P))
    cands = [j for j in range(P) if j not in forced]
    kfree = max(0, Ktot - len(forced))
    best, best_key = None, None
    for sub in itertools.combinations(cands, kfree):
        key = (sum(scores[j] for j in sub), [-j for j in sub])   # max sum, then lowest indices
        if best_key is None or key > best_key:
            best, best_key = sub, key
    return sorted(forced | set(best))


@pytest.mark.parametrize("seed", range(6))
def test_select_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    ps = 4
    lens = rng.integers(1, 11 * ps, size=5)
    P = (lens + ps - 1) // ps
    ind = np.zeros(6, np.int32)
    ind[1:] = np.cumsum(P)
    H = 2
    # integer scores give plenty of exact ties
    sc = rng.integers(-3, 4, size=(int(ind[-1]), H)).astype(np.float64)
    budget = rng.integers(0, 9, size=5)
    for n_sink, n_local in [(0, 0), (1, 2), (2, 1)]:
        sel, cnt, kth, nxt = O.select(sc, H, ps, ind, lens, budget, n_sink, n_local, 12)
        for i in range(5):
            for h in range(H):
                ref = _brute_force(sc[ind[i]:ind[i + 1], h], int(P[i]), int(budget[i]), n_sink, n_local)
                got = [int(x) for x in sel[i, h] if x >= 0]
                assert got == ref, (i, h, n_sink, n_local)
                assert cnt[i] == len(ref)
                assert all(x == -1 for x in sel[i, h, cnt[i]:])


def test_select_gap_values():
    """s_kth / s_next are the K_free-th and (K_free+1)-th best candidate scores."""
    sc = np.array([[5.0], [1.0], [4.0], [3.0], [2.0], [0.0]])
    sel, cnt, kth, nxt = O.select(sc, 1, 1, [0, 6], [6], [3], 1, 0, 4)
    assert sel[0, 0, :3].tolist() == [0, 2, 3] and cnt[0] == 3
    assert kth[0, 0] == 3.0 and nxt[0, 0] == 2.0
    sel, cnt, kth, nxt = O.select(sc, 1, 1, [0, 6], [6], [6], 1, 0, 6)
    assert cnt[0] == 6 and kth[0, 0] == math.inf and nxt[0, 0] == -math.inf


# --------------------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------------------
def _all_pages(pb, max_sel):
    B, H = pb.batch, pb.num_kv_heads
    sel = np.full((B, H, max_sel), -1, np.int32)
    cnt = np.zeros(B, np.int32)
    for i in range(B):
        P = int(pb.page_indptr[i + 1] - pb.page_indptr[i])
        sel[i, :, :P] = np.arange(P)
        cnt[i] = P
    return sel, cnt


@pytest.mark.parametrize("Hq,H,D,Dv,alias", [(8, 2, 64, 64, False), (6, 1, 128, 128, False),
                                             (16, 1, 576, 512, True)])
def test_dense_budget_equals_sdpa(Hq, H, D, Dv, alias):
    """With every page selected, Eq. 4 is ordinary softmax attention: compare with torch's
    fp64 scaled_dot_product_attention, query head r using KV head r // g."""
    pb = random_problem(6, [16 * 4 + 9, 16 * 2, 5], Hq=Hq, H=H, D=D, ps=16, Dv=Dv, alias_v=alias)
    scale = 1.0 / math.sqrt(D)
    sel, cnt = _all_pages(pb, 8)
    out = O.attend(pb.q, pb.k, pb.v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, sel, cnt, scale, Dv)
    g = Hq // H
    for i in range(pb.batch):
        Ks, Vs = zip(*[request_kv(pb, i, h) for h in range(H)])
        K = torch.stack(Ks).repeat_interleave(g, dim=0)      # [Hq][n][D]
        V = torch.stack(Vs).repeat_interleave(g, dim=0)
        qi = pb.q[i].to(torch.float64)[:, None, :]            # [Hq][1][D]
        ref = torch.nn.functional.scaled_dot_product_attention(qi, K, V, scale=scale)[:, 0]
        np.testing.assert_allclose(out[i], ref.numpy(), rtol=0, atol=1e-12)


def test_single_token_gives_its_value():
    pb = random_problem(7, [1, 17], Hq=4, H=1, D=64, ps=16)
    sel = np.full((2, 1, 2), -1, np.int32)
    sel[0, 0, 0] = 0
    sel[1, 0, 0] = 1          # the one-token last page of request 1
    cnt = np.array([1, 1], np.int32)
    out = O.attend(pb.q, pb.k, pb.v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, sel, cnt, 0.125)
    for i, j in [(0, 0), (1, 1)]:
        p = int(pb.page_indices[pb.page_indptr[i] + j])
        vt = pb.v[p, 0, 0].to(torch.float64).numpy()
        for r in range(4):
            np.testing.assert_allclose(out[i, r], vt, rtol=0, atol=1e-15)


def test_empty_selection_gives_zero():
    pb = random_problem(8, [40], Hq=4, H=1, D=64, ps=16)
    sc = np.zeros((3, 1))
    sel, cnt, _, _ = O.select(sc, 1, 16, pb.page_indptr, pb.seq_lens, [0], 0, 0, 4)
    assert cnt[0] == 0
    out = O.attend(pb.q, pb.k, pb.v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, sel, cnt, 0.125)
    assert (out == 0).all()


# --------------------------------------------------------------------------------------
# paged layout (Appendix A): physical placement and sharing do not change any result
# --------------------------------------------------------------------------------------
def _run(pb, kind=O.MEAN_DOT, budget=4, n_sink=1, n_local=1, max_sel=6):
    return O.pipeline(pb.q, pb.k, pb.v, kind, pb.page_size, pb.page_indptr, pb.page_indices, pb.seq_lens,
                      [budget] * pb.batch, n_sink, n_local, max_sel, 0.125, pb.head_dim_v)


@pytest.mark.parametrize("kind", [O.MEAN_DOT, O.QUEST, O.MAX_DOT])
def test_physical_permutation_invariance(kind):
    pb = random_problem(9, [16 * 11 + 3, 16 * 7], Hq=8, H=2, D=64, ps=16, extra_pages=4)
    a = _run(pb, kind)
    perm = np.random.default_rng(0).permutation(pb.k.shape[0])
    inv = np.argsort(perm)
    pb2 = random_problem(9, [16 * 11 + 3, 16 * 7], Hq=8, H=2, D=64, ps=16, extra_pages=4)
    pb2.k = pb.k[torch.from_numpy(inv)]          # new storage slot s holds old page inv[s]
    pb2.v = pb.v[torch.from_numpy(inv)]
    pb2.page_indices = perm[pb.page_indices].astype(np.int32)
    b = _run(pb2, kind)
    assert np.array_equal(a["sel"], b["sel"]) and np.array_equal(a["out"], b["out"])
    assert np.array_equal(a["scores"], b["scores"])


def test_prefix_sharing_equals_private_copies():
    """Two requests sharing their first 5 physical pages give the same results as private copies."""
    pb = random_problem(10, [16 * 8 + 2, 16 * 6 + 9], Hq=4, H=1, D=64, ps=16, extra_pages=5)
    shared = pb.page_indices.copy()
    shared[pb.page_indptr[1]:pb.page_indptr[1] + 5] = shared[:5]
    pb.page_indices = shared
    a = _run(pb, budget=5)
    # private copies: duplicate the shared pages into the unused storage slots
    used = set(shared.tolist())
    free = [p for p in range(pb.k.shape[0]) if p not in used]
    priv = shared.copy()
    k2, v2 = pb.k.clone(), pb.v.clone()
    for m in range(5):
        k2[free[m]] = pb.k[shared[m]]
        v2[free[m]] = pb.v[shared[m]]
        priv[pb.page_indptr[1] + m] = free[m]
    pb.k, pb.v, pb.page_indices = k2, v2, priv
    b = _run(pb, budget=5)
    assert np.array_equal(a["sel"], b["sel"]) and np.array_equal(a["out"], b["out"])


def test_requests_are_independent():
    """No operator transforms the batch dimension (Appendix B): perturbing request 1 leaves
    request 0 unchanged."""
    pb = random_problem(11, [16 * 9, 16 * 9], Hq=4, H=1, D=64, ps=16)
    a = _run(pb)
    q2 = pb.q.clone()
    q2[1] = -q2[1]
    pb.q = q2
    b = _run(pb)
    assert np.array_equal(a["sel"][0], b["sel"][0]) and np.array_equal(a["out"][0], b["out"][0])


# --------------------------------------------------------------------------------------
# preconditions
# --------------------------------------------------------------------------------------
def test_rejects_page_count_mismatch():
    pb = random_problem(12, [40], Hq=4, H=1, D=64, ps=16)
    with pytest.raises(ValueError):
        O.summarize(pb.k, 16, [0, 2], pb.page_indices[:2], pb.seq_lens)


def test_rejects_shared_page_with_different_lengths():
    pb = random_problem(13, [40, 40], Hq=4, H=1, D=64, ps=16)
    idx = pb.page_indices.copy()
    idx[5] = idx[1]          # request 1's partial last page aliases request 0's full page 1
    with pytest.raises(ValueError):
        O.summarize(pb.k, 16, pb.page_indptr, idx, pb.seq_lens)


# --------------------------------------------------------------------------------------
# approximate radix top-k (Sec. 5.2 stochastic early termination, Appendix D remapping)
# --------------------------------------------------------------------------------------
def _lowbias32(x):
    x &= 0xFFFFFFFF
    x ^= x >> 16
    x = (x * 0x7FEB352D) & 0xFFFFFFFF
    x ^= x >> 15
    x = (x * 0x846CA68B) & 0xFFFFFFFF
    x ^= x >> 16
    return x


def _order_key(f):
    u = int(np.array([f], np.float32).view(np.uint32)[0])
    if f != f:
        return 0
    if u == 0x80000000:
        u = 0
    return (~u) & 0xFFFFFFFF if u & 0x80000000 else u | 0x80000000


def _tau_q(tau):
    """The tolerate ratio in 16-bit fixed point, rounded in fp32 (round half away from zero)."""
    x = np.float32(np.float32(tau) * np.float32(65536.0))
    return int(math.floor(float(x) + 0.5))


def _exact_topk(row, P, Ktot, n_sink, n_local):
    if Ktot >= P:
        return set(range(P))
    forced = {j for j in range(P) if j < n_sink or j >= P - n_local}
    cand = [j for j in range(P) if j not in forced]
    kfree = max(0, Ktot - len(forced))
    order = sorted(cand, key=lambda j: (-float(row[j]), j))      # larger score, lower index first
    return forced | set(order[:kfree])


def _topk_case(seed, H=2, B=3, P_max=60, ints=True):
    rng = np.random.default_rng(seed)
    stride = P_max
    if ints:
        sc = rng.integers(-6, 7, size=(H, B, stride)).astype(np.float32)    # many ties
    else:
        sc = rng.standard_normal((H, B, stride)).astype(np.float32)
    n = rng.integers(1, P_max + 1, size=B)
    bud = rng.integers(0, P_max // 2, size=B)
    return sc, n, bud


def _hash_fill(seed, unit, members, need):
    """The seeded random order of the threshold bin, written from its definition: members
    sorted by the top 8 bits of lowbias32(z ^ j), larger first, equal hashes by page;
    z = lowbias32(seed ^ lowbias32(unit))."""
    z = _lowbias32(seed ^ _lowbias32(unit))
    order = sorted(members, key=lambda j: (-(_lowbias32(z ^ j) >> 24), j))
    return set(order[:need])


@pytest.mark.parametrize("section,remap", [("approx_topk_binade", 0), ("approx_topk_affine", 1)])
def test_golden_approx_topk(section, remap):
    """Hand-worked pass schedules (tests/golden/hand_examples.txt): which tolerate ratios end the
    walk early, the certain members at that pass, the threshold bin the rest is drawn from, and
    the exact result otherwise."""
    G = _golden()[section]
    sc = np.array(G["scores"], np.float32)[None, None, :]
    P, K, seed = sc.shape[-1], int(G["budget"][0]), int(G["seed"][0])
    exact, certain, binm = (set(int(x) for x in G[k]) for k in ("exact", "certain", "bin"))
    need = K - len(certain)
    fill = _hash_fill(seed, 0, sorted(binm), need)
    # the example discriminates: the random fill is neither the exact nor the page-order fill
    assert fill != exact - certain and fill != set(sorted(binm)[:need])
    for tau in G["exact_taus"]:
        sel, cnt = O.topk_select(sc, [P], [K], 0, 0, K, tau=tau, seed=seed, remap=remap)
        assert set(sel[0, 0, :cnt[0]].tolist()) == exact, tau
    for tau in G["early_taus"]:
        sel, cnt = O.topk_select(sc, [P], [K], 0, 0, K, tau=tau, seed=seed, remap=remap)
        assert set(sel[0, 0, :cnt[0]].tolist()) == certain | fill, tau


@pytest.mark.parametrize("remap", [0, 1])
def test_approx_topk_tau_one_is_one_pass_and_a_sample(remap):
    """tau = 1 ends the walk after the first pass whenever bits are left (c * 65536 >= 0): the
    members are the candidates above T's bin at the first pass boundary (8 bits from the highest
    differing key bit) plus a hash-ordered sample of that bin, for every (request, head) unit."""
    rng = np.random.default_rng(77)
    H, B, P = 2, 3, 300
    sc = rng.integers(0, 12, size=(H, B, P)).astype(np.float32) + rng.integers(0, 4, size=(H, B, P)) / 8.0
    sc = sc.astype(np.float32)
    bud = [40, 25, 61]
    sel, cnt = O.topk_select(sc, [P] * B, bud, 1, 2, 64, tau=1.0, seed=99, remap=remap)
    for i in range(B):
        for h in range(H):
            cand = list(range(1, P - 2))
            row = [float(x) for x in sc[h, i]]
            if remap:
                lo, hi = min(row[j] for j in cand), max(row[j] for j in cand)
                key = {j: int(math.floor((row[j] - lo) * (4294967295.0 / (hi - lo)))) for j in cand}
            else:
                key = {j: _order_key(row[j]) for j in cand}
            kfree = bud[i] - 3
            T = sorted(key.values(), reverse=True)[kfree - 1]
            t0 = (min(key.values()) ^ max(key.values())).bit_length() - 1
            b1 = max(t0 - 7, 0)
            assert b1 > 0
            top = {j for j in cand if key[j] >> b1 > T >> b1}
            binm = sorted(j for j in cand if key[j] >> b1 == T >> b1)
            if len(binm) == kfree - len(top):
                want = top | set(binm)
            else:
                want = top | _hash_fill(99, i * H + h, binm, kfree - len(top))
            got = set(int(x) for x in sel[i, h, :cnt[i]])
            assert got == want | {0, P - 2, P - 1}, (i, h)


@pytest.mark.parametrize("tau", [0.2, 0.6, 1.0])
@pytest.mark.parametrize("remap", [0, 1])
def test_approx_topk_fill_comes_only_from_one_first_pass_bin(tau, remap):
    """Whatever pass the walk ends at, an unchosen candidate can outrank a chosen one only when
    both share the key bits the first pass resolves (the random fill never reaches outside the
    threshold bin), and the count is exactly the budget."""
    for seed in range(4):
        sc, n, bud = _topk_case(900 + seed, P_max=400, ints=(seed % 2 == 0))
        H, B, _ = sc.shape
        sel, cnt = O.topk_select(sc, n, bud, 1, 2, 256, tau=tau, seed=seed, remap=remap)
        for i in range(B):
            P = int(n[i])
            for h in range(H):
                got = set(int(x) for x in sel[i, h, :cnt[i]])
                forced = {j for j in range(P) if j < 1 or j >= P - 2}
                if int(bud[i]) >= P:
                    assert got == set(range(P))
                    continue
                assert forced <= got and len(got) == len(forced) + max(0, int(bud[i]) - len(forced))
                cand = [j for j in range(P) if j not in forced]
                row = [float(x) for x in sc[h, i]]
                if remap:
                    lo, hi = min(row[j] for j in cand), max(row[j] for j in cand)
                    sc_ = 4294967295.0 / (hi - lo) if hi > lo else 0.0
                    key = {j: int(math.floor((row[j] - lo) * sc_)) for j in cand}
                else:
                    key = {j: _order_key(row[j]) for j in cand}
                t0 = (min(key.values()) ^ max(key.values())).bit_length() - 1
                b1 = max(t0 - 7, 0) if t0 >= 0 else 32
                for s_ in got - forced:
                    for u in set(cand) - got:
                        if key[u] > key[s_]:
                            assert key[u] >> b1 == key[s_] >> b1, (i, h, s_, u)


def test_approx_topk_sample_is_uniform_over_the_bin():
    """Over many seeds every member of the threshold bin is drawn about equally often
    (need / bin size), the sample stays inside the bin, and certain members are always kept."""
    sc = np.zeros((1, 1, 200), np.float32)          # 160 tied candidates form the bin
    sc[0, 0, 50:90] = 1.0                            # 40 certain members above it
    runs, need = 3000, 20
    freq = np.zeros(200)
    for seed in range(runs):
        sel, cnt = O.topk_select(sc, [200], [60], 0, 0, 60, tau=1.0, seed=seed, remap=0)
        got = sel[0, 0, :cnt[0]]
        assert set(range(50, 90)) <= set(got.tolist()) and cnt[0] == 60
        freq[got] += 1
    binm = [j for j in range(200) if not 50 <= j < 90]
    p = freq[binm] / runs
    expect = need / len(binm)
    sd = math.sqrt(expect * (1 - expect) / runs)
    assert abs(p.mean() - expect) < 1e-12
    assert np.abs(p - expect).max() < 5 * sd, (p.min(), p.max(), expect)


@pytest.mark.parametrize("remap", [0, 1])
def test_approx_topk_with_zero_tolerance_is_the_exact_selection(remap):
    for seed in range(6):
        sc, n, bud = _topk_case(100 + seed, P_max=300, ints=(remap == 0))
        H, B, _ = sc.shape
        sel, cnt = O.topk_select(sc, n, bud, 1, 4, 200, tau=0.0, seed=seed, remap=remap)
        for i in range(B):
            for h in range(H):
                exact = _exact_topk(sc[h, i], int(n[i]), int(bud[i]), 1, 4)
                assert set(int(x) for x in sel[i, h, : cnt[i]]) == exact
                assert (np.diff(sel[i, h, : cnt[i]]) > 0).all() and (sel[i, h, cnt[i]:] == -1).all()


@pytest.mark.parametrize("tau", [0.1, 0.25, 0.5, 0.9, 1.0])
def test_approx_topk_recall_is_at_least_one_minus_tau(tau):
    """Candidates in bins above the threshold bin are true members, and there are at least
    (1 - tau) K_free of them when refinement stops (tau in 16-bit fixed point)."""
    for seed in range(8):
        rng = np.random.default_rng(500 + seed)
        H, B, P = 2, 2, 2000
        dist = seed % 4
        if dist == 0:
            sc = rng.standard_normal((H, B, P))
        elif dist == 1:
            sc = rng.lognormal(0.0, 1.0, (H, B, P))
        elif dist == 2:
            sc = rng.uniform(-1, 1, (H, B, P))
        else:
            sc = np.where(rng.random((H, B, P)) < 0.1, rng.normal(4, 0.5, (H, B, P)), rng.normal(0, 1, (H, B, P)))
        sc = sc.astype(np.float32)
        n, bud = np.full(B, P), np.full(B, 130)
        for remap in (0, 1):
            sel, cnt = O.topk_select(sc, n, bud, 1, 4, 130, tau=tau, seed=seed, remap=remap)
            for i in range(B):
                for h in range(H):
                    exact = _exact_topk(sc[h, i], P, 130, 1, 4)
                    got = set(int(x) for x in sel[i, h, : cnt[i]])
                    assert len(got) == 130 and {0, P - 4, P - 3, P - 2, P - 1} <= got
                    kfree = 125
                    hits = len((got & exact) - {0, P - 4, P - 3, P - 2, P - 1})
                    assert hits * 65536 >= (65536 - _tau_q(tau)) * kfree, (tau, remap, hits)


def test_approx_topk_sample_depends_on_the_seed():
    sc = np.zeros((1, 1, 400), np.float32)          # one bin: every candidate ties
    sc[0, 0, 100:140] = 1.0                          # 40 certain members above it
    sel_a, _ = O.topk_select(sc, [400], [80], 0, 0, 80, tau=1.0, seed=1, remap=0)
    sel_b, _ = O.topk_select(sc, [400], [80], 0, 0, 80, tau=1.0, seed=2, remap=0)
    a, b = set(sel_a[0, 0].tolist()), set(sel_b[0, 0].tolist())
    assert set(range(100, 140)) <= a and set(range(100, 140)) <= b
    assert a != b                                    # a different window of the tied bin


# --------------------------------------------------------------------------------------
# 8-bit floating-point KV caches (Sec. 5.3; Appendix E: fp8_e4m3 and fp8_e5m2 cache dtypes)
# --------------------------------------------------------------------------------------
FP8 = [(torch.float8_e4m3fn, O.KV_FP8_E4M3), (torch.float8_e5m2, O.KV_FP8_E5M2)]


@pytest.mark.parametrize("dtype,fmt", FP8)
def test_fp8_codes_decode_like_torch(dtype, fmt):
    """Every one of the 256 codes decodes to torch's value for the same OCP format."""
    codes = np.arange(256, dtype=np.uint8)
    got = O.fp8_dequantize(codes, fmt, 1.0)
    ref = torch.from_numpy(codes).view(dtype).float().numpy()
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])


def test_fp8_closed_forms():
    """Values fixed by the format definitions: largest finite, smallest subnormal, one, the
    special codes."""
    e4 = O.fp8_dequantize(np.array([0x7E, 0x01, 0x08, 0x38, 0x80, 0xFE, 0x7F], np.uint8), O.KV_FP8_E4M3, 1.0)
    assert e4[:6].tolist() == [448.0, 2.0 ** -9, 2.0 ** -6, 1.0, 0.0, -448.0] and np.isnan(e4[6])
    assert math.copysign(1.0, e4[4]) == -1.0
    e5 = O.fp8_dequantize(np.array([0x7B, 0x01, 0x04, 0x3C, 0x7C, 0xFC, 0x7D], np.uint8), O.KV_FP8_E5M2, 1.0)
    assert e5[:6].tolist() == [57344.0, 2.0 ** -16, 2.0 ** -14, 1.0, math.inf, -math.inf] and np.isnan(e5[6])


@pytest.mark.parametrize("dtype,fmt", FP8)
def test_fp8_scale_is_one_fp32_product(dtype, fmt):
    """Cache value = fp32(scale * code value): compare with torch's fp32 multiply."""
    codes = np.arange(256, dtype=np.uint8)
    s = 0.0173
    got = O.fp8_dequantize(codes, fmt, s)
    ref = (torch.from_numpy(codes).view(dtype).float() * torch.tensor(s, dtype=torch.float32)).numpy()
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])


@pytest.mark.parametrize("dtype,fmt", FP8)
@pytest.mark.parametrize("k_scale,v_scale", [(1.0, 1.0), (0.25, 2.0)])
@pytest.mark.parametrize("kind", [O.MEAN_DOT, O.QUEST, O.MAX_DOT])
def test_fp8_pipeline_equals_the_bf16_pipeline_on_exact_values(dtype, fmt, k_scale, v_scale, kind):
    """With power-of-two scales every cache value is a bf16 value: the whole fp8 decode step must
    equal the (pinned) bf16 step run on those values."""
    from tests._problems import Problem, fp8_problem
    pb = random_problem(41, [16 * 5 + 3, 16 * 9, 7], Hq=8, H=2, D=64, ps=16, extra_pages=2)
    p8 = fp8_problem(pb, dtype, k_scale, v_scale)
    kd = (p8.k.float() * k_scale).to(torch.bfloat16)
    vd = (p8.v.float() * v_scale).to(torch.bfloat16)
    assert torch.equal(kd.float(), p8.k.float() * k_scale)          # exact in bf16
    args = (pb.page_size, pb.page_indptr, pb.page_indices, pb.seq_lens, [4, 6, 1], 1, 2, 8, 0.125)
    r8 = O.pipeline(pb.q, p8.k, p8.v, kind, *args, k_scale=k_scale, v_scale=v_scale)
    rb = O.pipeline(pb.q, kd, vd, kind, *args)
    for key in ("mean", "max", "min", "scores", "sel", "cnt", "out"):
        assert np.array_equal(r8[key], rb[key], equal_nan=key in ("mean", "max", "min", "scores")), key


@pytest.mark.parametrize("dtype,fmt", FP8)
@pytest.mark.parametrize("k_scale", [1.0, 0.25])
@pytest.mark.parametrize("kind", [O.MEAN_DOT, O.MEAN_DOT_CONTENT])
def test_fp8_mla_latent_pipeline_equals_the_bf16_pipeline_on_exact_values(dtype, fmt, k_scale, kind):
    """An fp8 MLA latent (Sec. 5.3, Appendix E cache dtypes; V aliased to the first 512 channels of
    the 576-channel latent): with a power-of-two scale every cache value is a bf16 value, so the
    whole fp8 step equals the bf16 step on those values; V takes the latent's (K) scale."""
    from tests._problems import fp8_problem
    pb = random_problem(51, [64 * 3 + 5, 64 * 5, 20], Hq=16, H=1, D=576, ps=64, Dv=512, alias_v=True, extra_pages=2)
    p8 = fp8_problem(pb, dtype, k_scale, 1.0)
    kd = (p8.k.float() * k_scale).to(torch.bfloat16)
    assert torch.equal(kd.float(), p8.k.float() * k_scale)          # exact in bf16
    args = (pb.page_size, pb.page_indptr, pb.page_indices, pb.seq_lens, [3, 2, 1], 1, 1, 4, 1.0 / 24, 512)
    r8 = O.pipeline(pb.q, p8.k, None, kind, *args, k_scale=k_scale, v_scale=7.0)   # v_scale unused: V is K
    rb = O.pipeline(pb.q, kd, None, kind, *args)
    for key in ("mean", "max", "min", "scores", "sel", "cnt", "out"):
        assert np.array_equal(r8[key], rb[key], equal_nan=key in ("mean", "max", "min", "scores")), key


@pytest.mark.parametrize("dtype,fmt", FP8)
def test_fp8_mla_latent_attention_equals_sdpa(dtype, fmt):
    """Every page selected, a general latent scale: torch fp64 attention over the fp32 cache values
    with V = the first 512 latent channels at the same scale, every head sharing the latent."""
    from tests._problems import fp8_problem
    ks = 0.0213
    pb = random_problem(53, [64 * 2 + 9, 40], Hq=16, H=1, D=576, ps=64, Dv=512, alias_v=True)
    p8 = fp8_problem(pb, dtype, ks, 1.0)
    sel, cnt = _all_pages(pb, 4)
    sm = 1.0 / 24
    out = O.attend(pb.q, p8.k, None, 64, pb.page_indptr, pb.page_indices, pb.seq_lens, sel, cnt, sm,
                   head_dim_v=512, k_scale=ks, v_scale=3.0)
    kd = (p8.k.float() * torch.tensor(ks, dtype=torch.float32)).double()
    for i in range(pb.batch):
        ks_ = []
        for j in range(int(pb.page_indptr[i + 1] - pb.page_indptr[i])):
            p = int(pb.page_indices[pb.page_indptr[i] + j])
            ks_.append(kd[p, 0, : min(64, int(pb.seq_lens[i]) - j * 64)])
        K = torch.cat(ks_)[None].expand(16, -1, -1)
        V = K[..., :512]
        qi = pb.q[i].to(torch.float64)[:, None, :]
        ref = torch.nn.functional.scaled_dot_product_attention(qi, K, V, scale=sm)[:, 0]
        np.testing.assert_allclose(out[i], ref.numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("dtype,fmt", FP8)
def test_fp8_summaries_with_a_general_scale(dtype, fmt):
    """scale 0.0173: Mean is the fp64 mean of the fp32 cache values; Max and Min are those
    values' max and min rounded to bf16 (torch's round-to-nearest-even conversion)."""
    from tests._problems import fp8_problem
    s = 0.0173
    pb = random_problem(43, [16 * 3 + 5, 16 * 2], Hq=4, H=2, D=64, ps=16)
    p8 = fp8_problem(pb, dtype, s, s)
    mean, mx, mn = O.summarize(p8.k, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, k_scale=s)
    deq = p8.k.float() * torch.tensor(s, dtype=torch.float32)
    for i in range(pb.batch):
        for j in range(int(pb.page_indptr[i + 1] - pb.page_indptr[i])):
            p = int(pb.page_indices[pb.page_indptr[i] + j])
            n = min(16, int(pb.seq_lens[i]) - j * 16)
            x = deq[p, :, :n]                                   # [H][n][D] fp32
            np.testing.assert_allclose(mean[p], x.double().mean(dim=1).numpy(), rtol=0, atol=1e-15)
            assert np.array_equal(mx[p], x.max(dim=1).values.to(torch.bfloat16).double().numpy())
            assert np.array_equal(mn[p], x.min(dim=1).values.to(torch.bfloat16).double().numpy())


@pytest.mark.parametrize("dtype,fmt", FP8)
def test_fp8_attention_equals_sdpa_on_the_cache_values(dtype, fmt):
    """Every page selected, different K and V scales: torch fp64 attention over the fp32
    cache values."""
    from tests._problems import fp8_problem
    ks, vs = 0.021, 0.0377
    pb = random_problem(47, [16 * 4 + 9, 16 * 2, 5], Hq=8, H=2, D=64, ps=16)
    p8 = fp8_problem(pb, dtype, ks, vs)
    sel, cnt = _all_pages(pb, 8)
    out = O.attend(pb.q, p8.k, p8.v, 16, pb.page_indptr, pb.page_indices, pb.seq_lens, sel, cnt, 0.125,
                   k_scale=ks, v_scale=vs)
    kd = (p8.k.float() * torch.tensor(ks, dtype=torch.float32)).double()
    vd = (p8.v.float() * torch.tensor(vs, dtype=torch.float32)).double()
    g = 4
    for i in range(pb.batch):
        Ks, Vs = [], []
        for h in range(2):
            kk, vv = [], []
            for j in range(int(pb.page_indptr[i + 1] - pb.page_indptr[i])):
                p = int(pb.page_indices[pb.page_indptr[i] + j])
                n = min(16, int(pb.seq_lens[i]) - j * 16)
                kk.append(kd[p, h, :n])
                vv.append(vd[p, h, :n])
            Ks.append(torch.cat(kk))
            Vs.append(torch.cat(vv))
        K = torch.stack(Ks).repeat_interleave(g, dim=0)
        V = torch.stack(Vs).repeat_interleave(g, dim=0)
        qi = pb.q[i].to(torch.float64)[:, None, :]
        ref = torch.nn.functional.scaled_dot_product_attention(qi, K, V, scale=0.125)[:, 0]
        np.testing.assert_allclose(out[i], ref.numpy(), rtol=0, atol=1e-12)
