"""Small random paged problems for the tests (input construction only, no method arithmetic)."""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np
import torch


@dataclass
class Problem:
    q: torch.Tensor            # bf16 [B][Hq][Dqk]
    k: torch.Tensor            # bf16 [P][H][ps][Dqk]
    v: Optional[torch.Tensor]  # bf16 [P][H][ps][Dv] or None (V = K[..., :Dv])
    seq_lens: np.ndarray
    page_indptr: np.ndarray
    page_indices: np.ndarray
    page_size: int
    head_dim_v: int

    @property
    def batch(self):
        return len(self.seq_lens)

    @property
    def num_kv_heads(self):
        return self.k.shape[1]

    @property
    def num_q_heads(self):
        return self.q.shape[1]


def random_problem(seed: int, lens: List[int], Hq: int, H: int, D: int, ps: int, Dv: Optional[int] = None,
                   alias_v: bool = False, extra_pages: int = 0, scale: float = 1.0) -> Problem:
    """Random bf16 q/K/V, physical pages in a seeded random order, ragged lengths."""
    g = torch.Generator().manual_seed(seed)
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens, dtype=np.int32)
    pages = (lens + ps - 1) // ps
    indptr = np.zeros(len(lens) + 1, np.int32)
    indptr[1:] = np.cumsum(pages)
    total = int(indptr[-1]) + extra_pages
    perm = rng.permutation(total)[: int(indptr[-1])].astype(np.int32)
    Dv = D if Dv is None else Dv
    q = (torch.randn(len(lens), Hq, D, generator=g) * scale).to(torch.bfloat16)
    k = (torch.randn(total, H, ps, D, generator=g) * scale).to(torch.bfloat16)
    v = None if alias_v else torch.randn(total, H, ps, Dv, generator=g).to(torch.bfloat16)
    return Problem(q=q, k=k, v=v, seq_lens=lens, page_indptr=indptr, page_indices=perm,
                   page_size=ps, head_dim_v=Dv)


def valid_keys(pb: Problem, i: int, h: int, j: int) -> torch.Tensor:
    """fp64 keys of the valid tokens of logical page j of request i, KV head h."""
    ps = pb.page_size
    p = int(pb.page_indices[pb.page_indptr[i] + j])
    n = min(ps, int(pb.seq_lens[i]) - j * ps)
    return pb.k[p, h, :n].to(torch.float64)


def request_kv(pb: Problem, i: int, h: int, pages=None):
    """fp64 (K, V) of request i, KV head h, over the given logical pages (all by default)."""
    ps = pb.page_size
    P = int(pb.page_indptr[i + 1] - pb.page_indptr[i])
    pages = range(P) if pages is None else pages
    ks, vs = [], []
    for j in pages:
        p = int(pb.page_indices[pb.page_indptr[i] + j])
        n = min(ps, int(pb.seq_lens[i]) - j * ps)
        ks.append(pb.k[p, h, :n].to(torch.float64))
        if pb.v is None:
            vs.append(pb.k[p, h, :n, : pb.head_dim_v].to(torch.float64))
        else:
            vs.append(pb.v[p, h, :n].to(torch.float64))
    return torch.cat(ks), torch.cat(vs)


def fp8_problem(pb: Problem, dtype, k_scale: float, v_scale: float) -> Problem:
    """The same problem with K and V stored as 8-bit floating-point codes of `dtype`
    (torch.float8_e4m3fn or torch.float8_e5m2): code = fp8(x * fp32(1 / scale)), rounded by
    torch's conversion."""
    def quant(x, s):
        return None if x is None else (x.float() * torch.tensor(1.0 / s, dtype=torch.float32)).to(dtype)
    return Problem(q=pb.q, k=quant(pb.k, k_scale), v=quant(pb.v, v_scale), seq_lens=pb.seq_lens,
                   page_indptr=pb.page_indptr, page_indices=pb.page_indices, page_size=pb.page_size,
                   head_dim_v=pb.head_dim_v)


def strip_last_token(pb: Problem, seed: int):
    """The cache without each request's newest token (its slot overwritten with other values),
    and the removed K and V rows [B][H][D] (V rows None when V is aliased)."""
    g = torch.Generator().manual_seed(seed)
    k, v = pb.k.clone(), None if pb.v is None else pb.v.clone()
    kn = torch.empty((pb.batch, pb.k.shape[1], pb.k.shape[3]), dtype=pb.k.dtype)
    vn = None if v is None else torch.empty((pb.batch, v.shape[1], v.shape[3]), dtype=v.dtype)
    for i in range(pb.batch):
        t = int(pb.seq_lens[i]) - 1
        p = int(pb.page_indices[pb.page_indptr[i] + t // pb.page_size])
        kn[i] = k[p, :, t % pb.page_size]
        k[p, :, t % pb.page_size] = torch.randn(k.shape[1], k.shape[3], generator=g).to(k.dtype)
        if v is not None:
            vn[i] = v[p, :, t % pb.page_size]
            v[p, :, t % pb.page_size] = torch.randn(v.shape[1], v.shape[3], generator=g).to(v.dtype)
    return k, v, kn, vn
