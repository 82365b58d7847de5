"""Seeded synthetic decode workloads shaped like the Vortex evaluation (arXiv 2606.06453).

This module only *generates inputs*.  It holds none of the method's arithmetic (no summaries,
scores, selection or attention); both the HIP path and the CPU oracle consume what it
produces, and neither is imported here.

Large tensors (q, K, V) come from a counter-based generator so that any slice of a
multi-gigabyte cache can be regenerated bit-identically on the host, without materialising
the rest.  That is what lets the oracle check sampled requests of a full-size workload.

Counter-based normal generator
------------------------------
* ``lowbias32`` is C. Wellons' 32-bit integer hash (hash-prospector, 2018):
  ``x ^= x>>16; x *= 0x7feb352d; x ^= x>>15; x *= 0x846ca68b; x ^= x>>16`` (mod 2**32).
* Element ``c`` of stream ``key`` draws ``u = lowbias32((c mod 2**32) ^ s) >> 16`` with
  ``s = lowbias32(key ^ lowbias32(c >> 32))``, a 16-bit uniform index.
* The normal value is ``TABLE[u]``, where ``TABLE[m] = Phi^-1((m + 0.5) / 65536)``. It is
  computed in fp64 by ``scipy.special.ndtri`` and rounded to fp32, so |x| <= 4.33.
* Values are rounded to bfloat16 with round-to-nearest-even, torch's ``.to(bfloat16)``.

Only integer operations, one table gather and IEEE-exact fp32 adds are involved, so CPU and
GPU produce identical bits.

Readings of the paper's workload wording (all recorded in the design doc):

* Contexts (C2) are integers ``L ~ U{8192..32768}``.
* C5 uses ``ln L ~ N(ln 16384, 0.6^2)``, clipped to ``[4096, 65536]`` and rounded.
* Physical pages are a seeded random permutation of ``[0, sum P_i)``.
* A planted ("relevant") page of request i and KV head h has keys
  ``k_t <- bf16(fp32(k_t) + fp32(0.5 * qbar_h))``, where ``qbar_h`` is the mean of the
  group's bf16 query heads (exact fp64 sum, one rounding to fp32).
* C2 plants ``round(0.02 * P_i)`` pages per (request, KV head), drawn from the non-forced
  pages. C1 plants 4 pages, drawn from all 64.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch

MEAN_DOT = 0   # score = mean over the group's heads of q_r . Mean_j   (block top-k)
QUEST = 1      # score = max over the group's heads of sum_c max(q*Max, q*Min)
MAX_DOT = 2    # score = mean over the group's heads of q_r . Max_j

KIND_NAMES = {MEAN_DOT: "mean_dot", QUEST: "quest", MAX_DOT: "max_dot", 3: "quest_consensus", 4: "envelope_lower",
              5: "quest_rectified", 6: "mean_dot_content", 7: "nsa", 8: "mean_dot_smooth"}   # the ABI's score kinds

_M32 = 0xFFFFFFFF


# ----------------------------------------------------------------------------------------
# counter-based generator (integer ops on int64 tensors; identical on CPU and GPU)
# ----------------------------------------------------------------------------------------
def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2**32 for 0 <= x < 2**32 held in int64, without int64 overflow."""
    c_lo, c_hi = c & 0xFFFF, c >> 16
    return (x * c_lo + (((x & 0xFFFF) * c_hi) << 16)) & _M32


def lowbias32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


_TABLE_CACHE: Dict[str, torch.Tensor] = {}


def normal_table(device) -> torch.Tensor:
    dev = str(device)
    if dev not in _TABLE_CACHE:
        from scipy.special import ndtri
        m = np.arange(65536, dtype=np.float64)
        t = ndtri((m + 0.5) / 65536.0).astype(np.float32)
        _TABLE_CACHE[dev] = torch.from_numpy(t).to(device)
    return _TABLE_CACHE[dev]


def counter_normals_at(key: int, counters: torch.Tensor) -> torch.Tensor:
    """fp32 N(0,1)-shaped values for the given int64 counters of stream ``key``."""
    c = counters.to(torch.int64)
    hi = c >> 32
    lo = c & _M32
    s = lowbias32((lowbias32(hi) ^ (key & _M32)) & _M32)
    u = lowbias32(lo ^ s) >> 16
    return normal_table(c.device)[u]


def counter_normals(key: int, start: int, count: int, device) -> torch.Tensor:
    ctr = torch.arange(start, start + count, dtype=torch.int64, device=device)
    return counter_normals_at(key, ctr)


def to_bf16(x32: torch.Tensor) -> torch.Tensor:
    return x32.to(torch.bfloat16)


# ----------------------------------------------------------------------------------------
# configurations
# ----------------------------------------------------------------------------------------
@dataclass(frozen=True)
class Config:
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim_qk: int
    head_dim_v: int
    page_size: int
    kind: int
    n_sink: int
    n_local: int
    lengths: Tuple            # ("const", L) | ("uniform", lo, hi) | ("lognormal", median, sigma, lo, hi)
    budget: Tuple             # ("pages", K) | ("frac", f, extra)
    planted: Tuple = ("none",)  # ("count", n, from_forced_ok) | ("frac", f) | ("none",)
    v_alias: bool = False     # MLA: V is the first head_dim_v channels of K
    seed: int = 0
    kv_dtype: str = "bf16"    # "bf16" | "fp8_e4m3" | "fp8_e5m2" (KV cache element type)
    k_scale: float = 1.0      # fp8 caches: value = scale * code
    v_scale: float = 1.0

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def sm_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim_qk)

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)

    def with_kv_dtype(self, kv_dtype: str) -> "Config":
        """The same workload with its KV cache stored in `kv_dtype`.  fp8 scales map the
        largest generated magnitude (|x| <= 6.5 for planted keys, 4.33 for values) near the
        top of the format's range."""
        if kv_dtype == "bf16":
            return self.replace(kv_dtype="bf16", k_scale=1.0, v_scale=1.0)
        top = {"fp8_e4m3": 448.0, "fp8_e5m2": 57344.0}[kv_dtype]
        return self.replace(kv_dtype=kv_dtype, k_scale=6.6 / top, v_scale=4.4 / top)


# The five workloads.  ``seed`` k selects numpy.random.SeedSequence(k).
CONFIGS: Dict[str, Config] = {
    "tiny_gqa": Config(
        name="tiny_gqa", batch=1, num_q_heads=4, num_kv_heads=1, head_dim_qk=64, head_dim_v=64,
        page_size=16, kind=MEAN_DOT, n_sink=0, n_local=0, lengths=("const", 1024),
        budget=("pages", 8), planted=("count", 4, True), seed=1),
    "llama3_8b_layer": Config(
        name="llama3_8b_layer", batch=64, num_q_heads=32, num_kv_heads=8, head_dim_qk=128,
        head_dim_v=128, page_size=16, kind=MEAN_DOT, n_sink=1, n_local=4,
        lengths=("uniform", 8192, 32768), budget=("pages", 128), planted=("frac", 0.02), seed=2),
    "long_gen_quest": Config(
        name="long_gen_quest", batch=16, num_q_heads=32, num_kv_heads=8, head_dim_qk=128,
        head_dim_v=128, page_size=32, kind=QUEST, n_sink=1, n_local=4,
        lengths=("const", 131072), budget=("pages", 128), seed=3),
    "mla_absorbed": Config(
        name="mla_absorbed", batch=32, num_q_heads=16, num_kv_heads=1, head_dim_qk=576,
        head_dim_v=512, page_size=64, kind=MEAN_DOT, n_sink=1, n_local=4,
        lengths=("const", 32768), budget=("pages", 32), v_alias=True, seed=4),
    "large_gqa": Config(
        name="large_gqa", batch=128, num_q_heads=48, num_kv_heads=8, head_dim_qk=128,
        head_dim_v=128, page_size=16, kind=MAX_DOT, n_sink=1, n_local=4,
        lengths=("lognormal", 16384, 0.6, 4096, 65536), budget=("frac", 0.01, 5), seed=5),
}
CONFIG_ORDER = ["tiny_gqa", "llama3_8b_layer", "long_gen_quest", "mla_absorbed", "large_gqa"]


# Small variants: same head geometry, page size and scoring as the full configs, with
# ragged lengths and budgets below the page count, so that top-K really selects.  The
# oracle finishes each of them in well under a second.
SMALL: Dict[str, Config] = {
    "tiny_gqa": CONFIGS["tiny_gqa"],
    "llama3_8b_layer": CONFIGS["llama3_8b_layer"].replace(
        batch=5, lengths=("uniform", 200, 2600), budget=("pages", 24), seed=12),
    "long_gen_quest": CONFIGS["long_gen_quest"].replace(
        batch=3, lengths=("uniform", 900, 4100), budget=("pages", 20), seed=13),
    "mla_absorbed": CONFIGS["mla_absorbed"].replace(
        batch=3, lengths=("uniform", 700, 3000), budget=("pages", 12), seed=14),
    "large_gqa": CONFIGS["large_gqa"].replace(
        batch=6, lengths=("lognormal", 1500, 0.6, 300, 4000), budget=("frac", 0.05, 5), seed=15),
}


# ----------------------------------------------------------------------------------------
# workload
# ----------------------------------------------------------------------------------------
def _u32(ss: np.random.SeedSequence) -> int:
    return int(ss.generate_state(1, dtype=np.uint32)[0])


@dataclass
class Workload:
    cfg: Config
    seq_lens: np.ndarray          # int32 [B]
    pages: np.ndarray             # int32 [B]  P_i = ceil(L_i / ps)
    page_indptr: np.ndarray       # int32 [B+1]
    page_indices: np.ndarray      # int32 [sum P]  physical page ids
    num_phys_pages: int
    pages_budget: np.ndarray      # int32 [B]  total pages incl. forced
    max_sel: int
    q: torch.Tensor               # bf16 [B][Hq][Dqk] (cpu)
    planted: Dict[Tuple[int, int], np.ndarray] = field(default_factory=dict)  # (i,h) -> logical pages
    key_k: int = 0
    key_v: int = 0

    # ---- derived ----
    @property
    def max_pages(self) -> int:
        return int(self.pages.max())

    @property
    def k_dims(self) -> Tuple[int, int, int, int]:
        c = self.cfg
        return (self.num_phys_pages, c.num_kv_heads, c.page_size, c.head_dim_qk)

    @property
    def v_dims(self) -> Tuple[int, int, int, int]:
        c = self.cfg
        return (self.num_phys_pages, c.num_kv_heads, c.page_size, c.head_dim_v)

    def qbar32(self) -> np.ndarray:
        """fp32 [B][Hkv][Dqk]: mean of each group's bf16 query heads (input construction only)."""
        c = self.cfg
        q64 = self.q.to(torch.float64).numpy().reshape(c.batch, c.num_kv_heads, c.group, c.head_dim_qk)
        return (q64.sum(axis=2) / c.group).astype(np.float32)

    def _planted_by_phys(self) -> Dict[int, List[Tuple[int, int]]]:
        """physical page -> list of (kv head, request) plants on it."""
        out: Dict[int, List[Tuple[int, int]]] = {}
        for (i, h), js in self.planted.items():
            base = int(self.page_indptr[i])
            for j in js:
                out.setdefault(int(self.page_indices[base + int(j)]), []).append((h, i))
        return out

    # ---- K / V generation ----
    def _gen_pages(self, key: int, dims, phys: torch.Tensor, device, apply_plants: bool) -> torch.Tensor:
        """bf16 [len(phys)][H][ps][D] for the given physical page ids."""
        _, H, ps, D = dims
        per_page = H * ps * D
        phys = phys.to(torch.int64).to(device)
        ctr = phys[:, None] * per_page + torch.arange(per_page, dtype=torch.int64, device=device)[None, :]
        x = counter_normals_at(key, ctr).view(-1, H, ps, D)
        if apply_plants and self.planted:
            x = self._apply_plants(x, phys)
        return to_bf16(x)

    def _apply_plants(self, x32: torch.Tensor, phys: torch.Tensor) -> torch.Tensor:
        by_phys = self._planted_by_phys()
        if not by_phys:
            return x32
        qbar = torch.from_numpy(self.qbar32()).to(x32.device)
        phys_list = phys.tolist()
        pos = {p: r for r, p in enumerate(phys_list)}
        half = torch.tensor(0.5, dtype=torch.float32, device=x32.device)
        for p, plants in by_phys.items():
            if p not in pos:
                continue
            r = pos[p]
            for (h, i) in plants:
                shift = qbar[i, h] * half          # exact scaling by 1/2
                x32[r, h] = x32[r, h] + shift[None, :]
        return x32

    def _stored(self, x: torch.Tensor, which: str) -> torch.Tensor:
        c = self.cfg
        return quantize_cache(x, c.kv_dtype, c.k_scale if which == "k" else c.v_scale)

    def k_pages(self, phys, device="cpu") -> torch.Tensor:
        phys = torch.as_tensor(np.asarray(phys, dtype=np.int64))
        return self._stored(self._gen_pages(self.key_k, self.k_dims, phys, device, apply_plants=True), "k")

    def v_pages(self, phys, device="cpu") -> torch.Tensor:
        if self.cfg.v_alias:
            raise ValueError("V aliases K for this config")
        phys = torch.as_tensor(np.asarray(phys, dtype=np.int64))
        return self._stored(self._gen_pages(self.key_v, self.v_dims, phys, device, apply_plants=False), "v")

    def head_pages(self, phys, h: int, which: str = "k", device="cpu") -> torch.Tensor:
        """bf16 [len(phys)][1][ps][D]: one KV head's slice of the given physical pages
        (bit-identical to the same slice of the full storage)."""
        c = self.cfg
        key, dims = (self.key_k, self.k_dims) if which == "k" else (self.key_v, self.v_dims)
        if which == "v" and c.v_alias:
            raise ValueError("V aliases K for this config")
        _, H, ps, D = dims
        phys = torch.as_tensor(np.asarray(phys, dtype=np.int64)).to(device)
        per_page, per_head = H * ps * D, ps * D
        ctr = (phys[:, None] * per_page + h * per_head
               + torch.arange(per_head, dtype=torch.int64, device=device)[None, :])
        x = counter_normals_at(key, ctr).view(-1, 1, ps, D)
        if which == "k" and self.planted:
            qbar = torch.from_numpy(self.qbar32()).to(device)
            pos = {int(p): r for r, p in enumerate(phys.tolist())}
            for p, plants in self._planted_by_phys().items():
                if p in pos:
                    for (hh, i) in plants:
                        if hh == h:
                            x[pos[p], 0] = x[pos[p], 0] + qbar[i, h][None, :] * 0.5
        return self._stored(to_bf16(x), which)

    def _materialize(self, key, dims, device, apply_plants, chunk_pages=None) -> torch.Tensor:
        P, H, ps, D = dims
        out = torch.empty((P, H, ps, D), dtype=torch.bfloat16, device=device)
        per_page = H * ps * D
        if chunk_pages is None:
            chunk_pages = max(1, (1 << 26) // per_page)
        for p0 in range(0, P, chunk_pages):
            p1 = min(P, p0 + chunk_pages)
            ctr = torch.arange(p0 * per_page, p1 * per_page, dtype=torch.int64, device=device)
            out[p0:p1] = to_bf16(counter_normals_at(key, ctr).view(p1 - p0, H, ps, D))
        if apply_plants and self.planted:
            by_phys = self._planted_by_phys()
            ids = sorted(by_phys)
            for s in range(0, len(ids), 4096):
                sub = torch.tensor(ids[s:s + 4096], dtype=torch.int64)
                out[sub.to(device)] = self._gen_pages(key, dims, sub, device, apply_plants=True)
        return out

    def k_storage(self, device="cpu") -> torch.Tensor:
        return self._stored(self._materialize(self.key_k, self.k_dims, device, apply_plants=True), "k")

    def v_storage(self, device="cpu") -> Optional[torch.Tensor]:
        if self.cfg.v_alias:
            return None
        return self._stored(self._materialize(self.key_v, self.v_dims, device, apply_plants=False), "v")

    def layer(self, l: int) -> "Workload":
        """Another attention layer of the same batch: same lengths, page table and budgets,
        independent q / K / V streams (planted pages keep their positions)."""
        if l == 0:
            return self
        ss = np.random.SeedSequence([self.cfg.seed, 1000 + l])
        s_q, s_k, s_v = ss.spawn(3)
        c = self.cfg
        q = to_bf16(counter_normals(_u32(s_q), 0, c.batch * c.num_q_heads * c.head_dim_qk, "cpu")
                    ).view(c.batch, c.num_q_heads, c.head_dim_qk)
        return dataclasses.replace(self, q=q, key_k=_u32(s_k), key_v=_u32(s_v))

    # ---- sub-batches for sampled checks ----
    def sub_batch(self, reqs) -> "SubBatch":
        """Compact host copy of the given requests: their pages renumbered 0..n-1."""
        reqs = [int(r) for r in reqs]
        c = self.cfg
        phys_all, indptr, lens = [], [0], []
        for i in reqs:
            b0, b1 = int(self.page_indptr[i]), int(self.page_indptr[i + 1])
            phys_all.extend(int(p) for p in self.page_indices[b0:b1])
            indptr.append(indptr[-1] + (b1 - b0))
            lens.append(int(self.seq_lens[i]))
        uniq = sorted(set(phys_all))
        remap = {p: r for r, p in enumerate(uniq)}
        k = self.k_pages(uniq)
        v = None if c.v_alias else self.v_pages(uniq)
        return SubBatch(
            reqs=reqs, seq_lens=np.array(lens, np.int32), page_indptr=np.array(indptr, np.int32),
            page_indices=np.array([remap[p] for p in phys_all], np.int32), k=k, v=v,
            q=self.q[reqs].contiguous(), pages_budget=self.pages_budget[reqs].copy(),
            num_phys_pages=len(uniq))


@dataclass
class SubBatch:
    reqs: List[int]
    seq_lens: np.ndarray
    page_indptr: np.ndarray
    page_indices: np.ndarray
    k: torch.Tensor
    v: Optional[torch.Tensor]
    q: torch.Tensor
    pages_budget: np.ndarray
    num_phys_pages: int


def _lengths(cfg: Config, rng: np.random.Generator) -> np.ndarray:
    spec = cfg.lengths
    if spec[0] == "const":
        return np.full(cfg.batch, spec[1], dtype=np.int32)
    if spec[0] == "uniform":
        return rng.integers(spec[1], spec[2] + 1, size=cfg.batch).astype(np.int32)
    if spec[0] == "lognormal":
        med, sigma, lo, hi = spec[1:]
        x = np.exp(rng.normal(math.log(med), sigma, size=cfg.batch))
        return np.clip(np.rint(x), lo, hi).astype(np.int32)
    raise ValueError(spec)


def _budget(cfg: Config, pages: np.ndarray) -> np.ndarray:
    spec = cfg.budget
    if spec[0] == "pages":
        return np.full(cfg.batch, spec[1], dtype=np.int32)
    if spec[0] == "frac":
        f, extra = spec[1], spec[2]
        return (np.ceil(f * pages) + extra).astype(np.int32)
    raise ValueError(spec)


def make(cfg: Config, seed: Optional[int] = None) -> Workload:
    """Build the host-side description of a workload (K/V are generated on demand)."""
    seed = cfg.seed if seed is None else seed
    ss = np.random.SeedSequence(seed)
    s_q, s_k, s_v, s_len, s_perm, s_plant = ss.spawn(6)
    B, H, ps = cfg.batch, cfg.num_kv_heads, cfg.page_size
    lens = _lengths(cfg, np.random.default_rng(s_len))
    pages = ((lens + ps - 1) // ps).astype(np.int32)
    indptr = np.zeros(B + 1, dtype=np.int32)
    indptr[1:] = np.cumsum(pages)
    total = int(indptr[-1])
    perm = np.random.default_rng(s_perm).permutation(total).astype(np.int32)
    budget = _budget(cfg, pages)
    max_sel = int(budget.max())
    q = to_bf16(counter_normals(_u32(s_q), 0, B * cfg.num_q_heads * cfg.head_dim_qk, "cpu")
                ).view(B, cfg.num_q_heads, cfg.head_dim_qk)
    wl = Workload(cfg=cfg, seq_lens=lens, pages=pages, page_indptr=indptr, page_indices=perm,
                  num_phys_pages=total, pages_budget=budget, max_sel=max_sel, q=q,
                  key_k=_u32(s_k), key_v=_u32(s_v))
    rng = np.random.default_rng(s_plant)
    if cfg.planted[0] != "none":
        for i in range(B):
            P = int(pages[i])
            forced = set(range(min(cfg.n_sink, P))) | set(range(max(0, P - cfg.n_local), P))
            if cfg.planted[0] == "count":
                n, allow_forced = cfg.planted[1], cfg.planted[2]
                pool = np.arange(P) if allow_forced else np.array([j for j in range(P) if j not in forced])
            else:
                pool = np.array([j for j in range(P) if j not in forced])
                n = int(round(cfg.planted[1] * P))
            for h in range(H):
                if n > 0:
                    wl.planted[(i, h)] = np.sort(rng.choice(pool, size=n, replace=False)).astype(np.int32)
    return wl


KV_DTYPES = ("bf16", "fp8_e4m3", "fp8_e5m2")


def torch_kv_dtype(name: str):
    return {"bf16": torch.bfloat16, "fp8_e4m3": torch.float8_e4m3fn, "fp8_e5m2": torch.float8_e5m2}[name]


def quantize_cache(x: torch.Tensor, kv_dtype: str, scale: float) -> torch.Tensor:
    """A generated bf16 cache stored as `kv_dtype`: code = fp8(x * fp32(1 / scale)), rounded by
    torch's conversion (input construction; both the HIP path and the oracle read the codes)."""
    if kv_dtype == "bf16":
        return x
    inv = torch.tensor(1.0 / scale, dtype=torch.float32, device=x.device)
    return (x.float() * inv).to(torch_kv_dtype(kv_dtype))


def forced_pages(P: int, n_sink: int, n_local: int) -> set:
    """Sink and local pages of a request with P pages (used by tests and planted-page choice)."""
    return set(range(min(n_sink, P))) | set(range(max(0, P - n_local), P))


def synthetic_scores(dist, H, B, stride, seed):
    """Seeded fp32 score rows ``[H][B][stride]`` for the top-k operator on its own.

    ``normal``, ``lognormal``, ``uniform`` and ``bimodal`` (10% of entries from N(4, 0.5^2))
    are the four score shapes of the paper's top-k study (Appendix D); ``ties`` draws integers
    in [-20, 20] so that most scores tie."""
    rng = np.random.default_rng(seed)
    shape = (H, B, stride)
    if dist == "normal":
        x = rng.standard_normal(shape)
    elif dist == "lognormal":
        x = rng.lognormal(0.0, 1.0, shape)
    elif dist == "uniform":
        x = rng.uniform(-1.0, 1.0, shape)
    elif dist == "bimodal":
        x = np.where(rng.random(shape) < 0.1, rng.normal(4.0, 0.5, shape), rng.normal(0.0, 1.0, shape))
    else:                                     # many exact ties
        x = rng.integers(-20, 21, shape).astype(np.float64)
    return x.astype(np.float32)
