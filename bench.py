"""Benchmark: one sparse decode step of one attention layer, on one MI355X.

A step is the whole hot path for a batch of decode tokens:
  vx_append_score_topk (write the new token's K/V rows and refresh the summaries of the page
  holding it, inside the top-K launch; then score and select) -> vx_sparse_paged_decode
(--cache-stage append: vx_kv_append_summarize as a launch of its own, then vx_page_score_topk;
--cache-stage summarize: vx_page_summarize of that page instead, with the token already in the
cache).  The appended rows are the step token's own rows, so every step sees the same cache.
on the 32-query / 8-KV-head, head_dim 128, page 16 workload with batch 64, contexts U[8k, 32k],
Mean summaries and a 128-page budget (1 sink + 4 local + 123 chosen).  Inputs are seeded and
synthetic, and already resident in HBM.  Successive steps rotate over `--layers`
independent layer caches (same batch and lengths, separate q/K/V/summaries).  Each step
therefore reads a different ~0.9 GB working set, which the 256 MB Infinity Cache cannot hold.

Every call is launched eagerly from Python.  --graph captures each layer's step once into two
HIP graphs (summarize + select, and decode) and replays them instead; on this ROCm stack the
replays run slower than eager launches, so it is not the default.

Prints one JSON line.  value = decode tokens per second = batch / step time.
roofline: the decode call (its split kernel, which also merges split GQA pairs; for MLA plus the
merge kernel), timed with HIP events recorded on the launch stream around it on every
`--decode-event-every`-th timed step.  The events are created with hipEventDisableSystemFence:
a default event performs a system-scope release (an L2 writeback) when it is recorded, which
inflates short intervals.  Algorithmic bytes are those of the selected K/V tokens plus q and
out.  traffic: HBM bytes per call from the committed counter profile of the workload, while
the decode sources still match it (else null).
cpu_baseline: the fp64 oracle's decode step on a bounded sample of the same workload (rank
0, N = 1 only), on the oracle's default thread count and on one thread, with the CPU model.
decode_by_workload: the same decode-call measurement on each of the five workloads (fewer
steps), so that the default run records the fraction of HBM peak on every one of them.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2606_06453_amd import vx, workloads as W  # noqa: E402
from paper_2606_06453_amd.decoder import SparseDecoder  # noqa: E402

HBM_PEAK_GBS = 8000.0
DECODE_SOURCES = ("decode.hip", "vx_device.h", "vx_internal.h")


def counted_decode_traffic(cfg_name: str):
    """HBM bytes per decode call from the committed rocprofv3 counter profile of this workload
    (FETCH_SIZE and WRITE_SIZE scaled by a plain copy's readings), or None when there is none
    or the decode sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"hbm_counters_{cfg_name}.md")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if ":" in line and line.split(":")[0] in ("decode_source_sha256", "decode_call_traffic_bytes"):
            k, v = line.split(":", 1)
            rec[k] = v.strip()
    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2606_06453_amd", "csrc", f), "rb").read())
    if rec.get("decode_source_sha256") != h.hexdigest()[:16] or "decode_call_traffic_bytes" not in rec:
        return None
    return float(rec["decode_call_traffic_bytes"])
METRIC = "sparse decode attn tokens/sec/GPU; achieved HBM GB/s vs MI355X peak"
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000


class HipEvent:
    """A HIP event recorded on a torch stream, created without the system-scope fence."""
    _hip = None

    def __init__(self):
        if HipEvent._hip is None:
            # the HIP runtime torch has already loaded (same soname, so the same instance)
            h = ctypes.CDLL("libamdhip64.so.7")
            h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventDestroy.argtypes = [ctypes.c_void_p]
            HipEvent._hip = h
        self.ev = ctypes.c_void_p()
        rc = HipEvent._hip.hipEventCreateWithFlags(ctypes.byref(self.ev), HIP_EVENT_DISABLE_SYSTEM_FENCE)
        assert rc == 0, f"hipEventCreateWithFlags failed ({rc})"

    def record(self, stream: torch.cuda.Stream):
        rc = HipEvent._hip.hipEventRecord(self.ev, ctypes.c_void_p(stream.cuda_stream))
        assert rc == 0, f"hipEventRecord failed ({rc})"

    def elapsed_ms(self, end: "HipEvent") -> float:
        ms = ctypes.c_float()
        rc = HipEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self.ev, end.ev)
        assert rc == 0, f"hipEventElapsedTime failed ({rc})"
        return float(ms.value)

    def __del__(self):
        if HipEvent._hip is not None and self.ev:
            HipEvent._hip.hipEventDestroy(self.ev)


def describe(cfg: W.Config) -> str:
    L = cfg.lengths
    ctx = {"const": lambda: f"{L[1]}", "uniform": lambda: f"U[{L[1]},{L[2]}]",
           "lognormal": lambda: f"lognormal median {L[1]} clip[{L[3]},{L[4]}]"}[L[0]]()
    bud = f"{cfg.budget[1]} pages" if cfg.budget[0] == "pages" else f"ceil({cfg.budget[1]}*P)+{cfg.budget[2]} pages"
    return (f"{cfg.name}: B={cfg.batch} Hq={cfg.num_q_heads} Hkv={cfg.num_kv_heads} Dqk={cfg.head_dim_qk} "
            f"Dv={cfg.head_dim_v} page={cfg.page_size} ctx={ctx} score={W.KIND_NAMES[cfg.kind]} budget={bud} "
            f"sink={cfg.n_sink} local={cfg.n_local}"
            + ("" if cfg.kv_dtype == "bf16" else f" kv={cfg.kv_dtype} k_scale={cfg.k_scale:.6g} v_scale={cfg.v_scale:.6g}"))


class Layer:
    def __init__(self, wl: W.Workload, dev: str, block_size: int = 0, topk_options=None, two_pass=None):
        c = wl.cfg
        self.wl = wl
        self.k = wl.k_storage(dev)
        self.v = wl.v_storage(dev)
        self.kv = vx.PagedKV(self.k, self.v, c.head_dim_v, k_scale=c.k_scale, v_scale=c.v_scale,
                             block_size=block_size)
        # blocks below the page size: r blocks per page; the budget, forced pages and selection
        # row keep their token counts (r blocks for each page)
        self.r = c.page_size // block_size if block_size else 1
        self.bs = c.page_size // self.r
        self.batch = vx.BatchSpec(torch.from_numpy(wl.page_indptr).to(dev),
                                  torch.from_numpy(wl.page_indices).to(dev),
                                  torch.from_numpy(wl.seq_lens).to(dev), wl.max_pages)
        self.q = wl.q.to(dev)
        self.budget = torch.from_numpy(wl.pages_budget * self.r).to(dev)
        self.first = torch.from_numpy(((wl.seq_lens - 1) // self.bs).astype(np.int32)).to(dev)
        # the step token's own K/V rows [B][H][D] (token seq_lens[i] - 1), appended every step
        last = torch.from_numpy(wl.page_indices[wl.page_indptr[:-1] + wl.pages - 1].astype(np.int64)).to(dev)
        slot = torch.from_numpy(((wl.seq_lens - 1) % c.page_size).astype(np.int64)).to(dev)
        def rows(t):     # gathered through an integer view (fp8 tensors have no index kernels)
            iv = t.view(torch.int16 if t.element_size() == 2 else torch.uint8)
            return iv[last, :, slot].contiguous().view(t.dtype)
        self.k_new = rows(self.k)
        self.v_new = None if self.v is None else rows(self.v)
        self.dec = SparseDecoder(self.kv, self.batch, c.num_q_heads, c.kind, c.n_sink * self.r, c.n_local * self.r,
                                 wl.max_sel * self.r, c.sm_scale, two_pass=two_pass, topk_options=topk_options)
        self.dec.summarize()             # prefill: every page's summary


def algorithmic_decode_bytes(layer: Layer) -> int:
    """Selected valid tokens x (Dqk + Dv) x 2 B per (request, KV head), plus q and out."""
    c = layer.wl.cfg
    sel = layer.dec.sel_pages.cpu().numpy()
    cnt = layer.dec.sel_count.cpu().numpy()
    lens = layer.wl.seq_lens
    tokens = 0
    for i in range(c.batch):
        j = sel[i, :, : cnt[i]].astype(np.int64)                  # blocks of layer.bs tokens
        n = np.minimum(layer.bs, lens[i] - j * layer.bs)
        tokens += int(n.sum())
    per_token = (c.head_dim_qk + (0 if c.v_alias else c.head_dim_v)) * (2 if c.kv_dtype == "bf16" else 1)
    qo = c.batch * c.num_q_heads * (c.head_dim_qk + c.head_dim_v) * 2
    return tokens * per_token + qo


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(layer: Layer, target_s: float = 10.0, one_core_s: float = 8.0) -> dict:
    """The oracle's decode step (incremental summary + score + select + attend) on the first
    requests of the same workload, repeated until ~target_s of wall time, on the oracle's
    default thread count and then on one thread."""
    from oracle import oracle as O
    wl, c = layer.wl, layer.wl.cfg
    n_req = min(4, c.batch)
    ind = wl.page_indptr[: n_req + 1].copy()
    phys = wl.page_indices[: ind[-1]]
    uniq, inv = np.unique(phys, return_inverse=True)
    idx = inv.astype(np.int32)
    sel_t = torch.from_numpy(uniq.astype(np.int64)).to(layer.k.device)
    k = layer.k[sel_t].cpu()
    v = layer.v[sel_t].cpu() if layer.v is not None else None
    q = wl.q[:n_req].contiguous()
    lens = wl.seq_lens[:n_req].copy()
    bud = wl.pages_budget[:n_req].copy()
    H = c.num_kv_heads
    mean, mx, mn = O.summarize(k, c.page_size, ind, idx, lens, k_scale=c.k_scale)       # prefill, untimed
    first = (wl.pages[:n_req] - 1).astype(np.int32)

    def step():
        m2, x2, n2 = O.summarize(k, c.page_size, ind, idx, lens, first_page=first, k_scale=c.k_scale)
        sc = O.flow_scores(c.kind, q, H, c.page_size, ind, idx, lens, mean, mx, mn, head_dim_v=c.head_dim_v)
        sel, cnt, _, _ = O.select(sc, H, c.page_size, ind, lens, bud, c.n_sink, c.n_local, wl.max_sel)
        return O.attend(q, k, v, c.page_size, ind, idx, lens, sel, cnt, c.sm_scale, c.head_dim_v,
                        k_scale=c.k_scale, v_scale=c.v_scale)

    def timed(budget_s):
        reps, t0 = 0, time.perf_counter()
        while True:
            step()
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s:
                return reps, el

    threads = O.num_threads()
    reps, el = timed(target_s)
    O.set_num_threads(1)
    reps1, el1 = timed(one_core_s)
    O.set_num_threads(threads)
    return {"value": n_req * reps / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "one_core": {"value": n_req * reps1 / el1, "unit": "tokens/s", "cores": 1,
                         "sample": f"{reps1} repetitions in {el1:.1f} s"},
            "sample": f"first {n_req} of {c.batch} requests of the same workload, full decode step "
                      f"(incremental summary + score + select + attention; the token's K/V row copy is left "
                      f"out), {reps} repetitions in {el:.1f} s on {threads} threads"}


def read_ceiling(dev: str, gib: float = 4.0, reps: int = 5, workgroups: int = 4096) -> dict:
    """The device's practical streaming-read rate: vx_stream_read (16-byte non-temporal loads,
    the decode kernels' load form) over a buffer far larger than the Infinity Cache, best of
    `reps`, timed with fence-free HIP events.  A context figure beside the nameplate peak, not
    the roofline's peak."""
    buf = torch.empty(int(gib * (1 << 30)), dtype=torch.uint8, device=dev).fill_(1)
    sink = torch.zeros(workgroups, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    best = 0.0
    for _ in range(reps):
        e0, e1 = HipEvent(), HipEvent()
        e0.record(stream)
        vx.stream_read(buf, sink)
        e1.record(stream)
        torch.cuda.synchronize()
        best = max(best, buf.numel() / (e0.elapsed_ms(e1) * 1e-3) / 1e9)
    del buf, sink
    return {"GB/s": best, "method": f"vx_stream_read over a {gib:g} GiB buffer, {workgroups} workgroups, "
                                     f"best of {reps}"}


def topk_study(args) -> None:
    """The approximate radix top-k against the exact select (Sec. 5.2; Appendix D study):
    seeded fp32 score rows of four shapes, (candidates, k) cells, 128 rows per call.  For each
    cell: the exact select's time and every approximate variant's time and mean recall@k
    against the exact selection; the fastest variant with recall >= 0.97 is reported.  Times
    are per call, averaged over 50 calls that run back to back on the GPU."""
    dev = "cuda"
    stream = torch.cuda.current_stream()
    H, B = 8, 16
    taus = [0.02, 0.05, 0.1, 0.2, 0.3]
    reps = 50
    # a few milliseconds of matrix products queued ahead of the timed calls: the host enqueues
    # all of them while the GPU is still busy, so the events see the kernels back to back
    # rather than the host's per-call marshalling
    ma = torch.randn(8192, 8192, device=dev, dtype=torch.bfloat16)
    mc = torch.empty_like(ma)

    def timed(sc, n, bud, k, tau, remap, sel, cnt):
        for _ in range(5):
            vx.topk_select(sc, n, bud, 0, 0, k, sel, cnt, tolerate_ratio=tau, seed=17, remap=remap)
        e0, e1 = HipEvent(), HipEvent()
        for _ in range(4):
            torch.mm(ma, ma, out=mc)
        e0.record(stream)
        for _ in range(reps):
            vx.topk_select(sc, n, bud, 0, 0, k, sel, cnt, tolerate_ratio=tau, seed=17, remap=remap)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_ms(e1) / reps * 1e3

    rows = []
    for dist in ("bimodal", "normal", "lognormal", "uniform"):
        for P in (2048, 8192):
            for k in (128, 512):
                sc = torch.from_numpy(W.synthetic_scores(dist, H, B, P, seed=P + k)).to(dev)
                n = torch.full((B,), P, dtype=torch.int32, device=dev)
                bud = torch.full((B,), k, dtype=torch.int32, device=dev)
                sel = torch.empty((B, H, k), dtype=torch.int32, device=dev)
                cnt = torch.empty((B,), dtype=torch.int32, device=dev)
                t_exact = timed(sc, n, bud, k, 0.0, 0, sel, cnt)
                exact = sel.cpu().numpy().copy()
                cell = {"dist": dist, "candidates": P, "k": k, "exact_us": t_exact, "variants": []}
                for remap in (0, 1):
                    for tau in [0.0] + taus:
                        if tau == 0.0 and remap == 0:
                            continue
                        t = timed(sc, n, bud, k, tau, remap, sel, cnt)
                        got = sel.cpu().numpy()
                        rec = float(np.mean([len(np.intersect1d(got[i, h], exact[i, h])) / k
                                             for i in range(B) for h in range(H)]))
                        cell["variants"].append({"tau": tau, "remap": remap, "us": t, "recall": rec})
                ok = [v for v in cell["variants"] if v["recall"] >= 0.97]
                best = min(ok, key=lambda v: v["us"]) if ok else None
                cell["best_at_recall_0.97"] = best
                cell["speedup"] = t_exact / best["us"] if best else None
                rows.append(cell)
                print(f"[topk] {dist:9s} P={P:5d} k={k:4d} exact {t_exact:6.2f} us  best "
                      f"{best['us'] if best else float('nan'):6.2f} us (tau {best['tau'] if best else '-'}, "
                      f"remap {best['remap'] if best else '-'}, recall {best['recall'] if best else float('nan'):.3f})",
                      file=sys.stderr, flush=True)
    sp = [r["speedup"] for r in rows if r["speedup"]]
    print(json.dumps({"topk_study": rows, "mean_speedup_at_recall_0.97": float(np.mean(sp)) if sp else None,
                      "rows_per_call": H * B}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=240)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="llama3_8b_layer", choices=W.CONFIG_ORDER)
    ap.add_argument("--layers", type=int, default=3)
    ap.add_argument("--kind", default=None, choices=sorted(W.KIND_NAMES.values()),
                    help="score the workload with this flow instead of its own (block mean, Quest, Max, the "
                         "envelope flows, the rope-unaware MLA score, NSA, positional smoothing)")
    ap.add_argument("--kv-dtype", default="bf16", choices=W.KV_DTYPES,
                    help="KV cache element type (fp8: per-tensor scales, values = scale * code)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--block-size", type=int, default=0,
                    help="summary / selection block in tokens below the page size (0: one block per page); "
                         "budget, sink and local pages keep their token counts")
    ap.add_argument("--cache-stage", default="fused", choices=("fused", "append", "summarize"),
                    help="append: the fused KV append + summary refresh; summarize: the summary refresh only")
    ap.add_argument("--decode-event-every", type=int, default=1,
                    help="bracket the decode call with HIP events on every n-th timed step")
    ap.add_argument("--graph", action="store_true",
                    help="replay each layer's step from captured HIP graphs instead of eager launches")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (to scale HBM byte counters)")
    ap.add_argument("--topk-study", action="store_true",
                    help="only run the approximate radix top-k study against the exact select")
    ap.add_argument("--tau", type=float, default=0.0,
                    help="approximate radix top-k in the indexer step (Sec. 5.2): tolerate ratio")
    ap.add_argument("--remap", type=int, default=0, choices=(0, 1),
                    help="approximate radix top-k: key remap (1: affine over the candidates' range)")
    ap.add_argument("--topk-seed", type=int, default=1, help="approximate radix top-k: seed of the sample")
    ap.add_argument("--block-mean-scoring", default="auto", choices=("auto", "one-pass", "two-pass"),
                    help="block mean: the fp32 Mean in one pass, or a bf16 bound pass and re-scoring "
                         "(auto: by the batch's size)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the per-workload decode measurement (decode_by_workload)")
    ap.add_argument("--sweep-steps", type=int, default=40)
    ap.add_argument("--sweep-warmup", type=int, default=10)
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU's share of the path only; --gpus must be 1 "
              "(the path shards by request and KV head with no exchange, see DESIGN.md)", file=sys.stderr)
        sys.exit(2)
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.topk_study:
        topk_study(args)
        return
    if args.copy_calibration:
        n = 1 << 30
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty(n, dtype=torch.uint8, device=dev)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_per_copy": n, "copies": 5}), flush=True)
        return
    cfg = W.CONFIGS[args.config].with_kv_dtype(args.kv_dtype)
    if args.kind is not None:
        cfg = cfg.replace(kind={v: k for k, v in W.KIND_NAMES.items()}[args.kind])
    m = measure(cfg, args, dev, args.steps, args.warmup, graph=args.graph)
    layers = m.pop("layers")

    res = {
        "metric": METRIC, "value": cfg.batch / (m["ms_step"] * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": m["ms_step"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.kv_dtype, "data": "synthetic",
        "config": {"workload": describe(cfg), "batch": cfg.batch, "layers_rotated": args.layers,
                   "launch": "hip_graph" if args.graph else "eager", "kv_cache": cfg.kv_dtype,
                   "cache_stage": args.cache_stage, "block_size": layers[0].bs,
                   "block_mean_scoring": "two-pass" if layers[0].dec.mean_bf16 is not None else "one-pass"},
        "stages_ms": {**({"append_score_topk": m["stage_ms"][1]} if args.cache_stage == "fused" else
                         {("kv_append_summarize" if args.cache_stage == "append" else "summarize_incremental"):
                          m["stage_ms"][0], "score_topk": m["stage_ms"][1]}), "decode": m["stage_ms"][2],
                      "note": "separate untimed pass with an event between stages"},
        "roofline": {"bound": "hbm", "achieved": m["achieved"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": m["achieved"] / HBM_PEAK_GBS,
                     "traffic": counted_decode_traffic(cfg.name if cfg.kv_dtype == "bf16" else
                                                       f"{cfg.name}_{cfg.kv_dtype}"),
                     "kernel": "vx_sparse_paged_decode (the split kernel; for MLA plus the merge kernel)",
                     "event_steps": m["event_steps"], "decode_call_ms": m["decode_call_ms"],
                     "algorithmic_bytes_per_launch": m["bytes_avg"]},
    }
    res["roofline"]["practical_read_ceiling"] = read_ceiling(dev)
    res["roofline"]["frac_of_practical_ceiling"] = m["achieved"] / res["roofline"]["practical_read_ceiling"]["GB/s"]
    if not args.no_cpu_baseline and layers[0].r == 1:      # the baseline step is the page-granular one
        print("[bench] timing the CPU oracle baseline", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(layers[0])
    del layers
    if m["recall"] is not None:
        res["approx_topk"] = {"tolerate_ratio": args.tau, "remap": args.remap, "seed": args.topk_seed,
                              "recall_at_k": m["recall"]}
    if not args.no_sweep and args.kind is None and args.block_size == 0 and not args.graph and m["recall"] is None:
        res["decode_by_workload"] = decode_sweep(cfg, m, args, dev)
    print(json.dumps(res), flush=True)


def measure(cfg: W.Config, args, dev: str, steps: int, warmup: int, graph: bool = False) -> dict:
    """`warmup` untimed steps, then `steps` timed ones over `args.layers` rotating layer caches;
    the decode call of every `--decode-event-every`-th timed step is bracketed by HIP events on
    its stream."""
    wl0 = W.make(cfg)
    print(f"[bench] generating {args.layers} layer(s) of {describe(cfg)}", file=sys.stderr, flush=True)
    opt = approx_options(args)
    two_pass = {"auto": None, "one-pass": False, "two-pass": True}[args.block_mean_scoring]
    layers = [Layer(wl0.layer(l), dev, args.block_size, opt, two_pass) for l in range(args.layers)]
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def cache_call(L: Layer):
        if args.cache_stage == "append":
            L.dec.append(L.k_new, L.v_new)
        else:
            L.dec.summarize(L.first)

    def select_call(L: Layer):
        if args.cache_stage == "fused":
            L.dec.append_select(L.k_new, L.v_new, L.q, L.budget)
            return
        cache_call(L)
        L.dec.select(L.q, L.budget)

    def decode_call(L: Layer):
        L.dec.decode(L.q)

    # one eager step per layer (first use of every kernel), then capture the two graphs
    for L in layers:
        select_call(L)
        decode_call(L)
    torch.cuda.synchronize()
    graphs = None
    if graph:
        graphs = []
        for L in layers:
            gs, gd = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
            with torch.cuda.graph(gs):
                select_call(L)
            with torch.cuda.graph(gd):
                decode_call(L)
            graphs.append((gs, gd))
        torch.cuda.synchronize()

    def run_step(s: int, ev=None):
        li = s % len(layers)
        if graphs is None:
            select_call(layers[li])
        else:
            graphs[li][0].replay()
        if ev is not None:
            ev[0].record(stream)
        if graphs is None:
            decode_call(layers[li])
        else:
            graphs[li][1].replay()
        if ev is not None:
            ev[1].record(stream)

    def stage_times(n: int) -> np.ndarray:
        """Per-stage times (ms) over n untimed eager steps, with an event between every stage.  A
        spin kernel runs first, so that the host has queued every stage before the GPU reaches
        it and no interval holds host launch time."""
        ev = [[HipEvent() for _ in range(4)] for _ in range(n)]
        torch.cuda._sleep(5_000_000)
        for s in range(n):
            L = layers[s % len(layers)]
            ev[s][0].record(stream)
            if args.cache_stage != "fused":
                cache_call(L)
            ev[s][1].record(stream)
            if args.cache_stage == "fused":
                L.dec.append_select(L.k_new, L.v_new, L.q, L.budget)
            else:
                L.dec.select(L.q, L.budget)
            ev[s][2].record(stream)
            L.dec.decode(L.q)
            ev[s][3].record(stream)
        torch.cuda.synchronize()
        return np.array([[e[0].elapsed_ms(e[1]), e[1].elapsed_ms(e[2]), e[2].elapsed_ms(e[3])] for e in ev])

    for s in range(warmup):
        run_step(s)
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({warmup} steps, {'eager' if graphs is None else 'HIP graphs'})",
          file=sys.stderr, flush=True)

    every = max(1, args.decode_event_every)
    events = [[HipEvent(), HipEvent()] if s % every == 0 else None for s in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        run_step(s, events[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / steps
    dec_ms = np.array([e[0].elapsed_ms(e[1]) for e in events if e is not None])
    t_dec = float(dec_ms.mean())
    stage_ms = stage_times(min(steps, 20))     # breakdown only, after the timed region

    dec_bytes = [algorithmic_decode_bytes(L) for L in layers]
    bytes_avg = float(np.mean([dec_bytes[s % len(layers)] for s in range(steps) if events[s] is not None]))
    achieved = bytes_avg / (t_dec * 1e-3) / 1e9
    print(f"[bench] {cfg.name}: step {ms_step:.4f} ms; decode {t_dec:.4f} ms ({achieved:.0f} GB/s); stage "
          f"breakdown (ms) {args.cache_stage} {stage_ms[:, 0].mean():.4f} "
          f"{'append+score_topk' if args.cache_stage == 'fused' else 'score_topk'} {stage_ms[:, 1].mean():.4f} "
          f"decode {stage_ms[:, 2].mean():.4f}", file=sys.stderr, flush=True)
    recall = approx_recall(layers[0]) if opt is not None else None
    return {"ms_step": ms_step, "achieved": achieved, "bytes_avg": bytes_avg, "t_dec": t_dec, "recall": recall,
            "event_steps": sum(e is not None for e in events),
            "decode_call_ms": {"mean": t_dec, "p10": float(np.percentile(dec_ms, 10)),
                               "p50": float(np.percentile(dec_ms, 50)), "p90": float(np.percentile(dec_ms, 90))},
            "stage_ms": [float(stage_ms[:, k].mean()) for k in range(3)], "layers": layers}


def approx_options(args):
    """The approximate radix top-k options of the indexer step (None: exact)."""
    if args.tau == 0.0 and args.remap == 0:
        return None
    return vx.topk_options(tolerate_ratio=args.tau, seed=args.topk_seed, remap=args.remap)


def approx_recall(L: Layer) -> float:
    """recall@k of the layer's approximate selection against the exact selection of the same
    step (forced pages excluded): |approx & exact| / |exact| over the chosen candidates."""
    c = L.wl.cfg
    exact = SparseDecoder(L.kv, L.batch, c.num_q_heads, c.kind, L.dec.n_sink, L.dec.n_local, L.dec.max_sel,
                          c.sm_scale)
    exact.summarize()
    exact.select(L.q, L.budget)
    L.dec.select(L.q, L.budget)
    torch.cuda.synchronize()
    a, e = L.dec.sel_pages.cpu().numpy(), exact.sel_pages.cpu().numpy()
    cnt = exact.sel_count.cpu().numpy()
    hit = tot = 0
    for i in range(a.shape[0]):
        P = int(L.wl.pages[i]) * L.r
        forced = set(range(min(L.dec.n_sink, P))) | set(range(max(0, P - L.dec.n_local), P))
        for h in range(a.shape[1]):
            ex = set(e[i, h, : cnt[i]].tolist()) - forced
            hit += len(ex & set(a[i, h, : cnt[i]].tolist()))
            tot += len(ex)
    return hit / tot if tot else 1.0


def decode_sweep(main_cfg: W.Config, main: dict, args, dev: str) -> dict:
    """The decode call's HBM rate on every workload (the same protocol, fewer steps), so that one
    default run records the fraction of peak on each.  The first workload reuses the main run."""
    out = {}
    for name in W.CONFIG_ORDER:
        cfg = W.CONFIGS[name].with_kv_dtype(main_cfg.kv_dtype)
        if cfg.name == main_cfg.name and cfg.kv_dtype == main_cfg.kv_dtype:
            m = main
        else:
            m = measure(cfg, args, dev, args.sweep_steps, args.sweep_warmup)
            del m["layers"]
            torch.cuda.empty_cache()
        out[name] = {"kv_cache": cfg.kv_dtype, "decode_call_us": m["t_dec"] * 1e3,
                     "decode_call_us_p50": m["decode_call_ms"]["p50"] * 1e3,
                     "algorithmic_bytes": m["bytes_avg"], "achieved_GBps": m["achieved"],
                     "frac": m["achieved"] / HBM_PEAK_GBS, "step_ms": m["ms_step"],
                     "tokens_per_s": cfg.batch / (m["ms_step"] * 1e-3),
                     "steps": m["event_steps"]}
    return out


if __name__ == "__main__":
    main()
