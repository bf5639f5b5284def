"""Benchmark: causal top-k sparse GQA prefill on one MI355X.

Default workload "headline_32k": S=32768, Hq=32, Hkv=8, d=128, d_idx=128,
top-k 2048, bf16, seeded synthetic inputs with 128 planted needles. One step
runs every stage of the path once, on one HIP stream, with inputs resident
in HBM:

  1. indexer mode, 64-query selection blocks: scores -> top-k -> sparse attn
  2. indexer mode, per-query selection:       scores -> top-k -> sparse attn,
     and the fused scores+top-k that never stores the S x S scores
  3. dense causal GQA attention (the library's own dense kernel)
  4. oracle mode, per-query: dense normalisers -> mass -> top-k -> sparse attn
  5. the indexer's KL distillation objective and gradient, with the oracle
     mass rows of (4) as teacher and the per-query scores of (2) as student
  0. (first) the indexer front end: projection of d_model=4096 hidden states,
     key LayerNorm and RoPE (random weights)
  and, beside (1), the same sparse attention reading K/V from a paged cache

`value` is the ms per layer of (1), the selection-block-shared sparse prefill;
the per-query and oracle-mode times, the dense time and the speedups are
reported beside it.

--workload picks another of the paper-shaped workloads, each with its own
selection and modes (one JSON line each; --workload all runs every one):

  oracle_tiny_512  fp32 oracle mode, per query, k=64 (value: oracle mode)
  indexer_4k       indexer per query, k=512, unfused and fused (value: unfused)
  block_16k        64-query blocks, k=2048, 128-token forced window, summed
                   (value) and max-aggregated scores
  stress_100k      102,400 tokens, 128-query blocks, k=4096, planted (value)
                   and untrained indexer vectors

Every stage is bracketed by HIP events on the launch stream; per-stage times
are medians over the timed steps, roofline figures use the mean launch time.
Prints one JSON line per workload. Only one GPU is used: --gpus above 1 exits.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

from paper_2606_07703_amd.traffic import stage_counters, stage_traffic  # noqa: E402

PROFILES = os.path.join(ROOT, "profiles")
TRAFFIC_SUMMARY = os.path.join(PROFILES, "traffic_headline_32k.md")
MFMA_SUMMARY = os.path.join(PROFILES, "mfma_headline_32k.md")
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
FP32_VALU_PEAK_TFLOPS = 157.3
METRIC = "ms/layer sparse GQA prefill @32K, speedup vs own dense, % HBM/MFMA roofline"
ALL_WORKLOADS = ("oracle_tiny_512", "indexer_4k", "block_16k", "headline_32k", "stress_100k",
                 "head256_32k")


def causal_pairs(S: int) -> int:
    return S * (S + 1) // 2


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="headline_32k",
                    help="one of " + ", ".join(ALL_WORKLOADS) + ", or all")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="rough CPU time per oracle leg (bounded samples)")
    ap.add_argument("--summary-out", default=None,
                    help="also write a Markdown table of the workloads' lines to this file")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run one device copy of this size (the calibration "
                         "kernel for rocprofv3 FETCH_SIZE/WRITE_SIZE runs)")
    return ap.parse_args()


def causal_support_pairs(idx: np.ndarray, S: int, b: int) -> np.ndarray:
    """Per selection block r: sum over its queries t of |{s in idx[r] : 0 <= s <= t}|."""
    R = idx.shape[0]
    out = np.zeros(R, dtype=np.int64)
    for r in range(R):
        row = np.sort(idx[r][idx[r] >= 0])
        t0, t1 = r * b, min(r * b + b, S) - 1
        out[r] = int(np.searchsorted(row, np.arange(t0, t1 + 1), side="right").sum())
    return out


class Plan:
    """Stages of one workload's step, their algorithmic work and the modes
    (sums of stages) reported as ms/layer."""

    def __init__(self, w):
        self.w = w
        self.stages = []       # (name, fn)
        self.work = {}         # name -> (bound, flops or None, bytes or None) (filled after timing)
        self.modes = {}        # mode -> [stage names]
        self.value_mode = None
        self.tables = {}       # stage prefix -> (idx tensor, b)
        self.extra = {}

    def add(self, name, fn):
        self.stages.append((name, fn))


def build_plan(w, dev, B, PL, make_inputs, make_projection_inputs):
    S, Hq, Hkv, d, di, k = w.seq_len, w.num_q_heads, w.num_kv_heads, w.head_dim, w.index_dim, w.topk
    plan = Plan(w)

    def indexer_mode(prefix, b, agg="max", W=0, q_idx=None, k_idx=None, fused=False,
                     paged=False):
        p = B.Problem(S, Hq, Hkv, d, index_dim=di, topk=k, block_q=b, local_window=W, agg=agg,
                      dtype=w.dtype)
        buf = PL.Buffers.for_problem(p)
        qi = dev.q_idx if q_idx is None else q_idx
        ki = dev.k_idx if k_idx is None else k_idx
        plan.add(f"{prefix}.indexer_scores", lambda: B.sp_indexer_scores(p, qi, ki, buf.scores))
        plan.add(f"{prefix}.topk", lambda: B.sp_topk_select(p, buf.scores, buf.idx))
        plan.add(f"{prefix}.sparse_attn",
                 lambda: B.sp_sparse_gqa_attn(p, dev.q, dev.k, dev.v, buf.idx, buf.o))
        plan.modes[prefix] = [f"{prefix}.indexer_scores", f"{prefix}.topk", f"{prefix}.sparse_attn"]
        plan.tables[prefix] = (buf, b)
        if paged:
            # the same K/V scattered over a paged cache of 64-token pages
            # (every logical page at a shuffled physical page, plus spares)
            PAGE = 64
            npg = (S + PAGE - 1) // PAGE
            perm = torch.from_numpy(
                np.random.default_rng(w.seed).permutation(npg + 8)[:npg].astype(np.int32))
            pad = npg * PAGE - S
            kk = torch.cat([dev.k, dev.k.new_zeros(pad, Hkv, d)]) if pad else dev.k
            vv = torch.cat([dev.v, dev.v.new_zeros(pad, Hkv, d)]) if pad else dev.v
            kpg = torch.zeros(npg + 8, PAGE, Hkv, d, dtype=dev.k.dtype, device="cuda")
            vpg = torch.zeros_like(kpg)
            kpg[perm.long().cuda()] = kk.view(npg, PAGE, Hkv, d)
            vpg[perm.long().cuda()] = vv.view(npg, PAGE, Hkv, d)
            ptab = perm.cuda()
            o_paged = torch.empty_like(dev.q)
            plan.add(f"{prefix}.sparse_attn_paged", lambda: B.sp_sparse_gqa_attn_paged(
                p, dev.q, kpg, vpg, ptab, buf.idx, o_paged))
        if fused:
            fz_idx = torch.empty(S, k, dtype=torch.int32, device="cuda")
            fz_ws = torch.empty(B.sp_workspace_bytes(p, "indexer_topk"), dtype=torch.uint8,
                                device="cuda")
            plan.add(f"{prefix}.fused_scores_topk",
                     lambda: B.sp_indexer_topk(p, qi, ki, fz_idx, fz_ws))
            plan.modes[prefix + "_fused"] = [f"{prefix}.fused_scores_topk", f"{prefix}.sparse_attn"]
        return p, buf

    def oracle_mode():
        p = B.Problem(S, Hq, Hkv, d, topk=k, block_q=1, dtype=w.dtype)
        buf = PL.Buffers.for_problem(p, oracle=True)
        plan.add("oracle.normalisers",
                 lambda: B.sp_dense_attn(p, dev.q, dev.k, dev.v, None, buf.lse))
        plan.add("oracle.mass", lambda: B.sp_oracle_support(p, dev.q, dev.k, buf.lse, buf.scores))
        plan.add("oracle.topk", lambda: B.sp_topk_select(p, buf.scores, buf.idx))
        plan.add("oracle.sparse_attn",
                 lambda: B.sp_sparse_gqa_attn(p, dev.q, dev.k, dev.v, buf.idx, buf.o))
        plan.modes["oracle"] = ["oracle.normalisers", "oracle.mass", "oracle.topk",
                                "oracle.sparse_attn"]
        plan.tables["oracle"] = (buf, 1)
        return p, buf

    def dense():
        p = B.Problem(S, Hq, Hkv, d, dtype=w.dtype)
        o = torch.empty(S, Hq, d, dtype=dev.q.dtype, device="cuda")
        plan.add("dense.attn", lambda: B.sp_dense_attn(p, dev.q, dev.k, dev.v, o, None))
        plan.modes["dense"] = ["dense.attn"]

    if w.name == "headline_32k":
        # indexer front end on Qwen-like hidden states (d_model 4096, random weights)
        D_MODEL = 4096
        pb0 = B.Problem(S, Hq, Hkv, d, index_dim=di, topk=k, block_q=64, dtype=w.dtype)
        px, pwq, pwk, pg, pbeta = (t.cuda() for t in make_projection_inputs(S, D_MODEL, di,
                                                                           seed=w.seed))
        pqo = torch.empty(S, di, dtype=torch.bfloat16, device="cuda")
        pko = torch.empty(S, di, dtype=torch.bfloat16, device="cuda")
        plan.add("frontend.project",
                 lambda: B.sp_indexer_project(pb0, px, pwq, pwk, pg, pbeta, pqo, pko))
        plan.extra["d_model"] = D_MODEL
        indexer_mode("block64", 64, paged=True)
        pq, buf_q = indexer_mode("perquery", 1, fused=True)
        dense()
        _, buf_o = oracle_mode()
        # KL distillation objective: teacher = oracle mass rows, student =
        # per-query indexer scores, every query row supervised
        kl_rows = torch.arange(S, dtype=torch.int32, device="cuda")
        kl_val = torch.empty(S, device="cuda")
        kl_loss = torch.empty(1, device="cuda")
        kl_grad = torch.empty(S, S, device="cuda")
        plan.add("kl.loss", lambda: B.sp_kl_loss(pq, kl_rows, buf_o.scores, buf_q.scores, kl_val,
                                                 kl_loss, kl_grad))
        plan.value_mode = "block64"
    elif w.name == "oracle_tiny_512":
        oracle_mode()
        dense()
        plan.value_mode = "oracle"
    elif w.name == "indexer_4k":
        indexer_mode("perquery", 1, fused=True)
        dense()
        plan.value_mode = "perquery"
    elif w.name == "block_16k":
        indexer_mode("block64sum", 64, agg="sum", W=w.local_window)
        indexer_mode("block64max", 64, agg="max", W=w.local_window)
        dense()
        plan.value_mode = "block64sum"
    elif w.name == "head256_32k":
        indexer_mode("block64", 64, paged=True)
        dense()
        plan.value_mode = "block64"
    elif w.name == "stress_100k":
        b = w.block_q[0]
        indexer_mode(f"block{b}", b)
        # untrained indexer: the same draws without the needles planted in
        # k_idx (i.i.d. Gaussian vectors, uncorrelated with K)
        un = make_inputs(S, Hq, Hkv, d, index_dim=di, dtype=w.dtype, needles=w.needles,
                         stratified=w.stratified, seed=w.seed, untrained=True)
        uq, uk = un.q_idx.cuda(), un.k_idx.cuda()
        plan.extra["untrained"] = (un.q_idx, un.k_idx)
        indexer_mode(f"untrained{b}", b, q_idx=uq, k_idx=uk)
        dense()
        plan.value_mode = f"block{b}"
    else:
        raise SystemExit(f"no bench plan for workload {w.name}")
    return plan


def work_model(plan, S, Hq, Hkv, d, di, k, elt):
    """Algorithmic work per launch of each stage: (bound, flops, bytes). Counts
    causal pairs and selected rows only, never the work the method avoids."""
    C = causal_pairs(S)
    work, counts = {}, {}
    for name, _ in plan.stages:
        prefix, stage = name.split(".", 1)
        if stage == "project":
            dm = plan.extra["d_model"]
            work[name] = ("hbm", 2.0 * S * dm * 2 * di,
                          2.0 * (S * dm + 2 * di * dm + 2 * S * di) + 8.0 * di)
        elif stage == "attn" and prefix == "dense":
            work[name] = ("mfma" if elt == 2 else "alu", 4.0 * d * Hq * C, None)
        elif stage == "normalisers":
            work[name] = ("mfma" if elt == 2 else "alu", 2.0 * d * Hq * C, None)
        elif stage == "mass":
            work[name] = ("mfma" if elt == 2 else "alu", 2.0 * d * Hq * C, 4.0 * C)
        elif stage in ("indexer_scores", "topk", "sparse_attn", "sparse_attn_paged",
                       "fused_scores_topk"):
            buf, b = plan.tables[prefix]
            R = (S + b - 1) // b
            lens = np.minimum(np.arange(R) * b + b, S).astype(np.float64)
            if stage == "indexer_scores":
                if b == 1:
                    work[name] = ("hbm", 2.0 * di * C, 4.0 * C + 2.0 * S * di * elt)
                else:
                    work[name] = ("mfma", 2.0 * di * C, None)
            elif stage == "topk":
                work[name] = ("hbm", None, 4.0 * lens.sum() + 4.0 * R * k)
            elif stage == "fused_scores_topk":
                # one scoring of every causal pair (the passes recompute it;
                # that is overhead, not work)
                work[name] = ("mfma", 2.0 * di * C, 2.0 * S * di * elt + 4.0 * S * k)
            else:
                if prefix not in counts:
                    idx_np = buf.idx.cpu().numpy()
                    counts[prefix] = (int((idx_np >= 0).sum()),
                                      causal_support_pairs(idx_np, S, b), idx_np.size)
                rows, pairs, nidx = counts[prefix]
                gather = rows * Hkv * 2 * d * elt      # K and V rows of every KV head
                qo = 2 * S * Hq * d * elt
                work[name] = ("hbm", 4.0 * d * Hq * pairs.sum(), gather + qo + 4.0 * nidx)
        elif stage == "loss":
            # read P and z on s <= t, write the full gradient rows
            work[name] = ("hbm", None, 2 * 4.0 * C + 4.0 * S * S + 8.0 * S)
        else:
            raise KeyError(name)
    return work, counts


def run_workload(args, name):
    from paper_2606_07703_amd import binding as B
    from paper_2606_07703_amd import pipeline as PL
    from synth import get_workload, make_inputs, make_projection_inputs

    w = get_workload(name)
    S, Hq, Hkv, d, di, k = w.seq_len, w.num_q_heads, w.num_kv_heads, w.head_dim, w.index_dim, w.topk
    torch.cuda.set_device(0)
    B.load()
    t_gen = time.time()
    inp = make_inputs(S, Hq, Hkv, d, index_dim=di, dtype=w.dtype, needles=w.needles,
                      stratified=w.stratified, seed=w.seed)
    dev = inp.to("cuda")
    print(f"[bench] {name}: inputs ready in {time.time() - t_gen:.1f}s", file=sys.stderr,
          flush=True)
    plan = build_plan(w, dev, B, PL, make_inputs, make_projection_inputs)
    stream = torch.cuda.current_stream()
    stages = plan.stages

    def step(events=None):
        for i, (_, fn) in enumerate(stages):
            if events is not None:
                events[i].record(stream)
            fn()
        if events is not None:
            events[-1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] {name}: warmup done", file=sys.stderr, flush=True)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3
    per_stage = {nm: [evs[s][i].elapsed_time(evs[s][i + 1]) for s in range(args.steps)]
                 for i, (nm, _) in enumerate(stages)}
    med = {n: float(np.median(v)) for n, v in per_stage.items()}
    mean = {n: float(np.mean(v)) for n, v in per_stage.items()}
    print(f"[bench] {name}: timed steps done", file=sys.stderr, flush=True)
    if args.copy_mib > 0:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    elt = 2 if w.dtype == "bf16" else 4
    work, counts = work_model(plan, S, Hq, Hkv, d, di, k, elt)
    headline = name == "headline_32k"
    kernels = {}
    for st, (bound, flops, nbytes) in work.items():
        ms = mean[st]
        ent = {"ms_median": round(med[st], 4), "ms_mean": round(ms, 4), "bound": bound}
        if flops is not None:
            ent["tflops"] = round(flops / (ms * 1e-3) / 1e12, 2)
            if elt == 2:
                ent["frac_mfma_bf16"] = round(ent["tflops"] / BF16_PEAK_TFLOPS, 4)
            else:
                ent["frac_valu_fp32"] = round(ent["tflops"] / FP32_VALU_PEAK_TFLOPS, 4)
        if nbytes is not None:
            ent["gbs"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
            if ent["gbs"] <= HBM_PEAK_GBS:
                ent["frac_hbm"] = round(ent["gbs"] / HBM_PEAK_GBS, 4)
            else:
                # gathered rows served from L2 and the Infinity Cache: the
                # algorithmic byte rate is a gather rate, not an HBM fraction
                ent["gather_gbs_above_hbm_peak"] = True
        if headline:
            tb = stage_traffic(TRAFFIC_SUMMARY, st)
            if tb is not None:
                # DRAM bytes from the counters
                ent["traffic_gb"] = round(tb / 1e9, 3)
                ent["dram_gbs"] = round(tb / (ms * 1e-3) / 1e9, 1)
                ent["frac_dram"] = round(ent["dram_gbs"] / HBM_PEAK_GBS, 4)
            mc = stage_counters(MFMA_SUMMARY, st)
            if mc is not None:
                # matrix-core busy cycles per SIMD over the launch, from the
                # committed counter run: at the running clock, and at the
                # published peak's 2.4 GHz
                ent["mfma_busy"] = round(mc["mfma_busy"], 4)
                ent["mfma_busy_vs_2p4ghz"] = round(mc["mfma_busy_peak"], 4)
                ent["clock_ghz"] = round(mc["clock_ghz"], 3)
        kernels[st] = ent

    modes = {m: round(sum(med[s] for s in sts), 4) for m, sts in plan.modes.items()}
    value_ms = modes[plan.value_mode]
    dense_ms = modes["dense"]
    # roofline of the dominant kernel of the measured mode
    dom = max(plan.modes[plan.value_mode], key=lambda n: mean[n])
    bound, flops, nbytes = work[dom]
    ms_dom = mean[dom]
    if bound == "mfma":
        roof = {"bound": "mfma", "achieved": round(flops / (ms_dom * 1e-3) / 1e12, 2),
                "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    elif bound == "alu":
        roof = {"bound": "alu", "achieved": round(flops / (ms_dom * 1e-3) / 1e12, 3),
                "peak": FP32_VALU_PEAK_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(nbytes / (ms_dom * 1e-3) / 1e9, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    # HBM bytes per launch from the committed rocprofv3 counter runs, only while
    # the kernel's sources are unchanged since they were taken
    roof["traffic"] = stage_traffic(TRAFFIC_SUMMARY, dom) if headline else None
    roof["kernel"] = dom
    roof["launch_ms"] = round(ms_dom, 4)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(plan, inp, counts, args.cpu_seconds)

    b_val = plan.tables[plan.value_mode][1] if plan.value_mode in plan.tables else 1
    cfg = {"workload": w.name, "seq_len": S, "num_q_heads": Hq, "num_kv_heads": Hkv,
           "head_dim": d, "index_dim": di, "topk": k, "block_q": b_val,
           "local_window": w.local_window, "selection": plan.value_mode}
    out = {
        "metric": METRIC,
        "value": value_ms,
        "unit": "ms/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms / args.steps, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded Gaussian Q/K/V and indexer vectors, planted needles)",
        "config": cfg,
        "speedup_vs_dense": round(dense_ms / value_ms, 3),
        "dense_ms": dense_ms,
        "modes_ms_per_layer": modes,
        "mode_speedups_vs_dense": {m: round(dense_ms / v, 3) for m, v in modes.items()
                                   if m != "dense"},
        "roofline": roof,
        "kernels": kernels,
        "cpu_baseline": cpu,
        "paper_context": {"ttft_speedup_npu_qwen3.5_0.8b_256k": 1.71,
                          "ttft_speedup_gpu80g_qwen3.5_9b_256k": 1.93},
    }
    if headline:
        # names kept from earlier bench lines
        out["per_query_ms_per_layer"] = modes["perquery"]
        out["per_query_speedup_vs_dense"] = round(dense_ms / modes["perquery"], 3)
        out["per_query_fused_ms_per_layer"] = modes["perquery_fused"]
        out["oracle_mode_ms_per_layer"] = modes["oracle"]
    print(json.dumps(out), flush=True)
    del plan, dev, inp
    torch.cuda.empty_cache()
    return out


def cpu_model() -> str:
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for ln in out.splitlines():
            if ln.strip().startswith("Model name:"):
                return ln.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _spread(n_total, n, include=()):
    return np.unique(np.concatenate([np.linspace(0, n_total - 1, n).round().astype(int),
                                     np.asarray(include, dtype=int)]))


def cpu_baseline(plan, inp, counts, seconds):
    """The fp64 oracle on the host, timed on bounded samples of the workload.

    Legs: the measured mode (indexer scores, top-k, restricted attention, or
    the oracle mode for the tiny workload), dense attention, and oracle mode
    where the workload runs it. Each stage runs on evenly spaced selection
    blocks (query rows for dense), and its time is scaled to the whole layer
    by that stage's own work: causal length for scoring, mass and top-k,
    causal pairs for dense, and kept (query, key) pairs for restricted
    attention (counted on the GPU's support tables, which hold the same
    number of pairs per block as a correct selection).
    """
    import oracle
    w = plan.w
    S, k = w.seq_len, w.topk
    q64, k64, v64 = oracle._f64(inp.q), oracle._f64(inp.k), oracle._f64(inp.v)
    oracle._load()
    legs = {}

    def timed(fn):
        t0 = time.perf_counter()
        r = fn()
        return r, time.perf_counter() - t0

    def run_units(mode, units, b, agg, W, qi, ki, R):
        if mode == "indexer":
            Y, t_sc = timed(lambda: oracle.support_scores("indexer", units, b, q_idx=qi, k_idx=ki,
                                                          agg=agg))
        else:
            Y, t_sc = timed(lambda: oracle.support_scores("oracle", units, b, q=q64, k=k64))
        sel, t_tk = timed(lambda: oracle.select(Y, units, b, S, k, W))
        table = np.full((R, k), -1, dtype=np.int32)
        table[units] = sel
        rows = np.concatenate([np.arange(u * b, min(u * b + b, S)) for u in units])
        _, t_sp = timed(lambda: oracle.sparse(q64, k64, v64, table, b, rows=rows))
        return table, t_sc, t_tk, t_sp

    def selection_leg(mode, prefix, b, agg="max", W=0, qi=None, ki=None):
        R = (S + b - 1) // b
        L = np.minimum(np.arange(R) * b + b, S).astype(np.float64)
        # sample size: time two blocks from the middle of the sequence, then
        # take as many evenly spaced blocks as fill about `seconds`
        probe = np.array([R // 2, min(R - 1, R // 2 + 1)])
        _, a, c, e = run_units(mode, probe, b, agg, W, qi, ki, R)
        per_unit = (a + c + e) / len(probe) * L.mean() / L[probe].mean()
        n = int(max(4, min(R, seconds / max(per_unit, 1e-9))))
        units = _spread(R, n)
        table, t_sc, t_tk, t_sp = run_units(mode, units, b, agg, W, qi, ki, R)
        # kept pairs of the sampled blocks under the oracle's own selection
        pairs_s = 0
        for u in units:
            srt = np.sort(table[u][table[u] >= 0])
            ts = np.arange(u * b, min(u * b + b, S))
            pairs_s += int(np.searchsorted(srt, ts, side="right").sum())
        pairs_all = counts[prefix][1].sum() if prefix in counts else pairs_s * R / len(units)
        scale_L = L.sum() / L[units].sum()
        ms = 1e3 * ((t_sc + t_tk) * scale_L + t_sp * pairs_all / max(pairs_s, 1))
        legs[prefix] = {"ms_per_layer": round(ms, 1),
                        "sample": f"{len(units)} of {R} {b}-query blocks",
                        "measured_s": round(t_sc + t_tk + t_sp, 2)}
        return ms

    def dense_leg():
        probe = np.array([S // 2, S // 2 + 1]) if S > 2 else np.arange(S)
        _, t = timed(lambda: oracle.dense(q64, k64, v64, rows=probe))
        per_row = t / len(probe) * (S / 2) / max(float(probe.mean()) + 1, 1.0)
        n = int(max(4, min(S, seconds / max(per_row, 1e-9))))
        rows = _spread(S, n, include=[S - 1])
        _, t = timed(lambda: oracle.dense(q64, k64, v64, rows=rows))
        scale = (S * (S + 1) / 2) / float((rows + 1).sum())
        legs["dense"] = {"ms_per_layer": round(1e3 * t * scale, 1),
                         "sample": f"{len(rows)} of {S} query rows", "measured_s": round(t, 2)}

    vm = plan.value_mode
    if vm == "oracle":
        selection_leg("oracle", "oracle", 1)
    else:
        buf, b = plan.tables[vm]
        agg = "sum" if vm.endswith("sum") else "max"
        if vm.startswith("untrained"):
            qi, ki = (oracle._f64(t) for t in plan.extra["untrained"])
        else:
            qi, ki = oracle._f64(inp.q_idx), oracle._f64(inp.k_idx)
        W = w.local_window if vm.startswith("block64") and w.name == "block_16k" else 0
        selection_leg("indexer", vm, b, agg=agg, W=W, qi=qi, ki=ki)
        if "oracle" in plan.modes:
            selection_leg("oracle", "oracle", 1)
    dense_leg()
    main = legs[vm]
    return {"value": main["ms_per_layer"], "unit": "ms/layer", "cores": oracle.num_threads(),
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{main['sample']} ({vm} mode), {main['measured_s']} s measured, each "
                      "stage scaled by its own work (causal length for scores and top-k, "
                      "kept pairs for restricted attention)",
            "legs": legs}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the path shards by selection blocks, see the design notes)", file=sys.stderr)
        sys.exit(2)
    names = ALL_WORKLOADS if args.workload == "all" else (args.workload,)
    lines = [run_workload(args, n) for n in names]
    if args.summary_out:
        write_summary(args, lines)


def write_summary(args, lines):
    """Markdown table of the workloads' bench lines (modes, rooflines, CPU legs)."""
    cmd = "python3 -u bench.py --workload " + args.workload + \
        f" --steps {args.steps} --warmup {args.warmup}" + \
        (" --no-cpu-baseline" if args.no_cpu_baseline else "")
    L = ["# Bench lines of every workload", "", "Command (repository root, one MI355X):", "",
         "    " + cmd, "",
         "ms/layer are medians of the timed steps (HIP events on the launch stream); the "
         "roofline fraction is the dominant kernel of the measured mode; CPU legs are the fp64 "
         "oracle on bounded samples of the same workload, scaled to a layer.", "",
         "| workload | measured mode | ms/layer | dense ms | speedup | other modes (ms/layer) "
         "| dominant kernel: roofline | CPU oracle ms/layer (cores) |",
         "|---|---|---:|---:|---:|---|---|---|"]
    for d in lines:
        cfg = d["config"]
        others = ", ".join(f"{m} {v}" for m, v in d["modes_ms_per_layer"].items()
                           if m not in (cfg["selection"], "dense"))
        r = d["roofline"]
        cpu = d["cpu_baseline"]
        cpu_s = "—" if not cpu else (f"{cpu['value']} ({cpu['cores']}); " + ", ".join(
            f"{k} {v['ms_per_layer']}" for k, v in cpu["legs"].items()))
        L.append(f"| {cfg['workload']} (S={cfg['seq_len']}, d={cfg['head_dim']}, b={cfg['block_q']}, "
                 f"k={cfg['topk']}) "
                 f"| {cfg['selection']} | {d['value']} | {d['dense_ms']} | {d['speedup_vs_dense']} "
                 f"| {others or '—'} | {r['kernel']}: {r['frac']} of {r['peak']} {r['unit']} "
                 f"| {cpu_s} |")
    L.append("")
    L.append("Per-kernel figures (ms median, roofline fractions) are in each line's `kernels` "
             "object; the CPU host was " + (lines[0]["cpu_baseline"] or {}).get("cpu_model", "—")
             + ".")
    open(args.summary_out, "w").write("\n".join(L) + "\n")


if __name__ == "__main__":
    main()
