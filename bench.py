"""Benchmark: causal top-k sparse GQA prefill at 32K on one MI355X.

Workload "headline_32k": S=32768, Hq=32, Hkv=8, d=128, d_idx=128, top-k 2048,
bf16, seeded synthetic inputs with 128 planted needles. One step runs every
stage of the path once, on one HIP stream, with inputs resident in HBM:

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
reported beside it. Every stage is bracketed by HIP events on the launch
stream; per-stage times are medians over the timed steps.

Prints one JSON line. Only one GPU is used: --gpus above 1 exits.
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

from paper_2606_07703_amd.traffic import stage_traffic  # noqa: E402

TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "traffic_headline_32k.md")
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
FP32_VALU_PEAK_TFLOPS = 157.3


def causal_pairs(S: int) -> int:
    return S * (S + 1) // 2


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="headline_32k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-units", type=int, default=256,
                    help="selection blocks the CPU oracle times (bounded sample)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run one device copy of this size (the calibration "
                         "kernel for rocprofv3 FETCH_SIZE/WRITE_SIZE runs)")
    return ap.parse_args()


def support_rows(idx: torch.Tensor) -> int:
    return int((idx >= 0).sum().item())


def causal_support_pairs(idx: np.ndarray, S: int, b: int) -> int:
    """Sum over queries t of |{s in idx[t//b] : 0 <= s <= t}|."""
    total = 0
    R, k = idx.shape
    for r in range(R):
        row = np.sort(idx[r][idx[r] >= 0])
        t0, t1 = r * b, min(r * b + b, S) - 1
        ts = np.arange(t0, t1 + 1)
        total += int(np.searchsorted(row, ts, side="right").sum())
    return total


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the path shards by selection blocks, see the design notes)", file=sys.stderr)
        sys.exit(2)
    from paper_2606_07703_amd import binding as B
    from paper_2606_07703_amd import pipeline as PL
    from synth import get_workload, make_inputs, make_projection_inputs

    w = get_workload(args.workload)
    S, Hq, Hkv, d, di, k = w.seq_len, w.num_q_heads, w.num_kv_heads, w.head_dim, w.index_dim, w.topk
    torch.cuda.set_device(0)
    B.load()
    t_gen = time.time()
    inp = make_inputs(S, Hq, Hkv, d, index_dim=di, dtype=w.dtype, needles=w.needles,
                      stratified=w.stratified, seed=w.seed)
    dev = inp.to("cuda")
    print(f"[bench] inputs ready in {time.time() - t_gen:.1f}s", file=sys.stderr, flush=True)

    pb = B.Problem(S, Hq, Hkv, d, index_dim=di, topk=k, block_q=64, dtype=w.dtype)
    pq = B.Problem(S, Hq, Hkv, d, index_dim=di, topk=k, block_q=1, dtype=w.dtype)
    buf_b = PL.Buffers.for_problem(pb)
    buf_q = PL.Buffers.for_problem(pq)
    buf_o = PL.Buffers.for_problem(pq, oracle=True)
    o_dense = torch.empty(S, Hq, d, dtype=dev.q.dtype, device="cuda")
    # KL distillation objective: teacher = oracle mass rows, student = per-query
    # indexer scores, every query row supervised
    kl_rows = torch.arange(S, dtype=torch.int32, device="cuda")
    kl_val = torch.empty(S, device="cuda")
    kl_loss = torch.empty(1, device="cuda")
    kl_grad = torch.empty(S, S, device="cuda")
    # the same K/V scattered over a paged cache of 64-token pages (every
    # logical page at a shuffled physical page, plus spare pages)
    PAGE = 64
    npg = (S + PAGE - 1) // PAGE
    perm = torch.from_numpy(np.random.default_rng(w.seed).permutation(npg + 8)[:npg].astype(np.int32))
    kpg = torch.zeros(npg + 8, PAGE, Hkv, d, dtype=dev.k.dtype, device="cuda")
    vpg = torch.zeros_like(kpg)
    kpg[perm.long().cuda()] = dev.k.view(npg, PAGE, Hkv, d)
    vpg[perm.long().cuda()] = dev.v.view(npg, PAGE, Hkv, d)
    ptab = perm.cuda()
    o_paged = torch.empty_like(dev.q)
    # fused per-query scoring + top-k (no S x S score buffer)
    fz_idx = torch.empty(S, k, dtype=torch.int32, device="cuda")
    fz_ws = torch.empty(B.sp_workspace_bytes(pq, "indexer_topk"), dtype=torch.uint8,
                        device="cuda")
    # indexer front end on Qwen-like hidden states (d_model 4096, random weights)
    D_MODEL = 4096
    px, pwq, pwk, pg, pb_ = (t.cuda() for t in make_projection_inputs(S, D_MODEL, di, seed=w.seed))
    pqo = torch.empty(S, di, dtype=torch.bfloat16, device="cuda")
    pko = torch.empty(S, di, dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()

    stages = [
        ("frontend.project", lambda: B.sp_indexer_project(pb, px, pwq, pwk, pg, pb_, pqo, pko)),
        ("block64.indexer_scores", lambda: B.sp_indexer_scores(pb, dev.q_idx, dev.k_idx, buf_b.scores)),
        ("block64.topk", lambda: B.sp_topk_select(pb, buf_b.scores, buf_b.idx)),
        ("block64.sparse_attn", lambda: B.sp_sparse_gqa_attn(pb, dev.q, dev.k, dev.v, buf_b.idx, buf_b.o)),
        ("block64.sparse_attn_paged", lambda: B.sp_sparse_gqa_attn_paged(
            pb, dev.q, kpg, vpg, ptab, buf_b.idx, o_paged)),
        ("perquery.indexer_scores", lambda: B.sp_indexer_scores(pq, dev.q_idx, dev.k_idx, buf_q.scores)),
        ("perquery.topk", lambda: B.sp_topk_select(pq, buf_q.scores, buf_q.idx)),
        ("perquery.sparse_attn", lambda: B.sp_sparse_gqa_attn(pq, dev.q, dev.k, dev.v, buf_q.idx, buf_q.o)),
        ("perquery.fused_scores_topk", lambda: B.sp_indexer_topk(pq, dev.q_idx, dev.k_idx, fz_idx,
                                                                 fz_ws)),
        ("dense.attn", lambda: B.sp_dense_attn(pq, dev.q, dev.k, dev.v, o_dense, None)),
        ("oracle.normalisers", lambda: B.sp_dense_attn(pq, dev.q, dev.k, dev.v, None, buf_o.lse)),
        ("oracle.mass", lambda: B.sp_oracle_support(pq, dev.q, dev.k, buf_o.lse, buf_o.scores)),
        ("oracle.topk", lambda: B.sp_topk_select(pq, buf_o.scores, buf_o.idx)),
        ("oracle.sparse_attn", lambda: B.sp_sparse_gqa_attn(pq, dev.q, dev.k, dev.v, buf_o.idx, buf_o.o)),
        ("kl.loss", lambda: B.sp_kl_loss(pq, kl_rows, buf_o.scores, buf_q.scores, kl_val, kl_loss,
                                         kl_grad)),
    ]

    def step(events=None):
        for i, (_, fn) in enumerate(stages):
            if events is not None:
                events[i].record(stream)
            fn()
        if events is not None:
            events[-1].record(stream)

    for i in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3
    per_stage = {name: [] for name, _ in stages}
    for s in range(args.steps):
        for i, (name, _) in enumerate(stages):
            per_stage[name].append(evs[s][i].elapsed_time(evs[s][i + 1]))
    med = {n: float(np.median(v)) for n, v in per_stage.items()}
    mean = {n: float(np.mean(v)) for n, v in per_stage.items()}
    print("[bench] timed steps done", file=sys.stderr, flush=True)
    if args.copy_mib > 0:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # ---------------------------------------------------------- algorithmic work
    C = causal_pairs(S)
    idx_b = buf_b.idx.cpu().numpy()
    idx_q = buf_q.idx.cpu().numpy()
    idx_o = buf_o.idx.cpu().numpy()
    elt = 2  # bf16

    def sparse_bytes(idx_np, b):
        rows = int((idx_np >= 0).sum())            # gathered support rows (per block or query)
        gather = rows * Hkv * 2 * d * elt            # K and V rows of every KV head
        qo = 2 * S * Hq * d * elt
        return gather + qo + idx_np.size * 4

    def sparse_flops(idx_np, b):
        return 4 * d * Hq * causal_support_pairs(idx_np, S, b)

    R_b = pb.num_blocks
    lens_b = np.array([min(r * 64 + 64, S) for r in range(R_b)])
    work = {
        "frontend.project": ("hbm", 2.0 * S * D_MODEL * 2 * di,
                             2.0 * (S * D_MODEL + 2 * di * D_MODEL + 2 * S * di) + 8.0 * di),
        "block64.indexer_scores": ("mfma", 2.0 * di * C, None),
        "block64.topk": ("hbm", None, 4.0 * lens_b.sum() + 4.0 * R_b * k),
        "block64.sparse_attn": ("hbm", sparse_flops(idx_b, 64), sparse_bytes(idx_b, 64)),
        "block64.sparse_attn_paged": ("hbm", sparse_flops(idx_b, 64), sparse_bytes(idx_b, 64)),
        "perquery.indexer_scores": ("hbm", 2.0 * di * C, 4.0 * C + 2.0 * S * di * elt),
        "perquery.topk": ("hbm", None, 4.0 * C + 4.0 * S * k),
        "perquery.sparse_attn": ("hbm", sparse_flops(idx_q, 1), sparse_bytes(idx_q, 1)),
        # algorithmic work of one scoring of every causal pair (the passes
        # recompute it; that is overhead, not work)
        "perquery.fused_scores_topk": ("mfma", 2.0 * di * C, 2.0 * S * di * elt + 4.0 * S * k),
        "dense.attn": ("mfma", 4.0 * d * Hq * C, None),
        "oracle.normalisers": ("mfma", 2.0 * d * Hq * C, None),
        "oracle.mass": ("mfma", 2.0 * d * Hq * C, 4.0 * C),
        "oracle.topk": ("hbm", None, 4.0 * C + 4.0 * S * k),
        "oracle.sparse_attn": ("hbm", sparse_flops(idx_o, 1), sparse_bytes(idx_o, 1)),
        # read P and z on s <= t, write the full gradient rows
        "kl.loss": ("hbm", None, 2 * 4.0 * C + 4.0 * S * S + 8.0 * S),
    }
    kernels = {}
    for name, (bound, flops, nbytes) in work.items():
        ms = mean[name]
        ent = {"ms_median": round(med[name], 4), "ms_mean": round(ms, 4), "bound": bound}
        if flops is not None:
            ent["tflops"] = round(flops / (ms * 1e-3) / 1e12, 2)
            ent["frac_mfma_bf16"] = round(ent["tflops"] / BF16_PEAK_TFLOPS, 4)
        if nbytes is not None:
            ent["gbs"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
            ent["frac_hbm"] = round(ent["gbs"] / HBM_PEAK_GBS, 4)
        tb = stage_traffic(TRAFFIC_SUMMARY, name)
        if tb is not None:
            # DRAM bytes from the counters: kernels whose gathers hit in L2 or the
            # Infinity Cache move far fewer bytes than the algorithmic count
            ent["traffic_gb"] = round(tb / 1e9, 3)
            ent["dram_gbs"] = round(tb / (ms * 1e-3) / 1e9, 1)
            ent["frac_dram"] = round(ent["dram_gbs"] / HBM_PEAK_GBS, 4)
        kernels[name] = ent

    block_ms = sum(med[n] for n in ("block64.indexer_scores", "block64.topk", "block64.sparse_attn"))
    pq_ms = sum(med[n] for n in ("perquery.indexer_scores", "perquery.topk", "perquery.sparse_attn"))
    pqf_ms = med["perquery.fused_scores_topk"] + med["perquery.sparse_attn"]
    or_ms = sum(med[n] for n in ("oracle.normalisers", "oracle.mass", "oracle.topk",
                                 "oracle.sparse_attn"))
    dense_ms = med["dense.attn"]

    # the roofline object covers the dominant kernel of the headline path (the
    # block-shared indexer mode that `value` times)
    headline = ("block64.indexer_scores", "block64.topk", "block64.sparse_attn")
    dom = max(headline, key=lambda n: mean[n])
    bound, flops, nbytes = work[dom]
    ms_dom = mean[dom]
    if bound == "mfma":
        roof = {"bound": "mfma", "achieved": round(flops / (ms_dom * 1e-3) / 1e12, 2),
                "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(nbytes / (ms_dom * 1e-3) / 1e9, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    # HBM bytes per launch from the committed rocprofv3 counter runs, only while
    # the kernel's sources are unchanged since they were taken
    roof["traffic"] = stage_traffic(TRAFFIC_SUMMARY, dom)
    roof["kernel"] = dom
    roof["launch_ms"] = round(ms_dom, 4)

    # ------------------------------------------------------------- CPU baseline
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(inp, S, Hq, d, k, args.cpu_units)

    out = {
        "metric": "ms/layer sparse GQA prefill @32K, speedup vs own dense, % HBM/MFMA roofline",
        "value": round(block_ms, 4),
        "unit": "ms/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms / args.steps, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Gaussian Q/K/V and indexer vectors, planted needles)",
        "config": {"workload": w.name, "seq_len": S, "num_q_heads": Hq, "num_kv_heads": Hkv,
                   "head_dim": d, "index_dim": di, "topk": k, "block_q": 64,
                   "selection": "indexer, 64-query blocks, max aggregation"},
        "speedup_vs_dense": round(dense_ms / block_ms, 3),
        "dense_ms": round(dense_ms, 4),
        "per_query_ms_per_layer": round(pq_ms, 4),
        "per_query_speedup_vs_dense": round(dense_ms / pq_ms, 3),
        "per_query_fused_ms_per_layer": round(pqf_ms, 4),
        "oracle_mode_ms_per_layer": round(or_ms, 4),
        "roofline": roof,
        "kernels": kernels,
        "cpu_baseline": cpu,
        "paper_context": {"ttft_speedup_npu_qwen3.5_0.8b_256k": 1.71,
                          "ttft_speedup_gpu80g_qwen3.5_9b_256k": 1.93},
    }
    print(json.dumps(out), flush=True)


def cpu_baseline(inp, S, Hq, d, k, n_units):
    """The fp64 oracle on the host, timed on a bounded sample of selection blocks.

    It runs the same three stages as `value` (indexer scores with 64-query
    max aggregation, top-k, restricted attention) for n_units blocks spread
    evenly over the sequence, and scales the time to the whole layer by the
    causal length of each block (the work of every stage grows with it).
    """
    import oracle
    b = 64
    R = (S + b - 1) // b
    units = np.unique(np.linspace(0, R - 1, n_units).round().astype(int))
    q64, k64, v64 = oracle._f64(inp.q), oracle._f64(inp.k), oracle._f64(inp.v)
    qi, ki = oracle._f64(inp.q_idx), oracle._f64(inp.k_idx)
    oracle._load()
    t0 = time.perf_counter()
    Y = oracle.support_scores("indexer", units, b, q_idx=qi, k_idx=ki, agg="max")
    sel = oracle.select(Y, units, b, S, k)
    table = np.full((R, k), -1, dtype=np.int32)
    table[units] = sel
    rows = np.concatenate([np.arange(u * b, min(u * b + b, S)) for u in units])
    oracle.sparse(q64, k64, v64, table, b, rows=rows)
    secs = time.perf_counter() - t0
    L = np.array([min(r * b + b, S) for r in range(R)], dtype=np.float64)
    scale = L.sum() / L[units].sum()
    ms_layer = secs * scale * 1e3
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": round(ms_layer, 1), "unit": "ms/layer", "cores": cores, "kind": "oracle",
            "sample": f"{len(units)} of {R} 64-query blocks (indexer scores, top-k, sparse "
                      f"attention), {secs:.1f}s measured, scaled by causal length"}


if __name__ == "__main__":
    main()
