"""HBM traffic per kernel launch from rocprofv3 counter runs.

Two `rocprofv3 --pmc` runs of the same bench command, one collecting
FETCH_SIZE and one WRITE_SIZE (KiB per dispatch, summed over the L2
channels), give the bytes each launch moves between L2 and memory. Each
counter is scaled by what it reads for a plain device copy of known size run
in the same process (`bench.py --copy-mib N`): factor = true bytes / counted
bytes, so a read of B bytes reports as B.

The summary is a Markdown file under profiles/ holding, per bench stage, the
raw counts, the scaled bytes per launch, and a digest of the sources the
stage's kernel is built from. bench.py reports a stage's traffic only while
that digest still matches the tree (a changed kernel reports null).

    python -m paper_2606_07703_amd.traffic \\
        --fetch DIR --write DIR --copy-mib 1024 --out profiles/traffic_....md \\
        --cmd-fetch "..." --cmd-write "..."
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import os
import re
from typing import Dict, List, Optional

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")

# bench stage -> HIP source of the kernel it launches
STAGE_KERNEL_FILE = {
    "frontend.project": "indexer_project.hip",
    "block64.indexer_scores": "indexer_mfma.hip",
    "block64.topk": "topk.hip",
    "block64.sparse_attn": "sparse_block_mfma.hip",
    "block64.sparse_attn_paged": "sparse_block_mfma.hip",
    "perquery.indexer_scores": "indexer_mfma.hip",
    "perquery.topk": "topk.hip",
    "perquery.sparse_attn": "sparse_query_mfma.hip",
    "perquery.fused_scores_topk": "indexer_topk.hip",
    "dense.attn": "dense_mfma.hip",
    "oracle.normalisers": "dense_mfma.hip",
    "oracle.mass": "mass_mfma.hip",
    "oracle.topk": "topk.hip",
    "oracle.sparse_attn": "sparse_query_mfma.hip",
    "kl.loss": "kl_loss.hip",
}
STAGES = list(STAGE_KERNEL_FILE)
# kernel launches per stage when not one (per-row KL, then the mean)
STAGE_DISPATCHES = {"kl.loss": 2, "perquery.fused_scores_topk": 10}

# kernels of the library (everything else in a trace is torch or the runtime)
LIB_KERNEL_RE = re.compile(r"sp::|_ZN2sp")
COPY_KERNEL_RE = re.compile(r"copy|elementwise", re.I)


def kernel_sources(hip_file: str) -> List[str]:
    """The kernel's source and every local header it includes (recursively),
    plus the dispatch layer and the build flags, as paths relative to ROOT."""
    seen: List[str] = []
    todo = [os.path.join(CSRC, hip_file)]
    while todo:
        f = todo.pop()
        if f in seen or not os.path.exists(f):
            continue
        seen.append(f)
        for m in re.finditer(r'^#include "([^"]+)"', open(f).read(), re.M):
            todo.append(os.path.join(os.path.dirname(f), m.group(1)))
    seen += [os.path.join(CSRC, "api.cpp"), os.path.join(PKG, "build.py")]
    return sorted(os.path.relpath(f, ROOT) for f in seen)


def sources_digest(files: List[str]) -> str:
    h = hashlib.sha256()
    for f in files:
        h.update(f.encode())
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()[:16]


def read_dispatches(run_dir: str, counter: str) -> List[Dict]:
    """[{id, name, value}] in dispatch order for one counter (KiB)."""
    paths = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not paths:
        raise FileNotFoundError(f"no counter_collection.csv under {run_dir}")
    per: Dict[int, Dict] = {}
    for p in paths:
        for r in csv.DictReader(open(p)):
            if r["Counter_Name"] != counter:
                continue
            did = int(r["Dispatch_Id"])
            e = per.setdefault(did, {"id": did, "name": r["Kernel_Name"], "value": 0.0})
            e["value"] += float(r["Counter_Value"])
    return [per[k] for k in sorted(per)]


def summarize(fetch_dir: str, write_dir: str, copy_bytes: int) -> Dict:
    out = {"copy_bytes": copy_bytes, "stages": {}}
    for counter, run_dir, key in (("FETCH_SIZE", fetch_dir, "fetch"),
                                  ("WRITE_SIZE", write_dir, "write")):
        ds = read_dispatches(run_dir, counter)
        lib = [d for d in ds if LIB_KERNEL_RE.search(d["name"])]
        copies = [d for d in ds if not LIB_KERNEL_RE.search(d["name"])
                  and COPY_KERNEL_RE.search(d["name"])]
        per_step = sum(STAGE_DISPATCHES.get(st, 1) for st in STAGES)
        if len(lib) % per_step:
            raise ValueError(f"{counter}: {len(lib)} library dispatches is not a whole number "
                             f"of {per_step}-dispatch steps")
        if not copies:
            raise ValueError(f"{counter}: no copy dispatch for calibration")
        # the calibration copy is the largest copy dispatch
        cal_kib = max(d["value"] for d in copies)
        factor = copy_bytes / (cal_kib * 1024.0)
        out[f"{key}_copy_kib"] = cal_kib
        out[f"{key}_factor"] = factor
        nsteps = len(lib) // per_step
        first = 0
        for st in STAGES:
            nd = STAGE_DISPATCHES.get(st, 1)
            vals = [sum(lib[s * per_step + first + x]["value"] for x in range(nd))
                    for s in range(nsteps)]
            kib = sum(vals) / len(vals)
            e = out["stages"].setdefault(st, {"kernel": _short(lib[first]["name"])})
            e[f"{key}_kib"] = kib
            e[f"{key}_bytes"] = kib * 1024.0 * factor
            first += nd
    for st, e in out["stages"].items():
        e["traffic_bytes"] = e["fetch_bytes"] + e["write_bytes"]
        files = kernel_sources(STAGE_KERNEL_FILE[st])
        e["sources"] = files
        e["digest"] = sources_digest(files)
    return out


def _short(name: str) -> str:
    m = re.search(r"(\w+_kernel)(<[^()]*>)?", name)
    return (m.group(1) + (m.group(2) or "")) if m else name[:80]


def write_md(path: str, s: Dict, cmd_fetch: str, cmd_write: str, parse_cmd: str) -> None:
    L = ["# HBM traffic per launch: headline 32K workload, every bench stage", "",
         "L2 <-> memory bytes per kernel launch from two rocprofv3 counter runs of one",
         "bench step (FETCH_SIZE, then WRITE_SIZE), each scaled by the same counter on a",
         f"device copy of {s['copy_bytes']} bytes run in the same process.", "",
         "Commands (repository root, one MI355X):", "",
         "    " + cmd_fetch, "    " + cmd_write, "    " + parse_cmd, "",
         f"Calibration: FETCH_SIZE read {s['fetch_copy_kib']:.1f} KiB for the copy "
         f"(factor {s['fetch_factor']:.4f}); WRITE_SIZE read {s['write_copy_kib']:.1f} KiB "
         f"(factor {s['write_factor']:.4f}).", "",
         "| stage | kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | read bytes | written bytes "
         "| traffic bytes | digest |",
         "|---|---|---:|---:|---:|---:|---:|---|"]
    for st in STAGES:
        e = s["stages"][st]
        L.append(f"| {st} | `{e['kernel']}` | {e['fetch_kib']:.1f} | {e['write_kib']:.1f} | "
                 f"{e['fetch_bytes']:.4g} | {e['write_bytes']:.4g} | {e['traffic_bytes']:.4g} "
                 f"| {e['digest']} |")
    L += ["", "Digest = first 16 hex digits of sha256 over these sources (path, then bytes):", ""]
    for st in STAGES:
        L.append(f"- {st}: " + ", ".join(s["stages"][st]["sources"]))
    L.append("")
    L.append("<!-- machine-readable: stage traffic_bytes digest -->")
    for st in STAGES:
        e = s["stages"][st]
        L.append(f"<!-- traffic {st} {e['traffic_bytes']:.6e} {e['digest']} -->")
    open(path, "w").write("\n".join(L) + "\n")


def load_traffic(path: str) -> Dict[str, Dict]:
    """{stage: {"bytes": float, "digest": str, "current": bool}} from a summary file."""
    out: Dict[str, Dict] = {}
    if not os.path.exists(path):
        return out
    for m in re.finditer(r"<!-- traffic (\S+) (\S+) (\S+) -->", open(path).read()):
        st, nbytes, dig = m.group(1), float(m.group(2)), m.group(3)
        cur = st in STAGE_KERNEL_FILE and \
            sources_digest(kernel_sources(STAGE_KERNEL_FILE[st])) == dig
        out[st] = {"bytes": nbytes, "digest": dig, "current": cur}
    return out


def stage_traffic(path: str, stage: str) -> Optional[float]:
    e = load_traffic(path).get(stage)
    return e["bytes"] if e and e["current"] else None


# ------------------------------------------------------- matrix-core counters
# gfx950: 256 CUs of 4 SIMDs; GRBM counters are summed over the 8 XCDs.
N_SIMD = 1024
N_XCD = 8
PUBLISHED_CLOCK_GHZ = 2.4
MFMA_COUNTERS = ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE")


def read_dispatch_counters(run_dir: str) -> List[Dict]:
    """[{id, name, ns, counters{name: value}}] in dispatch order."""
    paths = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not paths:
        raise FileNotFoundError(f"no counter_collection.csv under {run_dir}")
    per: Dict[int, Dict] = {}
    for p in paths:
        for r in csv.DictReader(open(p)):
            did = int(r["Dispatch_Id"])
            e = per.setdefault(did, {"id": did, "name": r["Kernel_Name"], "counters": {},
                                     "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
            c = r["Counter_Name"]
            e["counters"][c] = e["counters"].get(c, 0.0) + float(r["Counter_Value"])
    return [per[k] for k in sorted(per)]


def summarize_mfma(run_dir: str) -> Dict:
    """Per bench stage (the first dispatch of the stage's kernels, averaged
    over steps): MFMA busy cycles per SIMD as a fraction of the launch's
    cycles at the running shader clock (GRBM_GUI_ACTIVE per XCD over the
    launch duration) and at the published peak's clock."""
    ds = [d for d in read_dispatch_counters(run_dir) if LIB_KERNEL_RE.search(d["name"])]
    per_step = sum(STAGE_DISPATCHES.get(st, 1) for st in STAGES)
    if len(ds) % per_step:
        raise ValueError(f"{len(ds)} library dispatches is not a whole number of "
                         f"{per_step}-dispatch steps")
    nsteps = len(ds) // per_step
    out = {"stages": {}}
    first = 0
    for st in STAGES:
        nd = STAGE_DISPATCHES.get(st, 1)
        busy = cyc = ns = sqb = 0.0
        for s in range(nsteps):
            for x in range(nd):
                d = ds[s * per_step + first + x]
                busy += d["counters"].get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
                cyc += d["counters"].get("GRBM_GUI_ACTIVE", 0.0) / N_XCD
                sqb += d["counters"].get("SQ_BUSY_CYCLES", 0.0)
                ns += d["ns"]
        files = kernel_sources(STAGE_KERNEL_FILE[st])
        out["stages"][st] = {
            "kernel": _short(ds[first]["name"]),
            "ms": ns / nsteps / 1e6,
            "clock_ghz": cyc / ns,
            "mfma_busy": busy / (N_SIMD * cyc) if cyc else 0.0,
            "mfma_busy_peak": busy / (N_SIMD * PUBLISHED_CLOCK_GHZ * ns) if ns else 0.0,
            "se_busy": sqb / (32 * cyc) if cyc else 0.0,
            "mfma_busy_cycles": busy / nsteps,
            "sources": files,
            "digest": sources_digest(files),
        }
        first += nd
    return out


def write_mfma_md(path: str, s: Dict, cmd: str, parse_cmd: str) -> None:
    L = ["# Matrix-core utilisation per launch: headline 32K workload, every bench stage", "",
         "One rocprofv3 counter run of one bench step. Per launch: SQ_VALU_MFMA_BUSY_CYCLES",
         f"(summed over the {N_SIMD} SIMDs), GRBM_GUI_ACTIVE (summed over the {N_XCD} XCDs) "
         "and SQ_BUSY_CYCLES",
         "(summed over the 32 shader engines), with the launch duration from the trace.", "",
         "* clock = GRBM_GUI_ACTIVE / 8 / duration (the shader clock under this load);",
         f"* MFMA busy = MFMA busy cycles / ({N_SIMD} x GRBM_GUI_ACTIVE / 8): the share of the "
         "launch's cycles the matrix cores are busy, at the running clock;",
         f"* vs peak = MFMA busy cycles / ({N_SIMD} x {PUBLISHED_CLOCK_GHZ} GHz x duration): "
         "the same against the published 2.5 PFLOP/s bf16 peak's clock;",
         "* SE busy = SQ_BUSY_CYCLES / (32 x GRBM_GUI_ACTIVE / 8): cycles in which a shader "
         "engine holds any wave.", "",
         "A 32x32x16 bf16 MFMA keeps a SIMD's matrix core busy 32 cycles (1024 FLOP per busy "
         "cycle).", "",
         "Commands (repository root, one MI355X):", "", "    " + cmd, "    " + parse_cmd, "",
         "| stage | kernel | ms | clock GHz | MFMA busy | vs peak | SE busy | digest |",
         "|---|---|---:|---:|---:|---:|---:|---|"]
    for st in STAGES:
        e = s["stages"][st]
        L.append(f"| {st} | `{e['kernel']}` | {e['ms']:.4f} | {e['clock_ghz']:.3f} | "
                 f"{100 * e['mfma_busy']:.1f}% | {100 * e['mfma_busy_peak']:.1f}% | "
                 f"{100 * e['se_busy']:.1f}% | {e['digest']} |")
    L += ["", "<!-- machine-readable: stage mfma_busy mfma_busy_peak clock_ghz digest -->"]
    for st in STAGES:
        e = s["stages"][st]
        L.append(f"<!-- mfma {st} {e['mfma_busy']:.6f} {e['mfma_busy_peak']:.6f} "
                 f"{e['clock_ghz']:.6f} {e['digest']} -->")
    open(path, "w").write("\n".join(L) + "\n")


def stage_counters(path: str, stage: str) -> Optional[Dict]:
    """{mfma_busy, mfma_busy_peak, clock_ghz} of a stage from a summary file,
    while the digest of the kernel's sources still matches the tree."""
    if not os.path.exists(path):
        return None
    for m in re.finditer(r"<!-- mfma (\S+) (\S+) (\S+) (\S+) (\S+) -->", open(path).read()):
        if m.group(1) != stage or stage not in STAGE_KERNEL_FILE:
            continue
        if sources_digest(kernel_sources(STAGE_KERNEL_FILE[stage])) != m.group(5):
            return None
        return {"mfma_busy": float(m.group(2)), "mfma_busy_peak": float(m.group(3)),
                "clock_ghz": float(m.group(4))}
    return None


# ------------------------------------------------------------ kernel times
def write_stats_md(path: str, stats_csv: str, bench_json: str, cmd: str) -> None:
    """Kernel-time summary of a rocprofv3 --kernel-trace --stats run of the
    bench, with the bench line of the same run for the roofline cross-check."""
    import json
    rows = list(csv.DictReader(open(stats_csv)))
    line = json.loads([ln for ln in open(bench_json) if ln.startswith("{")][-1])
    roof = line["roofline"]
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    L = ["# Kernel-time summary: headline 32K workload, every bench stage", "",
         "Workload: S=32768, Hq=32, Hkv=8, d=128, d_idx=128, top-k 2048, bf16 (bench.py's "
         "headline_32k step: front end, indexer mode with 64-query blocks (contiguous and "
         "paged K/V), per query (unfused and fused), dense, oracle mode and the KL "
         "objective).", "",
         "Command (repository root, one MI355X):", "", "    " + cmd, "",
         f"Roofline cross-check: the bench line of this run measured `{roof['kernel']}` with HIP "
         f"events at {roof['launch_ms']} ms per launch; its kernel's average below comes from "
         "the trace of the same launches (warmup included).", "",
         "| kernel | calls | avg ms | min ms | max ms | share of GPU time |",
         "|---|---:|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = _short(r["Name"]) if "sp::" in r["Name"] else r["Name"].split("(")[0][:60]
        L.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.4f} | "
                 f"{float(r['MinNs']) / 1e6:.4f} | {float(r['MaxNs']) / 1e6:.4f} | "
                 f"{100 * float(r['TotalDurationNs']) / total:.2f}% |")
    open(path, "w").write("\n".join(L) + "\n")


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--fetch", help="rocprofv3 output dir of the FETCH_SIZE run")
    ap.add_argument("--write", help="rocprofv3 output dir of the WRITE_SIZE run")
    ap.add_argument("--copy-mib", type=int)
    ap.add_argument("--out", required=True)
    ap.add_argument("--cmd-fetch")
    ap.add_argument("--cmd-write")
    ap.add_argument("--mfma", help="rocprofv3 output dir of the matrix-core counter run "
                                   "(writes the utilisation summary instead)")
    ap.add_argument("--cmd-mfma")
    ap.add_argument("--stats", help="kernel_stats.csv of a --kernel-trace --stats run "
                                    "(writes the kernel-time summary instead)")
    ap.add_argument("--bench-json", help="the bench line of that run")
    ap.add_argument("--cmd-stats")
    a = ap.parse_args(argv)
    if a.stats:
        write_stats_md(a.out, a.stats, a.bench_json, a.cmd_stats or "")
        return
    if a.mfma:
        s = summarize_mfma(a.mfma)
        parse_cmd = (f"python3 -m paper_2606_07703_amd.traffic --mfma {a.mfma} --out {a.out} "
                     "--cmd-mfma '...'")
        write_mfma_md(a.out, s, a.cmd_mfma or "", parse_cmd)
        for st in STAGES:
            e = s["stages"][st]
            print(f"{st:26s} {e['ms']:8.4f} ms  MFMA busy {100 * e['mfma_busy']:5.1f}%  "
                  f"vs peak {100 * e['mfma_busy_peak']:5.1f}%  clock {e['clock_ghz']:.3f}")
        return
    s = summarize(a.fetch, a.write, a.copy_mib << 20)
    parse_cmd = (f"python3 -m paper_2606_07703_amd.traffic --fetch {a.fetch} --write {a.write} "
                 f"--copy-mib {a.copy_mib} --out {a.out} --cmd-fetch '...' --cmd-write '...'")
    write_md(a.out, s, a.cmd_fetch, a.cmd_write, parse_cmd)
    for st in STAGES:
        e = s["stages"][st]
        print(f"{st:26s} {e['traffic_bytes'] / 1e9:10.3f} GB  {e['kernel']}")


if __name__ == "__main__":
    main()
