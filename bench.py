"""Benchmark of the shifted non-local search path on one MI355X.

One step = snls_search (fused search + top-k) followed by snls_aggregate on
the 480 x 854 denoising workload (B=1, T=5, C=64, ws=9, wt=2, ps=7,
S_Q=1, inner product, k=10, softmax scale 1), inputs resident in HBM.
Prints one JSON line (see the design doc for the counting rules).

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
PEAK_FP32_VALU = 157.3e12  # MI355X fp32 vector peak (packed FMA), FLOP/s
PEAK_FP32_VALU_UNPACKED = 78.6e12  # 256 CUs x 4 SIMDs x 16 lanes x 2 flop x 2.4 GHz, unpacked FMA
PEAK_HBM = 8.0e12          # MI355X HBM3E, B/s


def frames_in_window(p):
    return sum(min(p["T"] - 1, t + p["wt"]) - max(0, t - p["wt"]) + 1 for t in range(p["T"]))


def work_counts(p):
    """Algorithmic work of one step: queries, candidates, flops, bytes."""
    nH, nW = (p["H"] - 1) // p["stride0"] + 1, (p["W"] - 1) // p["stride0"] + 1
    Ch = p["C"] // p["HD"]
    n_q = p["B"] * p["T"] * nH * nW
    n_cand = p["B"] * p["HD"] * nH * nW * p["ws"] ** 2 * frames_in_window(p)
    f_search = n_cand * p["ps"] ** 2 * Ch * (2 if p["dist_type"] == 0 else 3)
    f_agg = n_q * p["HD"] * p["k"] * p["ps"] ** 2 * Ch * 2
    vid = p["B"] * p["T"] * p["C"] * p["H"] * p["W"] * 4
    q_bytes = vid if p["ps"] > 1 or p["stride0"] == 1 else p["B"] * p["T"] * p["C"] * nH * nW * 4
    flow_bytes = p["B"] * p["T"] * 2 * p["wt"] * 2 * nH * nW * 4
    kept = n_q * p["HD"] * p["k"] * 16
    search_bytes = q_bytes + vid + flow_bytes + kept
    agg_bytes = vid + vid + kept
    return dict(queries=n_q, candidates=n_cand, f_search=f_search, f_agg=f_agg,
                bytes_total=q_bytes + 2 * vid + flow_bytes + vid + kept, search_bytes=search_bytes,
                agg_bytes=agg_bytes)


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2309_16849_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def measured_counters():
    """Counter record of one snls_search call (HBM bytes, fp32 FMA
    instructions) from the committed rocprofv3 summary, or None when missing
    or taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", "search_denoise480x854_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    return rec


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "search_denoise480x854_traffic.json")
# the two kernels of one snls_search call on this workload: scores, then top-k
SEARCH_KERNELS = ("search_tile_scores_kernel", "tile_topk_kernel")
COPY_KERNEL_HINT = "mulfunctor"  # torch.mul(src, 1, out=dst): one read and one write per element


def _read_csv(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def _find(dirpath, suffix):
    for root, _, files in os.walk(dirpath):
        for fn in files:
            if fn.endswith(suffix):
                return os.path.join(root, fn)
    raise FileNotFoundError("%s*%s" % (dirpath, suffix))


def summarize_profiles(outdir, copy_mib):
    """Turn the rocprofv3 outputs of the profiling commands (kernel trace,
    FETCH_SIZE pass, WRITE_SIZE pass, counter passes) into the summaries kept
    under profiles/.  HBM traffic per search launch = counter KiB scaled by
    what the same counter reads for a plain copy of copy_mib MiB."""
    import collections
    cmd = ("cd /tmp && rocprofv3 {opts} --output-format csv -d $R/gpurun_out/{d} -o run -- "
           "python3 $R/bench.py --steps {s} --warmup {w} --no-cpu-baseline --copy-probe-mib %d" % copy_mib)
    lines = ["# rocprofv3 summary: 480x854 denoising workload (search + top-k + aggregation)", "",
             "Commands (R = repository root on the GPU box):", ""]
    lines.append("    " + cmd.format(opts="--kernel-trace --stats", d="prof_trace", s=10, w=2))
    trace = _read_csv(_find(os.path.join(outdir, "prof_trace"), "kernel_stats.csv"))
    lines += ["", "| kernel | calls | avg us | min us | max us | total % |", "|---|---|---|---|---|---|"]
    for r in trace:
        name = r["Name"]
        short = name.split("(")[0].replace("void ", "")[:70]
        lines.append("| %s | %s | %.1f | %.1f | %.1f | %.1f |" % (
            short, r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
            float(r["Percentage"])))
    counters = collections.defaultdict(dict)
    for d in sorted(os.listdir(outdir)):
        if not d.startswith("prof_pmc") or not os.path.isdir(os.path.join(outdir, d)):
            continue
        rows = _read_csv(_find(os.path.join(outdir, d), "counter_collection.csv"))
        names = sorted({r["Counter_Name"] for r in rows})
        lines += ["", "    " + cmd.format(opts="--pmc " + " ".join(names), d=d, s=2, w=1)]
        acc = collections.defaultdict(list)
        for r in rows:
            acc[(r["Kernel_Name"], r["Counter_Name"])].append(float(r["Counter_Value"]))
        for (kn, cn), v in acc.items():
            counters[kn][cn] = sum(v) / len(v)
    lines += ["", "Counters, mean per dispatch:", "", "| kernel | counter | value |", "|---|---|---|"]
    for kn in sorted(counters):
        for cn in sorted(counters[kn]):
            lines.append("| %s | %s | %.6g |" % (kn.split("(")[0].replace("void ", "")[:60], cn, counters[kn][cn]))
    search = [kn for kn in counters if any(sk in kn for sk in SEARCH_KERNELS)]
    copy = [kn for kn in counters if COPY_KERNEL_HINT in kn.lower() and "FETCH_SIZE" in counters[kn]]
    rec = None
    if search and copy and all("FETCH_SIZE" in counters[kn] and "WRITE_SIZE" in counters[kn] for kn in search):
        cpy = counters[copy[0]]
        exp_kib = copy_mib * 1024.0
        f_fetch = exp_kib / cpy["FETCH_SIZE"]
        f_write = exp_kib / cpy["WRITE_SIZE"]
        fetch_kib = sum(counters[kn]["FETCH_SIZE"] for kn in search)
        write_kib = sum(counters[kn]["WRITE_SIZE"] for kn in search)
        fetch_b = fetch_kib * f_fetch * 1024.0
        write_b = write_kib * f_write * 1024.0
        fma = sum(counters[kn].get("SQ_INSTS_VALU_FMA_F32", 0.0) for kn in search)
        rec = {"kernels": search, "kernel_source_hash": kernel_source_hash(), "copy_kernel": copy[0],
               "copy_mib": copy_mib, "copy_fetch_kib": cpy["FETCH_SIZE"], "copy_write_kib": cpy["WRITE_SIZE"],
               "fetch_scale": f_fetch, "write_scale": f_write, "search_fetch_kib": fetch_kib,
               "search_write_kib": write_kib, "fetch_bytes_per_launch": fetch_b,
               "write_bytes_per_launch": write_b, "bytes_per_launch": fetch_b + write_b,
               "fma_f32_wave_insts_per_launch": fma}
        with open(TRAFFIC_FILE, "w") as f:
            json.dump(rec, f, indent=1)
        lines += ["", "HBM traffic of one snls_search call (%s): FETCH %.1f MB + WRITE %.1f MB = %.1f MB "
                  "(counter KiB x %.3f / %.3f, from a %d MiB copy)." % (
                      " + ".join(k.split("(")[0].replace("void ", "") for k in search), fetch_b / 1e6,
                      write_b / 1e6, (fetch_b + write_b) / 1e6, f_fetch, f_write, copy_mib)]
    md = os.path.join(ROOT, "profiles", "search_denoise480x854_rocprofv3.md")
    with open(md, "w") as f:
        f.write("\n".join(lines) + "\n")
    return md, rec


def cpu_baseline(c, budget_s=12.0):
    """The oracle on the host cores: search + top-k + aggregation for a band of
    query rows of the middle frame, scaled to queries/s."""
    import oracle
    p, scale = c["params"], c["scale"]
    nH, nW = (p["H"] - 1) // p["stride0"] + 1, (p["W"] - 1) // p["stride0"] + 1
    x64 = c["q"].astype(np.float64)
    fl64 = c["flows"].astype(np.float64)
    t_mid = p["T"] // 2
    r0 = nH // 2

    def band(nrows):
        rows = np.array([(t_mid * nH + r0 + i) * nW + j for i in range(nrows) for j in range(nW)], np.int64)
        return rows

    def run(nrows):
        rows = band(nrows)
        t0 = time.perf_counter()
        res = oracle.search(x64, x64, fl64, p, qids=rows, extra=0)
        t1 = time.perf_counter()
        d = np.zeros((p["B"] * p["HD"] * p["T"] * nH * nW, p["k"]))
        ind = np.zeros(d.shape + (3,))
        d[rows] = res["dists"]
        ind[rows] = res["inds"]
        lo = p["ps"] // 2
        inner = range(r0 + lo, r0 + nrows - (p["ps"] - 1 - lo))
        pix = np.array([(t_mid * p["H"] + y) * p["W"] + x for y in inner for x in range(p["W"])], np.int64)
        shp = (p["B"], p["HD"], p["T"], nH, nW, p["k"])
        t2 = time.perf_counter()
        oracle.aggregate_at(x64, d.reshape(shp), ind.reshape(shp + (3,)), p, pix, scale)
        t3 = time.perf_counter()
        per_q = (t1 - t0) / len(rows) + (t3 - t2) / max(len(pix), 1)
        return per_q, len(rows), len(pix), (t1 - t0) + (t3 - t2)

    oracle.build()
    per_q, _, _, _ = run(8)  # pilot
    nrows = int(max(8, min(nH // 2 - 1, budget_s / (per_q * nW))))
    per_q, nq, npix, wall = run(nrows)
    cores = int(os.environ.get("OMP_NUM_THREADS", 0)) or len(os.sched_getaffinity(0))
    return {"value": 1.0 / per_q, "unit": "queries/s", "cores": cores, "kind": "oracle",
            "sample": "%d query rows x %d (%d queries) of frame %d for search+top-k, aggregation at the %d output "
                      "pixels those queries cover alone; %.1f s wall, fp64" % (nrows, nW, nq, t_mid, npix, wall)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", default="denoise480x854",
                    help="workload name (default: the 480x854 denoising workload; paper320_s1, paper320_s2 and "
                         "paper152_mem are the paper's own benchmark shapes)")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run one plain device copy of this size (calibrates the HBM byte counters)")
    ap.add_argument("--summarize-profiles", metavar="DIR", default=None,
                    help="write profiles/ summaries from the rocprofv3 outputs under DIR and exit")
    args = ap.parse_args()
    if args.summarize_profiles:
        md, rec = summarize_profiles(args.summarize_profiles, args.copy_probe_mib or 256)
        print(md)
        print(json.dumps(rec, indent=1))
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the path has no multi-GPU mode in this build "
              "(see DESIGN.md for how it would shard)", file=sys.stderr)
        sys.exit(2)

    import torch
    sys.path.insert(0, ROOT)
    from paper_2309_16849_amd import snls as B
    from workloads import config_index, make_config

    B.load_library()
    dev = torch.device("cuda:0")
    c = make_config(config_index(args.workload))
    p, scale = c["params"], c["scale"]
    x = torch.from_numpy(c["q"]).to(dev)
    fl = torch.from_numpy(c["flows"]).to(dev)
    shp = B.out_shape(p)
    dists = torch.empty(shp, device=dev)
    inds = torch.empty(shp + (3,), device=dev)
    out = torch.empty(B.video_shape(p), device=dev)
    ws = B.workspace_for(B.SNLS_OP_AGGREGATE, p, dev)
    sws = B.workspace_for(B.SNLS_OP_SEARCH, p, dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        B.snls_search(x, x, fl, p, dists, inds, sws)
        if ev is not None:
            ev[1].record()
        B.snls_aggregate(x, dists, inds, p, scale, out, ws)
        if ev is not None:
            ev[2].record()

    if args.copy_probe_mib:
        src = torch.empty(args.copy_probe_mib * (1 << 20) // 4, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1.0)
        torch.cuda.synchronize()
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats(dev)
    step()
    torch.cuda.synchronize()
    peak_mem = torch.cuda.max_memory_allocated(dev)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    t_search = float(np.mean([e[0].elapsed_time(e[1]) for e in evs])) * 1e-3
    t_agg = float(np.mean([e[1].elapsed_time(e[2]) for e in evs])) * 1e-3

    w = work_counts(p)
    ms = elapsed / args.steps * 1e3
    value = w["queries"] * args.steps / elapsed
    achieved = w["f_search"] / t_search
    rec = measured_counters()
    traffic = rec["bytes_per_launch"] if rec else None
    # fp32 multiply-adds the search kernels issue (rocprofv3 counter, 64 lanes
    # per wave instruction), against the unpacked fp32 VALU peak this build
    # can reach (packed fp32 instructions are disabled)
    issued = None
    if rec and rec.get("fma_f32_wave_insts_per_launch"):
        fl = rec["fma_f32_wave_insts_per_launch"] * 64 * 2
        issued = {"fma_flop_per_launch": fl, "tflops": fl / t_search / 1e12,
                  "peak_unpacked": PEAK_FP32_VALU_UNPACKED / 1e12,
                  "frac_unpacked": fl / t_search / PEAK_FP32_VALU_UNPACKED}
    line = {
        "metric": "queries/s (search+top-k+aggregate) and % fp32 VALU/HBM roofline, config 2",
        "value": value, "unit": "queries/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": c["name"], "B": p["B"], "T": p["T"], "C": p["C"], "H": p["H"], "W": p["W"],
                   "HD": p["HD"], "ws": p["ws"], "wt": p["wt"], "ps": p["ps"], "stride0": p["stride0"],
                   "stride1": p["stride1"], "k": p["k"], "dist": "inner_product" if p["dist_type"] == 0 else "squared_l2", "softmax_scale": scale,
                   "parallelism": "single_gpu"},
        "roofline": {"bound": "alu", "kernel": "snls_search (scores + top-k kernels)", "achieved": achieved / 1e12,
                     "peak": PEAK_FP32_VALU / 1e12, "unit": "TFLOP/s", "frac": achieved / PEAK_FP32_VALU,
                     "traffic": traffic, "issued": issued},
        "candidates_per_s": w["candidates"] * args.steps / elapsed,
        "step_alg_tflops": (w["f_search"] + w["f_agg"]) / (elapsed / args.steps) / 1e12,
        "step_frac_fp32_valu": (w["f_search"] + w["f_agg"]) / (elapsed / args.steps) / PEAK_FP32_VALU,
        "step_frac_hbm": w["bytes_total"] / (elapsed / args.steps) / PEAK_HBM,
        "search_ms": t_search * 1e3, "aggregate_ms": t_agg * 1e3,
        "peak_mem_gb": peak_mem / 1e9, "search_workspace_gb": sws.numel() * 4 / 1e9,
        "aggregate_alg_tflops": w["f_agg"] / t_agg / 1e12,
    }
    if not args.no_cpu_baseline and args.workload == "denoise480x854":
        line["cpu_baseline"] = cpu_baseline(c, args.cpu_budget)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
