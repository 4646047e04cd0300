"""Benchmark of the shifted non-local search path on one MI355X.

One step = snls_search (search + top-k) followed by snls_aggregate, plus
snls_backward for a workload with a training step, inputs resident in HBM.
The default workload is the 480 x 854 denoising video (B=1, T=5, C=64,
ws=9, wt=2, ps=7, S_Q=1, inner product, k=10, softmax scale 1).  Prints one
JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

Roofline of the search call (the dominant call of every forward workload):
  achieved  fp32 FLOP/s the call's kernels issue: the SQ_INSTS_VALU_FMA_F32
            count of one call (rocprofv3, committed under profiles/ for this
            workload and these kernel sources) x 64 lanes x 2 flop, divided by
            the call time measured live here with HIP events;
  frac      achieved / 157.3 TFLOP/s (MI355X fp32 vector peak, packed FMA);
  frac_attainable  achieved / 78.6 TFLOP/s (the unpacked fp32 ceiling: the
            library is built without packed fp32 instructions);
  alg_tflops / alg_frac  the direct count of the method (every candidate
            scored from its P x P x C_h patch) per call time; the kernels
            compute the same scores with far fewer multiply-adds, so this
            ratio can exceed 1 and is not a hardware fraction;
  traffic   HBM bytes of one call (FETCH_SIZE + WRITE_SIZE counters, scaled
            by what the same counters read for a plain device copy).
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2309_16849_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
PEAK_FP32_VALU = 157.3e12  # MI355X fp32 vector peak (packed FMA), FLOP/s
PEAK_FP32_VALU_UNPACKED = 78.6e12  # 256 CUs x 4 SIMDs x 16 lanes x 2 flop x 2.4 GHz, unpacked FMA
PEAK_HBM = 8.0e12          # MI355X HBM3E, B/s
DEFAULT_WORKLOAD = "denoise480x854"
METRIC = "queries/s (search+top-k+aggregate) and % fp32 VALU/HBM roofline, config 2"

# Kernels of each library call, by name (no kernel is shared between the
# search call and the others).
SEARCH_PAT = re.compile(r"(search_\w+|tile_topk_kernel|wave_topk_kernel|topk_kernel|l2_pair_planes_kernel|"
                        r"l2_norms_kernel)$")


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
    # backward through the k kept neighbours: dq and dk of each similarity,
    # dv and the weight gradient of each aggregated read (2 flop each)
    f_bwd = n_q * p["HD"] * p["k"] * p["ps"] ** 2 * Ch * 8
    vid = p["B"] * p["T"] * p["C"] * p["H"] * p["W"] * 4
    q_bytes = vid if p["ps"] > 1 or p["stride0"] == 1 else p["B"] * p["T"] * p["C"] * nH * nW * 4
    flow_bytes = p["B"] * p["T"] * 2 * p["wt"] * 2 * nH * nW * 4
    kept = n_q * p["HD"] * p["k"] * 16
    search_bytes = q_bytes + vid + flow_bytes + kept
    agg_bytes = vid + vid + kept
    # q, k, v, grad_out and the kept neighbours read; dq, dk, dv, dflows written
    bwd_bytes = 4 * vid + kept + 3 * vid + 2 * flow_bytes
    return dict(queries=n_q, candidates=n_cand, f_search=f_search, f_agg=f_agg, f_bwd=f_bwd,
                bytes_total=q_bytes + 2 * vid + flow_bytes + vid + kept, search_bytes=search_bytes,
                agg_bytes=agg_bytes, bwd_bytes=bwd_bytes)


# ---------------------------------------------------------------- counters --

def _kernel_files():
    """Kernel name -> source file defining it (csrc/*.hip)."""
    out = {}
    for path in sorted(glob.glob(os.path.join(CSRC, "*.hip"))):
        with open(path) as f:
            text = f.read()
        for m in re.finditer(r"__global__\s+(?:void\s+)?(?:__launch_bounds__\([^)]*\)\s+)?(\w+)\s*\(", text):
            out[m.group(1)] = os.path.basename(path)
    return out


def _base_name(kernel):
    """'void snls::search_tile_scores_kernel<7>(float const*, ...)' -> 'search_tile_scores_kernel'."""
    s = kernel.split("(")[0].replace("void ", "").strip()
    s = s.split("<")[0]
    return s.split("::")[-1]


def source_hash(kernels):
    """Hash of the sources that define the given kernels, plus the shared
    header: a counter record stays valid while none of them changes."""
    files = _kernel_files()
    names = sorted({files.get(_base_name(k)) for k in kernels} - {None})
    h = hashlib.sha256()
    for fn in names + ["snls_internal.h"]:
        with open(os.path.join(CSRC, fn), "rb") as fh:
            h.update(fn.encode() + fh.read())
    return h.hexdigest()[:16]


def counters_path(workload):
    return os.path.join(PROFILES, "snls_step_%s_counters.json" % workload)


def measured_counters(workload):
    """Counter record of one step of this workload from the committed
    rocprofv3 summary, or None when missing or taken on other sources."""
    path = counters_path(workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("workload") != workload or rec.get("source_hash") != source_hash(rec.get("kernels", {})):
        return None
    return rec


# ------------------------------------------------------ profile summaries --

COPY_KERNEL_HINT = "mulfunctor"  # torch.mul(src, 1, out=dst): one read and one write per element


def _read_csv(path):
    with open(path) as f:
        return list(csv.DictReader(f))


def _find(dirpath, suffix):
    for root, _, files in os.walk(dirpath):
        for fn in files:
            if fn.endswith(suffix):
                return os.path.join(root, fn)
    raise FileNotFoundError("%s*%s" % (dirpath, suffix))


def _short(kernel, n=72):
    return kernel.split("(")[0].replace("void ", "")[:n]


def summarize_profiles(outdir, workload, copy_mib, extra_args=""):
    """Turn the rocprofv3 outputs of one workload (kernel trace under
    OUTDIR/prof_<workload>_trace, counter passes under
    OUTDIR/prof_<workload>_pmc*) into profiles/snls_step_<workload>_rocprofv3.md
    and the counter record bench.py reads.  HBM bytes per dispatch = counter
    KiB scaled by what the same counter reads for a plain copy of copy_mib MiB."""
    tag = "prof_%s" % workload
    args = "--workload %s --steps {s} --warmup {w} --no-cpu-baseline --copy-probe-mib %d%s" % (
        workload, copy_mib, extra_args)
    cmd = ("cd /tmp && rocprofv3 {opts} --output-format csv -d $R/$OUT/{d} -o run -- "
           "python3 $R/bench.py " + args)
    lines = ["# rocprofv3 summary: workload %s (one step: %s)" % (
        workload, "search + top-k, aggregation, backward" if "train" in workload else "search + top-k, aggregation"),
             "", "Commands (R = repository root, OUT = output folder under it):", ""]
    lines.append("    " + cmd.format(opts="--kernel-trace --stats", d=tag + "_trace", s=10, w=2))
    trace = _read_csv(_find(os.path.join(outdir, tag + "_trace"), "kernel_stats.csv"))
    lines += ["", "| kernel | calls | avg us | min us | max us | total % |", "|---|---|---|---|---|---|"]
    durations = {}
    for r in trace:
        durations[r["Name"]] = float(r["AverageNs"]) / 1e3
        lines.append("| %s | %s | %.1f | %.1f | %.1f | %.1f |" % (
            _short(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
            float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    counters = collections.defaultdict(dict)
    for d in sorted(os.listdir(outdir)):
        if not d.startswith(tag + "_pmc") or not os.path.isdir(os.path.join(outdir, d)):
            continue
        rows = _read_csv(_find(os.path.join(outdir, d), "counter_collection.csv"))
        names = sorted({r["Counter_Name"] for r in rows})
        lines += ["", "    " + cmd.format(opts="--pmc " + " ".join(names), d=d, s=2, w=1)]
        acc = collections.defaultdict(list)
        for r in rows:
            acc[(r["Kernel_Name"], r["Counter_Name"])].append(float(r["Counter_Value"]))
        for (kn, cn), v in acc.items():
            counters[kn][cn] = sum(v) / len(v)
    copy = [kn for kn in counters if COPY_KERNEL_HINT in kn.lower() and "FETCH_SIZE" in counters[kn]]
    f_fetch = f_write = None
    if copy and "WRITE_SIZE" in counters[copy[0]]:
        exp_kib = copy_mib * 1024.0
        f_fetch = exp_kib / counters[copy[0]]["FETCH_SIZE"]
        f_write = exp_kib / counters[copy[0]]["WRITE_SIZE"]
    lines += ["", "Counters, mean per dispatch (FETCH_SIZE / WRITE_SIZE in KiB as read; the copy of %d MiB reads "
              "FETCH x %s, WRITE x %s):" % (copy_mib, "%.3f" % f_fetch if f_fetch else "?",
                                            "%.3f" % f_write if f_write else "?"),
              "", "| kernel | counter | value |", "|---|---|---|"]
    for kn in sorted(counters):
        for cn in sorted(counters[kn]):
            lines.append("| %s | %s | %.6g |" % (_short(kn, 60), cn, counters[kn][cn]))
    ours = sorted(kn for kn in set(durations) | set(counters) if "snls::" in kn)
    kernels = {}
    for kn in ours:
        c = counters.get(kn, {})
        e = {"avg_us": durations.get(kn)}
        if f_fetch and "FETCH_SIZE" in c:
            e["fetch_bytes"] = c["FETCH_SIZE"] * f_fetch * 1024.0
        if f_write and "WRITE_SIZE" in c:
            e["write_bytes"] = c["WRITE_SIZE"] * f_write * 1024.0
        for cn in ("SQ_INSTS_VALU_FMA_F32", "SQ_INSTS_VALU", "SQ_BUSY_CYCLES", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT",
                   "SQ_LDS_IDX_ACTIVE", "SQ_WAVES", "GRBM_GUI_ACTIVE", "SQ_ACTIVE_INST_VALU"):
            if cn in c:
                e[cn] = c[cn]
        kernels[kn] = e
    search = [kn for kn in kernels if SEARCH_PAT.match(_base_name(kn))]

    def total(names, key):
        vals = [kernels[kn].get(key) for kn in names]
        return None if not names or any(v is None for v in vals) else float(sum(vals))

    rec = {"workload": workload, "source_hash": source_hash(kernels), "copy_mib": copy_mib,
           "fetch_scale": f_fetch, "write_scale": f_write, "kernels": kernels,
           "search_call": {"kernels": search, "avg_us": total(search, "avg_us"),
                           "fetch_bytes": total(search, "fetch_bytes"), "write_bytes": total(search, "write_bytes"),
                           "fma_f32_wave_insts": total(search, "SQ_INSTS_VALU_FMA_F32")}}
    sc = rec["search_call"]
    if sc["fetch_bytes"] is not None and sc["write_bytes"] is not None:
        lines += ["", "HBM traffic of one snls_search call (%s): FETCH %.1f MB + WRITE %.1f MB = %.1f MB." % (
            " + ".join(_short(k, 60) for k in search), sc["fetch_bytes"] / 1e6, sc["write_bytes"] / 1e6,
            (sc["fetch_bytes"] + sc["write_bytes"]) / 1e6)]
    if sc["fma_f32_wave_insts"] is not None and sc["avg_us"]:
        fl = sc["fma_f32_wave_insts"] * 128
        lines += ["", "Issued fp32 FMA flop of one snls_search call: %.4g (= %.4g wave FMAs x 64 x 2); at the "
                  "traced %.1f us: %.2f TFLOP/s = %.3f of 157.3, %.3f of 78.6." % (
                      fl, sc["fma_f32_wave_insts"], sc["avg_us"], fl / sc["avg_us"] / 1e6,
                      fl / sc["avg_us"] / 1e6 / 157.3, fl / sc["avg_us"] / 1e6 / 78.6)]
    os.makedirs(PROFILES, exist_ok=True)
    md = os.path.join(PROFILES, "snls_step_%s_rocprofv3.md" % workload)
    with open(md, "w") as f:
        f.write("\n".join(lines) + "\n")
    with open(counters_path(workload), "w") as f:
        json.dump(rec, f, indent=1)
    return md, rec


# ---------------------------------------------------------- CPU baseline --

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


def time_stacked(B, torch, x, dists, inds, p, scale, dev, reps=5):
    """The example's gather (weights = softmax over the row, computed by the
    caller as in the example) and the reduction over the k neighbours with a
    seeded (C, C, k) kernel: materialised stack, then the fused pass."""
    sign = 1.0 if p["dist_type"] == 0 else -1.0
    w = torch.softmax(sign * scale * dists, dim=-1).contiguous()
    g = torch.Generator(device="cpu").manual_seed(17)
    proj = (torch.randn((p["C"], p["C"], p["k"]), generator=g) / (p["C"] * p["k"]) ** 0.5).to(dev)
    st = torch.empty(B.stacked_shape(p), device=dev)
    gws = B.workspace_for(B.SNLS_OP_GATHER_STACKED, p, dev)
    fws = B.workspace_for(B.SNLS_OP_GATHER_REDUCE, p, dev)
    out = torch.empty((p["B"], p["T"], p["C"], p["H"], p["W"]), device=dev)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b_ in evs:
            a.record()
            fn()
            b_.record()
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b_) for a, b_ in evs]))

    t_gather = timed(lambda: B.snls_gather_stacked(x, w, inds, p, st, gws))
    t_reduce = timed(lambda: B.snls_stacked_reduce(st, proj, p, out))
    t_fused = timed(lambda: B.snls_gather_reduce(x, w, inds, proj, p, out, fws))
    pix = p["B"] * p["T"] * p["H"] * p["W"]
    red_flop = 2.0 * pix * p["C"] * p["k"] * p["C"]
    return {"gather_stacked_ms": t_gather, "stacked_reduce_ms": t_reduce, "gather_reduce_ms": t_fused,
            "stacked_gb": st.numel() * 4 / 1e9, "reduce_tflops_mfma": red_flop / (t_reduce * 1e-3) / 1e12,
            "reduce_flop": red_flop}


# ------------------------------------------------------------------ main --

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD,
                    help="workload name (default: the 480x854 denoising workload; tiny, motion, multihead, "
                         "train256 (with its backward pass), paper320_s1, paper320_s2, paper152_mem, "
                         "denoise480x854_sk05, denoise480x854_s2)")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run one plain device copy of this size (calibrates the HBM byte counters)")
    ap.add_argument("--stacked", action="store_true",
                    help="also time the code example's gather with caller weights and its reduction over the k "
                         "neighbours: snls_gather_stacked + snls_stacked_reduce, and the fused snls_gather_reduce "
                         "(Cout = C), outside the timed step")
    ap.add_argument("--summarize-profiles", metavar="DIR", default=None,
                    help="write the profiles/ summary of --workload from the rocprofv3 outputs under DIR and exit")
    args = ap.parse_args()
    if args.summarize_profiles:
        md, rec = summarize_profiles(args.summarize_profiles, args.workload, args.copy_probe_mib or 256)
        print(md)
        print(json.dumps(rec["search_call"], indent=1))
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the path has no multi-GPU mode", file=sys.stderr)
        sys.exit(2)

    import torch
    sys.path.insert(0, ROOT)
    from paper_2309_16849_amd import snls as B
    from workloads import CONFIGS, config_index, make_config

    B.load_library()
    dev = torch.device("cuda:0")
    wi = config_index(args.workload)
    c = make_config(wi)
    p, scale = c["params"], c["scale"]
    train = bool(CONFIGS[wi]["backward"])
    x = torch.from_numpy(c["q"]).to(dev)
    fl = torch.from_numpy(c["flows"]).to(dev)
    shp = B.out_shape(p)
    dists = torch.empty(shp, device=dev)
    inds = torch.empty(shp + (3,), device=dev)
    out = torch.empty(B.video_shape(p), device=dev)
    ws = B.workspace_for(B.SNLS_OP_AGGREGATE, p, dev)
    sws = B.workspace_for(B.SNLS_OP_SEARCH, p, dev)
    if train:
        go = torch.from_numpy(c["grad_out"]).to(dev)
        bws = B.workspace_for(B.SNLS_OP_BACKWARD, p, dev)

    # HIP events on torch's current stream, the stream every call is launched on
    def step(ev=None):
        if ev is not None:
            ev[0].record()
        B.snls_search(x, x, fl, p, dists, inds, sws)
        if ev is not None:
            ev[1].record()
        B.snls_aggregate(x, dists, inds, p, scale, out, ws)
        if ev is not None:
            ev[2].record()
        if train:
            B.snls_backward(x, x, x, fl, dists, inds, go, p, scale, workspace=bws)
            if ev is not None:
                ev[3].record()

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
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    t_search = float(np.mean([e[0].elapsed_time(e[1]) for e in evs])) * 1e-3
    t_agg = float(np.mean([e[1].elapsed_time(e[2]) for e in evs])) * 1e-3
    t_bwd = float(np.mean([e[2].elapsed_time(e[3]) for e in evs])) * 1e-3 if train else None

    w = work_counts(p)
    t_step = elapsed / args.steps
    value = w["queries"] / t_step
    rec = measured_counters(args.workload)
    sc = rec["search_call"] if rec else None
    issued = sc["fma_f32_wave_insts"] * 64 * 2 if sc and sc.get("fma_f32_wave_insts") else None
    traffic = sc["fetch_bytes"] + sc["write_bytes"] if sc and sc.get("fetch_bytes") is not None and \
        sc.get("write_bytes") is not None else None
    achieved = issued / t_search if issued else None
    roofline = {
        "bound": "alu", "kernel": "snls_search call: " + (" + ".join(_base_name(k) for k in sc["kernels"])
                                                          if sc else "kernels not profiled for these sources"),
        "achieved": achieved / 1e12 if achieved else None, "peak": PEAK_FP32_VALU / 1e12, "unit": "TFLOP/s",
        "frac": achieved / PEAK_FP32_VALU if achieved else None,
        "peak_attainable": PEAK_FP32_VALU_UNPACKED / 1e12,
        "frac_attainable": achieved / PEAK_FP32_VALU_UNPACKED if achieved else None,
        "traffic": traffic, "alg_bytes": w["search_bytes"],
        "alg_tflops": w["f_search"] / t_search / 1e12, "alg_frac": w["f_search"] / t_search / PEAK_FP32_VALU,
        "call_ms": t_search * 1e3, "profiled_call_ms": sc["avg_us"] / 1e3 if sc and sc.get("avg_us") else None,
    }
    metric = METRIC if args.workload == DEFAULT_WORKLOAD else \
        METRIC.replace("config 2", args.workload + (" (+backward)" if train else "")).replace(
            "search+top-k+aggregate", "search+top-k+aggregate" + ("+backward" if train else ""))
    line = {
        "metric": metric, "value": value, "unit": "queries/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": t_step * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": c["name"], "B": p["B"], "T": p["T"], "C": p["C"], "H": p["H"], "W": p["W"],
                   "HD": p["HD"], "ws": p["ws"], "wt": p["wt"], "ps": p["ps"], "stride0": p["stride0"],
                   "stride1": p["stride1"], "k": p["k"],
                   "dist": "inner_product" if p["dist_type"] == 0 else "squared_l2", "softmax_scale": scale,
                   "backward": train, "parallelism": "single_gpu"},
        "roofline": roofline,
        "candidates_per_s": w["candidates"] / t_step,
        "step_alg_tflops": (w["f_search"] + w["f_agg"]) / t_step / 1e12,
        "step_frac_hbm": w["bytes_total"] / t_step / PEAK_HBM,
        "search_ms": t_search * 1e3, "aggregate_ms": t_agg * 1e3,
        "peak_mem_gb": peak_mem / 1e9, "search_workspace_gb": sws.numel() * 4 / 1e9,
        "aggregate_alg_tflops": w["f_agg"] / t_agg / 1e12,
    }
    if train:
        line["backward_ms"] = t_bwd * 1e3
        line["backward_alg_tflops"] = w["f_bwd"] / t_bwd / 1e12
        line["backward_alg_frac_hbm"] = w["bwd_bytes"] / t_bwd / PEAK_HBM
    if args.stacked:
        line["stacked"] = time_stacked(B, torch, x, dists, inds, p, scale, dev)
    if not args.no_cpu_baseline and args.workload == DEFAULT_WORKLOAD:
        line["cpu_baseline"] = cpu_baseline(c, args.cpu_budget)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
