"""Synthetic workloads shaped like the paper's video benchmarks.

The paper evaluates on DAVIS / Set8 clips (480 x 854 frames, 32-192
features, 1-12 heads); those datasets are not available here, so seeded
synthetic videos stand in for them:

* ``tiny``      i.i.d. N(0,1) features used as q = k = v, i.i.d. U(-3,3) flows;
* ``motion``    a blurred random texture (N(0,1) noise, Gaussian sigma 1.5 px)
                warped by a smooth random velocity field (4 random
                low-frequency sinusoids per component, scaled so the largest
                velocity is A px per frame), plus N(0, 0.1^2) noise; the true
                flow between two frames is solved from the warp, and the
                predicted flow is the true flow plus N(0, 1.5^2) error.

Frames are produced by scipy's order-1 ``map_coordinates``; nothing here
touches the search, top-k or aggregation arithmetic.  Flow tensors are laid
out (B, T, 2*wt, 2, H, W): slot order dt = -wt..-1, +1..+wt, component 0 is
the row (h) offset and 1 the column (w) offset.
"""
from __future__ import annotations

import math
import os
import numpy as np
from scipy import ndimage

SEED_BASE = 230916849

# Search settings of the five workloads (B, T, C, H, W, heads; window ws,
# temporal radius wt, patch ps, query stride stride0, key stride stride1,
# neighbours k, distance 0 = inner product / 1 = squared L2).
CONFIGS = [
    dict(name="tiny", B=1, T=3, C=16, H=64, W=64, HD=1, ws=9, wt=1, ps=3, stride0=1, stride1=1.0, k=10,
         dist_type=0, scale=1.0, video="tiny", backward=False),
    dict(name="motion", B=1, T=5, C=32, H=128, W=128, HD=1, ws=9, wt=2, ps=7, stride0=1, stride1=1.0, k=10,
         dist_type=1, scale=1.0, video="motion", amp=8.0, backward=False),
    dict(name="denoise480x854", B=1, T=5, C=64, H=480, W=854, HD=1, ws=9, wt=2, ps=7, stride0=1, stride1=1.0,
         k=10, dist_type=0, scale=1.0, video="motion", amp=16.0, backward=False),
    dict(name="multihead", B=2, T=8, C=64, H=256, W=256, HD=4, ws=15, wt=3, ps=1, stride0=2, stride1=1.0,
         k=30, dist_type=0, scale=1.0, video="motion", amp=8.0, backward=False),
    dict(name="train256", B=1, T=5, C=64, H=256, W=256, HD=1, ws=9, wt=2, ps=3, stride0=1, stride1=1.0, k=10,
         dist_type=0, scale=1.0, video="motion", amp=8.0, backward=True),
    # The paper's own benchmark shapes (Sec. 4.4): runtime on 5 frames of
    # 320 x 320 with 32 features, ws = 9, ps = 1, query stride 1 or 2; peak
    # memory on 5 frames of 152 x 152 with 192 features, ps = 7, ws = 3.  The
    # temporal window and k are not stated there: the whole clip (wt = 2) and
    # k = 10 are used.
    dict(name="paper320_s1", B=1, T=5, C=32, H=320, W=320, HD=1, ws=9, wt=2, ps=1, stride0=1, stride1=1.0, k=10,
         dist_type=0, scale=1.0, video="motion", amp=8.0, backward=False),
    dict(name="paper320_s2", B=1, T=5, C=32, H=320, W=320, HD=1, ws=9, wt=2, ps=1, stride0=2, stride1=1.0, k=10,
         dist_type=0, scale=1.0, video="motion", amp=8.0, backward=False),
    dict(name="paper152_mem", B=1, T=5, C=192, H=152, W=152, HD=1, ws=3, wt=2, ps=7, stride0=1, stride1=1.0,
         k=10, dist_type=0, scale=1.0, video="motion", amp=8.0, backward=False),
    # Fractional key stride S_K = 1/2 (the paper's RVRT setting, Sec. 4.2,
    # Table 4) on the 480 x 854 denoising video: the window cells sit half a
    # pixel apart.
    dict(name="denoise480x854_sk05", B=1, T=5, C=64, H=480, W=854, HD=1, ws=9, wt=2, ps=7, stride0=1, stride1=0.5,
         k=10, dist_type=0, scale=1.0, video="motion", amp=16.0, backward=False, data_of="denoise480x854"),
    # Query stride 2 on the same video (a quarter of the queries, strided
    # patches overlapping by 5 of 7 pixels).
    dict(name="denoise480x854_s2", B=1, T=5, C=64, H=480, W=854, HD=1, ws=9, wt=2, ps=7, stride0=2, stride1=1.0,
         k=10, dist_type=0, scale=1.0, video="motion", amp=16.0, backward=False, data_of="denoise480x854"),
    # The settings of the paper's code example (App. B): 5 frames of
    # 128 x 128, 16 features in 2 heads, ws = 5, wt = 2, ps = 3, k = 10, key
    # stride 1/2 (its gather and reduction over the k neighbours follow).
    dict(name="example_appb", B=1, T=5, C=16, H=128, W=128, HD=2, ws=5, wt=2, ps=3, stride0=1, stride1=0.5,
         k=10, dist_type=0, scale=1.0, video="motion", amp=4.0, backward=False),
]

# The five workloads every parity test covers; the paper's benchmark shapes
# follow them.
N_MAIN_CONFIGS = 5


def config_index(name: str) -> int:
    """Index of the workload called name."""
    for i, c in enumerate(CONFIGS):
        if c["name"] == name:
            return i
    raise KeyError(name)

PARAM_KEYS = ("B", "T", "C", "H", "W", "HD", "ws", "wt", "ps", "stride0", "stride1", "k", "dist_type")


def config_params(idx: int, **override) -> dict:
    """The search parameters of workload idx as a plain dict (optionally overridden)."""
    c = dict(CONFIGS[idx])
    c.update(override)
    return {k: c[k] for k in PARAM_KEYS}


def small_params(**kw) -> dict:
    """A parameter dict with small defaults, for property sweeps."""
    p = dict(B=1, T=3, C=8, H=12, W=13, HD=1, ws=3, wt=1, ps=3, stride0=1, stride1=1.0, k=4, dist_type=0)
    p.update(kw)
    return p


def _velocity(rng, H: int, W: int, amp: float):
    """Smooth velocity field: per component a sum of 4 sinusoids with random
    frequencies in (-1, 1) cycles per frame extent and random phases, scaled so
    the largest velocity magnitude on the pixel grid is amp."""
    fh = rng.uniform(-1.0, 1.0, size=(2, 4))
    fw = rng.uniform(-1.0, 1.0, size=(2, 4))
    ph = rng.uniform(0.0, 2.0 * math.pi, size=(2, 4))

    def raw(y, x):
        u = np.zeros((2,) + np.shape(y))
        for c in range(2):
            for j in range(4):
                u[c] += np.sin(2.0 * math.pi * (fh[c, j] * y / H + fw[c, j] * x / W) + ph[c, j])
        return u

    def raw_jac(y, x):
        J = np.zeros((2, 2) + np.shape(y))
        for c in range(2):
            for j in range(4):
                arg = 2.0 * math.pi * (fh[c, j] * y / H + fw[c, j] * x / W) + ph[c, j]
                cs = np.cos(arg)
                J[c, 0] += cs * 2.0 * math.pi * fh[c, j] / H
                J[c, 1] += cs * 2.0 * math.pi * fw[c, j] / W
        return J

    yy, xx = np.meshgrid(np.arange(H, dtype=np.float64), np.arange(W, dtype=np.float64), indexing="ij")
    mag = np.sqrt((raw(yy, xx) ** 2).sum(0)).max()
    s = amp / mag if mag > 0 else 0.0
    return (lambda y, x: s * raw(y, x)), (lambda y, x: s * raw_jac(y, x))


def _true_flow(u, jac, H, W, s_from: float, s_to: float, iters: int = 20):
    """Displacement p' - p solving p' + s_to*u(p') = p + s_from*u(p) (Newton)."""
    yy, xx = np.meshgrid(np.arange(H, dtype=np.float64), np.arange(W, dtype=np.float64), indexing="ij")
    tgt = np.stack([yy, xx]) + s_from * u(yy, xx)
    pp = np.stack([yy, xx]).copy()
    for _ in range(iters):
        F = pp + s_to * u(pp[0], pp[1]) - tgt
        if np.abs(F).max() < 1e-6:
            break
        J = s_to * jac(pp[0], pp[1])
        a, b, c, d = 1.0 + J[0, 0], J[0, 1], J[1, 0], 1.0 + J[1, 1]
        det = a * d - b * c
        ok = np.abs(det) > 1e-3
        det = np.where(ok, det, 1.0)
        sy = np.where(ok, (d * F[0] - b * F[1]) / det, 0.5 * F[0])
        sx = np.where(ok, (-c * F[0] + a * F[1]) / det, 0.5 * F[1])
        pp = pp - np.clip(np.stack([sy, sx]), -4.0, 4.0)
    return pp - np.stack([yy, xx])


def make_motion_video(rng, T: int, C: int, H: int, W: int, wt: int, amp: float, noise: float = 0.1,
                      flow_err: float = 1.5):
    """One clip: frames (T, C, H, W) float32 and predicted flows (T, 2wt, 2, H, W) float32."""
    tc = (T - 1) // 2
    M = int(math.ceil(amp * max(abs(t - tc) for t in range(T)))) + 8
    base = rng.standard_normal((C, H + 2 * M, W + 2 * M), dtype=np.float32)
    base = ndimage.gaussian_filter(base, sigma=(0.0, 1.5, 1.5), mode="reflect", truncate=4.0)
    u, jac = _velocity(rng, H, W, amp)
    yy, xx = np.meshgrid(np.arange(H, dtype=np.float64), np.arange(W, dtype=np.float64), indexing="ij")
    vel = u(yy, xx)
    frames = np.empty((T, C, H, W), np.float32)
    for t in range(T):
        cy = yy + M + (t - tc) * vel[0]
        cx = xx + M + (t - tc) * vel[1]
        for c in range(C):
            frames[t, c] = ndimage.map_coordinates(base[c], [cy, cx], order=1, mode="nearest")
        frames[t] += noise * rng.standard_normal((C, H, W), dtype=np.float32)
    flows = np.zeros((T, 2 * wt, 2, H, W), np.float32)
    dts = list(range(-wt, 0)) + list(range(1, wt + 1))
    for t in range(T):
        for s, dt in enumerate(dts):
            t2 = t + dt
            if t2 < 0 or t2 >= T:
                continue  # no neighbour frame: the slot is never used
            fl = _true_flow(u, jac, H, W, float(t - tc), float(t2 - tc))
            flows[t, s] = fl + flow_err * rng.standard_normal(fl.shape, dtype=np.float32)
    return frames, flows


def _cache_dir():
    d = os.environ.get("SNLS_WORKLOAD_CACHE", os.path.join(os.path.expanduser("~"), ".cache", "snls_workloads"))
    os.makedirs(d, exist_ok=True)
    return d


def make_config(idx: int, seed: int | None = None, cache: bool = True) -> dict:
    """Inputs of workload idx: dict with 'params', 'scale', 'q', 'k', 'v', 'flows' (+ 'grad_out').

    Arrays are float32 numpy; q, k, v are (B,T,C,H,W), flows (B,T,2wt,2,H,W).
    Seeded by SEED_BASE + idx unless seed is given.  Large workloads are cached
    as .npy files (directory from $SNLS_WORKLOAD_CACHE or ~/.cache).
    """
    cfg = CONFIGS[idx]
    p = config_params(idx)
    # a workload that only changes search settings reuses another one's video
    didx = config_index(cfg["data_of"]) if "data_of" in cfg else idx
    seed = SEED_BASE + didx if seed is None else seed
    B, T, C, H, W, wt = p["B"], p["T"], p["C"], p["H"], p["W"], p["wt"]
    path = os.path.join(_cache_dir(), "cfg%d_seed%d.npz" % (didx, seed)) if cache else None
    if path and os.path.exists(path):
        with np.load(path, allow_pickle=False) as z:
            arrs = {k: z[k] for k in z.files}
    else:
        rng = np.random.default_rng(seed)
        if cfg["video"] == "tiny":
            x = rng.standard_normal((B, T, C, H, W), dtype=np.float32)
            flows = rng.uniform(-3.0, 3.0, size=(B, T, 2 * wt, 2, H, W)).astype(np.float32)
        else:
            xs, fs = [], []
            for _ in range(B):
                fr, fl = make_motion_video(rng, T, C, H, W, wt, cfg["amp"])
                xs.append(fr)
                fs.append(fl)
            x, flows = np.stack(xs), np.stack(fs)
        arrs = {"x": x, "flows": flows}
        if cfg["backward"]:
            arrs["grad_out"] = rng.standard_normal((B, T, C, H, W), dtype=np.float32)
        if path and x.size >= 1 << 20:
            tmp = path + ".tmp%d.npz" % os.getpid()
            np.savez(tmp, **arrs)
            os.replace(tmp, path)
    out = {"params": p, "scale": cfg["scale"], "name": cfg["name"], "q": arrs["x"], "k": arrs["x"],
           "v": arrs["x"], "flows": arrs["flows"]}
    if "grad_out" in arrs:
        out["grad_out"] = arrs["grad_out"]
    return out
