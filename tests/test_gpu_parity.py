"""Parity of the HIP library against the oracle on the same seeded inputs.

Small cases are compared element by element over whole outputs; the five
workloads at their full sizes are compared on sampled query rows and output
pixels that the oracle evaluates one by one.  Tolerances: see tests/parity.py.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2309_16849_amd import snls as B
from tests.parity import REL, assert_close, compare_topk, rms_finite
from workloads import config_params, make_config, small_params

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    return torch.device("cuda:0")


def _d(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)


def _h(t):
    return t.detach().cpu().numpy()


def _inputs(p, seed, flow_kind="frac", shared_qk=False):
    r = np.random.default_rng(seed)
    shp = (p["B"], p["T"], p["C"], p["H"], p["W"])
    q = r.standard_normal(shp, dtype=np.float32)
    k = q.copy() if shared_qk else r.standard_normal(shp, dtype=np.float32)
    v = r.standard_normal(shp, dtype=np.float32)
    fshp = (p["B"], p["T"], 2 * p["wt"], 2, p["H"], p["W"])
    if flow_kind == "frac":
        flows = r.uniform(-3, 3, fshp).astype(np.float32)
    elif flow_kind == "int":
        flows = r.integers(-2, 3, fshp).astype(np.float32)
    elif flow_kind == "far":
        flows = (r.choice([-1.0, 1.0], fshp) * 60.0).astype(np.float32)
    else:
        raise ValueError(flow_kind)
    return q, k, v, flows


def _sweep_cases(n=22, seed=7):
    r = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        ws = int(r.choice([1, 3, 5, 9]))
        wt = int(r.choice([0, 1, 2]))
        HD = int(r.choice([1, 2, 4]))
        p = small_params(
            B=int(r.choice([1, 2])), T=int(r.choice([1, 2, 3])), C=HD * int(r.choice([1, 3, 4])),
            H=int(r.choice([1, 7, 33])), W=int(r.choice([1, 7, 33])), HD=HD, ws=ws, wt=wt,
            ps=int(r.choice([1, 2, 3, 5])), stride0=int(r.choice([1, 2, 3])),
            stride1=float(r.choice([1.0, 0.5])), dist_type=int(r.choice([0, 1])))
        nc = (2 * wt + 1) * ws * ws
        p["k"] = int(min(nc, r.choice([1, 4, 10, 33])))
        kind = ["frac", "int", "far"][i % 3] if wt > 0 else "frac"
        cases.append((p, kind, bool(i % 4 == 0)))
    # fixed edge cases: frames shorter than the window, single pixel, big k
    cases.append((small_params(T=1, wt=2, ws=3, k=9, H=5, W=6), "frac", False))
    cases.append((small_params(T=2, H=1, W=1, ws=3, wt=1, ps=3, k=5), "frac", False))
    cases.append((small_params(T=3, H=20, W=19, ws=7, wt=1, ps=1, k=100, C=4), "frac", False))
    return cases


CASES = _sweep_cases()
IDS = ["c%d-ws%d-wt%d-ps%d-s%d-hd%d-%s" % (i, p["ws"], p["wt"], p["ps"], p["stride0"], p["HD"], kd)
       for i, (p, kd, _) in enumerate(CASES)]


@pytest.mark.parametrize("case", range(len(CASES)), ids=IDS)
def test_search_all_candidates(dev, case):
    p, kind, shared = CASES[case]
    p = dict(p, k=0)
    q, k, v, flows = _inputs(p, 1000 + case, kind, shared)
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    od, oi = oracle.search_all(q, k, flows, p)
    gd, gi = _h(gd).reshape(od.shape), _h(gi).reshape(oi.shape)
    assert np.array_equal(gi, oi.astype(np.float32)), "candidate positions differ"
    assert_close(gd, od, "all-candidate scores")


@pytest.mark.parametrize("case", range(len(CASES)), ids=IDS)
def test_fused_search_topk(dev, case):
    p, kind, shared = CASES[case]
    q, k, v, flows = _inputs(p, 2000 + case, kind, shared)
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    res = oracle.search(q, k, flows, p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])


@pytest.mark.parametrize("case", range(0, len(CASES), 2), ids=IDS[::2])
def test_standalone_topk(dev, case):
    p, kind, shared = CASES[case]
    q, k, v, flows = _inputs(p, 3000 + case, kind, shared)
    ad, ai = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), dict(p, k=0))
    gd, gi = B.snls_topk(ad, ai, p["k"], p["dist_type"])
    torch.cuda.synchronize()
    res = oracle.search(q, k, flows, p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])


@pytest.mark.parametrize("case", range(len(CASES)), ids=IDS)
def test_aggregate(dev, case):
    p, kind, shared = CASES[case]
    q, k, v, flows = _inputs(p, 4000 + case, kind, shared)
    scale = 0.25
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    out = B.snls_aggregate(_d(v, dev), gd, gi, p, scale)
    torch.cuda.synchronize()
    gd_h, gi_h, out_h = _h(gd), _h(gi), _h(out)
    # decoupled: the oracle aggregates the GPU's own neighbours
    ref = oracle.aggregate(v, gd_h, gi_h, p, scale)
    assert_close(out_h, ref, "aggregate (GPU neighbours)")
    # end to end: the oracle's own neighbours, pixels of rows with near-tie swaps masked
    res = oracle.search(q, k, flows, p)
    _, swaps = compare_topk(gd_h.reshape(-1, p["k"]), gi_h.reshape(-1, p["k"], 3), res, p["k"])
    nH, nW = oracle.grid(p)
    shp = (p["B"], p["HD"], p["T"], nH, nW, p["k"])
    ref2 = oracle.aggregate(v, res["dists"][:, :p["k"]].reshape(shp), res["inds"][:, :p["k"]].reshape(shp + (3,)),
                            p, scale)
    mask = _swap_mask(p, swaps.reshape(shp[:-1]))
    assert_close(out_h[~mask], ref2[~mask], "aggregate (end to end)", scale=rms_finite(ref2))


# ------------------------------------------------ tiled aggregation --
# Query stride 1 with up to 7 frames and 64 channels per head goes through
# the tiled gather: neighbours of smooth motion land in the per-slot bin
# boxes; scattered neighbours, frames outside the window and odd caller-given
# positions take its direct path.  (Single-pixel patches take the per-query
# gather at every stride.)

def _motion_inputs(p, seed, amp=4.0):
    from workloads import make_motion_video
    r = np.random.default_rng(seed)
    fr, fl = make_motion_video(r, p["T"], p["C"], p["H"], p["W"], p["wt"], amp)
    return fr[None].copy(), fl[None].copy()


@pytest.mark.parametrize("ps,k,C,HD,scale,stride0", [(7, 10, 64, 1, 1.0, 1), (3, 10, 64, 1, 1.0, 1),
                                                      (5, 16, 32, 2, 0.3, 1), (7, 4, 48, 1, 0.05, 1),
                                                      (1, 12, 64, 1, 1.0, 1), (7, 10, 64, 1, 1.0, 2),
                                                      (3, 10, 32, 2, 0.5, 2), (5, 8, 16, 1, 1.0, 3),
                                                      (4, 6, 16, 1, 1.0, 4), (2, 9, 8, 1, 1.0, 5)])
def test_aggregate_tiled_motion(dev, ps, k, C, HD, scale, stride0):
    p = small_params(T=5, C=C, HD=HD, H=37, W=53, ws=9, wt=2, ps=ps, k=k, stride0=stride0)
    x, flows = _motion_inputs(p, 9100 + ps + k)
    v = np.random.default_rng(9200 + ps).standard_normal(x.shape, dtype=np.float32)
    xd = _d(x, dev)
    gd, gi = B.snls_search(xd, xd, _d(flows, dev), p)
    out = B.snls_aggregate(_d(v, dev), gd, gi, p, scale)
    torch.cuda.synchronize()
    ref = oracle.aggregate(v, _h(gd), _h(gi), p, scale)
    assert_close(_h(out), ref, "tiled aggregate (motion neighbours)")


@pytest.mark.parametrize("seed,ps,stride0,HD", [(0, 5, 1, 1), (1, 5, 1, 1), (2, 1, 2, 2), (3, 1, 3, 1),
                                                (4, 3, 2, 1), (5, 1, 1, 4)])
def test_aggregate_tiled_odd_neighbours(dev, seed, ps, stride0, HD):
    """Caller-given neighbours: frames outside the window or the clip,
    non-integer frames, huge and non-finite displacements, non-finite scores,
    neighbours far from the others (direct path) and integer positions.
    Single-pixel patches take the per-query gather, other patches with query
    stride 1 the tiled gather, the rest the merged gather."""
    p = small_params(T=4, C=64, HD=HD, H=21, W=35, ws=5, wt=1, ps=ps, stride0=stride0, k=6)
    r = np.random.default_rng(9300 + seed)
    v = r.standard_normal((1, 4, 64, 21, 35), dtype=np.float32)
    nH, nW = oracle.grid(p)
    shp = (1, HD, 4, nH, nW, 6)
    d = r.standard_normal(shp).astype(np.float32)
    t_q = np.arange(4)[None, None, :, None, None, None]
    ind = np.zeros(shp + (3,), np.float32)
    ind[..., 0] = np.clip(t_q + r.integers(-1, 2, shp), 0, 3)
    ind[..., 1] = r.uniform(-2, 2, shp).astype(np.float32)
    ind[..., 2] = r.uniform(-2, 2, shp).astype(np.float32)
    m = r.random(shp)
    ind[..., 0] = np.where(m < 0.05, t_q + 2 * (t_q < 2) - (t_q >= 2) * 2, ind[..., 0])  # outside the window
    ind[..., 1] = np.where((m > 0.05) & (m < 0.1), r.uniform(-30, 30, shp), ind[..., 1])  # far: direct path
    ind[..., 2] = np.where((m > 0.1) & (m < 0.15), np.round(ind[..., 2]), ind[..., 2])  # integer columns
    ind[..., 0] = np.where((m > 0.15) & (m < 0.17), 1.5, ind[..., 0])  # not an integer frame
    ind[..., 0] = np.where((m > 0.17) & (m < 0.19), 7.0, ind[..., 0])  # outside the clip
    ind[..., 1] = np.where((m > 0.19) & (m < 0.21), 3.0e6, ind[..., 1])  # absurd displacement
    ind[..., 2] = np.where((m > 0.21) & (m < 0.22), np.nan, ind[..., 2])
    d = np.where((m > 0.22) & (m < 0.24), -np.inf, d).astype(np.float32)
    d[0, 0, 1, 3, 4 % nW, :] = -np.inf  # a row with no finite score
    out = B.snls_aggregate(_d(v, dev), _d(d, dev), _d(ind, dev), p, 0.7)
    torch.cuda.synchronize()
    ref = oracle.aggregate(v, d, ind, p, 0.7)
    assert_close(_h(out), ref, "tiled aggregate (odd neighbours)")


@pytest.mark.parametrize("stride0,HD,C,k,H,W", [(2, 4, 64, 30, 37, 29), (1, 1, 16, 7, 20, 23), (3, 2, 8, 5, 17, 16),
                                                (2, 1, 4, 1, 9, 10), (2, 2, 64, 12, 33, 40), (2, 1, 8, 60, 19, 21),
                                                (2, 1, 8, 61, 15, 14), (1, 3, 12, 3, 70, 9)])
def test_aggregate_p1(dev, stride0, HD, C, k, H, W):
    """Single-pixel patches: per-query gather of the searched neighbours,
    holes of the query grid cleared."""
    p = small_params(T=4, C=C, HD=HD, H=H, W=W, ws=7, wt=1, ps=1, stride0=stride0, k=k)
    x, flows = _motion_inputs(p, 9400 + stride0 + k)
    v = np.random.default_rng(9500 + k).standard_normal(x.shape, dtype=np.float32)
    xd = _d(x, dev)
    gd, gi = B.snls_search(xd, xd, _d(flows, dev), p)
    out = B.snls_aggregate(_d(v, dev), gd, gi, p, 0.5)
    torch.cuda.synchronize()
    ref = oracle.aggregate(v, _h(gd), _h(gi), p, 0.5)
    assert_close(_h(out), ref, "single-pixel aggregate")


def _swap_mask(p, swaps):
    """Output pixels covered by a query patch whose top-k had a near-tie swap."""
    mask = np.zeros((p["B"], p["T"], p["C"], p["H"], p["W"]), bool)
    lo = -(p["ps"] // 2)
    for b, hd, t, mh, mw in zip(*np.nonzero(swaps)):
        h, w = mh * p["stride0"], mw * p["stride0"]
        mask[b, t, :, max(h + lo, 0):max(h + lo + p["ps"], 0), max(w + lo, 0):max(w + lo + p["ps"], 0)] = True
    return mask


# ------------------------------------------------------ tiled kernel --
# Cases inside the tiled kernel's domain (inner product, S_K <= 1, P <= 7,
# Ws <= 9; query strides 1 to 5): every patch size, key strides 1, 3/4, 1/2 and
# 1/4, ragged tiles and channel chunks, narrow shift unions (few tasks:
# channel-split groups), wide ones (several rounds) and unions too wide for
# the LDS layout (the per-candidate fallback).

def _tile_cases(n=28, seed=31):
    r = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        HD = int(r.choice([1, 2]))
        ps = 1 + i % 7
        p = small_params(B=int(r.choice([1, 2])), T=int(r.choice([1, 2, 3, 5])), HD=HD,
                         C=HD * int(r.choice([1, 3, 4, 6, 9])), H=int(r.choice([5, 17, 23, 31])),
                         W=int(r.choice([6, 16, 19, 41])), ws=int(r.choice([1, 2, 4, 5, 7, 8, 9])),
                         wt=int(r.choice([0, 1, 2, 3, 4])), ps=ps, stride0=1,
                         stride1=float([1.0, 0.5, 0.75, 1.0, 0.25][i % 5 if i < 20 else (i + 1) % 5]), dist_type=0)
        nc = (2 * p["wt"] + 1) * p["ws"] ** 2
        p["k"] = int(min(nc, r.choice([1, 5, 10, 12, 13, 16])))
        kind = ["frac", "smooth", "int", "wide", "far"][i % 5]
        cases.append((p, kind))
    return cases


TILE_CASES = _tile_cases() + [
    (small_params(T=3, C=16, H=23, W=29, ws=9, wt=1, ps=7, k=10), "edge"),
    (small_params(T=3, C=8, H=17, W=19, ws=5, wt=1, ps=3, k=7, stride1=0.5), "edge"),
    # query strides above 1: smaller tiles of strided queries on the same halo
    (small_params(T=3, C=16, H=37, W=41, ws=9, wt=1, ps=7, k=10, stride0=2), "smooth"),
    (small_params(T=3, C=12, HD=2, H=29, W=33, ws=7, wt=2, ps=5, k=12, stride0=2), "frac"),
    (small_params(T=2, C=8, H=31, W=26, ws=5, wt=1, ps=3, k=9, stride0=3, stride1=0.5), "wide"),
    (small_params(T=3, C=8, H=23, W=25, ws=9, wt=1, ps=4, k=16, stride0=4), "edge"),
    (small_params(T=2, C=6, H=19, W=21, ws=8, wt=1, ps=6, k=20, stride0=2), "far"),
    (small_params(T=3, C=10, H=21, W=27, ws=9, wt=1, ps=2, k=10, stride0=5), "int"),
    # a key stride whose products S_K * (d - r) are not exact in fp32: the
    # displacement rounds twice (product, then sum), never as one fused
    # multiply-add, on both sides
    (small_params(T=3, C=8, H=23, W=26, ws=9, wt=1, ps=5, k=10, stride1=0.3), "frac"),
    (small_params(T=2, C=6, H=19, W=22, ws=7, wt=1, ps=3, k=8, stride1=0.7, stride0=2), "smooth"),
    # one query per tile 37 rows below its neighbours, one 5000 rows outside
    # the frame: the shift union is clipped to rows a valid cell can read
    (small_params(T=3, C=8, H=64, W=40, ws=9, wt=1, ps=7, k=10), "vspread"),
    (small_params(T=2, C=8, H=61, W=33, ws=5, wt=1, ps=3, k=8, stride1=0.5), "vspread"),
    (small_params(T=3, C=8, H=30, W=56, ws=9, wt=1, ps=5, k=10), "split"),
    # windows above 9 at P = 7 (the 15 x 15 window-table instance): every
    # window side class, key strides 1 and 1/2, strided queries, k past 16
    (small_params(T=3, C=16, H=29, W=33, ws=15, wt=1, ps=7, k=10), "smooth"),
    (small_params(T=2, C=8, H=24, W=27, ws=11, wt=1, ps=7, k=20, stride1=0.5), "frac"),
    (small_params(T=2, C=12, H=31, W=26, ws=13, wt=0, ps=7, k=12, stride0=2), "edge"),
    (small_params(T=3, C=8, H=20, W=40, ws=15, wt=1, ps=7, k=10), "wide"),
    # k above the 81 cells of the top-k's seeding spiral
    (small_params(T=2, C=8, H=21, W=23, ws=15, wt=1, ps=7, k=100), "smooth"),
]
TILE_IDS = ["t%d-ws%d-wt%d-ps%d-sk%g-k%d-%s" % (i, p["ws"], p["wt"], p["ps"], p["stride1"], p["k"], kd)
            for i, (p, kd) in enumerate(TILE_CASES)]


def _tile_flows(p, kind, r):
    fshp = (p["B"], p["T"], 2 * p["wt"], 2, p["H"], p["W"])
    if kind == "smooth":  # one offset per frame pair plus a little jitter: small union
        base = r.uniform(-4, 4, fshp[:4] + (1, 1))
        return (base + r.uniform(-0.4, 0.4, fshp)).astype(np.float32)
    if kind == "wide":  # spread of about 14 px: several rounds of shift rows
        return r.uniform(-7, 7, fshp).astype(np.float32)
    if kind == "far":  # +-60 px: the union exceeds the LDS layout
        return (r.choice([-1.0, 1.0], fshp) * 60.0 + r.uniform(-1, 1, fshp)).astype(np.float32)
    if kind == "split":  # column offsets of +-12 px alternating along each row: a union wider than 30 shifts
        fl = r.uniform(-0.5, 0.5, fshp)
        sign = np.where(np.arange(p["W"]) % 2 == 0, -1.0, 1.0)
        fl[:, :, :, 1] += 12.0 * sign
        return fl.astype(np.float32)
    if kind == "vspread":  # small offsets, but one query per tile far below and one far outside the frame
        fl = r.uniform(-2, 2, fshp)
        fl[:, :, :, 0, 0::10, 0::8] = 37.25
        fl[:, :, :, 0, 5::10, 3::8] = -5000.5
        return fl.astype(np.float32)
    if kind == "int":
        return r.integers(-3, 4, fshp).astype(np.float32)
    if kind == "edge":  # just below integers: adding a cell offset can round up to the next integer
        m = r.integers(-3, 4, fshp).astype(np.float32)
        below = np.nextafter(m, np.float32(-np.inf), dtype=np.float32)
        return np.where(r.random(fshp) < 0.7, below, r.uniform(-3, 3, fshp)).astype(np.float32)
    return r.uniform(-3, 3, fshp).astype(np.float32)


@pytest.mark.parametrize("case", range(len(TILE_CASES)), ids=TILE_IDS)
def test_tiled_search_topk(dev, case):
    p, kind = TILE_CASES[case]
    r = np.random.default_rng(8000 + case)
    shp = (p["B"], p["T"], p["C"], p["H"], p["W"])
    q = r.standard_normal(shp, dtype=np.float32)
    k = r.standard_normal(shp, dtype=np.float32)
    flows = _tile_flows(p, kind, r)
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    res = oracle.search(q, k, flows, p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])


# The tiled route at P = 7, S_Q = 1 with 64 channels per head (the 480x854
# workload's channel count: 16 chunks of 4 channels): smooth, wide (several
# shift-column blocks), far (scored directly) and tall (several rounds of
# shift rows) unions; two heads; key strides below 1; L2; windows of 5 to 9.
C64_CASES = [
    (small_params(T=3, C=64, H=30, W=33, ws=9, wt=1, ps=7, k=10), "smooth"),
    (small_params(T=3, C=64, H=27, W=31, ws=9, wt=1, ps=7, k=10), "wide"),
    (small_params(T=2, C=128, HD=2, H=23, W=26, ws=7, wt=1, ps=7, k=12, stride1=0.5), "frac"),
    (small_params(T=3, C=64, H=21, W=37, ws=9, wt=1, ps=7, k=20, dist_type=1), "edge"),
    (small_params(T=2, C=64, H=64, W=24, ws=9, wt=1, ps=7, k=10), "vspread"),
    (small_params(T=2, C=64, H=20, W=22, ws=9, wt=1, ps=7, k=10), "far"),
    (small_params(T=3, C=64, H=26, W=29, ws=5, wt=1, ps=7, k=8, stride1=0.3), "int"),
    (small_params(B=2, T=3, C=64, H=19, W=41, ws=9, wt=2, ps=7, k=16, dist_type=1, stride1=0.75), "split"),
]


@pytest.mark.parametrize("case", range(len(C64_CASES)),
                         ids=["c%d-ws%d-hd%d-sk%g-d%d-%s" % (i, p["ws"], p["HD"], p["stride1"], p["dist_type"], kd)
                              for i, (p, kd) in enumerate(C64_CASES)])
def test_tiled_search_c64(dev, case):
    p, kind = C64_CASES[case]
    r = np.random.default_rng(9500 + case)
    shp = (p["B"], p["T"], p["C"], p["H"], p["W"])
    q = r.standard_normal(shp, dtype=np.float32)
    k = (q + 0.5 * r.standard_normal(shp, dtype=np.float32)).astype(np.float32) if case % 2 else \
        r.standard_normal(shp, dtype=np.float32)
    flows = _tile_flows(p, kind, r)
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    res = oracle.search(q, k, flows, p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])


def test_tiled_nan_features_c64(dev):
    """NaN feature values away from the borders with 64 channels (P = 7):
    every candidate whose patch reads one is invalid, as in the oracle."""
    p = small_params(T=3, C=64, H=34, W=36, ws=9, wt=1, ps=7, k=10)
    r = np.random.default_rng(9600)
    q, k, v, flows = _inputs(p, 9601)
    m = 4 + 6
    for arr in (q, k):
        for _ in range(4):
            arr[0, r.integers(0, 3), r.integers(0, 64), r.integers(m, 34 - m), r.integers(m, 36 - m)] = np.nan
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    assert not np.isnan(_h(gd)).any()
    res = oracle.search(q, k, flows, p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])


# Task packing of the tiled scores kernel: every tile of every frame gets
# offsets whose integer parts span a chosen number of rows and columns, so
# the union of its windows is 10..22 shift rows by 10..26 shift columns.
# That runs every tail length (0-3 rows past the last whole quad of 4), every
# number of 6-column blocks (2-5), the channel split of the tail (1, 2 or 4
# parts) and unions that take two rounds of rows.
def _packing_flows(p, seed):
    r = np.random.default_rng(seed)
    tqh, tqw = 16 - p["ps"] + 1, 8  # query tile of the tiled kernel at query stride 1
    fl = np.zeros((p["B"], p["T"], 2 * p["wt"], 2, p["H"], p["W"]), np.float32)
    n = 0
    for t in range(p["T"]):
        for slot in range(2 * p["wt"]):
            for y0 in range(0, p["H"], tqh):
                for x0 in range(0, p["W"], tqw):
                    sh, sw = (n * 5) % 13, (n * 7) % 17
                    n += 1
                    yy, xx = np.mgrid[y0:min(y0 + tqh, p["H"]), x0:min(x0 + tqw, p["W"])]
                    j = (yy - y0) * tqw + (xx - x0)
                    base_h, base_w = r.integers(-2, 3, 2)
                    fl[:, t, slot, 0, yy, xx] = base_h + 0.3 + (j % (sh + 1))
                    fl[:, t, slot, 1, yy, xx] = base_w + 0.6 + ((j * 3) % (sw + 1))
    return fl


@pytest.mark.parametrize("ps,dist_type", [(7, 0), (7, 1), (3, 0)])
def test_tiled_task_packing(dev, ps, dist_type):
    p = small_params(T=3, C=8, H=40 if ps == 7 else 42, W=48, ws=9, wt=1, ps=ps, k=10, dist_type=dist_type)
    r = np.random.default_rng(9100 + ps + dist_type)
    shp = (p["B"], p["T"], p["C"], p["H"], p["W"])
    q = r.standard_normal(shp, dtype=np.float32)
    k = r.standard_normal(shp, dtype=np.float32)
    flows = _packing_flows(p, 9200 + ps)
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    res = oracle.search(q, k, flows, p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])


# Squared L2 through the tiled path (key stride 1): inner products from the
# tiled kernel, key and query norm terms from their own kernel; border queries
# (clipped patches), wide unions (norms read straight from memory) and every
# patch size.
L2_TILE_CASES = [
    (small_params(T=3, C=8, H=23, W=31, ws=9, wt=1, ps=7, k=10, dist_type=1), "frac"),
    (small_params(T=5, C=32, H=37, W=53, ws=9, wt=2, ps=7, k=10, dist_type=1), "smooth"),
    (small_params(T=2, C=5, H=17, W=19, ws=5, wt=1, ps=3, k=7, dist_type=1), "int"),
    (small_params(T=3, C=12, HD=2, H=20, W=41, ws=7, wt=1, ps=5, k=16, dist_type=1), "wide"),
    (small_params(T=2, C=4, H=13, W=16, ws=3, wt=1, ps=1, k=4, dist_type=1), "far"),
    (small_params(T=4, C=9, H=9, W=8, ws=8, wt=2, ps=6, k=13, dist_type=1), "frac"),
    (small_params(B=2, T=1, C=16, H=21, W=22, ws=9, wt=0, ps=4, k=12, dist_type=1), "frac"),
    (small_params(T=3, C=70, H=19, W=26, ws=9, wt=1, ps=2, k=10, dist_type=1), "smooth"),
    (small_params(T=3, C=16, H=21, W=26, ws=9, wt=1, ps=7, k=10, dist_type=1), "edge"),
    (small_params(T=3, C=16, H=25, W=30, ws=9, wt=1, ps=7, k=10, dist_type=1), "far"),
    (small_params(T=3, C=16, H=33, W=35, ws=9, wt=1, ps=7, k=10, dist_type=1, stride0=2), "smooth"),
    (small_params(T=2, C=8, H=27, W=22, ws=5, wt=1, ps=3, k=20, dist_type=1, stride0=3), "frac"),
    # in-frame candidates in tiles whose union is too wide for the LDS layout
    # (+-12 px alternating column offsets): scored per candidate as inner
    # products, ranked by the squared L2 distance
    (small_params(T=3, C=8, H=26, W=56, ws=9, wt=1, ps=7, k=10, dist_type=1), "split"),
    (small_params(T=3, C=8, H=64, W=40, ws=9, wt=1, ps=7, k=10, dist_type=1), "vspread"),
    # fractional key strides: the norm terms cell by cell (each cell its own
    # bilinear fractions), border queries, every patch size class
    (small_params(T=3, C=8, H=23, W=31, ws=9, wt=1, ps=7, k=10, dist_type=1, stride1=0.5), "frac"),
    (small_params(T=3, C=12, HD=2, H=21, W=26, ws=7, wt=1, ps=5, k=12, dist_type=1, stride1=0.75), "edge"),
    (small_params(T=2, C=5, H=17, W=19, ws=5, wt=1, ps=3, k=7, dist_type=1, stride1=0.3), "smooth"),
    (small_params(T=2, C=4, H=13, W=16, ws=9, wt=1, ps=1, k=6, dist_type=1, stride1=0.25), "int"),
    (small_params(T=3, C=8, H=25, W=30, ws=9, wt=1, ps=7, k=10, dist_type=1, stride1=0.5), "far"),
    (small_params(T=3, C=16, H=33, W=35, ws=9, wt=1, ps=7, k=10, dist_type=1, stride0=2, stride1=0.5), "wide"),
    # windows above 9 at P = 7 (15 x 15 window tables, norm terms per cell)
    (small_params(T=3, C=8, H=27, W=30, ws=15, wt=1, ps=7, k=10, dist_type=1), "smooth"),
    (small_params(T=2, C=8, H=22, W=25, ws=11, wt=1, ps=7, k=12, dist_type=1, stride1=0.5), "frac"),
    (small_params(T=2, C=8, H=19, W=22, ws=13, wt=1, ps=7, k=128, dist_type=1), "smooth"),
    # norm terms from the summed-area tables at the frame's edges: a frame
    # smaller than the patch, and a thin one at S_K = 1/4
    (small_params(T=2, C=8, H=5, W=6, ws=5, wt=1, ps=7, k=6, dist_type=1, stride1=0.5), "frac"),
    (small_params(T=3, C=4, H=9, W=40, ws=9, wt=1, ps=5, k=10, dist_type=1, stride1=0.25), "wide"),
]


@pytest.mark.parametrize("case", range(len(L2_TILE_CASES)),
                         ids=["l%d-ws%d-ps%d-sk%g-%s" % (i, p["ws"], p["ps"], p["stride1"], kd)
                              for i, (p, kd) in enumerate(L2_TILE_CASES)])
def test_tiled_search_l2(dev, case):
    p, kind = L2_TILE_CASES[case]
    r = np.random.default_rng(8500 + case)
    shp = (p["B"], p["T"], p["C"], p["H"], p["W"])
    q = r.standard_normal(shp, dtype=np.float32)
    k = (q + 0.3 * r.standard_normal(shp, dtype=np.float32)).astype(np.float32) if case % 2 else \
        r.standard_normal(shp, dtype=np.float32)
    flows = _tile_flows(p, kind, r)
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    res = oracle.search(q, k, flows, p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])


# Single-pixel patches at any query stride (the multi-head workload's path):
# windows up to 15, k up to 30, several heads, ragged query grids.
P1_CASES = [
    (small_params(T=4, C=64, HD=4, H=40, W=37, ws=15, wt=1, ps=1, stride0=2, k=30), "smooth"),
    (small_params(T=3, C=8, HD=2, H=31, W=26, ws=15, wt=1, ps=1, stride0=3, k=20), "frac"),
    (small_params(B=2, T=2, C=5, H=19, W=23, ws=9, wt=1, ps=1, stride0=2, k=12), "int"),
    (small_params(T=3, C=16, HD=1, H=22, W=30, ws=7, wt=1, ps=1, stride0=2, k=9), "wide"),
    (small_params(T=2, C=4, H=17, W=18, ws=5, wt=1, ps=1, stride0=2, k=6), "far"),
    (small_params(T=5, C=33, HD=1, H=25, W=21, ws=14, wt=2, ps=1, stride0=4, k=17), "frac"),
    (small_params(T=3, C=16, HD=2, H=21, W=27, ws=15, wt=1, ps=1, stride0=2, k=30), "edge"),
    (small_params(T=3, C=12, HD=1, H=16, W=19, ws=9, wt=1, ps=1, stride0=1, k=10), "edge"),
]


# The multi-head workload's settings at 40 x 56 on a smooth motion video:
# with k = 30 the single-pixel search selects inside its scoring kernel
# (query frame first: bisection of the first frame's cells, then merges of
# few cells per frame); with k = 40 the scores go through the workspace to
# the wave top-k, whose three selection paths this video reaches: about 94%
# of the rows have at most 64 candidates at or above the first threshold,
# about 6% between 65 and 128 (two entries per lane, 128-entry sort) and a
# few rows more than 128 (bisection for the exact k-th key).
@pytest.mark.parametrize("kk", [30, 40])
def test_wave_topk_paths(dev, kk):
    p = small_params(B=1, T=8, C=64, HD=4, H=40, W=56, ws=15, wt=3, ps=1, stride0=2, k=kk)
    x, flows = _motion_inputs(p, 3, 6.0)
    gd, gi = B.snls_search(_d(x, dev), _d(x, dev), _d(flows, dev), p)
    out = B.snls_aggregate(_d(x, dev), gd, gi, p, 1.0)
    torch.cuda.synchronize()
    res = oracle.search(x, x, flows, p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])
    assert_close(_h(out), oracle.aggregate(x, _h(gd), _h(gi), p, 1.0), "aggregate (P = 1)")


# Exact ties: 0/1 features and integer offsets make every score an exact
# integer on both sides, so the order (score, then smaller id) must match the
# oracle element for element -- the large-k selection's bisection path and
# its choice among keys equal to the k-th.
TIE_CASES = [
    small_params(T=3, C=4, H=20, W=21, ws=9, wt=1, ps=1, stride0=2, k=40),
    small_params(T=3, C=3, H=17, W=19, ws=7, wt=1, ps=3, k=20),
    small_params(T=3, C=3, H=17, W=19, ws=7, wt=1, ps=3, k=10),
    small_params(T=2, C=2, H=16, W=18, ws=5, wt=1, ps=3, k=30, dist_type=1),
    small_params(T=3, C=1, H=12, W=13, ws=9, wt=2, ps=1, k=64),
    # single-pixel patches with k <= 32 (selection inside the scoring
    # kernel): tied keys beyond 32 of a frame take the tie path of its
    # bisection; frames outside the clip fill with invalid candidates
    small_params(T=3, C=2, H=20, W=21, ws=9, wt=1, ps=1, stride0=2, k=20),
    small_params(T=2, C=1, H=19, W=17, ws=15, wt=2, ps=1, stride0=2, k=32),
    small_params(T=1, C=3, H=9, W=11, ws=3, wt=2, ps=1, stride0=2, k=25),
]


@pytest.mark.parametrize("case", range(len(TIE_CASES)))
def test_topk_exact_ties(dev, case):
    p = TIE_CASES[case]
    r = np.random.default_rng(8900 + case)
    shp = (p["B"], p["T"], p["C"], p["H"], p["W"])
    q = r.integers(0, 2, shp).astype(np.float32)
    k = r.integers(0, 2, shp).astype(np.float32)
    fshp = (p["B"], p["T"], 2 * p["wt"], 2, p["H"], p["W"])
    flows = r.integers(-2, 3, fshp).astype(np.float32)
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    res = oracle.search(q, k, flows, p)
    kk = p["k"]
    np.testing.assert_array_equal(_h(gd).reshape(-1, kk), res["dists"][:, :kk].astype(np.float32))
    np.testing.assert_array_equal(_h(gi).reshape(-1, kk, 3), res["inds"][:, :kk].astype(np.float32))


@pytest.mark.parametrize("case", range(len(P1_CASES)),
                         ids=["p%d-ws%d-s%d-%s" % (i, p["ws"], p["stride0"], kd) for i, (p, kd) in enumerate(P1_CASES)])
def test_p1_search(dev, case):
    p, kind = P1_CASES[case]
    r = np.random.default_rng(8700 + case)
    shp = (p["B"], p["T"], p["C"], p["H"], p["W"])
    q = r.standard_normal(shp, dtype=np.float32)
    k = r.standard_normal(shp, dtype=np.float32)
    flows = _tile_flows(p, kind, r)
    v = r.standard_normal(shp, dtype=np.float32)
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    out = B.snls_aggregate(_d(v, dev), gd, gi, p, 0.5)
    torch.cuda.synchronize()
    res = oracle.search(q, k, flows, p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])
    assert_close(_h(out), oracle.aggregate(v, _h(gd), _h(gi), p, 0.5), "aggregate (P = 1)")


# ------------------------------------------- the example's interface --

@pytest.mark.parametrize("nb,T,H,W,wt,kind", [(1, 5, 23, 31, 2, "frac"), (2, 4, 9, 14, 3, "frac"),
                                              (1, 6, 16, 16, 2, "int"), (1, 3, 1, 7, 2, "frac"),
                                              (1, 7, 12, 10, 4, "far")])
def test_chain_flows(dev, nb, T, H, W, wt, kind):
    """Flow chaining from one-step forward/backward flows against the oracle;
    then a search on the chained offsets against the oracle's."""
    r = np.random.default_rng(9400 + T + H)
    shp = (nb, T, 2, H, W)
    if kind == "int":
        ff, bf = r.integers(-2, 3, shp).astype(np.float32), r.integers(-2, 3, shp).astype(np.float32)
    elif kind == "far":  # large, smooth offsets: most reads clamp at the border (a rough field of this
        # size would amplify rounding by its gradient at every step of the chain)
        ff = (r.choice([-30.0, 30.0], (nb, T, 2, 1, 1)) + r.uniform(-0.5, 0.5, shp)).astype(np.float32)
        bf = (r.choice([-30.0, 30.0], (nb, T, 2, 1, 1)) + r.uniform(-0.5, 0.5, shp)).astype(np.float32)
    else:
        ff, bf = r.uniform(-2.5, 2.5, shp).astype(np.float32), r.uniform(-2.5, 2.5, shp).astype(np.float32)
    fl = B.snls_chain_flows(_d(ff, dev), _d(bf, dev), wt)
    torch.cuda.synchronize()
    ref = oracle.chain_flows(ff, bf, wt)
    assert_close(_h(fl), ref, "chained flows")
    p = small_params(B=nb, T=T, C=6, H=H, W=W, ws=5, wt=wt, ps=3, k=7)
    q = r.standard_normal((nb, T, 6, H, W), dtype=np.float32)
    gd, gi = B.snls_search(_d(q, dev), _d(q, dev), fl, p)
    torch.cuda.synchronize()
    res = oracle.search(q, q, _h(fl), p)
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])


@pytest.mark.parametrize("ps,stride0,HD,k,C", [(7, 1, 1, 10, 64), (3, 2, 2, 5, 12), (1, 2, 4, 30, 64),
                                                (5, 1, 1, 4, 20)])
def test_aggregate_stacked(dev, ps, stride0, HD, k, C):
    """Stacked aggregation against the oracle, and its sum over the neighbours
    against snls_aggregate on the same neighbours."""
    p = small_params(T=3, C=C, HD=HD, H=21, W=26, ws=9, wt=1, ps=ps, stride0=stride0, k=k)
    r = np.random.default_rng(9500 + ps + k)
    q, kk, v, flows = _inputs(p, 9600 + ps)
    gd, gi = B.snls_search(_d(q, dev), _d(kk, dev), _d(flows, dev), p)
    st = B.snls_aggregate_stacked(_d(v, dev), gd, gi, p, 0.3)
    out = B.snls_aggregate(_d(v, dev), gd, gi, p, 0.3)
    torch.cuda.synchronize()
    ref = oracle.aggregate_stacked(v, _h(gd), _h(gi), p, 0.3)
    assert_close(_h(st), ref, "stacked aggregation")
    summed = _h(st).astype(np.float64).sum(2).transpose(0, 2, 1, 3, 4, 5).reshape(tuple(out.shape))
    assert_close(summed, _h(out).astype(np.float64), "stacked aggregation summed over k", rel=1e-4)


# --------------------------------------------------- non-finite inputs --

@pytest.mark.parametrize("dist_type,ps,ws,k,stride0", [(0, 3, 5, 10, 1), (0, 7, 9, 10, 1), (1, 3, 5, 10, 1),
                                                       (0, 4, 8, 10, 1), (0, 7, 9, 20, 1), (0, 1, 9, 20, 2),
                                                       (0, 1, 15, 30, 2), (1, 5, 7, 24, 1), (0, 7, 9, 10, 2),
                                                       (1, 3, 5, 10, 3)])
def test_nan_features_match_oracle(dev, dist_type, ps, ws, k, stride0):
    """NaN feature values away from the borders: every candidate whose patch
    reads one is invalid (a NaN similarity ranks as an invalid candidate), as
    in the oracle; the tiled, single-pixel and direct kernels, and both top-k
    kernels."""
    p = small_params(T=3, C=8, H=40, W=42, ws=ws, wt=1, ps=ps, k=k, stride0=stride0, dist_type=dist_type)
    r = np.random.default_rng(8100 + ps)
    q, k, v, flows = _inputs(p, 8200 + ps)
    m = ws // 2 + 6
    for arr in (q, k):
        for _ in range(4):
            arr[0, r.integers(0, 3), r.integers(0, 8), r.integers(m, 40 - m), r.integers(m, 42 - m)] = np.nan
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    assert not np.isnan(_h(gd)).any()
    res = oracle.search(q, k, flows, p)
    assert np.isinf(res["all_dists"]).sum() > np.isinf(oracle.search(
        np.nan_to_num(q), np.nan_to_num(k), flows, p)["all_dists"]).sum()
    compare_topk(_h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3), res, p["k"])


@pytest.mark.parametrize("dist_type,ps,ws,stride0,k", [(0, 7, 9, 1, 12), (0, 3, 5, 1, 12), (1, 3, 5, 2, 12),
                                                       (0, 1, 15, 2, 30), (0, 7, 9, 1, 20)])
def test_nonfinite_inputs_stay_in_bounds(dev, dist_type, ps, ws, stride0, k):
    """NaN and +-inf anywhere in q, k and the flows (scores are then not
    specified): no NaN score is kept, and every kept neighbour is a distinct
    candidate of the query's own window."""
    p = small_params(T=4, C=8, H=23, W=30, ws=ws, wt=2, ps=ps, k=k, stride0=stride0, dist_type=dist_type)
    r = np.random.default_rng(8300 + ps + stride0)
    q, k, v, flows = _inputs(p, 8400 + ps)
    for arr in (q, k, flows):
        flat = arr.reshape(-1)
        idx = r.choice(flat.size, size=flat.size // 50, replace=False)
        flat[idx] = r.choice([np.nan, np.inf, -np.inf], size=idx.size)
    gd, gi = B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    gd_h, gi_h = _h(gd).reshape(-1, p["k"]), _h(gi).reshape(-1, p["k"], 3)
    assert not np.isnan(gd_h).any()
    _, cand = oracle.search_all(np.zeros_like(q), np.zeros_like(k), flows, p)
    cand = cand.reshape(gi_h.shape[0], -1, 3).astype(np.float32)
    key = lambda a: tuple("nan" if np.isnan(x) else float(x) for x in a)
    for row in range(gi_h.shape[0]):
        valid = {key(c): j for j, c in enumerate(cand[row])}
        ids = [valid.get(key(gi_h[row, i])) for i in range(p["k"])]
        assert None not in ids, "row %d keeps a position outside its window" % row
        if np.isfinite(gi_h[row]).all():  # non-finite offsets make positions of one frame coincide
            assert len(set(ids)) == p["k"], "row %d repeats a candidate" % row


def test_deterministic(dev):
    p = small_params(T=3, C=8, H=33, W=33, HD=2, ws=5, wt=1, ps=3, k=7)
    q, k, v, flows = _inputs(p, 5000)
    a = [B.snls_search(_d(q, dev), _d(k, dev), _d(flows, dev), p) for _ in range(2)]
    o = [B.snls_aggregate(_d(v, dev), a[0][0], a[0][1], p, 0.5) for _ in range(2)]
    torch.cuda.synchronize()
    assert torch.equal(a[0][0], a[1][0]) and torch.equal(a[0][1], a[1][1])
    assert torch.equal(o[0], o[1])


# ------------------------------------------------------------ workloads --

_CFG_CACHE = {}


def _cfg(idx):
    if idx not in _CFG_CACHE:
        _CFG_CACHE.clear()
        _CFG_CACHE[idx] = make_config(idx)
    return _CFG_CACHE[idx]


def _sample_rows(p, n, rng):
    nH, nW = oracle.grid(p)
    rows = []
    for b in range(p["B"]):
        for hd in range(p["HD"]):
            for t in range(p["T"]):
                for mh, mw in ((0, 0), (0, nW - 1), (nH - 1, 0), (nH - 1, nW - 1), (nH // 2, 0), (0, nW // 2)):
                    rows.append((((b * p["HD"] + hd) * p["T"] + t) * nH + mh) * nW + mw)
    total = oracle.n_queries(p)
    rows += list(rng.choice(total, size=min(n, total), replace=False))
    return np.unique(np.array(rows, np.int64))


def _covering_rows(p, pix):
    nH, nW = oracle.grid(p)
    lo, S = -(p["ps"] // 2), p["stride0"]
    rows = set()
    for pi in pix:
        x = pi % p["W"]
        y = (pi // p["W"]) % p["H"]
        t = (pi // (p["W"] * p["H"])) % p["T"]
        b = pi // (p["W"] * p["H"] * p["T"])
        for ph in range(lo, lo + p["ps"]):
            for pw in range(lo, lo + p["ps"]):
                h, w = y - ph, x - pw
                if h < 0 or w < 0 or h % S or w % S or h // S >= nH or w // S >= nW:
                    continue
                for hd in range(p["HD"]):
                    rows.add((((b * p["HD"] + hd) * p["T"] + t) * nH + h // S) * nW + w // S)
    return np.array(sorted(rows), np.int64)


@pytest.mark.parametrize("idx", [0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10])
def test_workload_parity(dev, idx):
    """Search + top-k + aggregation of each workload at its full size (the
    launch configuration bench.py times), on sampled rows and pixels: the five
    workloads, then the paper's own benchmark shapes (320 x 320 at query
    strides 1 and 2, the 152 x 152 x 192 memory shape), the 480 x 854
    workload at key stride 1/2 and at query stride 2, and the settings of
    the paper's code example."""
    c = _cfg(idx)
    p, scale = c["params"], c["scale"]
    print("workload %d (%s) %s" % (idx, c["name"], p), flush=True)
    rng = np.random.default_rng(77 + idx)
    qd, fd = _d(c["q"], dev), _d(c["flows"], dev)
    gd, gi = B.snls_search(qd, qd, fd, p)
    out = B.snls_aggregate(qd, gd, gi, p, scale)
    torch.cuda.synchronize()
    kk = p["k"]
    gd_h, gi_h, out_h = _h(gd).reshape(-1, kk), _h(gi).reshape(-1, kk, 3), _h(out)
    assert np.isfinite(out_h).all()
    # search + top-k on sampled rows
    rows = _sample_rows(p, 400 if idx else 4000, rng)
    res = oracle.search(c["q"], c["k"], c["flows"], p, qids=rows)
    n_sw, _ = compare_topk(gd_h[rows], gi_h[rows], res, kk, scale=rms_finite(gd_h))
    print("  rows %d, near-tie swaps %d" % (len(rows), n_sw), flush=True)
    # aggregation on sampled pixels, decoupled and end to end
    total_pix = p["B"] * p["T"] * p["H"] * p["W"]
    pix = np.unique(np.concatenate([rng.choice(total_pix, 60, replace=False), [0, total_pix - 1, p["W"] - 1]]))
    nH, nW = oracle.grid(p)
    shp = (p["B"], p["HD"], p["T"], nH, nW, kk)
    ref = oracle.aggregate_at(c["v"], gd_h.reshape(shp), gi_h.reshape(shp + (3,)), p, pix, scale)
    got = out_h.transpose(0, 1, 3, 4, 2).reshape(-1, p["C"])[pix]
    assert_close(got, ref, "aggregate at sampled pixels (GPU neighbours)", scale=rms_finite(out_h))
    cov = _covering_rows(p, pix[:24])
    res2 = oracle.search(c["q"], c["k"], c["flows"], p, qids=cov)
    _, sw2 = compare_topk(gd_h[cov], gi_h[cov], res2, kk, scale=rms_finite(gd_h))
    d_all = gd_h.astype(np.float64).copy()
    i_all = gi_h.astype(np.float64).copy()
    d_all[cov] = res2["dists"][:, :kk]
    i_all[cov] = res2["inds"][:, :kk]
    ref2 = oracle.aggregate_at(c["v"], d_all.reshape(shp), i_all.reshape(shp + (3,)), p, pix[:24], scale)
    swapped_pix = set()
    for r in cov[sw2]:
        swapped_pix.add(int(r))
    keep = [i for i, pi in enumerate(pix[:24]) if not (set(_covering_rows(p, [pi]).tolist()) & swapped_pix)]
    assert_close(got[:24][keep], ref2[keep], "aggregate at sampled pixels (end to end)", scale=rms_finite(out_h))


# ------------------------------------------------------------- backward --

def test_backward_matches_oracle(dev):
    """Gradients w.r.t. q, k, v and flows (train256 settings on a 40 x 44 crop
    size), with an upstream gradient on the scores as well."""
    p = config_params(4, H=40, W=44)
    r = np.random.default_rng(11)
    q, k, v, flows = _inputs(p, 6000)
    q *= 0.3
    k *= 0.3
    go = r.standard_normal(q.shape, dtype=np.float32)
    scale = 0.5
    qd, kd, vd, fd = (_d(a, dev) for a in (q, k, v, flows))
    gd, gi = B.snls_search(qd, kd, fd, p)
    nH, nW = oracle.grid(p)
    gdist = r.standard_normal((p["B"], p["HD"], p["T"], nH, nW, p["k"]), dtype=np.float32)
    grads = B.snls_backward(qd, kd, vd, fd, gd, gi, _d(go, dev), p, scale, grad_dists=_d(gdist, dev))
    torch.cuda.synchronize()
    ref = oracle.backward(q, k, v, flows, _h(gd), _h(gi), go, p, scale, grad_dists=gdist)
    for name, g_gpu, g_ref in zip(("dq", "dk", "dv", "dflows"), grads, ref):
        assert_close(_h(g_gpu), g_ref, name)
    assert np.any(_h(grads[3]) != 0)


@pytest.mark.parametrize("kw", [dict(dist_type=1, ps=3, ws=5, k=6), dict(HD=2, C=40, ps=5, ws=5, k=5),
                                dict(C=96, ps=3, ws=3, k=4, H=17, W=19), dict(stride0=2, ps=1, ws=7, k=9, HD=4, C=16),
                                dict(stride0=2, ps=3, ws=5, k=7, dist_type=1, wt=2, T=5),
                                dict(ps=7, ws=9, k=10, C=32, H=23, W=26), dict(ps=2, ws=4, k=6, C=8),
                                dict(ps=4, ws=5, k=8, HD=2, C=16, stride0=2), dict(ps=6, ws=3, k=5, C=64, H=19, W=21),
                                dict(ps=5, ws=5, k=12, C=24, dist_type=1)],
                         ids=["l2", "heads", "c96", "p1-s2", "l2-s2", "p7", "p2", "p4-s2", "p6", "p5-l2"])
def test_backward_shapes(dev, kw):
    """Gradients against the oracle over distances, heads, channel counts
    above one wave and query strides."""
    p = small_params(T=3, C=8, H=20, W=23, ws=5, wt=1, ps=3, k=5)
    p.update(kw)
    r = np.random.default_rng(6100 + len(str(kw)))
    q, k, v, flows = _inputs(p, 6200 + p["C"] + p["ps"])
    q *= 0.3
    k *= 0.3
    go = r.standard_normal(q.shape, dtype=np.float32)
    scale = 0.4
    qd, kd, vd, fd = (_d(a, dev) for a in (q, k, v, flows))
    gd, gi = B.snls_search(qd, kd, fd, p)
    grads = B.snls_backward(qd, kd, vd, fd, gd, gi, _d(go, dev), p, scale)
    torch.cuda.synchronize()
    ref = oracle.backward(q, k, v, flows, _h(gd), _h(gi), go, p, scale)
    for name, g_gpu, g_ref in zip(("dq", "dk", "dv", "dflows"), grads, ref):
        assert_close(_h(g_gpu), g_ref, name)


def test_backward_full_size_matches_oracle(dev):
    """train256 at its full size (256 x 256, T = 5, C = 64, P = 3, k = 10):
    dq, dk, dv and the flow gradients of the GPU against the oracle's
    gradients for the GPU's own neighbours, element by element.  q and k
    are separate tensors (scaled copies of the video) so that every
    gradient is checked on its own."""
    c = _cfg(4)
    p, scale = c["params"], c["scale"]
    q = np.ascontiguousarray(c["q"] * np.float32(0.5))
    k = np.ascontiguousarray(c["k"] * np.float32(0.4))
    print("backward at full size %s" % p, flush=True)
    qd, kd, vd, fd = (_d(a, dev) for a in (q, k, c["v"], c["flows"]))
    gd, gi = B.snls_search(qd, kd, fd, p)
    grads = B.snls_backward(qd, kd, vd, fd, gd, gi, _d(c["grad_out"], dev), p, scale)
    torch.cuda.synchronize()
    ref = oracle.backward(q, k, c["v"], c["flows"], _h(gd), _h(gi), c["grad_out"], p, scale)
    for name, g_gpu, g_ref in zip(("dq", "dk", "dv", "dflows"), grads, ref):
        assert_close(_h(g_gpu), g_ref, name)
        print("  %s ok" % name, flush=True)


def test_backward_adjoint_full_size(dev):
    """train256 at full size: v -> out is linear for fixed neighbours, so
    <out(x), y> = <x, grad_v(y)> with both sides from the GPU."""
    c = _cfg(4)
    p = c["params"]
    qd, fd = _d(c["q"], dev), _d(c["flows"], dev)
    gd, gi = B.snls_search(qd, qd, fd, p)
    r = np.random.default_rng(12)
    x = _d(r.standard_normal(c["q"].shape, dtype=np.float32), dev)
    y = _d(c["grad_out"], dev)
    out = B.snls_aggregate(x, gd, gi, p, c["scale"])
    _, _, gv, _ = B.snls_backward(qd, qd, x, fd, gd, gi, y, p, c["scale"])
    torch.cuda.synchronize()
    lhs = float((out.double() * y.double()).sum())
    rhs = float((x.double() * gv.double()).sum())
    assert abs(lhs - rhs) <= REL * max(abs(lhs), 1.0)


# ------------------------------------- the example's gather and reduction --

@pytest.mark.parametrize("ps,stride0,HD,C,k,stride1", [(3, 1, 2, 16, 10, 0.5), (7, 1, 1, 64, 6, 1.0),
                                                       (1, 2, 4, 64, 12, 1.0), (5, 2, 1, 8, 5, 1.0),
                                                       (3, 3, 2, 12, 4, 1.0), (3, 1, 1, 70, 4, 1.0),
                                                       (2, 1, 2, 6, 3, 1.0)],
                         ids=["example", "p7", "p1-heads", "p5-s2", "p3-s3", "c70-plain", "c3-plain"])
def test_gather_stacked_and_reduce(dev, ps, stride0, HD, C, k, stride1):
    """The example's gather with caller weights (weights with zeros, negative
    values, neighbours outside the clip or with non-finite offsets), the
    reduction over the k neighbours (MFMA) from the gathered stack, and the
    fused gather + reduction, against the oracle."""
    p = small_params(T=5, C=C, HD=HD, H=21, W=19, ws=5, wt=2, ps=ps, stride0=stride0, stride1=stride1, k=k)
    q, kk_, v, flows = _inputs(p, 7100 + ps * 10 + C)
    r = np.random.default_rng(7200 + C + ps)
    gd, gi = B.snls_search(_d(q, dev), _d(kk_, dev), _d(flows, dev), p)
    torch.cuda.synchronize()
    inds = _h(gi).copy()
    shp = _h(gd).shape
    wts = r.standard_normal(shp).astype(np.float32)
    wts[r.random(shp) < 0.2] = 0.0
    flat = inds.reshape(-1, 3)
    sel = r.choice(flat.shape[0], 7, replace=False)
    flat[sel[:3], 0] = np.array([5.0, -1.0, 2.5], np.float32)  # outside the clip / not an integer
    flat[sel[3:5], 1] = np.nan
    flat[sel[5:], 2] = np.inf
    vd, wd, idd = _d(v, dev), _d(wts, dev), _d(inds, dev)
    st = B.snls_gather_stacked(vd, wd, idd, p)
    torch.cuda.synchronize()
    ref = oracle.gather_stacked(v, wts, inds, p)
    assert_close(_h(st), ref, "stacked gather")
    if C // HD % 4 == 0 and C // HD <= 64:
        for cout in (C, 20, 128):
            proj = r.standard_normal((cout, C, k)).astype(np.float32) / np.sqrt(C * k)
            pd = _d(proj, dev)
            red = B.snls_stacked_reduce(st, pd, p)
            fused = B.snls_gather_reduce(vd, wd, idd, pd, p)
            torch.cuda.synchronize()
            ref_red = oracle.stacked_reduce(ref, proj, p)
            assert_close(_h(red), oracle.stacked_reduce(_h(st), proj, p), "reduction of the GPU stack (cout %d)" % cout)
            assert_close(_h(fused), ref_red, "fused gather + reduction (cout %d)" % cout)
    else:
        proj = _d(np.zeros((8, C, k), np.float32), dev)
        with pytest.raises(B.SnlsError):
            B.snls_gather_reduce(vd, wd, idd, proj, p)


def test_gather_reduce_example_full_size(dev):
    """The code example's pipeline at its own size (5 x 128 x 128, 16
    features in 2 heads, k = 10, key stride 1/2): search, weights = a softmax
    over the row with temperature 10 computed by the caller as in the example
    (+10 for the inner product, larger is better; invalid neighbours, -inf,
    get weight 0), the gather that keeps the neighbours apart, and the fused
    gather + reduction with a (16, 16, 10) kernel, element by element against
    the oracle."""
    from workloads import config_index
    c = _cfg(config_index("example_appb"))
    p = c["params"]
    qd, fd = _d(c["q"], dev), _d(c["flows"], dev)
    gd, gi = B.snls_search(qd, qd, fd, p)
    w = torch.softmax(10.0 * gd, dim=-1).contiguous()
    assert torch.isfinite(w).all()
    proj = torch.from_numpy(np.random.default_rng(31).standard_normal((16, 16, 10)).astype(np.float32) / 12.0).to(dev)
    st = B.snls_gather_stacked(qd, w, gi, p)
    out = B.snls_gather_reduce(qd, w, gi, proj, p)
    torch.cuda.synchronize()
    ref = oracle.gather_stacked(c["v"], _h(w), _h(gi), p)
    assert_close(_h(st), ref, "stacked gather (example size)")
    assert_close(_h(out), oracle.stacked_reduce(ref, _h(proj), p), "gather + reduction (example size)")
