"""Oracle for the Shifted Non-Local Search path (test infrastructure only).

This package is the plain, slow CPU reference that the HIP library is checked
against.  Only the test suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the library and its Python
binding never do, and the two share no code.

The arithmetic lives in ``snls_oracle.c`` (double precision, OpenMP over
queries).  This module only builds that file with gcc, converts numpy arrays to
float64 and back, and calls it through ctypes.  Section references are to
"Space-Time Attention with Shifted Non-Local Search" (Gauen & Chan, 2024):
Sec. 3.1 (non-local search), Sec. 3.2 (shifted search, top-L, aggregation).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "snls_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


class _Params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("B", "T", "C", "H", "W", "HD", "ws", "wt", "ps", "stride0")] + [
        ("stride1", ctypes.c_double),
        ("k", ctypes.c_int),
        ("dist_type", ctypes.c_int),
        ("fp32_positions", ctypes.c_int),
    ]


def build(force: bool = False) -> str:
    """Compile snls_oracle.c into liboracle.so (gcc, -O2, OpenMP, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-shared", "-fPIC",
             "-Wall", "-Wextra", "-Wno-unused-parameter", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i64 = ctypes.c_int64
        lib.oracle_search.argtypes = [P, P, P, P, P, i64, P, P]
        lib.oracle_topk.argtypes = [P, i64, ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P]
        lib.oracle_aggregate.argtypes = [P, P, P, P, ctypes.c_double, P]
        lib.oracle_aggregate_at.argtypes = [P, P, P, P, ctypes.c_double, P, i64, P]
        lib.oracle_search_fixed.argtypes = [P, P, P, P, P, P, P]
        lib.oracle_backward.argtypes = [P] * 9 + [ctypes.c_double, P, P, P, P]
        lib.oracle_bilinear_image.argtypes = [P, ctypes.c_int, ctypes.c_int, P, P, i64, P]
        ci = ctypes.c_int
        lib.oracle_chain_flows.argtypes = [P, P, ci, ci, ci, ci, ci, P]
        lib.oracle_aggregate_stacked.argtypes = [P, P, P, P, ctypes.c_double, P]
        lib.oracle_gather_stacked.argtypes = [P, P, P, P, P]
        lib.oracle_stacked_reduce.argtypes = [P, P, P, ci, P]
        for f in ("oracle_search", "oracle_topk", "oracle_aggregate", "oracle_aggregate_at",
                  "oracle_search_fixed", "oracle_backward", "oracle_bilinear_image", "oracle_chain_flows",
                  "oracle_aggregate_stacked", "oracle_gather_stacked", "oracle_stacked_reduce"):
            getattr(lib, f).restype = None
        _lib = lib
    return _lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _params(p: dict, fp32_positions: bool = True) -> _Params:
    s = _Params()
    for n in ("B", "T", "C", "H", "W", "HD", "ws", "wt", "ps", "stride0", "k", "dist_type"):
        setattr(s, n, int(p[n]))
    s.stride1 = float(p["stride1"])
    s.fp32_positions = 1 if fp32_positions else 0
    return s


def grid(p: dict):
    """Query grid (nH, nW) = ((H-1)//S_Q + 1, (W-1)//S_Q + 1) (appendix example)."""
    return (p["H"] - 1) // p["stride0"] + 1, (p["W"] - 1) // p["stride0"] + 1


def n_queries(p: dict) -> int:
    nH, nW = grid(p)
    return p["B"] * p["HD"] * p["T"] * nH * nW


def n_cand(p: dict) -> int:
    return (2 * p["wt"] + 1) * p["ws"] ** 2


def search_all(q, k, flows, p: dict, qids=None, fp32_positions: bool = True):
    """Every candidate of the listed query rows (all rows if qids is None).

    Returns (dists, inds): float64 arrays (nq, n_cand) and (nq, n_cand, 3), in
    candidate-id order ((dt+wt)*Ws + d_h)*Ws + d_w.  Sec. 3.2.
    """
    lib = _load()
    if qids is None:
        qids = np.arange(n_queries(p), dtype=np.int64)
    qids = np.ascontiguousarray(qids, dtype=np.int64)
    nc = n_cand(p)
    d = np.empty((len(qids), nc), np.float64)
    ind = np.empty((len(qids), nc, 3), np.float64)
    qq, kk, ff = _f64(q), _f64(k), _f64(flows)
    prm = _params(p, fp32_positions)
    lib.oracle_search(_ptr(qq), _ptr(kk), _ptr(ff), ctypes.byref(prm), _ptr(qids), len(qids), _ptr(d), _ptr(ind))
    return d, ind


def topk(dists, kk: int, dist_type: int):
    """top-L per row (Sec. 3.2): (values, column ids), best first, ties to the smaller id."""
    lib = _load()
    dd = _f64(dists)
    rows, ncols = dd.shape
    od = np.empty((rows, kk), np.float64)
    oi = np.empty((rows, kk), np.int64)
    lib.oracle_topk(_ptr(dd), rows, ncols, kk, dist_type, _ptr(od), _ptr(oi))
    return od, oi


def search(q, k, flows, p: dict, qids=None, extra: int = 1, fp32_positions: bool = True):
    """Search + top-k for the listed rows.

    Returns a dict with the top-(k+extra) values 'dists', column ids 'ids',
    positions 'inds' (rows, k+extra, 3) and the full rows 'all_dists',
    'all_inds'.  The entries past k let a comparison judge swaps at the k-th
    boundary.
    """
    ad, ai = search_all(q, k, flows, p, qids, fp32_positions)
    kk = min(p["k"] + extra, ad.shape[1])
    d, ids = topk(ad, kk, p["dist_type"])
    inds = np.take_along_axis(ai, ids[:, :, None], axis=1)
    return {"dists": d, "ids": ids, "inds": inds, "all_dists": ad, "all_inds": ai}


def aggregate(v, dists, inds, p: dict, scale: float = 1.0):
    """Weighted patch aggregation over the whole video (Sec. 3.2), float64 (B,T,C,H,W)."""
    lib = _load()
    vv, dd, ii = _f64(v), _f64(dists), _f64(inds)
    out = np.empty(vv.shape, np.float64)
    prm = _params(p)
    lib.oracle_aggregate(_ptr(vv), _ptr(dd), _ptr(ii), ctypes.byref(prm), float(scale), _ptr(out))
    return out


def aggregate_at(v, dists, inds, p: dict, pixels, scale: float = 1.0):
    """The aggregation at listed output pixels (flattened (b,t,y,x) indices); returns (npix, C)."""
    lib = _load()
    vv, dd, ii = _f64(v), _f64(dists), _f64(inds)
    pix = np.ascontiguousarray(pixels, dtype=np.int64)
    out = np.empty((len(pix), p["C"]), np.float64)
    prm = _params(p)
    lib.oracle_aggregate_at(_ptr(vv), _ptr(dd), _ptr(ii), ctypes.byref(prm), float(scale), _ptr(pix), len(pix),
                            _ptr(out))
    return out


def search_fixed(q, k, flows, p: dict, sel, fp32_positions: bool = False):
    """Distances and positions of a fixed candidate choice sel (rows, k, 3) = (dt, d_h, d_w)."""
    lib = _load()
    rows = n_queries(p)
    s = np.ascontiguousarray(sel, dtype=np.int32)
    assert s.shape == (rows, p["k"], 3)
    d = np.empty((rows, p["k"]), np.float64)
    ind = np.empty((rows, p["k"], 3), np.float64)
    qq, kk, ff = _f64(q), _f64(k), _f64(flows)
    prm = _params(p, fp32_positions)
    lib.oracle_search_fixed(_ptr(qq), _ptr(kk), _ptr(ff), ctypes.byref(prm), _ptr(s), _ptr(d), _ptr(ind))
    return d, ind


def backward(q, k, v, flows, dists, inds, grad_out, p: dict, scale: float = 1.0, grad_dists=None):
    """Gradients (dq, dk, dv, dflows) of the search + aggregation (top-k set held fixed), float64."""
    lib = _load()
    qq, kk, vv, ff = _f64(q), _f64(k), _f64(v), _f64(flows)
    dd, ii, go = _f64(dists), _f64(inds), _f64(grad_out)
    gd = _f64(grad_dists) if grad_dists is not None else None
    gq, gk, gv = np.empty(qq.shape), np.empty(kk.shape), np.empty(vv.shape)
    gf = np.empty(ff.shape)
    prm = _params(p)
    lib.oracle_backward(_ptr(qq), _ptr(kk), _ptr(vv), _ptr(ff), _ptr(dd), _ptr(ii), _ptr(go), _ptr(gd),
                        ctypes.byref(prm), float(scale), _ptr(gq), _ptr(gk), _ptr(gv), _ptr(gf))
    return gq, gk, gv, gf


def bilinear_image(img, ys, xs):
    """Bilinear reads of a 2-D image at (ys, xs); zero outside, pixel centres on integers."""
    lib = _load()
    im = _f64(img)
    y, x = _f64(ys).ravel(), _f64(xs).ravel()
    out = np.empty(len(y), np.float64)
    lib.oracle_bilinear_image(_ptr(im), im.shape[0], im.shape[1], _ptr(y), _ptr(x), len(y), _ptr(out))
    return out


def chain_flows(fflow, bflow, wt: int):
    """Offsets to frames t-wt..t+wt composed from one-step flows (B,T,2,H,W); returns (B,T,2wt,2,H,W)."""
    lib = _load()
    ff, bf = _f64(fflow), _f64(bflow)
    B, T, _, H, W = ff.shape
    out = np.empty((B, T, 2 * wt, 2, H, W), np.float64)
    lib.oracle_chain_flows(_ptr(ff), _ptr(bf), B, T, H, W, int(wt), _ptr(out))
    return out


def aggregate_stacked(v, dists, inds, p: dict, scale: float = 1.0):
    """The aggregation with the k neighbours kept apart: (B, HD, k, T, C/HD, H, W), float64."""
    lib = _load()
    vv, dd, ii = _f64(v), _f64(dists), _f64(inds)
    out = np.empty((p["B"], p["HD"], p["k"], p["T"], p["C"] // p["HD"], p["H"], p["W"]), np.float64)
    prm = _params(p)
    lib.oracle_aggregate_stacked(_ptr(vv), _ptr(dd), _ptr(ii), ctypes.byref(prm), float(scale), _ptr(out))
    return out


def gather_stacked(v, weights, inds, p: dict):
    """The example's gather with the caller's weights (B,HD,T,nH,nW,k):
    returns (B, HD, k, T, C/HD, H, W), float64."""
    lib = _load()
    vv, ww, ii = _f64(v), _f64(weights), _f64(inds)
    out = np.empty((p["B"], p["HD"], p["k"], p["T"], p["C"] // p["HD"], p["H"], p["W"]), np.float64)
    prm = _params(p)
    lib.oracle_gather_stacked(_ptr(vv), _ptr(ww), _ptr(ii), ctypes.byref(prm), _ptr(out))
    return out


def stacked_reduce(stacked, proj, p: dict):
    """The reduction over the k neighbours with kernel proj (Cout, C, k):
    returns (B, T, Cout, H, W), float64."""
    lib = _load()
    ss, pp = _f64(stacked), _f64(proj)
    cout = pp.shape[0]
    assert pp.shape == (cout, p["C"], p["k"]), pp.shape
    out = np.empty((p["B"], p["T"], cout, p["H"], p["W"]), np.float64)
    prm = _params(p)
    lib.oracle_stacked_reduce(_ptr(ss), _ptr(pp), ctypes.byref(prm), cout, _ptr(out))
    return out
