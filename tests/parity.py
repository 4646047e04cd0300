"""Comparison rules between the HIP library and the oracle.

* scores, aggregated outputs, gradients: |gpu - oracle| <= REL * max(|oracle|,
  rms(oracle tensor)) element by element (REL = 1e-4, fp32 computation);
* top-k: the kept scores match rank by rank within that tolerance; every
  kept position (frame, disp_h, disp_w) must be bit-identical to a candidate
  of the oracle's full row, and where the chosen candidate differs from the
  oracle's at that rank, its oracle score must lie within the tolerance of the
  oracle's score at that rank (a near-tie, where either choice is correct).
"""
from __future__ import annotations

import numpy as np

REL = 1e-4


def rms_finite(a) -> float:
    a = np.asarray(a, np.float64)
    f = a[np.isfinite(a)]
    return float(np.sqrt(np.mean(f * f))) if f.size else 0.0


def assert_close(gpu, ref, what: str, rel: float = REL, scale: float | None = None):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    inf_ref = ~np.isfinite(ref)
    if inf_ref.any():
        assert np.array_equal(gpu[inf_ref], ref[inf_ref]), "%s: non-finite entries differ" % what
    s = rms_finite(ref) if scale is None else scale
    fin = ~inf_ref
    err = np.abs(gpu[fin] - ref[fin])
    tol = rel * np.maximum(np.abs(ref[fin]), s)
    bad = err > tol
    if bad.any():
        i = int(np.argmax(err - tol))
        raise AssertionError("%s: %d of %d entries out of tolerance; worst gpu=%r ref=%r tol=%r" % (
            what, int(bad.sum()), bad.size, gpu[fin][i], ref[fin][i], tol[i]))
    return float(err.max() / max(s, 1e-30)) if err.size else 0.0


def compare_topk(gd, gi, res, k: int, rel: float = REL, scale: float | None = None):
    """gd (rows, k), gi (rows, k, 3) from the GPU; res from oracle.search on the
    same rows.  Returns (number of near-tie swaps, per-row swap flags)."""
    gd = np.asarray(gd, np.float64)
    gi = np.asarray(gi, np.float64)
    od, ad, ai = res["dists"], res["all_dists"], res["all_inds"]
    s = rms_finite(od[:, :k]) if scale is None else scale
    rows = gd.shape[0]
    # ranked scores
    assert_close(gd, od[:, :k], "top-k scores", rel, s)
    swaps = np.zeros(rows, bool)
    n_swaps = 0
    for r in range(rows):
        lookup = {tuple(ai[r, j]): j for j in range(ai.shape[1])}
        seen = set()
        for j in range(k):
            key = tuple(gi[r, j])
            assert key in lookup, "row %d rank %d: position %r is not a candidate of the oracle row" % (r, j, key)
            cid = lookup[key]
            assert cid not in seen, "row %d: candidate %d kept twice" % (r, cid)
            seen.add(cid)
            if cid != res["ids"][r, j]:
                ref = od[r, j]
                got = ad[r, cid]
                assert np.isfinite(ref) and np.isfinite(got), (
                    "row %d rank %d: invalid candidates must follow id order (%d vs %d)" % (
                        r, j, cid, res["ids"][r, j]))
                tol = rel * max(abs(ref), s)
                assert abs(got - ref) <= tol, (
                    "row %d rank %d: kept candidate %d (oracle score %r) but oracle has %d (%r), tol %r" % (
                        r, j, cid, got, res["ids"][r, j], ref, tol))
                swaps[r] = True
                n_swaps += 1
    return n_swaps, swaps
