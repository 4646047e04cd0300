"""Pins of the oracle against facts that do not come from the oracle itself.

The paper prints no worked numeric example for the search, so every part of
the oracle is pinned by a special case that reduces to an independent library
routine (torch grid_sample / unfold / fold, a dense matrix product, a sort),
by a closed form, by an invariant, or by finite differences.  Each test names
the passage of "Space-Time Attention with Shifted Non-Local Search" it pins.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from workloads import small_params

rng_seed = 1234


def _rng(i=0):
    return np.random.default_rng(rng_seed + i)


def _grid_sample(img, ys, xs):
    """Bilinear reads of a (C,H,W) image at real positions via torch grid_sample
    (align_corners=True: pixel centres on integers; zeros outside)."""
    C, H, W = img.shape
    t = torch.from_numpy(np.asarray(img, np.float64))[None]
    gx = 2.0 * torch.from_numpy(np.asarray(xs, np.float64)) / max(W - 1, 1) - 1.0
    gy = 2.0 * torch.from_numpy(np.asarray(ys, np.float64)) / max(H - 1, 1) - 1.0
    g = torch.stack([gx.reshape(-1), gy.reshape(-1)], -1)[None, None]
    out = F.grid_sample(t, g, mode="bilinear", padding_mode="zeros", align_corners=True)
    return out[0, :, 0].numpy()  # (C, n)


def _unfold(img, ps, stride=1):
    """Zero-padded ps x ps patches of a (C,H,W) image centred on the grid (odd ps)."""
    t = torch.from_numpy(np.asarray(img, np.float64))[None]
    u = F.unfold(t, kernel_size=ps, padding=ps // 2, stride=stride)[0]  # (C*ps*ps, L)
    return u.numpy()


def _qrow(p, b, hd, t, mh, mw):
    nH, nW = oracle.grid(p)
    return (((b * p["HD"] + hd) * p["T"] + t) * nH + mh) * nW + mw


def _cid(p, dt, dh, dw):
    return ((dt + p["wt"]) * p["ws"] + dh) * p["ws"] + dw


# ---------------------------------------------------------------- bilinear --

def test_bilinear_matches_grid_sample(oracle_lib):
    """Sec. 3.2 "bilinear interpolation ... for efficient indexing": the
    oracle's read equals torch grid_sample (align_corners=True, zero padding),
    including integer positions, exact borders and positions off the frame."""
    r = _rng(1)
    H, W = 7, 9
    img = r.standard_normal((H, W))
    ys = np.concatenate([r.uniform(-2.5, H + 1.5, 400), np.arange(-1, H + 1), [0.0, H - 1.0, -1e-9, H - 1 + 1e-9]])
    xs = np.concatenate([r.uniform(-2.5, W + 1.5, 400), np.arange(-1, W + 1)[: H + 2], [W - 1.0, 0.0, 3.0, 2.0]])
    n = min(len(ys), len(xs))
    ys, xs = ys[:n], xs[:n]
    got = oracle.bilinear_image(img, ys, xs)
    ref = _grid_sample(img[None], ys, xs)[0]
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-13)
    # integer positions read the pixel itself
    iy, ix = r.integers(0, H, 50), r.integers(0, W, 50)
    np.testing.assert_array_equal(oracle.bilinear_image(img, iy, ix), img[iy, ix])


# ------------------------------------------------------ similarity / window --

def test_zero_flow_pixel_search_is_masked_dense_product(oracle_lib):
    """Sec. 3.1 neighbourhood attention: with ps=1, wt=0 and no offsets the
    scores are the in-window entries of the dense product Q_M K_M^T."""
    r = _rng(2)
    p = small_params(T=2, C=5, H=6, W=7, ws=5, wt=0, ps=1, k=3)
    q = r.standard_normal((1, 2, 5, 6, 7))
    k = r.standard_normal((1, 2, 5, 6, 7))
    flows = np.zeros((1, 2, 0, 2, 6, 7))
    d, ind = oracle.search_all(q, k, flows, p)
    rr = p["ws"] // 2
    for t in range(2):
        QM = q[0, t].reshape(5, -1).T
        KM = k[0, t].reshape(5, -1).T
        S = QM @ KM.T
        for h in range(6):
            for w in range(7):
                row = _qrow(p, 0, 0, t, h, w)
                for dh in range(5):
                    for dw in range(5):
                        y, x = h + dh - rr, w + dw - rr
                        got = d[row, _cid(p, 0, dh, dw)]
                        if 0 <= y < 6 and 0 <= x < 7:
                            assert got == pytest.approx(S[h * 7 + w, y * 7 + x], abs=1e-12)
                            assert tuple(ind[row, _cid(p, 0, dh, dw)]) == (t, dh - rr, dw - rr)
                        else:
                            assert got == -np.inf


@pytest.mark.parametrize("ps,stride0,HD", [(3, 1, 1), (5, 1, 2), (3, 2, 2)])
def test_zero_flow_patch_search_is_unfold_product(oracle_lib, ps, stride0, HD):
    """Sec. 3.1 non-local search with query stride S_Q: inner-product scores
    are dot products of zero-padded unfolded patches (query pixels outside
    the frame contribute nothing), per head of C/HD channels."""
    r = _rng(3)
    C, H, W = 4, 9, 8
    p = small_params(T=1, C=C, H=H, W=W, HD=HD, ws=3, wt=0, ps=ps, stride0=stride0, k=2)
    q = r.standard_normal((1, 1, C, H, W))
    k = r.standard_normal((1, 1, C, H, W))
    flows = np.zeros((1, 1, 0, 2, H, W))
    d, _ = oracle.search_all(q, k, flows, p)
    nH, nW = oracle.grid(p)
    Ch = C // HD
    rr = 1
    for hd in range(HD):
        Qp = _unfold(q[0, 0, hd * Ch:(hd + 1) * Ch], ps)
        Kp = _unfold(k[0, 0, hd * Ch:(hd + 1) * Ch], ps)
        for mh in range(nH):
            for mw in range(nW):
                h, w = mh * stride0, mw * stride0
                row = _qrow(p, 0, hd, 0, mh, mw)
                for dh in range(3):
                    for dw in range(3):
                        y, x = h + dh - rr, w + dw - rr
                        if 0 <= y < H and 0 <= x < W:
                            ref = Qp[:, h * W + w] @ Kp[:, y * W + x]
                            assert d[row, _cid(p, 0, dh, dw)] == pytest.approx(ref, abs=1e-12)


def test_zero_flow_l2_interior_is_unfold_distance(oracle_lib):
    """Squared L2 patch distance (the distance the workloads add to the
    paper's inner product) equals ||unfold(q) - unfold(k)||^2 where the query
    patch lies inside the frame."""
    r = _rng(4)
    C, H, W, ps = 3, 9, 9, 3
    p = small_params(T=1, C=C, H=H, W=W, ws=3, wt=0, ps=ps, k=2, dist_type=1)
    q = r.standard_normal((1, 1, C, H, W))
    k = r.standard_normal((1, 1, C, H, W))
    d, _ = oracle.search_all(q, k, np.zeros((1, 1, 0, 2, H, W)), p)
    Qp, Kp = _unfold(q[0, 0], ps), _unfold(k[0, 0], ps)
    for h in range(1, H - 1):
        for w in range(1, W - 1):
            for dh in range(3):
                for dw in range(3):
                    y, x = h + dh - 1, w + dw - 1
                    ref = ((Qp[:, h * W + w] - Kp[:, y * W + x]) ** 2).sum()
                    assert d[_qrow(p, 0, 0, 0, h, w), _cid(p, 0, dh, dw)] == pytest.approx(ref, abs=1e-12)


@pytest.mark.parametrize("wt,T", [(1, 3), (2, 4)])
def test_integer_flows_shift_the_window(oracle_lib, wt, T):
    """Sec. 3.2: the window centre moves from (h, w) to (h + dh, w + dw) with
    (dh, dw) = F_in at the query.  With integer offsets (distinct per slot,
    rows != columns) every score equals the unfolded-patch product at the
    shifted centre; candidates whose centre leaves the frame, or whose frame
    lies outside the clip, are invalid.  Flow slots run dt = -wt..-1, 1..wt."""
    r = _rng(5)
    C, H, W, ps, ws = 3, 10, 11, 3, 3
    p = small_params(T=T, C=C, H=H, W=W, ws=ws, wt=wt, ps=ps, k=2)
    q = r.standard_normal((1, T, C, H, W))
    k = r.standard_normal((1, T, C, H, W))
    flows = r.integers(-3, 4, size=(1, T, 2 * wt, 2, H, W)).astype(np.float64)
    d, ind = oracle.search_all(q, k, flows, p)
    Kp = [_unfold(k[0, t], ps) for t in range(T)]
    slots = [(dt, s) for s, dt in enumerate(list(range(-wt, 0)) + list(range(1, wt + 1)))] + [(0, None)]
    for t in range(T):
        Qp = _unfold(q[0, t], ps)
        for h in range(H):
            for w in range(W):
                row = _qrow(p, 0, 0, t, h, w)
                for dt, slot in slots:
                    t2 = t + dt
                    sh = 0 if slot is None else int(flows[0, t, slot, 0, h, w])
                    sw = 0 if slot is None else int(flows[0, t, slot, 1, h, w])
                    for dh in range(ws):
                        for dw in range(ws):
                            c = _cid(p, dt, dh, dw)
                            y, x = h + sh + dh - 1, w + sw + dw - 1
                            assert tuple(ind[row, c]) == (t2, sh + dh - 1, sw + dw - 1)
                            if 0 <= t2 < T and 0 <= y < H and 0 <= x < W:
                                assert d[row, c] == pytest.approx(Qp[:, h * W + w] @ Kp[t2][:, y * W + x], abs=1e-12)
                            else:
                                assert d[row, c] == -np.inf


@pytest.mark.parametrize("dist_type,stride1", [(0, 1.0), (1, 1.0), (0, 0.5), (1, 0.75)])
def test_fractional_flows_match_grid_sample_patches(oracle_lib, dist_type, stride1):
    """Sec. 3.2 with fractional offsets and key stride S_K: the key patch is
    read at h + p + dh + S_K*(d - Ws//2) with bilinear interpolation; scores
    computed from torch grid_sample reads agree (query pixels outside the
    frame skipped)."""
    r = _rng(6)
    C, H, W, ps, ws, wt, T = 2, 7, 8, 3, 3, 1, 2
    p = small_params(T=T, C=C, H=H, W=W, ws=ws, wt=wt, ps=ps, k=2, dist_type=dist_type, stride1=stride1)
    q = r.standard_normal((1, T, C, H, W))
    k = r.standard_normal((1, T, C, H, W))
    flows = r.uniform(-2.5, 2.5, size=(1, T, 2, 2, H, W)).astype(np.float32).astype(np.float64)
    d, ind = oracle.search_all(q, k, flows, p)
    for t in range(T):
        for h in range(H):
            for w in range(W):
                row = _qrow(p, 0, 0, t, h, w)
                for dt in (-1, 0, 1):
                    t2 = t + dt
                    if not 0 <= t2 < T:
                        continue
                    slot = 0 if dt < 0 else 1
                    sh = 0.0 if dt == 0 else flows[0, t, slot, 0, h, w]
                    sw = 0.0 if dt == 0 else flows[0, t, slot, 1, h, w]
                    for dh in range(ws):
                        for dw in range(ws):
                            c = _cid(p, dt, dh, dw)
                            disp_h = float(np.float32(sh) + np.float32(np.float32(stride1) * np.float32(dh - 1)))
                            disp_w = float(np.float32(sw) + np.float32(np.float32(stride1) * np.float32(dw - 1)))
                            assert ind[row, c, 1] == disp_h and ind[row, c, 2] == disp_w
                            if not (0 <= h + disp_h <= H - 1 and 0 <= w + disp_w <= W - 1):
                                assert d[row, c] == (-np.inf if dist_type == 0 else np.inf)
                                continue
                            ys, xs, qv = [], [], []
                            for ph in (-1, 0, 1):
                                for pw in (-1, 0, 1):
                                    if 0 <= h + ph < H and 0 <= w + pw < W:
                                        ys.append(h + ph + disp_h)
                                        xs.append(w + pw + disp_w)
                                        qv.append(q[0, t, :, h + ph, w + pw])
                            kv = _grid_sample(k[0, t2], ys, xs).T
                            qv = np.array(qv)
                            ref = (qv * kv).sum() if dist_type == 0 else ((qv - kv) ** 2).sum()
                            assert d[row, c] == pytest.approx(ref, abs=1e-12)


def test_integer_shifted_video_recovers_true_offset(oracle_lib):
    """Sec. 3.3 motivation (a grid search around a predicted offset corrects
    its error): frames cropped from one canvas at integer offsets, flows =
    truth + integer error within the window radius.  In every frame block the
    best L2 candidate is the true displacement with distance exactly 0, and
    with unit-norm pixels the inner product of the true match equals the
    number of in-frame patch pixels and is the block maximum."""
    r = _rng(7)
    C, H, W, ps, ws, wt, T = 4, 12, 13, 3, 5, 1, 3
    canvas = r.standard_normal((C, H + 20, W + 20))
    offs = [(10, 10), (7, 12), (12, 6)]  # crop origin of each frame
    frames = np.stack([canvas[:, a:a + H, b:b + W] for a, b in offs])[None]
    unit = frames / np.linalg.norm(frames, axis=2, keepdims=True)
    rr = ws // 2
    flows = np.zeros((1, T, 2, 2, H, W))
    for t in range(T):
        for slot, dt in enumerate((-1, 1)):
            t2 = t + dt
            if 0 <= t2 < T:
                true = (offs[t][0] - offs[t2][0], offs[t][1] - offs[t2][1])
                err = r.integers(-rr, rr + 1, size=(2, H, W))
                flows[0, t, slot, 0] = true[0] + err[0]
                flows[0, t, slot, 1] = true[1] + err[1]
    for dist_type, vid in ((1, frames), (0, unit)):
        p = small_params(T=T, C=C, H=H, W=W, ws=ws, wt=wt, ps=ps, k=3, dist_type=dist_type)
        d, ind = oracle.search_all(vid, vid, flows, p)
        for t in range(T):
            for dt in (-1, 1):
                t2 = t + dt
                if not 0 <= t2 < T:
                    continue
                true = (offs[t][0] - offs[t2][0], offs[t][1] - offs[t2][1])
                for h in range(1, H - 1):
                    for w in range(1, W - 1):
                        if not (1 <= h + true[0] < H - 1 and 1 <= w + true[1] < W - 1):
                            continue
                        row = _qrow(p, 0, 0, t, h, w)
                        blk = slice(_cid(p, dt, 0, 0), _cid(p, dt, 0, 0) + ws * ws)
                        best = int(np.argmin(d[row, blk]) if dist_type else np.argmax(d[row, blk]))
                        assert tuple(ind[row, blk][best, 1:]) == true
                        if dist_type == 1:
                            assert d[row, blk][best] == 0.0
                        else:
                            assert d[row, blk][best] == pytest.approx(ps * ps, abs=1e-12)


@pytest.mark.parametrize("stride1", [1.0, 0.5])
def test_self_match_is_the_extremum(oracle_lib, stride1):
    """q = k, zero offsets: the zero-displacement candidate scores 0 for L2
    (the minimum) and, with unit-norm pixels, the count of in-frame patch
    pixels for the inner product (the maximum, by Cauchy-Schwarz and the
    convexity of bilinear weights), also on a half-pixel key grid."""
    r = _rng(8)
    C, H, W = 3, 8, 9
    x = r.standard_normal((1, 2, C, H, W))
    u = x / np.linalg.norm(x, axis=2, keepdims=True)
    for dist_type, vid in ((1, x), (0, u)):
        p = small_params(T=2, C=C, H=H, W=W, ws=5, wt=0, ps=3, k=2, dist_type=dist_type, stride1=stride1)
        d, _ = oracle.search_all(vid, vid, np.zeros((1, 2, 0, 2, H, W)), p)
        self_id = _cid(p, 0, 2, 2)
        for t in range(2):
            for h in range(H):
                for w in range(W):
                    row = _qrow(p, 0, 0, t, h, w)
                    npix = (min(h + 1, H - 1) - max(h - 1, 0) + 1) * (min(w + 1, W - 1) - max(w - 1, 0) + 1)
                    if dist_type == 1:
                        assert d[row, self_id] == 0.0
                        assert np.all(d[row] >= 0.0)
                    else:
                        assert d[row, self_id] == pytest.approx(npix, abs=1e-12)
                        others = np.delete(d[row], self_id)
                        assert np.all(others[np.isfinite(others)] < npix - 1e-9)


def test_frames_outside_the_video_are_skipped(oracle_lib):
    """Sec. 3.2 temporal window W_t = 2wt+1 around the query frame: frames
    beyond the clip (T < W_t here) are never scored; a single-pixel video has
    exactly one valid candidate per frame."""
    r = _rng(9)
    p = small_params(T=2, C=2, H=1, W=1, ws=3, wt=2, ps=3, k=2)
    x = r.standard_normal((1, 2, 2, 1, 1))
    flows = np.zeros((1, 2, 4, 2, 1, 1))
    d, ind = oracle.search_all(x, x, flows, p)
    for t in range(2):
        row = _qrow(p, 0, 0, t, 0, 0)
        finite = np.isfinite(d[row])
        assert finite.sum() == 2  # the zero-displacement cell of frames 0 and 1
        assert set(ind[row, finite, 0].astype(int)) == {0, 1}


# -------------------------------------------------------------------- top-k --

def test_topk_is_a_stable_sort(oracle_lib):
    """top-L (Sec. 3.2): the k best columns, best first, ties to the smaller
    column id -- equal to a lexicographic sort on (-score, id) / (score, id)."""
    r = _rng(10)
    d = r.integers(-3, 4, size=(50, 37)).astype(np.float64)
    d[r.random(d.shape) < 0.1] = -np.inf
    d[r.random(d.shape) < 0.05] = np.inf
    for dist_type in (0, 1):
        vals, ids = oracle.topk(d, 11, dist_type)
        for i in range(50):
            key = -d[i] if dist_type == 0 else d[i]
            order = np.lexsort((np.arange(37), key))[:11]
            np.testing.assert_array_equal(ids[i], order)
            np.testing.assert_array_equal(vals[i], d[i, order])


# -------------------------------------------------------------- aggregation --

@pytest.mark.parametrize("HD,scale", [(1, 1.0), (2, 0.3)])
def test_pixel_aggregation_is_masked_softmax_attention(oracle_lib, HD, scale):
    """Sec. 3.1 global attention A = softmax(S) V restricted to the window
    (neighbourhood attention): ps = 1, S_Q = 1, wt = 0, zero offsets and
    k = Ws^2 give out = softmax(scale * Q K^T + mask) V per head, exactly,
    borders included (the mask removes keys outside the frame)."""
    r = _rng(11)
    C, H, W, ws = 4, 6, 7, 3
    p = small_params(T=1, C=C, H=H, W=W, HD=HD, ws=ws, wt=0, ps=1, k=ws * ws)
    q, k, v = (r.standard_normal((1, 1, C, H, W)) for _ in range(3))
    res = oracle.search(q, k, np.zeros((1, 1, 0, 2, H, W)), p, extra=0)
    out = oracle.aggregate(v, res["dists"], res["inds"], p, scale)
    Ch = C // HD
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    yy, xx = yy.ravel(), xx.ravel()
    mask = np.where((np.abs(yy[:, None] - yy[None]) <= 1) & (np.abs(xx[:, None] - xx[None]) <= 1), 0.0, -np.inf)
    for hd in range(HD):
        cs = slice(hd * Ch, (hd + 1) * Ch)
        QM = q[0, 0, cs].reshape(Ch, -1).T
        KM = k[0, 0, cs].reshape(Ch, -1).T
        VM = v[0, 0, cs].reshape(Ch, -1).T
        S = scale * QM @ KM.T + mask
        A = np.exp(S - S.max(1, keepdims=True))
        A /= A.sum(1, keepdims=True)
        ref = (A @ VM).T.reshape(Ch, H, W)
        np.testing.assert_allclose(out[0, 0, cs], ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("ps,stride0", [(3, 1), (5, 1), (3, 2)])
def test_patch_aggregation_is_fold_of_weighted_patches(oracle_lib, ps, stride0):
    """Sec. 3.2 aggregation with integer offsets: summing each query's
    softmax-weighted neighbour patches into the output and dividing by the
    number of contributions equals torch fold(sum_l w_l unfold(V)) / fold(1)."""
    r = _rng(12)
    C, H, W, T, kk = 3, 9, 10, 3, 4
    p = small_params(T=T, C=C, H=H, W=W, ps=ps, stride0=stride0, k=kk)
    nH, nW = oracle.grid(p)
    v = r.standard_normal((1, T, C, H, W))
    dists = r.standard_normal((1, 1, T, nH, nW, kk)) * 2
    inds = np.zeros((1, 1, T, nH, nW, kk, 3))
    inds[..., 0] = r.integers(0, T, size=inds.shape[:-1])
    inds[..., 1:] = r.integers(-3, 4, size=inds.shape[:-1] + (2,))
    scale = 0.7
    out = oracle.aggregate(v, dists, inds, p, scale)
    wts = np.exp(scale * dists - (scale * dists).max(-1, keepdims=True))
    wts /= wts.sum(-1, keepdims=True)
    unf = [_unfold(v[0, t], ps) for t in range(T)]
    for t in range(T):
        cols = np.zeros((C * ps * ps, nH * nW))
        for mh in range(nH):
            for mw in range(nW):
                h, w = mh * stride0, mw * stride0
                for l in range(kk):
                    t2, dh, dw = inds[0, 0, t, mh, mw, l].astype(int)
                    y, x = h + dh, w + dw
                    if 0 <= y < H and 0 <= x < W:
                        patch = unf[t2][:, y * W + x]
                    else:  # centre off the frame: slice the zero-padded frame instead
                        m = ps + 4
                        pad = np.pad(v[0, t2], ((0, 0), (m, m), (m, m)))
                        y0, x0 = y + m - ps // 2, x + m - ps // 2
                        patch = pad[:, y0:y0 + ps, x0:x0 + ps].reshape(C * ps * ps)
                    cols[:, mh * nW + mw] += wts[0, 0, t, mh, mw, l] * patch
        folded = F.fold(torch.from_numpy(cols)[None], (H, W), ps, padding=ps // 2, stride=stride0)[0]
        ones = F.fold(torch.ones(1, ps * ps, nH * nW, dtype=torch.float64), (H, W), ps, padding=ps // 2,
                      stride=stride0)[0, 0]
        ref = torch.where(ones > 0, folded / ones.clamp(min=1), torch.zeros_like(folded)).numpy()
        np.testing.assert_allclose(out[0, t], ref, rtol=0, atol=1e-12)


def test_constant_value_video_is_reproduced(oracle_lib):
    """Sec. 3.2 normalisation by the number of contributing terms: with
    V = const, fractional offsets |d| <= 2 and any scores, every pixel at least
    2 px inside the frame comes out as the constant (weights sum to one);
    with ps = 1 and S_Q = 2 the pixels off the query grid stay 0 (holes)."""
    r = _rng(13)
    C, H, W, T, kk = 2, 11, 12, 2, 5
    for ps, stride0 in ((3, 1), (1, 2)):
        p = small_params(T=T, C=C, H=H, W=W, ps=ps, stride0=stride0, k=kk)
        nH, nW = oracle.grid(p)
        v = np.full((1, T, C, H, W), 3.25)
        dists = r.standard_normal((1, 1, T, nH, nW, kk))
        inds = np.zeros((1, 1, T, nH, nW, kk, 3))
        inds[..., 0] = r.integers(0, T, size=inds.shape[:-1])
        inds[..., 1:] = r.uniform(-2, 2, size=inds.shape[:-1] + (2,))
        out = oracle.aggregate(v, dists, inds, p, 1.0)
        inner = out[..., 2:H - 2, 2:W - 2]
        if stride0 == 1:
            np.testing.assert_allclose(inner, 3.25, rtol=0, atol=1e-12)
        else:
            on = np.zeros((H, W), bool)
            on[::2, ::2] = True
            assert np.all(out[..., ~on] == 0.0)
            np.testing.assert_allclose(inner[..., on[2:H - 2, 2:W - 2]], 3.25, rtol=0, atol=1e-12)


def test_aggregate_at_pixels_equals_full_scatter(oracle_lib):
    """The per-pixel evaluation used for sampled comparisons at full size
    agrees with the literal scatter form of the aggregation."""
    r = _rng(14)
    p = small_params(T=3, C=4, H=9, W=8, HD=2, ps=3, stride0=1, k=3, wt=1)
    nH, nW = oracle.grid(p)
    v = r.standard_normal((1, 3, 4, 9, 8))
    dists = r.standard_normal((1, 2, 3, nH, nW, 3))
    inds = np.zeros((1, 2, 3, nH, nW, 3, 3))
    inds[..., 0] = r.integers(0, 3, size=inds.shape[:-1])
    inds[..., 1:] = r.uniform(-3, 3, size=inds.shape[:-1] + (2,))
    full = oracle.aggregate(v, dists, inds, p, 0.5)
    pix = np.arange(3 * 9 * 8)
    at = oracle.aggregate_at(v, dists, inds, p, pix, 0.5)
    np.testing.assert_allclose(at, full[0].transpose(0, 2, 3, 1).reshape(-1, 4), rtol=0, atol=1e-13)


# ----------------------------------------------------------------- backward --

def _fixed_problem(seed, dist_type, HD=1, ps=3, stride0=1, stride1=1.0):
    r = _rng(100 + seed)
    C, H, W, T, wt, ws, kk = 4, 7, 8, 3, 1, 3, 3
    p = small_params(T=T, C=C, H=H, W=W, HD=HD, ws=ws, wt=wt, ps=ps, stride0=stride0, stride1=stride1, k=kk,
                     dist_type=dist_type)
    q, k, v = (r.standard_normal((1, T, C, H, W)) * 0.5 for _ in range(3))
    # offsets well away from integers so the bilinear weights stay smooth
    # (with key stride 1/2 the cells add multiples of 0.5: fractions 0.1-0.4
    # give positions 0.1-0.4 or 0.6-0.9 past an integer)
    lo, hi = (0.2, 0.8) if stride1 == 1.0 else (0.1, 0.4)
    flows = r.integers(-1, 2, size=(1, T, 2 * wt, 2, H, W)) + r.uniform(lo, hi, size=(1, T, 2 * wt, 2, H, W))
    nq = oracle.n_queries(p)
    sel = np.zeros((nq, kk, 3), np.int32)
    sel[:, :, 0] = r.integers(-wt, wt + 1, size=(nq, kk))
    sel[:, :, 1:] = r.integers(0, ws, size=(nq, kk, 2))
    # make sure every row selects in-range frames
    qt = (np.arange(nq) // (oracle.grid(p)[0] * oracle.grid(p)[1])) % T
    sel[:, :, 0] = np.clip(sel[:, :, 0] + qt[:, None], 0, T - 1) - qt[:, None]
    g = r.standard_normal(q.shape)
    nH, nW = oracle.grid(p)
    gd = r.standard_normal((1, HD, T, nH, nW, kk))
    return p, q, k, v, flows, sel, g, gd


def _loss(p, q, k, v, flows, sel, g, gd, scale):
    d, ind = oracle.search_fixed(q, k, flows, p, sel, fp32_positions=False)
    d = d.reshape(gd.shape)
    ind = ind.reshape(gd.shape + (3,))
    out = oracle.aggregate(v, d, ind, p, scale)
    fin = np.isfinite(d)
    return (g * out).sum() + (gd[fin] * d[fin]).sum(), d, ind


BWD_SHAPES = [  # dist_type, HD, P, S_Q, S_K
    (0, 1, 3, 1, 1.0), (1, 1, 3, 1, 1.0), (0, 2, 3, 1, 1.0),
    (0, 1, 1, 2, 1.0), (1, 1, 5, 2, 1.0), (0, 1, 5, 1, 0.5), (1, 2, 1, 1, 0.5), (0, 1, 3, 2, 0.5),
]


@pytest.mark.parametrize("dist_type,HD,ps,stride0,stride1", BWD_SHAPES)
def test_backward_matches_finite_differences(oracle_lib, dist_type, HD, ps, stride0, stride1):
    """Sec. 1 / 3.2 differentiable search: the chain-rule gradients w.r.t. q,
    k, v and the offsets F_in match central finite differences of the
    forward map (top-k set held fixed, positions in double precision), for
    single-pixel and 5 x 5 patches, query stride 2 and key stride 1/2."""
    p, q, k, v, flows, sel, g, gd = _fixed_problem(dist_type + 3 * HD + 7 * ps + 11 * stride0, dist_type, HD=HD,
                                                   ps=ps, stride0=stride0, stride1=stride1)
    scale = 0.2
    L0, d, ind = _loss(p, q, k, v, flows, sel, g, gd, scale)
    gq, gk, gv, gf = oracle.backward(q, k, v, flows, d, ind, g, p, scale, grad_dists=gd)
    r = _rng(200 + dist_type)
    eps = 1e-5
    for name, arr, grad in (("q", q, gq), ("k", k, gk), ("v", v, gv), ("flows", flows, gf)):
        flat = arr.reshape(-1)
        idx = r.choice(flat.size, 25, replace=False)
        if name == "flows":  # include entries that carry gradient
            nz = np.flatnonzero(gf.reshape(-1))
            idx = np.concatenate([idx, r.choice(nz, 15, replace=False)])
        for i in idx:
            old = flat[i]
            flat[i] = old + eps
            Lp = _loss(p, q, k, v, flows, sel, g, gd, scale)[0]
            flat[i] = old - eps
            Lm = _loss(p, q, k, v, flows, sel, g, gd, scale)[0]
            flat[i] = old
            fd = (Lp - Lm) / (2 * eps)
            assert grad.reshape(-1)[i] == pytest.approx(fd, rel=1e-6, abs=1e-7), (name, i)


@pytest.mark.parametrize("ps,stride0,stride1", [(3, 1, 1.0), (1, 2, 1.0), (5, 2, 1.0), (5, 1, 0.5)])
def test_backward_adjoint_identities(oracle_lib, ps, stride0, stride1):
    """Adjoint checks of the linear pieces: v -> out is linear for fixed
    scores and positions, and q -> d, k -> d are linear for the inner product,
    so <J x, y> = <x, J^T y> with J^T y from the backward pass."""
    p, q, k, v, flows, sel, g, gd = _fixed_problem(7 + ps + stride0, 0, ps=ps, stride0=stride0, stride1=stride1)
    scale = 0.4
    d, ind = oracle.search_fixed(q, k, flows, p, sel)
    d = d.reshape(gd.shape)
    ind = ind.reshape(gd.shape + (3,))
    r = _rng(300)
    x = r.standard_normal(v.shape)
    y = r.standard_normal(v.shape)
    lhs = (oracle.aggregate(x, d, ind, p, scale) * y).sum()
    _, _, gv, _ = oracle.backward(q, k, x, flows, d, ind, y, p, scale)
    assert lhs == pytest.approx((x * gv).sum(), rel=1e-10)
    zero = np.zeros_like(v)
    gq, gk, _, _ = oracle.backward(q, k, v, flows, d, ind, zero, p, scale, grad_dists=gd)
    dq = oracle.search_fixed(x, k, flows, p, sel)[0].reshape(gd.shape)
    dk = oracle.search_fixed(q, x, flows, p, sel)[0].reshape(gd.shape)
    fin = np.isfinite(dq)
    assert (dq[fin] * gd[fin]).sum() == pytest.approx((x * gq).sum(), rel=1e-10)
    assert (dk[fin] * gd[fin]).sum() == pytest.approx((x * gk).sum(), rel=1e-10)


def test_nan_similarity_scores_as_invalid():
    """A NaN feature makes the similarity of every candidate reading it NaN;
    those candidates score like invalid ones (-inf / +inf) so that every score
    is ordered, and all other candidates are unchanged."""
    p = small_params(T=2, C=3, H=9, W=10, ws=3, wt=1, ps=3, k=4)
    r = np.random.default_rng(5)
    q = r.standard_normal((1, 2, 3, 9, 10))
    k = r.standard_normal((1, 2, 3, 9, 10))
    flows = r.uniform(-1, 1, (1, 2, 2, 2, 9, 10))
    k_nan = k.copy()
    k_nan[0, 1, 2, 4, 5] = np.nan
    for dist in (0, 1):
        pp = dict(p, dist_type=dist)
        d0, _ = oracle.search_all(q, k, flows, pp)
        d1, _ = oracle.search_all(q, k_nan, flows, pp)
        assert not np.isnan(d1).any()
        changed = d1 != d0
        assert changed.any()
        assert np.all(d1[changed] == (-np.inf if dist == 0 else np.inf))
        assert np.all(np.isfinite(d0[changed]))


# ------------------------------------------- flow chaining (front-end) --

def _one_step_flows(r, B, T, H, W, kind):
    shp = (B, T, 2, H, W)
    if kind == "int":
        return r.integers(-2, 3, shp).astype(np.float64), r.integers(-2, 3, shp).astype(np.float64)
    return r.uniform(-3, 3, shp), r.uniform(-3, 3, shp)


def test_chain_flows_one_step_is_the_input(oracle_lib):
    """wt = 1: the +-1 slots are the forward and backward flows themselves;
    steps whose frame is outside the clip stay 0."""
    r = _rng(40)
    ff, bf = _one_step_flows(r, 2, 4, 7, 9, "frac")
    out = oracle.chain_flows(ff, bf, 1)
    np.testing.assert_array_equal(out[:, 1:, 0], bf[:, 1:])
    np.testing.assert_array_equal(out[:, :-1, 1], ff[:, :-1])
    assert not out[:, 0, 0].any() and not out[:, -1, 1].any()


def test_chain_flows_constant_motion_adds_up(oracle_lib):
    """A uniform translation composes to s times the one-step offset."""
    B, T, H, W, wt = 1, 6, 8, 10, 3
    ff = np.broadcast_to(np.array([0.75, -1.25]).reshape(1, 1, 2, 1, 1), (B, T, 2, H, W)).copy()
    bf = -ff
    out = oracle.chain_flows(ff, bf, wt)
    for t in range(T):
        for s in range(1, wt + 1):
            for sign, slot in ((1, wt + s - 1), (-1, wt - s)):
                if 0 <= t + sign * s < T:
                    np.testing.assert_array_equal(out[0, t, slot, 0], np.full((H, W), sign * s * 0.75))
                    np.testing.assert_array_equal(out[0, t, slot, 1], np.full((H, W), -sign * s * 1.25))
                else:
                    assert not out[0, t, slot].any()


def test_chain_flows_integer_composition_is_a_gather(oracle_lib):
    """Integer one-step flows: F_{+2}(x) = f_t(x) + f_{t+1}(x + f_t(x)), read
    by integer indexing (positions clamped into the frame)."""
    r = _rng(41)
    B, T, H, W = 1, 5, 9, 11
    ff, bf = _one_step_flows(r, B, T, H, W, "int")
    out = oracle.chain_flows(ff, bf, 2)
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    for t in range(T - 2):
        f1 = ff[0, t]
        py = np.clip(yy + f1[0], 0, H - 1).astype(int)
        px = np.clip(xx + f1[1], 0, W - 1).astype(int)
        ref = f1 + ff[0, t + 1][:, py, px]
        np.testing.assert_array_equal(out[0, t, 3], ref)
    for t in range(2, T):
        b1 = bf[0, t]
        py = np.clip(yy + b1[0], 0, H - 1).astype(int)
        px = np.clip(xx + b1[1], 0, W - 1).astype(int)
        ref = b1 + bf[0, t - 1][:, py, px]
        np.testing.assert_array_equal(out[0, t, 0], ref)


def test_chain_flows_fractional_composition_matches_grid_sample(oracle_lib):
    """Fractional flows: the second step is a bilinear read of the next flow
    field at the displaced position, clamped into the frame -- torch
    grid_sample with align_corners=True and border padding (fp64)."""
    r = _rng(42)
    B, T, H, W = 1, 4, 8, 13
    ff, bf = _one_step_flows(r, B, T, H, W, "frac")
    out = oracle.chain_flows(ff, bf, 3)
    yy, xx = np.meshgrid(np.arange(H, dtype=np.float64), np.arange(W, dtype=np.float64), indexing="ij")

    def sample(field, py, px):  # field (2, H, W) at positions (H, W)
        gx = 2 * px / (W - 1) - 1
        gy = 2 * py / (H - 1) - 1
        grid = torch.from_numpy(np.stack([gx, gy], -1)[None])
        return F.grid_sample(torch.from_numpy(field[None]), grid, mode="bilinear", padding_mode="border",
                             align_corners=True)[0].numpy()

    acc = ff[0, 0].copy()
    np.testing.assert_array_equal(out[0, 0, 3], acc)
    for s in (2, 3):
        acc = acc + sample(ff[0, s - 1], yy + acc[0], xx + acc[1])
        np.testing.assert_allclose(out[0, 0, 3 + s - 1], acc, rtol=0, atol=1e-12)


# ---------------------------------------- aggregation, neighbours apart --

@pytest.mark.parametrize("ps,stride0,HD", [(1, 1, 2), (3, 1, 1), (3, 2, 1)])
def test_stacked_aggregation_keeps_neighbours_apart(oracle_lib, ps, stride0, HD):
    """Integer offsets: slice l of the stacked aggregation is the fold of the
    queries' w_l-weighted l-th neighbour patches divided by the cover count
    (torch fold), per head."""
    r = _rng(43 + ps + stride0)
    Ch, H, W, T, kk = 2, 9, 8, 3, 4
    C = Ch * HD
    p = small_params(T=T, C=C, HD=HD, H=H, W=W, ps=ps, stride0=stride0, k=kk)
    nH, nW = oracle.grid(p)
    v = r.standard_normal((1, T, C, H, W))
    dists = r.standard_normal((1, HD, T, nH, nW, kk))
    inds = np.zeros((1, HD, T, nH, nW, kk, 3))
    inds[..., 0] = r.integers(0, T, size=inds.shape[:-1])
    inds[..., 1:] = r.integers(-2, 3, size=inds.shape[:-1] + (2,))
    scale = 0.8
    st = oracle.aggregate_stacked(v, dists, inds, p, scale)
    assert st.shape == (1, HD, kk, T, Ch, H, W)
    wts = np.exp(scale * dists - (scale * dists).max(-1, keepdims=True))
    wts /= wts.sum(-1, keepdims=True)
    m = ps + 4
    pad = np.pad(v[0], ((0, 0), (0, 0), (m, m), (m, m)))
    ones = F.fold(torch.ones(1, ps * ps, nH * nW, dtype=torch.float64), (H, W), ps, padding=ps // 2,
                  stride=stride0)[0, 0]
    for hd in range(HD):
        for l in range(kk):
            for t in range(T):
                cols = np.zeros((Ch * ps * ps, nH * nW))
                for mh in range(nH):
                    for mw in range(nW):
                        t2, dh, dw = inds[0, hd, t, mh, mw, l].astype(int)
                        y0 = mh * stride0 + dh + m - ps // 2
                        x0 = mw * stride0 + dw + m - ps // 2
                        patch = pad[t2, hd * Ch:(hd + 1) * Ch, y0:y0 + ps, x0:x0 + ps].reshape(-1)
                        cols[:, mh * nW + mw] = wts[0, hd, t, mh, mw, l] * patch
                folded = F.fold(torch.from_numpy(cols)[None], (H, W), ps, padding=ps // 2, stride=stride0)[0]
                ref = torch.where(ones > 0, folded / ones.clamp(min=1), torch.zeros_like(folded)).numpy()
                np.testing.assert_allclose(st[0, hd, l, t], ref, rtol=0, atol=1e-12)


# ------------------------------------------- gather with caller weights --

@pytest.mark.parametrize("ps,stride0,HD", [(3, 1, 1), (1, 2, 2), (5, 2, 1)])
def test_gather_stacked_caller_weights_fold(oracle_lib, ps, stride0, HD):
    """App. B example, gather with the caller's weights: with integer offsets
    slice l is the fold of the queries' w_l-weighted l-th neighbour patches
    divided by the cover count (torch fold), for arbitrary weights
    (negative, zero, unnormalised) -- the weights are used as given."""
    r = _rng(61 + ps + stride0 + HD)
    Ch, H, W, T, kk = 2, 9, 10, 3, 3
    C = Ch * HD
    p = small_params(T=T, C=C, HD=HD, H=H, W=W, ps=ps, stride0=stride0, k=kk)
    nH, nW = oracle.grid(p)
    v = r.standard_normal((1, T, C, H, W))
    wts = r.standard_normal((1, HD, T, nH, nW, kk))
    wts[..., 1] = np.where(r.random(wts.shape[:-1]) < 0.3, 0.0, wts[..., 1])
    inds = np.zeros((1, HD, T, nH, nW, kk, 3))
    inds[..., 0] = r.integers(0, T, size=inds.shape[:-1])
    inds[..., 1:] = r.integers(-2, 3, size=inds.shape[:-1] + (2,))
    st = oracle.gather_stacked(v, wts, inds, p)
    assert st.shape == (1, HD, kk, T, Ch, H, W)
    m = ps + 4
    pad = np.pad(v[0], ((0, 0), (0, 0), (m, m), (m, m)))
    ones = F.fold(torch.ones(1, ps * ps, nH * nW, dtype=torch.float64), (H, W), ps, padding=ps // 2,
                  stride=stride0)[0, 0]
    for hd in range(HD):
        for l in range(kk):
            for t in range(T):
                cols = np.zeros((Ch * ps * ps, nH * nW))
                for mh in range(nH):
                    for mw in range(nW):
                        t2, dh, dw = inds[0, hd, t, mh, mw, l].astype(int)
                        y0 = mh * stride0 + dh + m - ps // 2
                        x0 = mw * stride0 + dw + m - ps // 2
                        patch = pad[t2, hd * Ch:(hd + 1) * Ch, y0:y0 + ps, x0:x0 + ps].reshape(-1)
                        cols[:, mh * nW + mw] = wts[0, hd, t, mh, mw, l] * patch
                folded = F.fold(torch.from_numpy(cols)[None], (H, W), ps, padding=ps // 2, stride=stride0)[0]
                ref = torch.where(ones > 0, folded / ones.clamp(min=1), torch.zeros_like(folded)).numpy()
                np.testing.assert_allclose(st[0, hd, l, t], ref, rtol=0, atol=1e-12)


def test_gather_stacked_softmax_weights_is_stacked_aggregation(oracle_lib):
    """With the weights the aggregation forms itself (softmax of sign*scale*d,
    0 for non-finite scores), the caller-weight gather is the stacked
    aggregation at fractional offsets, including neighbours whose frame
    lies outside the clip or whose offset is not finite."""
    r = _rng(71)
    p = small_params(T=3, C=6, HD=2, H=11, W=12, ps=3, stride0=1, k=4, dist_type=1)
    nH, nW = oracle.grid(p)
    v = r.standard_normal((1, 3, 6, 11, 12))
    d = r.standard_normal((1, 2, 3, nH, nW, 4))
    d[0, 0, 1, 2, 3, 2] = np.inf
    inds = np.zeros((1, 2, 3, nH, nW, 4, 3))
    inds[..., 0] = r.integers(0, 3, size=inds.shape[:-1])
    inds[..., 1:] = r.uniform(-3, 3, size=inds.shape[:-1] + (2,))
    inds[0, 1, 0, 1, 1, 0, 0] = 5.0            # frame outside the clip
    inds[0, 1, 2, 3, 4, 1, 2] = np.nan         # offset not finite
    scale = 0.7
    s = -scale * d  # squared L2: smaller is better
    fin = np.isfinite(s)
    e = np.where(fin, np.exp(s - np.where(fin, s, -np.inf).max(-1, keepdims=True)), 0.0)
    w = e / e.sum(-1, keepdims=True)
    np.testing.assert_allclose(oracle.gather_stacked(v, w, inds, p), oracle.aggregate_stacked(v, d, inds, p, scale),
                               rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("HD,cout", [(1, 5), (2, 6)])
def test_stacked_reduce_is_strided_conv3d(oracle_lib, HD, cout):
    """App. B example: the reduction over the k neighbours is torch's conv3d
    with a (Cout, C, k, 1, 1) kernel at stride (k, 1, 1) after the example's
    rearrangement (b hd k t f h w -> (b t) (hd f) k h w)."""
    r = _rng(81 + HD)
    B, T, Ch, H, W, kk = 2, 3, 3, 5, 4, 4
    C = Ch * HD
    p = small_params(B=B, T=T, C=C, HD=HD, H=H, W=W, k=kk)
    st = r.standard_normal((B, HD, kk, T, Ch, H, W))
    proj = r.standard_normal((cout, C, kk))
    got = oracle.stacked_reduce(st, proj, p)
    x = torch.from_numpy(st).permute(0, 3, 1, 4, 2, 5, 6).reshape(B * T, C, kk, H, W)
    ref = F.conv3d(x, torch.from_numpy(proj)[..., None, None], stride=(kk, 1, 1))
    ref = ref.reshape(B, T, cout, H, W).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_reduce_of_gather_with_identity_kernel_is_aggregation(oracle_lib):
    """Sum over the neighbours: with proj[o, i, l] = [o == i] for every l the
    reduction of the gathered stack is the plain aggregation of Sec. 3.2
    (softmax weights)."""
    r = _rng(91)
    p = small_params(T=3, C=4, HD=2, H=10, W=9, ps=3, stride0=2, k=3)
    nH, nW = oracle.grid(p)
    v = r.standard_normal((1, 3, 4, 10, 9))
    d = r.standard_normal((1, 2, 3, nH, nW, 3))
    inds = np.zeros((1, 2, 3, nH, nW, 3, 3))
    inds[..., 0] = r.integers(0, 3, size=inds.shape[:-1])
    inds[..., 1:] = r.uniform(-2, 2, size=inds.shape[:-1] + (2,))
    w = np.exp(0.5 * d - (0.5 * d).max(-1, keepdims=True))
    w /= w.sum(-1, keepdims=True)
    proj = np.repeat(np.eye(4)[:, :, None], 3, axis=2)
    out = oracle.stacked_reduce(oracle.gather_stacked(v, w, inds, p), proj, p)
    np.testing.assert_allclose(out, oracle.aggregate(v, d, inds, p, 0.5), rtol=1e-12, atol=1e-12)
