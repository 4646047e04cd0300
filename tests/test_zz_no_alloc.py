"""snls_aggregate_static (the allocation-free aggregation) against
snls_aggregate, through the C ABI: two calls in a row on the library's static
scratch array, the second with a smaller problem, each compared with the
workspace entry point on the same inputs (same kernels: bit-identical), and
with the oracle to the parity tolerance."""
import numpy as np
import pytest
import torch

import oracle
from paper_2309_16849_amd import snls as B
from tests.parity import assert_close
from workloads import small_params

pytestmark = pytest.mark.gpu


def _case(p, seed, dev):
    r = np.random.default_rng(seed)
    shp = (p["B"], p["T"], p["C"], p["H"], p["W"])
    q = r.standard_normal(shp, dtype=np.float32)
    v = r.standard_normal(shp, dtype=np.float32)
    fl = r.uniform(-3, 3, (p["B"], p["T"], 2 * p["wt"], 2, p["H"], p["W"])).astype(np.float32)
    qd, vd, fd = (torch.from_numpy(a).to(dev) for a in (q, v, fl))
    d, i = B.snls_search(qd, qd, fd, p)
    return vd, d, i, v


@pytest.mark.parametrize("first,second", [
    # tiled aggregation (P = 7), then a smaller single-pixel problem
    (dict(T=3, C=16, H=48, W=52, ws=9, wt=1, ps=7, k=10),
     dict(T=2, C=16, HD=4, H=20, W=23, ws=7, wt=1, ps=1, stride0=2, k=12)),
    # more than 7 frames per window: softmax weights in the scratch, plain gather; then smaller
    (dict(T=9, C=8, H=30, W=31, ws=3, wt=4, ps=3, k=6), dict(T=3, C=8, H=17, W=15, ws=3, wt=1, ps=3, k=5)),
])
def test_aggregate_static_matches_workspace_entry(first, second):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dev = torch.device("cuda:0")
    B.load_library()
    scale = 0.3
    for n, kw in enumerate((first, second)):
        p = small_params(**kw)
        need = B.snls_workspace_size(B.SNLS_OP_AGGREGATE, p)
        assert 0 < need <= B.SNLS_STATIC_SCRATCH_BYTES
        vd, d, i, v = _case(p, 900 + n, dev)
        print("static aggregation call %d: %s (workspace %d bytes)" % (n, p, need), flush=True)
        ref = B.snls_aggregate(vd, d, i, p, scale)
        out = B.snls_aggregate_static(vd, d, i, p, scale)
        torch.cuda.synchronize()
        got, want = out.cpu().numpy(), ref.cpu().numpy()
        assert np.array_equal(got, want), "static-scratch aggregation differs from the workspace entry point"
        assert_close(got, oracle.aggregate(v, d.cpu().numpy(), i.cpu().numpy(), p, scale), "aggregate")
