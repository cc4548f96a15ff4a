"""fftsplit_conv2d captured in a HIP graph and replayed.

The library allocates nothing, clears nothing with a memset and never
synchronises, so a whole convolution (forward, contraction, inverse, and the
seam or pooling pass where the plan has one) can be captured on the caller's
stream.  Each replay runs on new input written into the captured buffer by
eager work between replays, and must equal, element for element, an eager
call on the same input (every kernel sums in a fixed order); one replay per
case is also checked against the oracle.
"""
import numpy as np
import pytest

import oracle
from workloads import make_random_bias, small_layer

from spectra_layout import rel_l2

torch = pytest.importorskip("torch")
fs = pytest.importorskip("paper_2003_12621_amd")

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


CASES = [
    # (n, cin, h, w, cout, k), tile, mode, pool
    ((2, 16, 30, 28, 32, 3), 14, "os", False),     # band kernels
    ((2, 16, 30, 28, 32, 3), 14, "os", True),      # max-pool in the inverse
    ((1, 5, 19, 23, 20, 5), 12, "oaa", False),     # overlap-add: general kernels + seam pass
    ((2, 3, 17, 19, 6, 3), 3, "oaa", False),       # OaAConv configuration
    ((1, 3, 32, 32, 16, 3), 6, "os", False),       # channel sum inside the inverse
]


@pytest.mark.parametrize("shape,tile,mode,pool", CASES, ids=[f"{s}-T{t}-{m}-p{int(p)}" for s, t, m, p in CASES])
def test_conv2d_graph_replays(shape, tile, mode, pool):
    n, cin, h, w, cout, k = shape
    print(f"[case] graph {shape} T={tile} {mode} pool={pool}", flush=True)
    plan = fs.Plan(n, cin, h, w, cout, k, tile=tile, mode=mode, bias=True, relu=True, pool=pool)
    xs, wt = [], None
    for seed in range(3):
        x_np, w_np = small_layer(n, cin, h, w, cout, k, seed=40 + seed)
        xs.append(x_np)
        wt = w_np if wt is None else wt
    b_np = make_random_bias(cout, cin, k, seed=43)
    wspec = plan.transform_weights(_dev(wt))
    bias = _dev(b_np)
    x = _dev(xs[0])
    out = plan.new_output()
    ws = plan.new_workspace()
    plan.conv2d(x, wspec, bias, out=out, workspace=ws)   # eager once before capture
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        plan.conv2d(x, wspec, bias, out=out, workspace=ws)
    torch.cuda.synchronize()

    ref_ws = plan.new_workspace()
    for i in range(5):
        xi = xs[i % 3]
        x.copy_(_dev(xi))
        g.replay()
        torch.cuda.synchronize()
        got = out.clone()
        eager = plan.conv2d(_dev(xi), wspec, bias, workspace=ref_ws)
        torch.cuda.synchronize()
        assert torch.equal(got, eager), f"replay {i} differs from the eager call"
        if i == 1:
            ref = oracle.direct_xcorr2d(xi, wt, b_np, relu=True)
            if pool:
                ref = oracle.maxpool2x2(ref)
            assert rel_l2(got.cpu().numpy(), ref) <= 1e-4
