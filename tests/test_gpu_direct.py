"""Parity of the spatial (direct) convolution, fftsplit_direct_conv2d,
against the oracle's float64 cross-correlation (eq. 1).

Same gate as the split path: relative L2 error <= 1e-4 on the fp32 output,
over every image, output channel and pixel.
"""
import numpy as np
import pytest

import oracle
from workloads import CONFIGS, make_random_bias, small_layer

from config_reference import config_inputs, config_reference
from spectra_layout import rel_l2, rel_max

torch = pytest.importorskip("torch")
fs = pytest.importorskip("paper_2003_12621_amd")

pytestmark = pytest.mark.gpu

GATE = 1e-4


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def run_direct(x, w, b, relu=False):
    n, cin, h, wd = x.shape
    cout, _, k, _ = w.shape
    plan = fs.Plan(n, cin, h, wd, cout, k, bias=b is not None, relu=relu)
    wdir = plan.direct_transform_weights(_dev(w))
    y = plan.direct_conv2d(_dev(x), wdir, None if b is None else _dev(b))
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("name", list(CONFIGS))
def test_direct_config_parity(name):
    x, w, b = config_inputs(name)
    print(f"[case] direct {name}", flush=True)
    y = run_direct(x, w, b)
    ref = config_reference(name)
    err = rel_l2(y, ref)
    print(f"[case] direct {name} rel_l2={err:.3e} rel_max={rel_max(y, ref):.3e}", flush=True)
    assert err <= GATE
    per_channel = [rel_l2(y[:, c], ref[:, c]) for c in range(ref.shape[1])]
    assert max(per_channel) <= GATE, int(np.argmax(per_channel))


EDGE = [
    # (n, cin, h, w, cout, k)
    (1, 1, 1, 1, 1, 1),       # one pixel, one channel
    (1, 3, 5, 5, 4, 7),       # filter wider than the image
    (2, 3, 13, 29, 4, 3),     # ragged, H != W, pixels not a multiple of the 64-pixel tile
    (1, 17, 9, 11, 65, 3),    # Cin and Cout just above 16 / 64
    (3, 9, 33, 35, 5, 5),
    (1, 130, 8, 8, 3, 3),     # Cin not a multiple of 16
    (1, 4, 20, 20, 128, 1),   # pointwise
]


@pytest.mark.parametrize("shape", EDGE, ids=[str(s) for s in EDGE])
@pytest.mark.parametrize("relu", [False, True])
def test_direct_edge_shapes(shape, relu):
    n, cin, h, wd, cout, k = shape
    print(f"[case] direct edge {shape} relu={relu}", flush=True)
    x, w = small_layer(n, cin, h, wd, cout, k, seed=sum(shape))
    b = make_random_bias(cout, cin, k, seed=7)
    y = run_direct(x, w, b, relu=relu)
    ref = oracle.direct_xcorr2d(x, w, b, relu=relu)
    err = rel_l2(y, ref)
    assert err <= GATE, err


def test_direct_matches_split_path():
    """The two methods agree with each other on the same layer."""
    x, w = small_layer(2, 24, 30, 30, 40, 5, seed=3)
    plan = fs.Plan(2, 24, 30, 30, 40, 5, tile=12)
    ys = plan.conv2d(_dev(x), plan.transform_weights(_dev(w)))
    yd = plan.direct_conv2d(_dev(x), plan.direct_transform_weights(_dev(w)))
    torch.cuda.synchronize()
    ref = oracle.direct_xcorr2d(x, w)
    assert rel_l2(ys.cpu().numpy(), ref) <= GATE
    assert rel_l2(yd.cpu().numpy(), ref) <= GATE
