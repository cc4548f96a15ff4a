"""Parity of the OaAConv configuration (the paper's comparison method,
Section 2 and Fig. 1): the library's overlap-add pipeline with patches of
the filter's size, T = K, at the odd transform sizes L = 2K - 1.

Same gate as the split path: relative L2 error <= 1e-4 against the oracle's
float64 cross-correlation on the same seeded inputs, over every image,
output channel and pixel.
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


def run_oaaconv(x, w, b, relu=False):
    n, cin, h, wd = x.shape
    cout, _, k, _ = w.shape
    plan = fs.Plan(n, cin, h, wd, cout, k, tile=k, mode="oaa", bias=b is not None, relu=relu)
    assert plan.nfft == 2 * k - 1
    y = plan.conv2d(_dev(x), plan.transform_weights(_dev(w)), None if b is None else _dev(b))
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("name", list(CONFIGS))
def test_oaaconv_config_parity(name):
    x, w, b = config_inputs(name)
    print(f"[case] oaaconv {name}", flush=True)
    y = run_oaaconv(x, w, b)
    ref = config_reference(name)
    err = rel_l2(y, ref)
    print(f"[case] oaaconv {name} rel_l2={err:.3e} rel_max={rel_max(y, ref):.3e}", flush=True)
    assert err <= GATE
    per_channel = [rel_l2(y[:, c], ref[:, c]) for c in range(ref.shape[1])]
    assert max(per_channel) <= GATE, int(np.argmax(per_channel))


EDGE = [
    # (n, cin, h, w, cout, k)
    (1, 1, 1, 1, 1, 3),       # one pixel: a single patch, all seams outside
    (1, 2, 2, 2, 3, 5),       # image smaller than a patch
    (2, 3, 13, 29, 4, 3),     # ragged, H != W, n > 1
    (1, 17, 9, 11, 65, 5),    # Cin and Cout just above 16 / 64
    (3, 9, 33, 35, 5, 7),
    (1, 130, 8, 8, 3, 3),     # Cin not a multiple of 16
]


@pytest.mark.parametrize("shape", EDGE, ids=[str(s) for s in EDGE])
@pytest.mark.parametrize("relu", [False, True])
def test_oaaconv_edge_shapes(shape, relu):
    n, cin, h, wd, cout, k = shape
    print(f"[case] oaaconv edge {shape} relu={relu}", flush=True)
    x, w = small_layer(n, cin, h, wd, cout, k, seed=sum(shape) + 1)
    b = make_random_bias(cout, cin, k, seed=9)
    y = run_oaaconv(x, w, b, relu=relu)
    ref = oracle.direct_xcorr2d(x, w, b, relu=relu)
    assert rel_l2(y, ref) <= GATE


def test_oaaconv_vgg16_stack():
    """The VGG-16 stack with every layer in the OaAConv configuration (T = 3,
    L = 5), batch 2, against the float64 chain."""
    from paper_2003_12621_amd.vgg import VGG16Stack
    from workloads import make_vgg16
    x, layers = make_vgg16(batch=32, seed=0)
    xs = np.ascontiguousarray(x[:2])
    stack = VGG16Stack(layers, batch=2, tiles=[3] * 13, mode="oaa")
    assert stack.tiles == [3] * 13
    out = stack.forward(_dev(xs))
    torch.cuda.synchronize()
    ref = oracle.vgg16_forward(xs, layers)
    err = rel_l2(out.cpu().numpy(), ref)
    print(f"[vgg] oaaconv stack final rel_l2 = {err:.3e}", flush=True)
    assert err <= GATE
