"""fftsplit_conv2d_noalloc (the workspace is the library's static device
scratch) against fftsplit_conv2d (a caller workspace): same kernels, so the
outputs must be bit-identical, and both within the gate of the oracle.

Calls run back to back on the one shared scratch, each smaller than the
one before, so each finds the previous call's data in it."""
import numpy as np
import pytest

import oracle
from workloads import make_random_bias, small_layer

from config_reference import config_inputs, config_reference
from spectra_layout import rel_l2

torch = pytest.importorskip("torch")
fs = pytest.importorskip("paper_2003_12621_amd")

pytestmark = pytest.mark.gpu

GATE = 1e-4


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _both(plan, x, w, b):
    """(conv2d with its own workspace, conv2d_noalloc) outputs on the device."""
    wspec = plan.transform_weights(_dev(w))
    xd = _dev(x)
    bd = None if b is None else _dev(b)
    ref = plan.conv2d(xd, wspec, bd)
    out = torch.full(plan.out_shape, float("nan"), dtype=torch.float32, device="cuda")
    plan.conv2d_noalloc(xd, wspec, bd, out=out)
    torch.cuda.synchronize()
    return ref, out


def test_noalloc_matches_conv2d_on_successive_smaller_layers():
    # 1. the 16 x 256 x 56^2 -> 256, K = 5 layer at T = 28: 134 MB of the
    #    scratch's 256 MiB
    x, w, b = config_inputs("c4_56x256_k5")
    plan = fs.Plan(16, 256, 56, 56, 256, 5, tile=28)
    assert plan.info.workspace_bytes <= fs.NOALLOC_MAX_WORKSPACE
    print(f"[case] noalloc c4 T=28 workspace={plan.info.workspace_bytes}", flush=True)
    ref, out = _both(plan, x, w, b)
    assert torch.equal(out, ref)
    assert rel_l2(out.cpu().numpy(), config_reference("c4_56x256_k5")) <= GATE

    # 2. a smaller layer with bias and ReLU, ragged tiles
    x, w = small_layer(2, 12, 45, 38, 20, 3, seed=71)
    b = make_random_bias(20, 12, 3, seed=72)
    plan = fs.Plan(2, 12, 45, 38, 20, 3, tile=14, bias=True, relu=True)
    print(f"[case] noalloc small os workspace={plan.info.workspace_bytes}", flush=True)
    ref, out = _both(plan, x, w, b)
    assert torch.equal(out, ref)
    assert rel_l2(out.cpu().numpy(), oracle.direct_xcorr2d(x, w, b, relu=True)) <= GATE

    # 3. smaller still, overlap-add with a max-pool: the seam partials and the
    #    unpooled staging buffer live in the scratch too
    x, w = small_layer(1, 3, 30, 30, 5, 3, seed=77)
    b = make_random_bias(5, 3, 3, seed=78)
    plan = fs.Plan(1, 3, 30, 30, 5, 3, tile=14, mode="oaa", bias=True, relu=True, pool=True)
    assert plan.info.aux_bytes > 0
    print(f"[case] noalloc small oaa+pool workspace={plan.info.workspace_bytes}", flush=True)
    ref, out = _both(plan, x, w, b)
    assert torch.equal(out, ref)
    assert rel_l2(out.cpu().numpy(), oracle.maxpool2x2(oracle.direct_xcorr2d(x, w, b, relu=True))) <= GATE


def test_noalloc_rejects_plans_beyond_the_scratch():
    # 32 x 64 x 224^2 -> 64 (the second VGG-16 layer at batch 32) needs about
    # 1 GiB of workspace: rejected before anything is enqueued
    plan = fs.Plan(32, 64, 224, 224, 64, 3, tile=14)
    assert plan.info.workspace_bytes > fs.NOALLOC_MAX_WORKSPACE
    x = torch.zeros((32, 64, 224, 224), dtype=torch.float32, device="cuda")
    wspec = torch.zeros(plan.info.wspec_bytes // 4, dtype=torch.float32, device="cuda")
    out = torch.full(plan.out_shape, 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(fs.FftsplitError) as e:
        plan.conv2d_noalloc(x, wspec, out=out)
    assert e.value.status == fs.ERROR_INSUFFICIENT_WORKSPACE
    assert "static scratch" in fs.last_error()
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    # and the next call that fits still works
    x1, w1 = small_layer(1, 4, 20, 20, 8, 3, seed=5)
    p1 = fs.Plan(1, 4, 20, 20, 8, 3, tile=6)
    ref, got = _both(p1, x1, w1, None)
    assert torch.equal(got, ref)
