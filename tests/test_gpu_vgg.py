"""The VGG-16 stack (13 convolutions with bias+ReLU, 5 max-pools) on the
split-FFT convolution at batch 32, each layer's tile chosen by its plan.

Against the float64 oracle (images are independent, so a subset of the
batch is an exact check of those images):
  * the final activation of all 32 images, as a chain from the input --
    the gate rel-L2 <= 1e-4, over the batch and per image;
  * every layer's output on images spread over the batch (first, second,
    middle, last), as a chain from the input (the gate) and fed the GPU's
    own previous activation, which localises drift to a layer (each layer
    alone within 1e-5);
  * the default stack, whose stage-ending layers pool inside their inverse
    stage, bit for bit against the stack with separate pooling passes, on
    all 32 images.
"""
import numpy as np
import pytest

import oracle
from workloads import make_vgg16

from spectra_layout import rel_l2

torch = pytest.importorskip("torch")
fs = pytest.importorskip("paper_2003_12621_amd")

pytestmark = pytest.mark.gpu

BATCH = 32
SAMPLE = [0, 1, 15, 31]


@pytest.fixture(scope="module")
def vgg_run():
    from paper_2003_12621_amd.vgg import VGG16Stack, POOL_AFTER
    x, layers = make_vgg16(batch=BATCH, seed=0)
    stack = VGG16Stack(layers, batch=BATCH, fuse_pool=False)
    out, outs = stack.forward(torch.from_numpy(x).cuda(), keep=True)
    torch.cuda.synchronize()
    print(f"[vgg] tiles per layer: {stack.tiles}", flush=True)
    got = [o[SAMPLE].cpu().numpy() for o in outs]
    final = out.cpu().numpy()
    return x, layers, got, final, POOL_AFTER


@pytest.fixture(scope="module")
def vgg_ref():
    """Every layer's output for the sampled images (float64 chain)."""
    x, layers = make_vgg16(batch=BATCH, seed=0)
    return oracle.vgg16_forward(x[SAMPLE], layers, return_all=True)


@pytest.fixture(scope="module")
def vgg_ref_final():
    """The final activation of the whole batch (float64 chain, eight images
    at a time to bound host memory)."""
    x, layers = make_vgg16(batch=BATCH, seed=0)
    return np.concatenate([oracle.vgg16_forward(x[i:i + 8], layers) for i in range(0, BATCH, 8)])


def test_vgg16_chain_matches_oracle(vgg_run, vgg_ref, vgg_ref_final):
    x, layers, got, final, _ = vgg_run
    ref_outs, ref_final_sample = vgg_ref
    assert final.shape == (BATCH, 512, 7, 7)
    for i, (g, r) in enumerate(zip(got, ref_outs), start=1):
        err = rel_l2(g, r)
        print(f"[vgg] layer {i:2d} chain rel_l2 = {err:.3e} (images {SAMPLE})", flush=True)
        assert err <= 1e-4, i
    np.testing.assert_array_equal(vgg_ref_final[SAMPLE], ref_final_sample)
    err = rel_l2(final, vgg_ref_final)
    per_image = [rel_l2(final[i], vgg_ref_final[i]) for i in range(BATCH)]
    print(f"[vgg] final rel_l2 = {err:.3e} over {BATCH} images, worst image {max(per_image):.3e}", flush=True)
    assert err <= 1e-4
    assert max(per_image) <= 1e-4, int(np.argmax(per_image))


def test_vgg16_each_layer_on_gpu_input(vgg_run):
    x, layers, got, _, pool_after = vgg_run
    a = x[SAMPLE].astype(np.float64)
    for i, (w, b) in enumerate(layers, start=1):
        ref = oracle.direct_xcorr2d(a, w, b, relu=True)
        err = rel_l2(got[i - 1], ref)
        assert err <= 1e-5, (i, err)
        a = got[i - 1].astype(np.float64)
        if i in pool_after:
            a = oracle.maxpool2x2(a)


def test_vgg16_direct_stack_matches_oracle(vgg_ref):
    """The same stack on the spatial convolution (method="direct"), on the
    sampled images as a batch: final activation against the float64 chain."""
    from paper_2003_12621_amd.vgg import VGG16Stack
    x, layers = make_vgg16(batch=BATCH, seed=0)
    xs = np.ascontiguousarray(x[SAMPLE])
    stack = VGG16Stack(layers, batch=len(SAMPLE), method="direct")
    out = stack.forward(torch.from_numpy(xs).cuda())
    torch.cuda.synchronize()
    err = rel_l2(out.cpu().numpy(), vgg_ref[1])
    print(f"[vgg] direct stack final rel_l2 = {err:.3e}", flush=True)
    assert err <= 1e-4


def test_vgg16_fused_pool_stack(vgg_run, vgg_ref_final):
    """The stack as it runs by default: the stage-ending layers write pooled
    activations (FFTSPLIT_MAXPOOL); same final output as with separate
    pooling passes, bit for bit on every image, and within the gate of the
    oracle chain."""
    from paper_2003_12621_amd.vgg import VGG16Stack
    x, layers, _, final_unfused, _ = vgg_run
    stack = VGG16Stack(layers, batch=BATCH)
    assert [p.pool for p in stack.plans] == [i in (2, 4, 7, 10, 13) for i in range(1, 14)]
    out = stack.forward(torch.from_numpy(x).cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    np.testing.assert_array_equal(got, final_unfused)
    assert rel_l2(got, vgg_ref_final) <= 1e-4
