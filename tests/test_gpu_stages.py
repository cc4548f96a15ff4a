"""Stage-by-stage parity of the HIP kernels against the oracle's steps.

Each kernel is fed inputs the oracle also sees and compared element by
element, so a failure names the stage:
  weights  -- eq. 8: conj(DFT(zero-padded filter)) / L^2 at the stored bins
  forward  -- eqs. 4-6 + forward DFT of every padded patch
  contract -- eq. 9 summed over input channels, on the GPU's own spectra
  inverse  -- eq. 10 (inverse DFT, crop/concatenate), bias, ReLU, on the
              GPU's own output spectra
Tolerances: spectra evaluated in double and rounded once (weights) must be
within 1e-6 relative; fp32 transforms and sums within 2e-6 relative L2.
"""
import numpy as np
import pytest

import oracle
from workloads import make_config, small_layer, make_random_bias

from spectra_layout import full_to_stored, stored_to_full, rel_l2, rel_max

torch = pytest.importorskip("torch")
fs = pytest.importorskip("paper_2003_12621_amd")

pytestmark = pytest.mark.gpu

CASES = [
    # name, (n, cin, h, w, cout, k), tile, mode
    ("c1_L8", (1, 3, 32, 32, 16, 3), 6),
    ("ragged_L16_k5", (2, 5, 19, 23, 10, 5), 12),
    ("ragged_L32", (3, 4, 37, 30, 7, 3), 30),
    ("k1_L8", (1, 2, 17, 9, 3, 1), 8),
    ("k7_L16", (1, 3, 21, 20, 5, 7), 10),
    # the OaAConv configuration (overlap-add, T = K, odd L = 2K - 1)
    ("oaa_k3_L5", (2, 5, 19, 23, 10, 3), 3),
    ("oaa_k5_L9", (1, 3, 21, 20, 70, 5), 5),
    ("oaa_k7_L13", (2, 17, 17, 30, 7, 7), 7),
]


def _oaaconv(shape, tile):
    return tile == shape[5] and tile in (3, 5, 7)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _setup(shape, tile, mode="os", seed=5):
    n, cin, h, w, cout, k = shape
    if _oaaconv(shape, tile):
        mode = "oaa"
    x, wt = small_layer(n, cin, h, w, cout, k, seed=seed)
    plan = fs.Plan(n, cin, h, w, cout, k, tile=tile, mode=mode)
    return x, wt, plan


@pytest.mark.parametrize("name,shape,tile", CASES)
def test_weight_spectra(name, shape, tile):
    x, wt, plan = _setup(shape, tile)
    L = plan.nfft
    wspec = plan.transform_weights(_dev(wt))
    torch.cuda.synchronize()
    got = plan.wspec_view(wspec).cpu().numpy()                     # [bins, cin, coutp]
    ref = full_to_stored(np.conj(oracle.filter_spectra(wt, L)) / (L * L))   # [bins, cout, cin]
    ref = ref.transpose(0, 2, 1)
    cout = shape[4]
    assert rel_max(got[:, :, :cout], ref) < 1e-6
    assert np.all(got[:, :, cout:] == 0)


@pytest.mark.parametrize("mode", ["os", "oaa"])
@pytest.mark.parametrize("name,shape,tile", CASES)
def test_forward_spectra(name, shape, tile, mode):
    n, cin, h, w, cout, k = shape
    if mode == "oaa" and tile < k - 1:
        pytest.skip("overlap-add needs T >= K - 1")
    if mode == "os" and _oaaconv(shape, tile):
        pytest.skip("the OaAConv configuration is overlap-add only")
    x, wt, plan = _setup(shape, tile, mode)
    ws = plan.new_workspace()
    plan.forward(_dev(x), ws)
    torch.cuda.synchronize()
    got = plan.xspec_view(ws).cpu().numpy()                        # [bins, cin, ntp]
    ref = oracle.patch_spectra(x, tile, k, mode)                   # [n, th, tw, cin, L, L]
    nt = plan.info.tiles
    ref = full_to_stored(ref.reshape(nt, cin, plan.nfft, plan.nfft))  # [bins, nt, cin]
    ref = ref.transpose(0, 2, 1)
    assert rel_l2(got[:, :, :nt], ref) < 2e-6
    assert rel_max(got[:, :, :nt], ref) < 1e-5
    assert np.all(got[:, :, nt:] == 0), "padding patches must have zero spectra"


@pytest.mark.parametrize("name,shape,tile", CASES)
def test_contraction(name, shape, tile):
    n, cin, h, w, cout, k = shape
    x, wt, plan = _setup(shape, tile)
    ws = plan.new_workspace()
    wspec = plan.transform_weights(_dev(wt))
    plan.forward(_dev(x), ws)
    plan.contract(wspec, ws)
    torch.cuda.synchronize()
    X = plan.xspec_view(ws).cpu().numpy().astype(np.complex128)     # [bins, cin, ntp]
    W = plan.wspec_view(wspec).cpu().numpy().astype(np.complex128)  # [bins, cin, coutp]
    Y = plan.yspec_view(ws).cpu().numpy()                           # [bins, coutp, ntp]
    # oracle step 4 with xs [t, ci, bins] and ws [co, ci, bins]; the stored
    # filter spectra are already conjugated, so they enter as conj(W).
    ref = oracle.hadamard_channel_sum(X.transpose(2, 1, 0), np.conj(W).transpose(2, 1, 0))  # [t, co, bins]
    ref = ref.transpose(2, 1, 0)                                    # [bins, co, t]
    # for even L the last two slots each hold two real bins (real and
    # imaginary part): their products are taken part by part
    for f in ((-2, -1) if plan.nfft % 2 == 0 else ()):
        ref[f] = (np.einsum("ic,it->ct", W[f].real, X[f].real)
                  + 1j * np.einsum("ic,it->ct", W[f].imag, X[f].imag))
    assert rel_l2(Y, ref) < 2e-6
    assert rel_max(Y, ref) < 1e-5


@pytest.mark.parametrize("mode", ["os", "oaa"])
@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("name,shape,tile", CASES)
def test_inverse_placement(name, shape, tile, relu, mode):
    n, cin, h, w, cout, k = shape
    if mode == "os" and _oaaconv(shape, tile):
        pytest.skip("the OaAConv configuration is overlap-add only")
    x, wt = small_layer(n, cin, h, w, cout, k, seed=6)
    plan = fs.Plan(n, cin, h, w, cout, k, tile=tile, bias=True, relu=relu, mode=mode)
    L = plan.nfft
    b = make_random_bias(cout, cin, k, seed=7)
    ws = plan.new_workspace()
    wspec = plan.transform_weights(_dev(wt))
    plan.forward(_dev(x), ws)
    plan.contract(wspec, ws)
    y = plan.inverse(ws, bias=_dev(b))
    torch.cuda.synchronize()
    Y = plan.yspec_view(ws).cpu().numpy()                            # [bins, coutp, ntp]
    nt = plan.info.tiles
    th, tw = plan.info.tiles_h, plan.info.tiles_w
    full = stored_to_full(Y[:, :cout, :nt], L)                       # [cout, nt, L, L]
    full = full.transpose(1, 0, 2, 3).reshape(n, th, tw, cout, L, L)
    # The stored output spectra carry the 1/L^2 of the inverse already; the
    # oracle's inverse divides by L^2 itself.
    ref = oracle.inverse_place(full * (L * L), h, w, tile, k, mode, b, relu)
    got = y.cpu().numpy()
    assert rel_l2(got, ref) < 2e-6
    assert rel_max(got, ref) < 1e-5


def test_maxpool_exact():
    rng = np.random.default_rng(8)
    for shape in [(2, 3, 8, 8), (1, 5, 7, 9), (4, 64, 224, 224), (1, 1, 2, 2)]:
        x = rng.standard_normal(shape).astype(np.float32)
        got = fs.maxpool2x2(_dev(x)).cpu().numpy()
        np.testing.assert_array_equal(got, oracle.maxpool2x2(x))


@pytest.mark.parametrize("prefetch", ["1", "2", "3"])
@pytest.mark.parametrize("cin", [16, 32, 40, 48, 64, 80, 100])
@pytest.mark.parametrize("cout", [64, 128])
def test_contraction_stage_pipeline(cin, cout, prefetch, monkeypatch):
    """The contraction's input-channel pipeline (stages of 16 channels loaded
    one, two or three stages ahead; a partial last stage; 64 x 64 tiles, and
    128 x 32 where 32 patches are padded) against the oracle's channel sum,
    and bit-identical across prefetch depths (same products, same order)."""
    monkeypatch.setenv("FFTSPLIT_CONTRACT_PREFETCH", prefetch)
    shape = (2, cin, 24, 24, cout, 3)
    x, wt = small_layer(*shape, seed=cin)
    plan = fs.Plan(*shape, tile=14)
    print(f"[case] cin={cin} cout={cout} prefetch={plan.info.contract_prefetch} "
          f"tile={plan.info.contract_tile_m}x{plan.info.contract_tile_n}", flush=True)
    ws = plan.new_workspace()
    wspec = plan.transform_weights(_dev(wt))
    plan.forward(_dev(x), ws)
    plan.contract(wspec, ws)
    torch.cuda.synchronize()
    X = plan.xspec_view(ws).cpu().numpy().astype(np.complex128)
    W = plan.wspec_view(wspec).cpu().numpy().astype(np.complex128)
    Y = plan.yspec_view(ws).cpu().numpy()
    ref = oracle.hadamard_channel_sum(X.transpose(2, 1, 0), np.conj(W).transpose(2, 1, 0)).transpose(2, 1, 0)
    for f in (-2, -1):
        ref[f] = (np.einsum("ic,it->ct", W[f].real, X[f].real)
                  + 1j * np.einsum("ic,it->ct", W[f].imag, X[f].imag))
    assert rel_l2(Y, ref) < 2e-6
    monkeypatch.setenv("FFTSPLIT_CONTRACT_PREFETCH", "1")
    plan1 = fs.Plan(*shape, tile=14)
    ws1 = plan1.new_workspace()
    plan1.forward(_dev(x), ws1)
    plan1.contract(plan1.transform_weights(_dev(wt)), ws1)
    torch.cuda.synchronize()
    assert np.array_equal(plan1.yspec_view(ws1).cpu().numpy(), Y)


@pytest.mark.parametrize("cin", [4, 8, 12, 20, 40, 64, 100])
def test_contraction_eight_channel_stages(cin, monkeypatch):
    """The 64 x 64 tile with 8-channel stages (the plan's choice for few
    input channels and many workgroups), loaded one, two and three stages
    ahead, partial last stages included: against the oracle's channel sum,
    and equal to the 16-channel stages' result (the same products added in
    the same channel order)."""
    shape = (2, cin, 24, 24, 64, 3)
    x, wt = small_layer(*shape, seed=100 + cin)
    outs = []
    for tile_env, pf in (("g3:64x64x16", "2"), ("g3:64x64x8", "1"), ("g3:64x64x8", "2"), ("g3:64x64x8", "3")):
        monkeypatch.setenv("FFTSPLIT_CONTRACT_TILE", tile_env)
        monkeypatch.setenv("FFTSPLIT_CONTRACT_PREFETCH", pf)
        plan = fs.Plan(*shape, tile=14)
        info = plan.info
        assert (info.contract_tile_m, info.contract_tile_n, info.contract_prefetch) == (64, 64, int(pf))
        print(f"[case] cin={cin} {tile_env} prefetch={pf}", flush=True)
        ws = plan.new_workspace()
        wspec = plan.transform_weights(_dev(wt))
        plan.forward(_dev(x), ws)
        plan.contract(wspec, ws)
        torch.cuda.synchronize()
        outs.append(plan.yspec_view(ws).cpu().numpy())
    X = plan.xspec_view(ws).cpu().numpy().astype(np.complex128)
    W = plan.wspec_view(wspec).cpu().numpy().astype(np.complex128)
    ref = oracle.hadamard_channel_sum(X.transpose(2, 1, 0), np.conj(W).transpose(2, 1, 0)).transpose(2, 1, 0)
    for f in (-2, -1):
        ref[f] = (np.einsum("ic,it->ct", W[f].real, X[f].real)
                  + 1j * np.einsum("ic,it->ct", W[f].imag, X[f].imag))
    for o in outs:
        assert rel_l2(o, ref) < 2e-6
        assert np.array_equal(o, outs[0])


@pytest.mark.parametrize("tile_env,n", [("g3:128x64x16", 16), ("g3:64x128x16", 32)])
def test_contraction_other_tiles(tile_env, n, monkeypatch):
    """The 128 x 64 and 64 x 128 tiles (plan options), both prefetch depths,
    against the oracle's channel sum and bit-identical to each other."""
    monkeypatch.setenv("FFTSPLIT_CONTRACT_TILE", tile_env)
    shape = (n, 40, 24, 24, 128, 3)
    x, wt = small_layer(*shape, seed=11)
    outs = []
    for pf in ("1", "2"):
        monkeypatch.setenv("FFTSPLIT_CONTRACT_PREFETCH", pf)
        plan = fs.Plan(*shape, tile=14)
        print(f"[case] {tile_env} n={n} prefetch={plan.info.contract_prefetch}", flush=True)
        ws = plan.new_workspace()
        wspec = plan.transform_weights(_dev(wt))
        plan.forward(_dev(x), ws)
        plan.contract(wspec, ws)
        torch.cuda.synchronize()
        outs.append(plan.yspec_view(ws).cpu().numpy())
    X = plan.xspec_view(ws).cpu().numpy().astype(np.complex128)
    W = plan.wspec_view(wspec).cpu().numpy().astype(np.complex128)
    ref = oracle.hadamard_channel_sum(X.transpose(2, 1, 0), np.conj(W).transpose(2, 1, 0)).transpose(2, 1, 0)
    for f in (-2, -1):
        ref[f] = (np.einsum("ic,it->ct", W[f].real, X[f].real)
                  + 1j * np.einsum("ic,it->ct", W[f].imag, X[f].imag))
    assert rel_l2(outs[1], ref) < 2e-6
    assert np.array_equal(outs[0], outs[1])
