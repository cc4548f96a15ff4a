"""The plan's cost model against the paper's operation counts (Section 3.2,
eqs. 13-14), host-only (plans for the architecture name, no GPU).

* Contraction work: eq. 13 minus eq. 14 is the Hadamard term,
  N^2/s^2 * (s+k-1)^2 complex products per channel pair and image.  The
  plan's model counts 8 real flops per complex multiply-add over the L^2/2
  stored bins of a real input (half of the L^2 complex bins eq. 13 counts),
  i.e. 4 flops per Hadamard product of eq. 13, for every (image, input,
  output) triple -- exactly, where the tile divides the image and nothing
  is padded; otherwise scaled by the padding of patches and channels.
* Tile choice: over L in {8, 16, 32}, the L that minimises eqs. 13 + 14
  per channel pair is the L the plan's time model picks on every workload
  but the smallest (1x3x32x32 -> 16), where padding 36 patches to 64 and 16
  channels to 64 dominates a model that prices padded work.
"""
import pytest

from oracle import opcount
from workloads import CONFIGS, VGG16_LAYERS, VGG_BATCH

fs = pytest.importorskip("paper_2003_12621_amd")


def _plan(n, cin, h, w, cout, k, tile=0):
    return fs.Plan(n, cin, h, w, cout, k, tile=tile, arch="gfx950")


def _hadamard(n_img, k, s):
    return opcount.mul_splitconv(n_img, k, s) - opcount.add_splitconv(n_img, k, s)


@pytest.mark.parametrize("name,tile", [("c2_224x64", 14), ("c3_112x128", 14), ("c4_56x256_k5", 28),
                                       ("c2_224x64", 30), ("c4_56x256_k5", 12), ("c1_32x3", 6)])
def test_model_contraction_flops_match_eq13_hadamard_term(name, tile):
    L = CONFIGS[name]["layer"]
    p = _plan(L.n, L.cin, L.h, L.w, L.cout, L.k, tile=tile)
    i = p.info
    exact = 4.0 * L.n * L.cin * L.cout * _hadamard(L.h, L.k, tile)
    # padding: patches (ceil(h/T)^2 per image, rounded up to the contraction
    # granule) against eq. 13's h^2/T^2, output channels against cout
    pad = (i.tiles_padded / (L.n * L.h * L.h / tile ** 2)) * (i.cout_padded / L.cout)
    assert i.model_contract_flops == pytest.approx(exact * pad, rel=1e-12)
    if L.h % tile == 0 and i.tiles_padded == i.tiles and i.cout_padded == L.cout:
        assert i.model_contract_flops == pytest.approx(exact, rel=1e-12)


def _eq13_14_argmin(h, k):
    tot = {}
    for nfft in (8, 16, 32):
        s = nfft - k + 1
        if s >= 1:
            tot[nfft] = opcount.mul_splitconv(h, k, s) + opcount.add_splitconv(h, k, s)
    return min(tot, key=tot.get)


@pytest.mark.parametrize("name", ["c2_224x64", "c3_112x128", "c4_56x256_k5"])
def test_tile_choice_matches_eq13_14_on_the_layers(name):
    L = CONFIGS[name]["layer"]
    assert _plan(L.n, L.cin, L.h, L.w, L.cout, L.k).nfft == _eq13_14_argmin(L.h, L.k)


@pytest.mark.parametrize("cin,cout,hw", VGG16_LAYERS)
def test_tile_choice_matches_eq13_14_on_vgg16(cin, cout, hw):
    assert _plan(VGG_BATCH, cin, hw, hw, cout, 3).nfft == _eq13_14_argmin(hw, 3)


def test_smallest_layer_is_where_they_differ():
    L = CONFIGS["c1_32x3"]["layer"]
    p = _plan(L.n, L.cin, L.h, L.w, L.cout, L.k)
    assert _eq13_14_argmin(L.h, L.k) == 16 and p.nfft == 8
    # padded work at L = 8: 36 patches -> 64, 16 channels -> 64
    assert (p.info.tiles, p.info.tiles_padded, p.info.cout_padded) == (36, 64, 64)


def test_model_transform_bytes():
    # forward: x once + patch spectra once; inverse: output spectra once +
    # y once (8 bytes per stored bin, L^2/2 bins per patch and channel)
    L = CONFIGS["c4_56x256_k5"]["layer"]
    i = _plan(L.n, L.cin, L.h, L.w, L.cout, L.k, tile=28).info
    img = L.n * L.h * L.w * 4
    spectra = 8 * (32 * 32 // 2) * 64
    assert i.model_transform_bytes == img * (L.cin + L.cout) + spectra * (L.cin + L.cout)


def test_fig3_table():
    """tests/golden/fig3_opcounts.txt (written from oracle.opcount by
    tests/golden/make_golden.py) states Fig. 3's outcome in numbers: SplitConv
    with s = 16 and s = 32 needs fewer operations than OaAConv at every
    kernel size 3..11, and for s = 32 the saving grows from k = 3 to 9."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "fig3_opcounts.txt")
    rows = [[float(v) for v in l.split()] for l in open(path) if l.strip() and not l.startswith("#")]
    assert [int(r[0]) for r in rows] == [3, 5, 7, 9, 11]
    for k, oaa, s16, s32, r16, r32 in rows:
        k = int(k)
        assert oaa == pytest.approx(opcount.mul_oaaconv(224, k) + opcount.add_oaaconv(224, k), rel=1e-12)
        assert s16 == pytest.approx(opcount.mul_splitconv(224, k, 16) + opcount.add_splitconv(224, k, 16),
                                    rel=1e-12)
        assert s32 == pytest.approx(opcount.mul_splitconv(224, k, 32) + opcount.add_splitconv(224, k, 32),
                                    rel=1e-12)
        assert oaa > s16 and oaa > s32
    r32 = [r[5] for r in rows]
    assert r32[0] < r32[1] < r32[2] < r32[3]
