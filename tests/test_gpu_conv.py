"""End-to-end parity of fftsplit_conv2d against the oracle.

The gate (stated for the method's fp32 output): relative L2 error
||y - y_ref|| / ||y_ref|| <= 1e-4 against the float64 direct
cross-correlation on the same seeded inputs, over every image, output
channel and pixel of each workload.
"""
import numpy as np
import pytest

import oracle
from workloads import CONFIGS, make_config, make_random_bias, small_layer

from config_reference import config_inputs, config_reference
from spectra_layout import rel_l2, rel_max

torch = pytest.importorskip("torch")
fs = pytest.importorskip("paper_2003_12621_amd")

pytestmark = pytest.mark.gpu

GATE = 1e-4


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def run_layer(x, w, b, tile, mode="os", relu=False):
    n, cin, h, wd = x.shape
    cout, _, k, _ = w.shape
    plan = fs.Plan(n, cin, h, wd, cout, k, tile=tile, mode=mode, bias=b is not None, relu=relu)
    wspec = plan.transform_weights(_dev(w))
    y = plan.conv2d(_dev(x), wspec, None if b is None else _dev(b))
    torch.cuda.synchronize()
    return plan, y.cpu().numpy()


def config_cases():
    for name, cfg in CONFIGS.items():
        for t in cfg["tiles"]:
            for mode in ("os", "oaa"):
                yield pytest.param(name, t, mode, id=f"{name}-T{t}-{mode}")


@pytest.mark.parametrize("name,tile,mode", list(config_cases()))
def test_config_parity(name, tile, mode):
    x, w, b = config_inputs(name)
    print(f"[case] {name} T={tile} {mode}", flush=True)
    plan, y = run_layer(x, w, b, tile, mode=mode)
    assert plan.tile == tile
    ref = config_reference(name)
    assert y.shape == ref.shape
    err = rel_l2(y, ref)
    print(f"[case] {name} T={tile} {mode} rel_l2={err:.3e} rel_max={rel_max(y, ref):.3e}", flush=True)
    assert err <= GATE
    # every output channel on its own (a fault confined to one contraction
    # tile would hide in the layer-wide norm)
    per_channel = [rel_l2(y[:, c], ref[:, c]) for c in range(ref.shape[1])]
    assert max(per_channel) <= GATE, int(np.argmax(per_channel))


EDGE = [
    # (n, cin, h, w, cout, k), tile
    ((1, 3, 19, 17, 4, 5), 4),     # overlap-add with T = K - 1 (no core)
    ((1, 2, 5, 5, 3, 3), 6),       # image smaller than a tile
    ((1, 2, 6, 6, 3, 3), 6),       # image equal to a tile
    ((2, 3, 13, 29, 4, 3), 6),     # ragged, H != W, n > 1
    ((1, 1, 40, 33, 1, 3), 14),    # Cin = Cout = 1
    ((1, 7, 31, 31, 65, 5), 12),   # Cout just above the 64-channel granule
    ((3, 9, 33, 35, 5, 5), 28),    # K = 5 at L = 32, ragged
    ((1, 4, 20, 20, 6, 1), 16),    # K = 1 (pointwise), L = 16
    ((2, 3, 30, 30, 4, 7), 26),    # K = 7 at L = 32
    ((1, 130, 17, 17, 3, 3), 14),  # Cin not a multiple of the contraction's K step
    ((32, 16, 14, 14, 128, 3), 14),  # one patch per image: patches padded to 32, 128x32 tiles
    ((3, 20, 28, 28, 256, 3), 14),   # 12 patches padded to 32
    ((5, 8, 40, 40, 130, 3), 30),    # output channels not in 128s: padded to 64
    ((1, 5, 23, 300, 7, 3), 30),     # width beyond the row-band kernels' 256: general forward / inverse, L = 32
    ((2, 4, 19, 264, 9, 5), 12),     # the same at L = 16, K = 5
    ((1, 3, 9, 258, 4, 3), 6),       # the same at L = 8
    ((1, 4, 20, 20, 5, 9), 8),       # K = 9 at L = 16
    ((2, 3, 17, 23, 4, 15), 2),      # K = 15: two-pixel tiles at L = 16 (overlap-save only)
    ((1, 2, 40, 40, 3, 31), 2),      # K = 31, the largest kernel: two-pixel tiles at L = 32
    ((1, 3, 9, 9, 2, 7), 26),        # one tile larger than the image, K = 7
    ((3, 5, 1, 37, 6, 3), 6),        # one-row images
    ((2, 4, 29, 1, 3, 5), 12),       # one-column images
]


@pytest.mark.parametrize("mode", ["os", "oaa"])
@pytest.mark.parametrize("shape,tile", EDGE)
@pytest.mark.parametrize("bias,relu", [(False, False), (True, True)])
def test_edge_shapes(shape, tile, bias, relu, mode):
    n, cin, h, w, cout, k = shape
    if mode == "oaa" and tile < k - 1:
        pytest.skip("overlap-add needs T >= K - 1")
    x, wt = small_layer(n, cin, h, w, cout, k, seed=31)
    b = make_random_bias(cout, cin, k, seed=32) if bias else None
    _, y = run_layer(x, wt, b, tile, mode=mode, relu=relu)
    ref = oracle.direct_xcorr2d(x, wt, b, relu=relu)
    assert rel_l2(y, ref) <= GATE
    assert rel_max(y, ref) <= 1e-5


def test_first_config_with_bias_and_relu():
    x, w, _ = make_config("c1_32x3")
    b = make_random_bias(16, 3, 3, seed=3)
    _, y = run_layer(x, w, b, 6, relu=True)
    ref = oracle.direct_xcorr2d(x, w, b, relu=True)
    assert rel_l2(y, ref) <= GATE


def test_overlap_save_is_deterministic():
    x, w, _ = make_config("c1_32x3")
    n, cin, h, wd = x.shape
    plan = fs.Plan(n, cin, h, wd, 16, 3, tile=6)
    wspec = plan.transform_weights(_dev(w))
    xd = _dev(x)
    outs = [plan.conv2d(xd, wspec).cpu().numpy() for _ in range(3)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_tile_sizes_agree():
    x, w = small_layer(2, 16, 61, 58, 24, 3, seed=41)
    ys = [run_layer(x, w, None, t)[1] for t in (6, 14, 30)]
    assert rel_l2(ys[1], ys[0]) <= 1e-5
    assert rel_l2(ys[2], ys[0]) <= 1e-5


def test_error_paths():
    x, w = small_layer(1, 3, 32, 32, 16, 3, seed=51)
    plan = fs.Plan(1, 3, 32, 32, 16, 3, tile=6)
    wspec = plan.transform_weights(_dev(w))
    xd = _dev(x)
    ws = plan.new_workspace()
    small = ws[: ws.numel() // 2]
    with pytest.raises(fs.FftsplitError) as e:
        plan.conv2d(xd, wspec, workspace=small)
    assert e.value.status == fs.ERROR_INSUFFICIENT_WORKSPACE
    # misaligned output pointer
    big = torch.empty(16 * 32 * 32 + 1, dtype=torch.float32, device="cuda")
    with pytest.raises(fs.FftsplitError) as e:
        plan.conv2d(xd, wspec, out=big[1:])
    assert e.value.status == fs.ERROR_INVALID_VALUE
    # output overlapping the input
    buf = torch.empty(3 * 32 * 32 + 16 * 32 * 32, dtype=torch.float32, device="cuda")
    buf[: 3 * 32 * 32].copy_(xd.view(-1))
    x_alias = buf[: 3 * 32 * 32].view(1, 3, 32, 32)
    y_alias = buf[1024: 1024 + 16 * 32 * 32].view(1, 16, 32, 32)
    with pytest.raises(fs.FftsplitError) as e:
        plan.conv2d(x_alias, wspec, out=y_alias)
    assert e.value.status == fs.ERROR_INVALID_VALUE
    # bias without the flag
    with pytest.raises(fs.FftsplitError) as e:
        plan.conv2d(xd, wspec, bias=torch.zeros(16, device="cuda"))
    assert e.value.status == fs.ERROR_INVALID_VALUE
    # after the failures, a good call still works
    y = plan.conv2d(xd, wspec)
    torch.cuda.synchronize()
    assert rel_l2(y.cpu().numpy(), oracle.direct_xcorr2d(x, w)) <= GATE



def test_timing_events_bracket_the_kernels():
    x, w = small_layer(2, 16, 40, 40, 32, 3, seed=61)
    plan = fs.Plan(2, 16, 40, 40, 32, 3, tile=14)
    wspec = plan.transform_weights(_dev(w))
    xd = _dev(x)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in ev:
        e.record()
    ws = plan.new_workspace()
    fs.set_timing_events(ev[0], ev[1])
    y = plan.conv2d(xd, wspec, workspace=ws)
    fs.set_timing_events(ev[2], ev[3])
    plan.contract(wspec, ws)
    fs.set_timing_events()
    torch.cuda.synchronize()
    t_conv = ev[0].elapsed_time(ev[1])
    t_con = ev[2].elapsed_time(ev[3])
    assert 0 < t_con < t_conv < 1000.0
    assert rel_l2(y.cpu().numpy(), oracle.direct_xcorr2d(x, w)) <= GATE
    with pytest.raises(ValueError):
        fs.set_timing_events(torch.cuda.Event(enable_timing=True), None)


@pytest.mark.parametrize("tile", [6, 14, 30])
def test_overlap_save_equals_overlap_add(tile):
    x, w = small_layer(2, 12, 45, 38, 20, 3, seed=71)
    b = make_random_bias(20, 12, 3, seed=72)
    _, y_os = run_layer(x, w, b, tile, mode="os", relu=True)
    _, y_oaa = run_layer(x, w, b, tile, mode="oaa", relu=True)
    assert rel_l2(y_oaa, y_os) <= 1e-6


def test_overlap_add_is_deterministic():
    x, w = small_layer(1, 8, 40, 40, 16, 5, seed=73)
    plan = fs.Plan(1, 8, 40, 40, 16, 5, tile=12, mode="oaa")
    wspec = plan.transform_weights(_dev(w))
    xd = _dev(x)
    outs = [plan.conv2d(xd, wspec).cpu().numpy() for _ in range(3)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


POOL_CASES = [
    # (n, cin, h, w, cout, k), tile, mode: which path pools
    ((2, 5, 28, 28, 9, 3), 14, "os"),     # band inverse, pooled in its store phase
    ((3, 4, 56, 56, 70, 5), 28, "os"),    # band, items spanning images
    ((1, 3, 60, 40, 6, 3), 6, "os"),      # band, T/2 odd and items starting mid tile-row: straddles
    ((2, 3, 26, 44, 5, 3), 14, "os"),     # band, ragged last tile rows and columns
    ((1, 2, 27, 28, 4, 3), 14, "os"),     # band, odd height: staged output + pooling pass
    ((3, 6, 14, 14, 7, 3), 14, "os"),     # general inverse (width 14), pooled in its store phase
    ((2, 3, 30, 26, 5, 3), 14, "os"),     # general, ragged last tiles
    ((1, 2, 27, 30, 4, 3), 6, "os"),      # general, L = 8, odd height: floor in the store phase
    ((2, 3, 22, 18, 5, 5), 12, "os"),     # general, K = 5
    ((1, 2, 21, 34, 3, 3), 30, "os"),     # general, L = 32, one partial tile per row
    ((1, 3, 30, 30, 5, 3), 14, "oaa"),    # overlap-add: staged output + pooling pass
    ((2, 3, 17, 19, 4, 3), 3, "oaa"),     # OaAConv configuration, odd sizes
]


@pytest.mark.parametrize("shape,tile,mode", POOL_CASES, ids=[f"{s}-T{t}-{m}" for s, t, m in POOL_CASES])
@pytest.mark.parametrize("relu", [False, True])
def test_fused_maxpool(shape, tile, mode, relu):
    n, cin, h, w, cout, k = shape
    print(f"[case] maxpool {shape} T={tile} {mode} relu={relu}", flush=True)
    x, wt = small_layer(n, cin, h, w, cout, k, seed=77)
    b = make_random_bias(cout, cin, k, seed=78)
    plan = fs.Plan(n, cin, h, w, cout, k, tile=tile, mode=mode, bias=True, relu=relu, pool=True)
    y = plan.conv2d(_dev(x), plan.transform_weights(_dev(wt)), _dev(b))
    torch.cuda.synchronize()
    assert tuple(y.shape) == (n, cout, h // 2, w // 2)
    ref = oracle.maxpool2x2(oracle.direct_xcorr2d(x, wt, b, relu=relu))
    assert rel_l2(y.cpu().numpy(), ref) <= GATE


FUSED_CIN_CASES = [
    # (n, cin, h, w, cout, k), tile, pool
    ((2, 3, 56, 56, 20, 3), 14, False),    # L = 16, three channels (an RGB input)
    ((1, 1, 40, 44, 70, 3), 14, True),     # L = 16, one channel, pooled
    ((3, 2, 30, 28, 9, 5), 4, False),      # L = 8, K = 5
    ((2, 4, 24, 36, 66, 3), 6, True),      # L = 8, four channels, pooled
    ((4, 3, 28, 28, 16, 3), 6, False),     # L = 8, items of 64 patches spanning images
]


@pytest.mark.parametrize("shape,tile,pool", FUSED_CIN_CASES,
                         ids=[f"{s}-T{t}-pool{int(p)}" for s, t, p in FUSED_CIN_CASES])
def test_fused_channel_sum(shape, tile, pool, monkeypatch):
    """conv2d with the channel sum inside the inverse against the oracle, and
    against the same plan with the contraction (FFTSPLIT_FUSE_CIN=0)."""
    n, cin, h, w, cout, k = shape
    print(f"[case] fused channel sum {shape} T={tile} pool={pool}", flush=True)
    x, wt = small_layer(n, cin, h, w, cout, k, seed=91)
    b = make_random_bias(cout, cin, k, seed=92)
    outs = []
    for fuse in ("1", "0"):
        monkeypatch.setenv("FFTSPLIT_FUSE_CIN", fuse)
        plan = fs.Plan(n, cin, h, w, cout, k, tile=tile, bias=True, relu=True, pool=pool)
        assert plan.info.fused_channel_sum == int(fuse)
        y = plan.conv2d(_dev(x), plan.transform_weights(_dev(wt)), _dev(b))
        torch.cuda.synchronize()
        outs.append(y.cpu().numpy())
    ref = oracle.direct_xcorr2d(x, wt, b, relu=True)
    if pool:
        ref = oracle.maxpool2x2(ref)
    assert rel_l2(outs[0], ref) <= GATE
    assert rel_l2(outs[0], outs[1]) <= 1e-6


def test_streams_and_concurrent_plans():
    """Launches go to the caller's current stream: two layers on two
    streams, each with its own workspace, give the results they give alone."""
    x1, w1 = small_layer(2, 16, 40, 40, 32, 3, seed=101)
    x2, w2 = small_layer(4, 8, 28, 36, 24, 5, seed=102)
    p1 = fs.Plan(2, 16, 40, 40, 32, 3, tile=14)
    p2 = fs.Plan(4, 8, 28, 36, 24, 5, tile=12)
    ws1, ws2 = p1.transform_weights(_dev(w1)), p2.transform_weights(_dev(w2))
    xd1, xd2 = _dev(x1), _dev(x2)
    ref1 = p1.conv2d(xd1, ws1).clone()
    ref2 = p2.conv2d(xd2, ws2).clone()
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for _ in range(3):
        with torch.cuda.stream(s1):
            y1 = p1.conv2d(xd1, ws1)
        with torch.cuda.stream(s2):
            y2 = p2.conv2d(xd2, ws2)
        outs.append((y1, y2))
    torch.cuda.synchronize()
    for y1, y2 in outs:
        assert torch.equal(y1, ref1) and torch.equal(y2, ref2)
    assert rel_l2(ref1.cpu().numpy(), oracle.direct_xcorr2d(x1, w1)) <= GATE
    assert rel_l2(ref2.cpu().numpy(), oracle.direct_xcorr2d(x2, w2)) <= GATE


def test_deterministic_output():
    """Overlap-save results are bitwise reproducible run to run (no atomics;
    every sum in a fixed order); overlap-add's seam sums too."""
    x, w = small_layer(3, 20, 33, 35, 40, 5, seed=103)
    for mode in ("os", "oaa"):
        plan = fs.Plan(3, 20, 33, 35, 40, 5, tile=12, mode=mode)
        wspec = plan.transform_weights(_dev(w))
        xd = _dev(x)
        a = plan.conv2d(xd, wspec).clone()
        b = plan.conv2d(xd, wspec).clone()
        torch.cuda.synchronize()
        assert torch.equal(a, b), mode


def _random_cases(count=48, seed=2024):
    """Seeded random layer shapes over the whole plan space: every kernel
    size, every FFT size that fits, both placements, bias / ReLU / max-pool,
    channel counts around the 16 / 64 / 128 granules."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < count:
        k = int(rng.choice([1, 3, 5, 7]))
        L = int(rng.choice([8, 16, 32]))
        t = L - k + 1
        mode = str(rng.choice(["os", "oaa"]))
        if mode == "oaa" and t < k - 1:
            continue
        if rng.random() < 0.15 and k > 1:          # the OaAConv configuration
            t, mode = k, "oaa"
        n = int(rng.integers(1, 4))
        h = int(rng.integers(1, 3 * t + 5))
        w = int(rng.integers(1, 3 * t + 5))
        if rng.random() < 0.5:
            w = max(4, w - w % 4)                  # widths the row-band kernels take
        cin = int(rng.choice([1, 2, 3, 4, 5, 16, 17, 33]))
        cout = int(rng.choice([1, 3, 16, 64, 65, 128, 130]))
        pool = bool(rng.random() < 0.25) and h >= 2 and w >= 2
        cases.append(((n, cin, h, w, cout, k), t, mode, bool(rng.random() < 0.5), bool(rng.random() < 0.5), pool))
    return cases


@pytest.mark.parametrize("shape,tile,mode,bias,relu,pool", _random_cases(),
                         ids=[f"{s}-T{t}-{m}-b{int(b)}r{int(r)}p{int(p)}" for s, t, m, b, r, p in _random_cases()])
def test_random_layers(shape, tile, mode, bias, relu, pool):
    n, cin, h, w, cout, k = shape
    print(f"[case] random {shape} T={tile} {mode} bias={bias} relu={relu} pool={pool}", flush=True)
    x, wt = small_layer(n, cin, h, w, cout, k, seed=sum(shape) + tile)
    b = make_random_bias(cout, cin, k, seed=5) if bias else None
    plan = fs.Plan(n, cin, h, w, cout, k, tile=tile, mode=mode, bias=bias, relu=relu, pool=pool)
    y = plan.conv2d(_dev(x), plan.transform_weights(_dev(wt)), None if b is None else _dev(b))
    torch.cuda.synchronize()
    ref = oracle.direct_xcorr2d(x, wt, b, relu=relu)
    if pool:
        ref = oracle.maxpool2x2(ref)
    assert rel_l2(y.cpu().numpy(), ref) <= GATE


def test_large_layer_general_kernels():
    """512 x 256 x 56 x 56 -> 256, K = 5, T = 28: 2.15 GB of patch spectra,
    past the 2 GiB the row-band kernels address, so the general forward and
    inverse kernels run at full size; checked on sampled images and channels.
    Inputs are drawn on the device from a seeded generator and the sampled
    images copied to the host for the oracle."""
    n, cin, h, w, cout, k = 512, 256, 56, 56, 256, 5
    g = torch.Generator(device="cuda")
    g.manual_seed(77)
    xd = torch.relu(torch.randn((n, cin, h, w), generator=g, device="cuda"))
    wd = torch.randn((cout, cin, k, k), generator=g, device="cuda") * float(np.sqrt(2.0 / (cin * k * k)))
    plan = fs.Plan(n, cin, h, w, cout, k, tile=28)
    assert plan.info.xspec_bytes >= 2 ** 31
    y = plan.conv2d(xd, plan.transform_weights(wd))
    torch.cuda.synchronize()
    wt = wd.cpu().numpy()
    sel = [3, 97, 200, 255]
    for img in (0, 257, 511):
        xi = xd[img:img + 1].cpu().numpy()
        ref = oracle.direct_xcorr2d(xi, wt[sel])
        got = y[img:img + 1, sel].cpu().numpy()
        assert rel_l2(got, ref) <= GATE, img


SWEEP_CASES = [
    # (n, cin, h, w, cout, k), tile -- 2560 to 4096 forward work items, so
    # that every workgroup runs several (at L = 16 not all the same number:
    # 2560 items, 3 per workgroup, for the forward and the inverse alike)
    ((16, 256, 48, 48, 16, 3), 6),
    ((16, 256, 56, 60, 256, 3), 14),
    ((16, 512, 56, 56, 16, 5), 28),
]


@pytest.mark.parametrize("shape,tile", SWEEP_CASES, ids=[f"{s}-T{t}" for s, t in SWEEP_CASES])
def test_forward_sweep_order(shape, tile, monkeypatch):
    """The row-band forward with its items a grid apart per workgroup
    (FFTSPLIT_FORWARD_SWEEP=1) and in contiguous runs (=0) against the
    oracle; the order changes no arithmetic, so both outputs are identical."""
    n, cin, h, w, cout, k = shape
    print(f"[case] forward sweep order {shape} T={tile}", flush=True)
    x, wt = small_layer(n, cin, h, w, cout, k, seed=111)
    outs = []
    for sweep in ("1", "0"):
        monkeypatch.setenv("FFTSPLIT_FORWARD_SWEEP", sweep)
        plan = fs.Plan(n, cin, h, w, cout, k, tile=tile)
        y = plan.conv2d(_dev(x), plan.transform_weights(_dev(wt)))
        torch.cuda.synchronize()
        outs.append(y.cpu().numpy())
    assert rel_l2(outs[0], oracle.direct_xcorr2d(x, wt)) <= GATE
    assert np.array_equal(outs[0], outs[1])


def test_pooled_inverse_uneven_item_counts():
    """Bias, ReLU and the fused 2x2 max-pool on a layer whose inverse runs
    2560 work items, three per workgroup but not on every workgroup (items a
    grid apart), against the oracle."""
    n, cin, h, w, cout, k, tile = 16, 64, 56, 60, 256, 3, 14
    print(f"[case] pooled inverse, uneven items ({n},{cin},{h},{w},{cout},{k}) T={tile}", flush=True)
    x, wt = small_layer(n, cin, h, w, cout, k, seed=121)
    b = make_random_bias(cout, cin, k, seed=122)
    plan = fs.Plan(n, cin, h, w, cout, k, tile=tile, bias=True, relu=True, pool=True)
    assert plan.info.inverse_band == 1
    y = plan.conv2d(_dev(x), plan.transform_weights(_dev(wt)), _dev(b))
    torch.cuda.synchronize()
    ref = oracle.maxpool2x2(oracle.direct_xcorr2d(x, wt, b, relu=True))
    assert rel_l2(y.cpu().numpy(), ref) <= GATE
