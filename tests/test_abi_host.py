"""Host-side checks of the C ABI: the library loads, exports what the header
declares, and plans validate arguments and report the documented geometry.
No kernel is launched (no GPU needed)."""
import ctypes
import os
import re

import pytest

import paper_2003_12621_amd as fs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fftsplit.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fftsplit_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 12
    handle = ctypes.CDLL(fs.LIB_PATH)
    for name in names:
        assert hasattr(handle, name), name
    # and the binding knows a signature for each of them
    assert set(names) == set(fs._SIGNATURES)


def plan(**kw):
    base = dict(n=1, cin=3, h=32, w=32, cout=16, k=3, tile=6)
    base.update(kw)
    return fs.Plan(arch="gfx950:sramecc+:xnack-", **base)


def status_of(**kw):
    try:
        plan(**kw)
    except fs.FftsplitError as e:
        return e.status
    return fs.SUCCESS


def test_first_config_geometry():
    p = plan()
    i = p.info
    assert (i.tile, i.nfft, i.tiles_h, i.tiles_w, i.tiles) == (6, 8, 6, 6, 36)
    assert i.bins == 8 * 8 // 2
    assert i.tiles_padded % 64 == 0 and i.tiles_padded >= 36
    assert i.cout_padded >= 16
    assert i.wspec_bytes == 8 * i.bins * 3 * i.cout_padded
    assert i.xspec_bytes == 8 * i.bins * 16 * i.tiles_padded   # channels in blocks of 16
    assert i.yspec_bytes == 8 * i.bins * i.cout_padded * i.tiles_padded
    assert i.yspec_offset >= i.xspec_offset + i.xspec_bytes
    assert i.workspace_bytes >= i.yspec_offset + i.yspec_bytes
    assert i.spec_group == 64 and i.tiles_padded % i.spec_group == 0


@pytest.mark.parametrize("t,group", [(6, 64), (14, 32), (30, 16)])
def test_output_spectra_group(t, group):
    """The inverse's unit of work, G patches, by FFT size 8 / 16 / 32."""
    i = plan(h=64, w=64, tile=t).info
    assert i.spec_group == group and i.tiles_padded % group == 0


@pytest.mark.parametrize("h,w,t,k", [(56, 56, 28, 5), (56, 56, 12, 5), (224, 224, 30, 3), (224, 224, 6, 3),
                                     (112, 112, 14, 3), (7, 9, 6, 3), (5, 5, 8, 1)])
def test_tile_grid_and_fft_size(h, w, t, k):
    p = plan(n=2, cin=4, h=h, w=w, cout=8, k=k, tile=t)
    assert p.info.nfft == t + k - 1
    assert p.info.tiles_h == -(-h // t) and p.info.tiles_w == -(-w // t)
    assert p.info.tiles == 2 * p.info.tiles_h * p.info.tiles_w


def test_status_codes():
    assert status_of() == fs.SUCCESS
    assert status_of(k=4, tile=5) == fs.ERROR_NOT_SUPPORTED          # even kernel
    assert status_of(tile=7) == fs.ERROR_NOT_SUPPORTED               # L = 9
    assert status_of(n=0) == fs.ERROR_INVALID_VALUE
    assert status_of(cin=-1) == fs.ERROR_INVALID_VALUE
    assert status_of(tile=-2) == fs.ERROR_INVALID_VALUE
    assert status_of(stride=2) == fs.ERROR_NOT_SUPPORTED
    assert status_of(pad=0) == fs.ERROR_NOT_SUPPORTED
    assert status_of(k=33, tile=0) == fs.ERROR_NOT_SUPPORTED
    assert status_of(k=5, tile=4, mode="oaa") == fs.SUCCESS          # T = K - 1
    assert status_of(k=7, tile=2, mode="oaa") == fs.ERROR_NOT_SUPPORTED  # T < K - 1
    assert status_of(cin=70000, tile=6) == fs.ERROR_NOT_SUPPORTED


def test_wrong_architecture_is_rejected():
    with pytest.raises(fs.FftsplitError) as e:
        fs.Plan(n=1, cin=3, h=32, w=32, cout=16, k=3, tile=6, arch="gfx942:sramecc+:xnack-")
    assert e.value.status == fs.ERROR_ARCH
    assert "gfx942" in str(e.value)


def test_status_strings_and_last_error():
    for code in range(6):
        assert fs.status_string(code)
    assert fs.status_string(99) == "unknown status"
    status_of(tile=7)
    assert "8, 16 or 32" in fs.last_error()
    plan()
    assert fs.last_error() == ""


def test_unknown_flags_rejected():
    prob = fs.problem(1, 3, 32, 32, 16, 3, 6)
    prob.flags = 64
    h = ctypes.c_void_p()
    st = fs.lib().fftsplit_plan_for_arch(ctypes.byref(prob), b"gfx950", ctypes.byref(h))
    assert st == fs.ERROR_INVALID_VALUE


def test_null_arguments():
    h = ctypes.c_void_p()
    L = fs.lib()
    assert L.fftsplit_plan_for_arch(None, b"gfx950", ctypes.byref(h)) == fs.ERROR_INVALID_VALUE
    prob = fs.problem(1, 3, 32, 32, 16, 3, 6)
    assert L.fftsplit_plan_for_arch(ctypes.byref(prob), None, ctypes.byref(h)) == fs.ERROR_INVALID_VALUE
    assert L.fftsplit_plan_info(None, ctypes.byref(fs.PlanInfo())) == fs.ERROR_INVALID_VALUE
    L.fftsplit_plan_destroy(None)


def test_arch_only_plan_cannot_launch():
    p = plan()
    L = fs.lib()
    fake = ctypes.c_void_p(1 << 20)
    st = L.fftsplit_conv2d(p._h, fake, fake, None, fake, fake, 1 << 30, None)
    assert st == fs.ERROR_INVALID_VALUE
    assert "architecture name only" in fs.last_error()
    assert L.fftsplit_forward(p._h, fake, fake, 1 << 30, None) == fs.ERROR_INVALID_VALUE
    assert L.fftsplit_direct_conv2d(p._h, fake, fake, None, fake, None) == fs.ERROR_INVALID_VALUE
    assert L.fftsplit_direct_transform_weights(p._h, fake, fake, None) == fs.ERROR_INVALID_VALUE
    assert L.fftsplit_probe_matrix(p._h, fake, None) == fs.ERROR_INVALID_VALUE


def test_auto_tile_choice_and_env_override(monkeypatch):
    monkeypatch.delenv("FFTSPLIT_TILE", raising=False)
    p = plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=0)
    assert p.info.nfft in (8, 16, 32) and p.info.tile == p.info.nfft - 4
    monkeypatch.setenv("FFTSPLIT_TILE", "12")
    p = plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=0)
    assert p.info.tile == 12
    # an explicit tile wins over the environment
    p = plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28)
    assert p.info.tile == 28
    monkeypatch.setenv("FFTSPLIT_TILE", "abc")
    assert status_of(tile=0) == fs.ERROR_INVALID_VALUE


def test_bin_order_matches_header():
    from spectra_layout import stored_coords, real_pairs
    for L in (8, 16, 32):
        coords = fs.bin_coords(L)
        assert len(coords) == L * L // 2
        assert coords[:-2] == stored_coords(L) and coords[-2:] == real_pairs(L)
        stored = set(coords[:-2]) | {b for pair in coords[-2:] for b in pair}
        assert len(stored) == L * L // 2 + 2
        # the packed slots hold exactly the real bins: both indices in {0, L/2}
        assert all(k in (0, L // 2) for pair in coords[-2:] for b in pair for k in b)
        # every (k1, k2) with k2 in [0, L/2] is stored or is the conjugate of a stored bin
        for k1 in range(L):
            for k2 in range(L // 2 + 1):
                mirror = ((-k1) % L, (-k2) % L)
                assert (k1, k2) in stored or mirror in stored


@pytest.mark.parametrize("L", [5, 9, 13])
def test_odd_bin_order(L):
    """The OaAConv sizes: (L*L+1)/2 complex bins, every bin of the real
    transform stored once or as the conjugate of a stored one."""
    from spectra_layout import stored_coords
    coords = fs.bin_coords(L)
    assert coords == stored_coords(L)
    assert len(coords) == (L * L + 1) // 2 == len(set(coords))
    for k1 in range(L):
        for k2 in range(L):
            mirror = ((-k1) % L, (-k2) % L)
            assert ((k1, k2) in coords) != (mirror in coords) or (k1, k2) == mirror == (0, 0)


@pytest.mark.parametrize("k", [3, 5, 7])
def test_oaaconv_plan(k):
    """Overlap-add with tile = k gives the OaAConv transform size 2k - 1."""
    p = plan(n=2, cin=8, h=30, w=31, cout=8, k=k, tile=k, mode="oaa")
    i = p.info
    L = 2 * k - 1
    assert (i.tile, i.nfft, i.bins) == (k, L, (L * L + 1) // 2)
    assert (i.tiles_h, i.tiles_w) == (-(-30 // k), -(-31 // k))
    assert i.aux_bytes == 4 * 8 * i.tiles_padded * L * L
    # odd sizes exist only for that configuration
    assert status_of(n=2, cin=8, h=30, w=31, cout=8, k=k, tile=k) == fs.ERROR_NOT_SUPPORTED
    assert status_of(n=2, cin=8, h=30, w=31, cout=8, k=k, tile=k + 2, mode="oaa") == fs.ERROR_NOT_SUPPORTED


def test_spectra_layout_helpers_roundtrip():
    import numpy as np
    from spectra_layout import full_to_stored, stored_to_full, rel_l2
    rng = np.random.default_rng(3)
    for L in (8, 16, 32, 5, 9, 13):
        a = rng.standard_normal((2, 3, L, L))
        full = np.fft.fft2(a)
        st = full_to_stored(full)
        assert st.shape == ((L * L + 1) // 2, 2, 3)
        np.testing.assert_allclose(stored_to_full(st, L), full, rtol=0, atol=1e-12)
    # the error measure sees imaginary parts
    assert rel_l2(np.array([1 + 1j]), np.array([1 + 0j])) == 1.0


@pytest.mark.parametrize("cin,tile,fused", [(3, 6, 1), (4, 6, 1), (5, 6, 0), (3, 14, 1), (4, 14, 0), (3, 30, 0)])
def test_fused_channel_sum_choice(cin, tile, fused):
    """Tiny-Cin layers sum their channels in the inverse (registers allow 4
    at L = 8, 3 at L = 16, none at L = 32); overlap-add never does."""
    assert plan(n=2, cin=cin, h=56, w=56, cout=16, k=3, tile=tile).info.fused_channel_sum == fused
    assert plan(n=2, cin=cin, h=56, w=56, cout=16, k=3, tile=tile, mode="oaa").info.fused_channel_sum == 0


def test_fused_channel_sum_env_off(monkeypatch):
    monkeypatch.setenv("FFTSPLIT_FUSE_CIN", "0")
    assert plan(n=2, cin=3, h=56, w=56, cout=16, k=3, tile=6).info.fused_channel_sum == 0


def test_maxpool_flag():
    """FFTSPLIT_MAXPOOL halves the output (floor); it needs a 2 x 2 image."""
    p = plan(n=2, cin=8, h=28, w=28, cout=8, k=3, tile=14, pool=True)
    assert p.out_shape == (2, 8, 14, 14)
    assert plan(n=1, cin=2, h=27, w=29, cout=3, k=3, tile=14, pool=True).out_shape == (1, 3, 13, 14)
    assert status_of(n=1, cin=2, h=1, w=8, cout=3, k=3, tile=6, pool=True) == fs.ERROR_INVALID_VALUE
    # a plan that cannot pool inside the inverse stages the unpooled output
    # in its workspace: odd height needs n*cout*h*w*4 more bytes
    a = plan(n=1, cin=2, h=28, w=28, cout=3, k=3, tile=14).info.workspace_bytes
    b = plan(n=1, cin=2, h=27, w=28, cout=3, k=3, tile=14, pool=True).info.workspace_bytes
    assert b >= a + 1 * 3 * 27 * 28 * 4 - 4096


def test_small_patch_granule():
    """Few patches and output channels in 128s: patches padded to 32 and the
    contraction in 128 x 32 tiles; otherwise 64 and 64 x 64."""
    i = plan(n=32, cin=512, h=14, w=14, cout=512, k=3, tile=14).info
    assert (i.tiles, i.tiles_padded, i.contract_tile_m, i.contract_tile_n) == (32, 32, 128, 32)
    i = plan(n=32, cin=512, h=14, w=14, cout=64, k=3, tile=14).info      # channels not in 128s
    assert (i.tiles_padded, i.contract_tile_m, i.contract_tile_n) == (64, 64, 64)
    i = plan(n=8, cin=64, h=14, w=14, cout=128, k=3, tile=6).info        # L = 8 groups 64 patches
    assert i.tiles_padded % 64 == 0 and i.contract_tile_n == 64
    i = plan(n=16, cin=8, h=56, w=56, cout=256, k=5, tile=28).info       # 64 patches: unchanged
    assert (i.tiles_padded, i.contract_tile_m, i.contract_tile_n) == (64, 64, 64)


def test_size_limits():
    """Largest problems the 32-bit offsets allow are accepted; beyond them
    NOT_SUPPORTED (arch-only plans: nothing is allocated)."""
    # 2.15 GB of patch spectra: accepted (above 2 GiB the general kernels run)
    assert status_of(n=512, cin=256, h=56, w=56, cout=256, k=5, tile=28) == fs.SUCCESS
    # patch spectra above 4 GiB
    assert status_of(n=1100, cin=256, h=56, w=56, cout=256, k=5, tile=28) == fs.ERROR_NOT_SUPPORTED
    # input tensor above 2^29 elements
    assert status_of(n=700, cin=256, h=56, w=56, cout=16, k=5, tile=28) == fs.ERROR_NOT_SUPPORTED
    # image plane above 2^31 pixels
    assert status_of(n=1, cin=1, h=50000, w=50000, cout=1, k=3, tile=6) == fs.ERROR_NOT_SUPPORTED


def test_contraction_prefetch_choice(monkeypatch):
    """The 3-product tiles with 16-channel stages (64x64, 128x32, 128x64,
    64x128) load two input-channel stages ahead through LDS; other tiles
    one, through registers; the environment variable overrides within what
    the tile has."""
    monkeypatch.delenv("FFTSPLIT_CONTRACT_PREFETCH", raising=False)
    monkeypatch.delenv("FFTSPLIT_CONTRACT_TILE", raising=False)
    assert plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28).info.contract_prefetch == 2
    assert plan(n=32, cin=512, h=14, w=14, cout=512, k=3, tile=14).info.contract_prefetch == 2   # 128 x 32
    monkeypatch.setenv("FFTSPLIT_CONTRACT_TILE", "g4:64x64x16")
    assert plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28).info.contract_prefetch == 1
    monkeypatch.setenv("FFTSPLIT_CONTRACT_TILE", "g3:128x64x16")
    assert plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28).info.contract_prefetch == 2
    monkeypatch.setenv("FFTSPLIT_CONTRACT_TILE", "g4:64x64x32")
    assert plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28).info.contract_prefetch == 1
    monkeypatch.delenv("FFTSPLIT_CONTRACT_TILE")
    monkeypatch.setenv("FFTSPLIT_CONTRACT_PREFETCH", "1")
    assert plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28).info.contract_prefetch == 1
    monkeypatch.setenv("FFTSPLIT_CONTRACT_PREFETCH", "3")
    assert plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28).info.contract_prefetch == 3
    assert plan(n=32, cin=512, h=14, w=14, cout=512, k=3, tile=14).info.contract_prefetch == 2


def test_contraction_stage_choice(monkeypatch):
    """8-channel stages three ahead where a layer has at most 128 input
    channels and at least 8192 64 x 64 workgroups (the VGG-16 layers at 224^2
    and 112^2); 16-channel stages two ahead elsewhere; a tile override
    restores the two-ahead default, and the prefetch override still applies."""
    monkeypatch.delenv("FFTSPLIT_CONTRACT_PREFETCH", raising=False)
    monkeypatch.delenv("FFTSPLIT_CONTRACT_TILE", raising=False)
    def choice(**kw):
        i = plan(**kw).info
        return (i.contract_tile_m, i.contract_tile_n, i.contract_stage_k, i.contract_prefetch)
    assert choice(n=32, cin=64, h=224, w=224, cout=64, k=3, tile=14) == (64, 64, 8, 3)
    assert choice(n=32, cin=64, h=112, w=112, cout=128, k=3, tile=14) == (64, 64, 8, 3)
    assert choice(n=32, cin=128, h=112, w=112, cout=128, k=3, tile=14) == (64, 64, 8, 3)
    assert choice(n=32, cin=128, h=56, w=56, cout=256, k=3, tile=14) == (64, 64, 16, 2)   # 4096 workgroups
    assert choice(n=32, cin=256, h=56, w=56, cout=256, k=3, tile=14) == (64, 64, 16, 2)
    assert choice(n=1, cin=64, h=224, w=224, cout=64, k=3, tile=14) == (64, 64, 16, 2)
    assert choice(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28) == (64, 64, 16, 2)
    monkeypatch.setenv("FFTSPLIT_CONTRACT_TILE", "g3:64x64x16")
    assert choice(n=32, cin=64, h=224, w=224, cout=64, k=3, tile=14) == (64, 64, 16, 2)
    monkeypatch.setenv("FFTSPLIT_CONTRACT_TILE", "g3:64x64x8")
    assert choice(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28) == (64, 64, 8, 2)
    monkeypatch.setenv("FFTSPLIT_CONTRACT_PREFETCH", "3")
    assert choice(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28) == (64, 64, 8, 3)
    monkeypatch.delenv("FFTSPLIT_CONTRACT_TILE")
    monkeypatch.setenv("FFTSPLIT_CONTRACT_PREFETCH", "1")
    assert choice(n=32, cin=64, h=224, w=224, cout=64, k=3, tile=14) == (64, 64, 8, 1)


@pytest.mark.parametrize("value", ["0x0x0", "-64x64x16", "g3:64x64x32", "g3:256x64x16", "64x64x16junk",
                                   "64x64", "g5:64x64x16", "96x64x16"])
def test_contraction_tile_override_is_validated(value, monkeypatch):
    """FFTSPLIT_CONTRACT_TILE is checked at plan time against the kernel
    variants the contraction has: anything else is INVALID_VALUE, so that a
    later conv2d cannot fail after its forward stage has been enqueued."""
    monkeypatch.setenv("FFTSPLIT_CONTRACT_TILE", value)
    assert status_of(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28) == fs.ERROR_INVALID_VALUE
    assert "FFTSPLIT_CONTRACT_TILE" in fs.last_error()


def test_probe_argument_checks():
    """The measurement hooks reject bad arguments before touching a device."""
    L = fs.lib()
    a, b = ctypes.c_void_p(1 << 20), ctypes.c_void_p(1 << 24)
    assert L.fftsplit_probe_matrix(None, a, None) == fs.ERROR_INVALID_VALUE
    assert L.fftsplit_probe_matrix(plan()._h, None, None) == fs.ERROR_INVALID_VALUE
    assert L.fftsplit_probe_stream(None, b, 16, 16, None) == fs.ERROR_INVALID_VALUE         # NULL source
    assert L.fftsplit_probe_stream(a, b, 24, 16, None) == fs.ERROR_INVALID_VALUE            # size not x16
    assert L.fftsplit_probe_stream(ctypes.c_void_p((1 << 20) + 8), b, 16, 16, None) == fs.ERROR_INVALID_VALUE
    assert L.fftsplit_probe_stream(a, ctypes.c_void_p((1 << 20) + 16), 64, 64, None) == fs.ERROR_INVALID_VALUE  # overlap
    assert L.fftsplit_probe_stream(None, None, 0, 0, None) == fs.SUCCESS                  # nothing to do


@pytest.mark.skipif(not os.path.isdir("/opt/rocm/include"), reason="no HIP headers")
def test_struct_layouts_match_header(tmp_path):
    """The binding's ctypes structures have the header's layout: a C program
    built here against include/fftsplit.h prints sizeof and every field's
    offsetof, which must equal ctypes' (a mismatch would garble fields
    silently)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = {"fftsplit_plan_info_t": fs.PlanInfo, "fftsplit_problem_t": fs.Problem}
    lines = []
    for cname, cls in structs.items():
        lines.append(f'printf("%zu\\n", sizeof({cname}));')
        lines += [f'printf("%zu\\n", offsetof({cname}, {f}));' for f, _ in cls._fields_]
    src = tmp_path / "layout.c"
    src.write_text("#include <stddef.h>\n#include <stdio.h>\n#include \"fftsplit.h\"\nint main(void) {\n"
                   + "\n".join(lines) + "\nreturn 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-x", "c", "-std=c11", "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                    "-D__HIP_PLATFORM_AMD__", str(src), "-o", str(exe)], check=True, capture_output=True)
    got = [int(v) for v in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()]
    want = []
    for cls in structs.values():
        want.append(ctypes.sizeof(cls))
        want += [getattr(cls, f).offset for f, _ in cls._fields_]
    assert got == want


def test_transform_variant_choice(monkeypatch):
    """Row-band transforms where the width allows them; the forward's items
    a grid apart only where input and patch spectra exceed 256 MB (the
    VGG-16 layer 2 at batch 32: 411 + 537 MB), contiguous runs otherwise;
    the environment forces either.  The input read non-temporally only
    where it alone exceeds 256 MB (layer 2's 411 MB; not layer 4's 205 MB,
    whose items are swept too)."""
    big = plan(n=32, cin=64, h=224, w=224, cout=64, k=3, tile=14).info
    assert (big.forward_band, big.forward_sweep, big.inverse_band) == (1, 1, 1)
    k5 = plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28).info
    assert (k5.forward_band, k5.forward_sweep, k5.inverse_band) == (1, 0, 1)
    narrow = plan(n=32, cin=512, h=14, w=14, cout=512, k=3, tile=14).info   # width not a multiple of 4
    assert (narrow.forward_band, narrow.forward_sweep, narrow.inverse_band) == (0, 0, 0)
    assert (big.forward_stream, k5.forward_stream, narrow.forward_stream) == (1, 0, 0)
    l4 = plan(n=32, cin=128, h=112, w=112, cout=128, k=3, tile=14).info
    assert (l4.forward_sweep, l4.forward_stream) == (1, 0)
    monkeypatch.setenv("FFTSPLIT_FORWARD_SWEEP", "1")
    assert plan(n=16, cin=256, h=56, w=56, cout=256, k=5, tile=28).info.forward_sweep == 1
    monkeypatch.setenv("FFTSPLIT_FORWARD_SWEEP", "0")
    assert plan(n=32, cin=64, h=224, w=224, cout=64, k=3, tile=14).info.forward_sweep == 0
