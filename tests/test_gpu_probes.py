"""The measurement hooks (fftsplit_probe_matrix, fftsplit_probe_stream):
the streaming probe moves exactly the bytes it states, and the matrix probe
of a plan runs its contraction's launch in no less time than the datasheet
peak allows for the contraction's executed operations."""
import pytest

torch = pytest.importorskip("torch")
fs = pytest.importorskip("paper_2003_12621_amd")

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rbytes,wbytes", [(4096, 8192), (8192, 4096), (1 << 20, 1 << 20), (0, 256), (256, 0)])
def test_stream_probe_moves_the_stated_bytes(rbytes, wbytes):
    src = torch.arange(max(rbytes, 16) // 4, dtype=torch.float32, device="cuda") + 1.0
    dst = torch.full((max(wbytes, 16) // 4 + 64,), -7.0, dtype=torch.float32, device="cuda")
    fs.probe_stream(src, dst, rbytes, wbytes)
    torch.cuda.synchronize()
    n = min(rbytes, wbytes) // 4
    assert torch.equal(dst[:n], src[:n])
    assert torch.all(dst[n:wbytes // 4] == 0)
    assert torch.all(dst[wbytes // 4:] == -7.0)        # nothing past write_bytes


def test_matrix_probe_respects_the_peak():
    print("[case] matrix probe, 16x256x56x56 K=5 T=28 launch", flush=True)
    plan = fs.Plan(16, 256, 56, 56, 256, 5, tile=28)
    i = plan.info
    sink = plan.probe_matrix()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    plan.probe_matrix(sink)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) * 1e3
    # executed fp32 matrix operations of the contraction: 3 real products
    # per complex multiply-add (Gauss), 2 flops each, over the padded tile
    flops = 6 * i.bins * i.cout_padded * i.tiles_padded * (-(-plan.cin // 16) * 16)
    assert i.contract_real_products == 3
    ideal_us = flops / 157.3e12 * 1e6
    assert us >= 0.95 * ideal_us, (us, ideal_us)
    assert sink.item() == 0.0


def test_matrix_probe_rejects_a_plan_without_contraction():
    plan = fs.Plan(1, 3, 32, 32, 16, 3, tile=6)
    if not plan.info.fused_channel_sum:
        pytest.skip("this plan runs a contraction")
    with pytest.raises(fs.FftsplitError):
        plan.probe_matrix()
