"""dsi_profile_stream: the streaming read rate the GEMM and attention
roofline figures are compared with (diagnostics, through the C ABI)."""
import pytest

from paper_2405_14105_amd import dsi

pytestmark = pytest.mark.gpu


def test_stream_read_rate_and_argument_checks():
    torch = pytest.importorskip("torch")
    dev = torch.device("cuda:0")
    slice_bytes, slices = 80 << 20, 4          # 320 MiB: more than the Infinity Cache
    buf = torch.ones(slice_bytes * slices, dtype=torch.uint8, device=dev)
    sink = torch.zeros(16, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    rates = {}
    for nt in (False, True):
        nb, ms = dsi.dsi_profile_stream(buf, slice_bytes * slices, slices, nt, 8, sink)
        # each slice rounded down to whole 8 KB runs of the 2048 waves
        assert slice_bytes - 2048 * 8192 < nb <= slice_bytes and nb % (2048 * 8192) == 0
        rates[nt] = nb / (ms * 1e-3) / 1e9
        print(f"nontemporal={nt}: {nb >> 20} MiB per launch, {ms * 1e3:.1f} us, {rates[nt]:.0f} GB/s")
        assert 500.0 < rates[nt] < 8000.0     # below the HBM peak: every launch reads HBM
    with pytest.raises(dsi.DsiError) as ei:    # misaligned buffer
        dsi.dsi_profile_stream(buf.data_ptr() + 4, slice_bytes, 1, False, 1, sink)
    assert ei.value.status == dsi.DSI_EINVAL
    with pytest.raises(dsi.DsiError) as ei:    # slices under 16 MiB
        dsi.dsi_profile_stream(buf, 32 << 20, 4, False, 1, sink)
    assert ei.value.status == dsi.DSI_EINVAL
    with pytest.raises(dsi.DsiError) as ei:    # no sink
        dsi.dsi_profile_stream(buf, slice_bytes, 1, False, 1, None)
    assert ei.value.status == dsi.DSI_EINVAL
    assert int(sink.sum().item()) == 0         # the all-ones data never matches the pattern
