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
    for nt, wg in ((False, 0), (True, 0), (True, 192), (True, 32)):
        nb, ms = dsi.dsi_profile_stream(buf, slice_bytes * slices, slices, nt, 8, sink, workgroups=wg)
        # each slice rounded down to whole 8 KB runs of the launch's waves
        waves = (wg or 256) * 8
        assert slice_bytes - waves * 8192 < nb <= slice_bytes and nb % (waves * 8192) == 0
        rates[nt, wg] = nb / (ms * 1e-3) / 1e9
        print(f"nontemporal={nt} workgroups={wg or 256}: {nb >> 20} MiB per launch, {ms * 1e3:.1f} us, "
              f"{rates[nt, wg]:.0f} GB/s")
        assert 500.0 < rates[nt, wg] < 8000.0     # below the HBM peak: every launch reads HBM
    for bad in (-1, 4097):                         # workgroups outside 0..4096
        with pytest.raises(dsi.DsiError) as ei:
            dsi.dsi_profile_stream(buf, slice_bytes, 1, False, 1, sink, workgroups=bad)
        assert ei.value.status == dsi.DSI_EINVAL
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
