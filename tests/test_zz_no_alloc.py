"""dsi_accept_noalloc, the accept/reject entry point that allocates nothing
(its workspace is a fixed device array): through the C ABI its decisions
equal dsi_accept's on the same inputs, on two calls in a row whose second is
smaller (the array keeps the first call's contents), in sampling and greedy
mode; sizes beyond the array are rejected on the host."""
import numpy as np
import pytest
import torch

from paper_2405_14105_amd import dsi

pytestmark = pytest.mark.gpu


def inputs(rng, B, k, V, dev):
    z = (rng.standard_normal((B * (k + 1), V)) * 1.3).astype(np.float32)
    g = rng.standard_normal((B, k, V)) * 2.0
    q = np.exp(g - g.max(axis=-1, keepdims=True))
    q = (q / q.sum(axis=-1, keepdims=True)).astype(np.float32)
    toks = rng.integers(0, V, size=(B, k + 1)).astype(np.int32)
    u = (rng.integers(0, 1 << 24, size=(B, k + 1)) / float(1 << 24)).astype(np.float32)
    t = lambda a: torch.from_numpy(a).to(dev)
    return t(z), t(toks), t(q), t(u)


def run(fn, stream, B, k, V, z, toks, q, u, mode, dev):
    n = torch.full((B,), -7, dtype=torch.int32, device=dev)
    tok = torch.full((B,), -7, dtype=torch.int32, device=dev)
    fn(stream, B, k, V, z, toks, q if mode == dsi.DSI_SAMPLE else None,
       u if mode == dsi.DSI_SAMPLE else None, n, tok, 1.0, mode)
    torch.cuda.synchronize()
    return n.cpu().numpy(), tok.cpu().numpy()


@pytest.mark.parametrize("mode", [dsi.DSI_SAMPLE, dsi.DSI_GREEDY])
def test_noalloc_accept_equals_accept_on_two_calls(dev, mode):
    stream = torch.cuda.current_stream().cuda_stream
    rng = np.random.default_rng(11)
    # the 64-row maximum over a 128256 vocabulary, then a smaller call
    for B, k, V in ((4, 15, 128256), (2, 3, 32000)):
        args = inputs(rng, B, k, V, dev)
        a = run(dsi.dsi_accept, stream, B, k, V, *args, mode, dev)
        b = run(dsi.dsi_accept_noalloc, stream, B, k, V, *args, mode, dev)
        print(f"B={B} k={k} V={V} mode={mode}: n {b[0].tolist()} token {b[1].tolist()}")
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
        assert ((b[0] >= 0) & (b[0] <= k)).all() and ((b[1] >= 0) & (b[1] < V)).all()


def test_noalloc_accept_rejects_sizes_beyond_its_array(dev):
    stream = torch.cuda.current_stream().cuda_stream
    # 64 rows over a 2^20-entry vocabulary need ~410 KB of workspace; the
    # call is rejected on the host before anything is enqueued, so the small
    # buffers below are never read
    B, k, V = 4, 15, 1 << 20
    z = torch.zeros((1, 16), dtype=torch.float32, device=dev)
    toks = torch.zeros((B, k + 1), dtype=torch.int32, device=dev)
    q = torch.zeros((1, 16), dtype=torch.float32, device=dev)
    u = torch.zeros((B, k + 1), dtype=torch.float32, device=dev)
    n = torch.zeros(B, dtype=torch.int32, device=dev)
    with pytest.raises(dsi.DsiError) as ei:
        dsi.dsi_accept_noalloc(stream, B, k, V, z, toks, q, u, n, n, 1.0, dsi.DSI_SAMPLE)
    assert ei.value.status == dsi.DSI_ECAPACITY
