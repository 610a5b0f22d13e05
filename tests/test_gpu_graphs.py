"""Graph replay of dsi_verify against eager launches.

A model created on a non-null stream captures each verification step into a
HIP graph the first time it sees a combination of arguments and replays it
afterwards.  Two models with the same weights -- one with graphs disabled
(DSI_GRAPHS=0 when it is created) -- run the same sequence of verifications
with the same persistent device buffers (so later calls are replays), with
fresh inputs copied in, commits and rollbacks between the calls; every call
must give bit-identical logits, decisions and cache lengths.
"""
import os

import numpy as np
import pytest
import torch

import dsi_synth as S
from paper_2405_14105_amd import dsi

from gpu_rig import Rig

pytestmark = pytest.mark.gpu

SEED = 0


def make_rig(shape, graphs: bool, n_windows, max_len):
    old = os.environ.get("DSI_GRAPHS")
    os.environ["DSI_GRAPHS"] = "1" if graphs else "0"
    try:
        return Rig(shape, SEED, n_windows, max_len)
    finally:
        if old is None:
            del os.environ["DSI_GRAPHS"]
        else:
            os.environ["DSI_GRAPHS"] = old


class Buffers:
    """Persistent device buffers for one (B, k) verification shape."""

    def __init__(self, dev, B, k, V, M):
        self.tok = torch.zeros((B, k + 1), dtype=torch.int32, device=dev)
        self.q = torch.zeros((B, k, V), dtype=torch.float32, device=dev)
        self.u = torch.zeros((B, k + 1), dtype=torch.float32, device=dev)
        self.n = torch.zeros(B, dtype=torch.int32, device=dev)
        self.t = torch.zeros(B, dtype=torch.int32, device=dev)
        self.z = torch.zeros((M, V), dtype=torch.float32, device=dev)

    def load(self, wi):
        self.tok.copy_(torch.from_numpy(wi["tokens"]))
        self.q.copy_(torch.from_numpy(wi["q"]))
        self.u.copy_(torch.from_numpy(wi["u"]))


def run(rig, buf, window0, B, k, mode, commit):
    dsi.dsi_verify(rig.model, rig.kv, window0, B, k, buf.tok, buf.q, buf.u, buf.n, buf.t,
                   1.0, mode, commit, buf.z)
    torch.cuda.synchronize()
    return buf.z.cpu().numpy().copy(), buf.n.cpu().numpy().copy(), buf.t.cpu().numpy().copy()


# lens, cache capacity: one key chunk; or 256-key chunks with the chunk
# launch and the combine inside the graph, the longest window 1010 keys so
# that commits take its key range past 1024 (a fifth chunk: a new plan and
# a new graph) between replays
# ... and o_ring_hd128 with 16-row windows: the three windows together run
# the three-row-tile kernels (48 rows), one window alone the one-row-tile ones
@pytest.mark.parametrize("name,lens,cap,kbig", [("ragged_bf16", [17, 40, 29], 200, 4),
                                                ("gqa_hd64", [17, 40, 29], 200, 4),
                                                ("gqa_hd64", [300, 1010, 250], 1600, 4),
                                                ("o_ring_hd128", [40, 70, 25], 300, 15)])
def test_graph_replays_match_eager(name, lens, cap, kbig):
    shape = S.SHAPES[name]
    B = len(lens)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        eager = make_rig(shape, False, B, cap)
        graph = make_rig(shape, True, B, cap)
        try:
            for b in range(B):
                p = S.prefix_tokens(shape, SEED, b, lens[b])
                eager.prefill(b, p)
                graph.prefill(b, p)
            bufs = {}
            schedule = []
            # same shapes repeatedly (replays), interleaved with other shapes,
            # greedy mode, single windows, commits and rollbacks
            for it in range(14):
                k = (kbig, kbig, kbig, 2, kbig, kbig, 2, kbig, kbig, kbig, kbig, 2, kbig, kbig)[it]
                mode = dsi.DSI_GREEDY if it in (5, 9) else dsi.DSI_SAMPLE
                w0, nb = (1, 1) if it in (6, 11) else (0, B)
                schedule.append((k, mode, w0, nb, it % 3 != 2))
            for it, (k, mode, w0, nb, commit) in enumerate(schedule):
                wi = S.window_inputs(shape, SEED + 100 + it, nb, k)
                key = (k, nb)
                if key not in bufs:
                    bufs[key] = (Buffers(eager.dev, nb, k, shape.vocab, nb * (k + 1)),
                                 Buffers(graph.dev, nb, k, shape.vocab, nb * (k + 1)))
                be, bg = bufs[key]
                be.load(wi)
                bg.load(wi)
                ze, ne, te = run(eager, be, w0, nb, k, mode, commit)
                zg, ng, tg = run(graph, bg, w0, nb, k, mode, commit)
                assert np.array_equal(ze, zg), it
                assert np.array_equal(ne, ng) and np.array_equal(te, tg), it
                for b in range(B):
                    assert eager.length(b) == graph.length(b), (it, b)
                if it % 4 == 3:
                    for b in range(B):
                        dsi.dsi_kv_rollback(eager.kv, b, lens[b])
                        dsi.dsi_kv_rollback(graph.kv, b, lens[b])
        finally:
            eager.close()
            graph.close()


def test_tree_graph_replays_match_eager():
    """dsi_verify_tree through replayed graphs (same buffers, fresh tokens and
    parent arrays copied in, commits with KV compaction and rollbacks in
    between) against eager launches, bit-identical including the cache."""
    shape = S.SHAPES["ragged_bf16"]
    B, R, lens = 2, 7, [23, 31]
    rng = np.random.default_rng(4)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        eager = make_rig(shape, False, B, 120)
        graph = make_rig(shape, True, B, 120)
        try:
            for b in range(B):
                p = S.prefix_tokens(shape, SEED, b, lens[b])
                eager.prefill(b, p)
                graph.prefill(b, p)
            bufs = []
            for rig in (eager, graph):
                d = rig.dev
                bufs.append({"tok": torch.zeros((B, R), dtype=torch.int32, device=d),
                             "par": torch.zeros((B, R), dtype=torch.int32, device=d),
                             "path": torch.zeros((B, R), dtype=torch.int32, device=d),
                             "n": torch.zeros(B, dtype=torch.int32, device=d),
                             "t": torch.zeros(B, dtype=torch.int32, device=d),
                             "z": torch.zeros((B * R, shape.vocab), dtype=torch.float32, device=d)})
            for it in range(10):
                toks = rng.integers(0, shape.vocab, (B, R)).astype(np.int32)
                par = np.full((B, R), -1, np.int32)
                for b in range(B):
                    for i in range(1, R):
                        par[b, i] = rng.integers(0, i)
                commit = it % 3 != 1
                outs = []
                for rig, bf in zip((eager, graph), bufs):
                    bf["tok"].copy_(torch.from_numpy(toks))
                    bf["par"].copy_(torch.from_numpy(par))
                    dsi.dsi_verify_tree(rig.model, rig.kv, 0, B, R, bf["tok"], bf["par"], bf["path"],
                                        bf["n"], bf["t"], commit, bf["z"])
                    torch.cuda.synchronize()
                    outs.append({k: v.cpu().numpy().copy() for k, v in bf.items() if k in ("path", "n", "t", "z")})
                for key in ("z", "path", "n", "t"):
                    assert np.array_equal(outs[0][key], outs[1][key]), (it, key)
                for b in range(B):
                    Lb = eager.length(b)
                    assert Lb == graph.length(b), (it, b)
                    for layer in (0, shape.n_layers - 1):
                        ke, ve = eager.export_kv(b, layer, Lb)
                        kg, vg = graph.export_kv(b, layer, Lb)
                        assert np.array_equal(ke, kg) and np.array_equal(ve, vg), (it, b, layer)
                if it % 4 == 3:
                    for b in range(B):
                        dsi.dsi_kv_rollback(eager.kv, b, lens[b])
                        dsi.dsi_kv_rollback(graph.kv, b, lens[b])
        finally:
            eager.close()
            graph.close()
