"""Dead cache rows never reach the logits (the KV-state pin; Section 3.1,
"KV cache": rows of terminated threads are dead after a rollback).

After a verification is rolled back, dsi_kv_poison fills the window's dead
rows [length, capacity) of every layer with NaN.  The same verification (or
token tree) run again must give bit-identical, finite logits and the same
decisions: no kernel reads a row past the window's rows into a result, and
the masked keys of a partial 32-key step (probability 0) cannot turn a NaN
value row into a NaN output.  Covers bf16 and fp32 caches, one and several
key chunks, 4-wave and pipelined attention plans (with nontemporal key and
value loads), and the ring O projection.
"""
import numpy as np
import pytest

import dsi_synth as S
from paper_2405_14105_amd import dsi

from gpu_rig import Rig

pytestmark = pytest.mark.gpu

SEED = 0


# cap: cache capacity (None: the window plus slack).  gqa_hd64 at 1600:
# 256-key chunks over a 1200-key prefix; at 11300: 4-wave workgroups and
# 128-key chunks; many_kv at 6000 with a 2000-key prefix: 4-wave 128-key
# chunks for the 4-row window, two 1280-key chunks of five steps per wave
# for the 9-node tree; mha_hd128 at 70000: 768-key chunks of three steps
# per wave with nontemporal key and value loads (one query tile);
# o_ring_hd128 at 8000 with k 10: three query tiles in one 1024-key chunk
# of four steps per wave.
@pytest.mark.parametrize("name,L,k,cap", [("ragged_bf16", 45, 5, None), ("ragged_f32", 37, 4, None),
                                          ("gqa_hd64", 1200, 3, 1600), ("gqa_hd64", 1200, 3, 11300),
                                          ("many_kv", 2000, 3, 6000), ("mha_hd128", 2000, 5, 70000),
                                          ("o_ring_hd128", 1000, 10, 8000),
                                          ("o_ring_hd128", 300, 10, None)])
def test_poisoned_dead_rows_do_not_reach_logits(name, L, k, cap):
    shape = S.SHAPES[name]
    cap = cap or L + 2 * (k + 1) + 40
    prefix = S.prefix_tokens(shape, SEED, 0, L)
    wi = S.window_inputs(shape, SEED, 1, k)
    rng = np.random.default_rng(5)
    toks = rng.integers(0, shape.vocab, size=9).astype(np.int32)[None]
    par = np.array([[-1, 0, 0, 1, 1, 2, 3, 5, 5]], np.int32)
    with Rig(shape, SEED, 1, cap) as rig:
        rig.prefill(0, prefix)
        a = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=True)
        dsi.dsi_kv_rollback(rig.kv, 0, L)
        ta = rig.verify_tree(0, toks, par, commit=False)   # on the same prefix
        dsi.dsi_kv_poison(rig.kv, 0)
        for layer in (0, shape.n_layers - 1):
            for x in rig.export_kv(0, layer, cap):   # [position, head, dim]
                assert np.isfinite(x[:L]).all()
                assert np.isnan(x[L:]).all()
        b = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=True)
        assert np.isfinite(b["logits"]).all()
        for key in a:
            assert np.array_equal(a[key], b[key]), key
        assert rig.length(0) == L + int(b["n"][0]) + 1
        dsi.dsi_kv_rollback(rig.kv, 0, L)
        dsi.dsi_kv_poison(rig.kv, 0)
        tb = rig.verify_tree(0, toks, par, commit=False)
        assert np.isfinite(tb["logits"]).all()
        for key in ta:
            assert np.array_equal(ta[key], tb[key]), key
