"""End-to-end parity over many seeds (weights, prefixes, drafts, q, u all
re-drawn per seed) on the fp32 tiny model: 32 seeds x 2 windows, sampling
and greedy verification of the same windows.

Gates per window: logits within 1e-4 of the oracle; the GPU's decision on
its own logits equals the oracle's on the same logits (split check), and
the oracle's on its own logits (end to end) unless a flag margin applies.
The share of windows compared without a flag is reported and must stay
high: a real disagreement shows as a failed comparison, not as a flag."""
import numpy as np
import pytest

import dsi_synth as S
from paper_2405_14105_amd import dsi

from gpu_rig import Rig
from parity import TOL, e2e_check, oracle_logits, split_check

pytestmark = pytest.mark.gpu


def test_tiny_32_seeds():
    shape = S.SHAPES["tiny"]
    L, k, B = 64, 5, 2
    compared = {"sample": 0, "greedy": 0}
    total = 0
    worst = 0.0
    for seed in range(32):
        with Rig(shape, seed, B, L + 2 * (k + 1) + 4) as rig:
            prefixes = [S.prefix_tokens(shape, seed, b, L) for b in range(B)]
            for b in range(B):
                rig.prefill(b, prefixes[b])
            wi = S.window_inputs(shape, seed, B, k)
            out = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=False)
            g = rig.verify(0, wi["tokens"], mode=dsi.DSI_GREEDY, commit=False)
        z = out["logits"].reshape(B, k + 1, -1)
        assert np.array_equal(g["logits"], out["logits"])
        for b in range(B):
            total += 1
            zo = oracle_logits(shape, prefixes[b], wi["tokens"][b], seed=seed)
            delta = float(np.abs(z[b] - zo).max())
            worst = max(worst, delta)
            assert delta <= TOL["f32"], (seed, b, delta)
            toks, q, u = wi["tokens"][b], wi["q"][b], wi["u"][b]
            split_check(z[b], toks, q, u, out["n"][b], out["token"][b])
            if e2e_check(zo, delta, toks, q, u, out["n"][b], out["token"][b]) is not None:
                compared["sample"] += 1
            split_check(z[b], toks, None, None, g["n"][b], g["token"][b], mode="greedy")
            if e2e_check(zo, delta, toks, None, None, g["n"][b], g["token"][b], mode="greedy") is not None:
                compared["greedy"] += 1
    print(f"{total} windows over 32 seeds: max|dz| = {worst:.3g}; compared end to end without a flag: "
          f"sample {compared['sample']}/{total}, greedy {compared['greedy']}/{total}")
    assert compared["sample"] >= 0.9 * total and compared["greedy"] >= 0.9 * total
