"""Write the fp64 oracle's window logits at the full 8B workload sizes.

Speculative inference hands the target the k+1 prompts x'_{<=i} as one batch
and reads k+1 logit rows back (Section 2, "Speculative Inference"); those rows
are what the GPU verification step computes.  At 32 layers over a 2059-token
sequence the oracle needs minutes, so its rows are computed once here and
stored; the GPU test (tests/test_gpu_endtoend8b.py) compares its own logits
with them element by element and checks the accept/reject decisions taken on
them.

This script calls only `oracle/` (the fp64 decoder: embedding, decoder layers,
final norm and LM head) and `dsi_synth` (the seeded weights and inputs).
Every layer runs over the whole sequence prefix + window at once, with the
cached K/V rounded to bf16 where the cache is bf16, as the oracle defines it.

    python tests/golden/make_fullsize_logits.py            # all cases
    python tests/golden/make_fullsize_logits.py l2048      # one case

Output: tests/golden/<case>_logits.npz with `logits` (float32 [k+1, V], the
fp64 values rounded to fp32), `tokens`, `prefix_len`, `seed`, `window`.
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import dsi_synth as S                                   # noqa: E402
from oracle.model import embed64, head64, layer64       # noqa: E402

SEED = 0
# (case name, workload, window index inside the workload's batch)
CASES = {
    "llama8b_L2048_k10_w0": ("llama8b_L2048_k10", 0),
    "llama8b_x7_L1024_k5_w0": ("llama8b_x7_L1024_k5", 0),
    "llama8b_x7_L1024_k5_w6": ("llama8b_x7_L1024_k5", 6),
}


def window_logits(wl_name: str, window: int, seed: int = SEED, log=print) -> dict:
    wl = S.WORKLOADS[wl_name]
    s = wl.shape
    L = wl.prefix_lens[window]
    prefix = S.prefix_tokens(s, seed, window, L)
    wi = S.window_inputs(s, seed, wl.n_windows, wl.k)
    toks = wi["tokens"][window]
    seq = np.concatenate([prefix.astype(np.int64), toks.astype(np.int64)])
    T = len(seq)

    def get(layer, name):
        return S.weight(s, seed, layer, name)

    t0 = time.time()
    x = embed64(get, seq)
    pos = np.arange(T)
    for l in range(s.n_layers):
        x, _, _ = layer64(s, get, l, x, pos)
        log(f"  {wl_name} window {window}: layer {l + 1}/{s.n_layers} "
            f"({time.time() - t0:.0f}s)")
    z = head64(s, get, x[L:])
    return {"logits": z.astype(np.float32), "tokens": toks.astype(np.int32),
            "prefix_len": np.int32(L), "seed": np.int32(seed), "window": np.int32(window)}


def main(argv):
    names = [c for c in CASES if not argv or any(a in c for a in argv)]
    for name in names:
        wl_name, window = CASES[name]
        out = window_logits(wl_name, window, log=lambda m: print(m, flush=True))
        path = os.path.join(HERE, f"{name}_logits.npz")
        np.savez(path, **out)
        print(f"wrote {path}: logits {out['logits'].shape}, "
              f"max|z| {float(np.abs(out['logits']).max()):.4g}", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:])
