"""Shared parity helpers for the GPU tests: oracle weight access, the
oracle's logits for a window, and the flag rules under which the GPU's
accept/reject decisions must equal the oracle's.

Decision rules (the accepted count n and the emitted token are compared
bit-exactly except where rounding may legitimately decide them):
  * split check: the GPU's accept/reject on its own logits against the
    oracle's verification of those same logits; a window is skipped when
    some compared acceptance has |a_i - u_i| < 1e-4 or the draw lies within
    1e-9 R of a CDF boundary;
  * end-to-end: against the oracle's verification of the oracle's logits;
    a window is also skipped when the measured logit error delta could flip
    a decision (|ln a_i - ln u_i| < 2 delta, draw margin < 4 delta, greedy
    top-2 gap <= 2 delta), since |delta ln p_v| <= 2 delta.
"""
from __future__ import annotations

import numpy as np

import dsi_synth as S
from oracle import forward64, verify64

TOL = {"f32": 1e-4, "bf16": 2e-2}


def tol_of(shape) -> float:
    """Logit tolerance of a shape: the bf16 one as soon as weights or the KV
    cache are stored in bf16 (rounding of a cached K/V element near a
    rounding boundary may go either way on the two sides)."""
    return TOL["bf16"] if "bf16" in (shape.wdtype, shape.kvdtype) else TOL["f32"]


def getter(shape, seed=0, cache=True):
    """get(layer, name) -> fp64 weights for the oracle (memoised if cache)."""
    memo = {}

    def get(layer, name):
        if not cache:
            return S.weight(shape, seed, layer, name).astype(np.float64)
        if (layer, name) not in memo:
            memo[(layer, name)] = S.weight(shape, seed, layer, name).astype(np.float64)
        return memo[(layer, name)]
    return get


def oracle_logits(shape, prefix, window_tokens, return_hidden=False, seed=0, cache=True):
    toks = np.concatenate([np.asarray(prefix, np.int64), np.asarray(window_tokens, np.int64)])
    res = forward64(shape, getter(shape, seed, cache), toks, return_hidden=return_hidden)
    L = len(prefix)
    if return_hidden:
        return res[0][L:], res[2][:, L:]
    return res[0][L:]


def split_check(z, tokens, q, u, n, tok, mode="sample"):
    r = verify64(z, tokens[1:], q, u, mode=mode)
    if r.accept_margin < 1e-4 or r.draw_margin < 1e-9:
        return None
    assert (int(n), int(tok)) == (r.n, r.token)
    return r


def e2e_check(zo, delta, tokens, q, u, n, tok, mode="sample"):
    r = verify64(zo, tokens[1:], q, u, mode=mode)
    if mode == "sample":
        lnflag = 2.0 * delta + 1e-6
        if any(abs(np.log(max(r.a[i], 1e-300)) - np.log(max(float(u[i]), 1e-300))) < lnflag
               for i in range(min(r.n + 1, len(r.a)))):
            return None
        if r.accept_margin < 1e-4 or r.draw_margin < 4.0 * delta + 1e-9:
            return None
    else:
        if r.accept_margin <= 2.0 * delta:
            return None
    assert (int(n), int(tok)) == (r.n, r.token)
    return r
