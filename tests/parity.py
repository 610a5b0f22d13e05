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

# Regression gates, about ten times the logit error measured on the small
# parity shapes (bf16 cache: 5e-5..2.3e-4; bf16 weights over an fp32 cache:
# ~5e-6; fp32 throughout: 2-3e-7), so a change that moves the logits by far
# less than the contract tolerance above still fails.
REG = {"bf16kv": 2e-3, "bf16w": 5e-5, "f32": 3e-6}


def tol_of(shape) -> float:
    """Logit tolerance of a shape: the bf16 one as soon as weights or the KV
    cache are stored in bf16 (rounding of a cached K/V element near a
    rounding boundary may go either way on the two sides)."""
    return TOL["bf16"] if "bf16" in (shape.wdtype, shape.kvdtype) else TOL["f32"]


def reg_of(shape) -> float:
    """Regression gate on the logit error of a small parity shape."""
    if shape.kvdtype == "bf16":
        return REG["bf16kv"]
    return REG["bf16w"] if shape.wdtype == "bf16" else REG["f32"]


def settle_u(zo, tokens, q, u, delta, temperature=1.0):
    """Uniforms (multiples of 2^-24, in [0, 1)) for which every decision the
    oracle takes on its logits zo is decided by a margin that a logit error
    up to delta cannot flip: |ln a_i - ln u_i| >= 4 delta and |a_i - u_i| >=
    2e-4 at the compared acceptance positions, and a draw margin >= 8 delta.
    A uniform that sits too close is moved away from its threshold, so the
    single-window tests compare every decision instead of skipping a
    flagged window; where no uniform reaches the draw margin, the one in the
    middle of the draw's widest CDF interval is taken.  Nothing here depends
    on the GPU's output."""
    u = np.array(u, dtype=np.float64).copy()
    tokens = np.asarray(tokens)
    k = len(tokens) - 1
    q2 = 2.0 ** 24
    for _ in range(64):
        r = verify64(zo, tokens[1:], q, u, temperature=temperature)
        moved = False
        for i in range(min(r.n + 1, k)):
            a = float(r.a[i])
            lo, hi = a * np.exp(-4.0 * delta) - 2e-4, a * np.exp(4.0 * delta) + 2e-4
            if lo < u[i] < hi:
                down, up = lo - 1e-3, hi + 1e-3
                ok_down, ok_up = down >= 0.0, up < 1.0
                if not (ok_down or ok_up):
                    raise AssertionError("no uniform clears the acceptance threshold")
                u[i] = down if (ok_down and (u[i] < a or not ok_up)) else up
                u[i] = np.floor(u[i] * q2) / q2
                moved = True
                break
        if moved:
            continue
        if r.draw_margin < 8.0 * delta + 1e-9:
            # the middle of the widest interval of the draw's CDF: the
            # largest margin any uniform can have for this draw
            t = int(np.argmax(r.r))
            c0 = float(np.sum(r.r[:t]))
            u[k] = np.floor((c0 + 0.5 * float(r.r[t])) / r.R * q2) / q2
        return u.astype(np.float32)
    raise AssertionError("could not settle the uniforms")


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


def oracle_greedy_continuation(shape, prompt, w0, N, seed=0, delta=None):
    """The target's own greedy tokens after prompt + w0, by the oracle: N
    steps of an fp64 forward over the whole sequence, argmax of the last row
    (ties to the lowest id).  Returns (tokens, n_sure): the first n_sure
    tokens are decided by a top-2 logit gap above 2 delta (delta: the logit
    tolerance of the shape), so a GPU path within that tolerance must
    reproduce them exactly; later ones may legitimately diverge."""
    delta = tol_of(shape) if delta is None else delta
    get = getter(shape, seed, cache=True)
    # one token per step on the oracle's own fp64 cache (cached = uncached
    # forward is one of the oracle's pins)
    zz, cache = forward64(shape, get, np.asarray([int(t) for t in prompt] + [int(w0)], np.int64))
    z = zz[-1]
    out, n_sure = [], None
    for i in range(N):
        t = int(np.argmax(z))
        top2 = np.sort(z)[-2:]
        if n_sure is None and top2[1] - top2[0] <= 2.0 * delta:
            n_sure = i
        out.append(t)
        if i + 1 < N:
            zz, cache = forward64(shape, get, np.asarray([t], np.int64), cache)
            z = zz[-1]
    return out, (N if n_sure is None else n_sure)


def e2e_check_parts(zo, delta, tokens, q, u, n, tok, mode="sample"):
    """End-to-end check split into its two decisions, for logit errors delta
    at which the draw itself is often within reach (full vocabularies): the
    accepted count n is compared unless an acceptance it depends on is
    flagged (|ln a_i - ln u_i| < 2 delta or |a_i - u_i| < 1e-4; greedy: a
    top-2 gap <= 2 delta in a row that decides an acceptance), and the token
    is compared when n is and its own decision is not flagged (draw margin
    < 4 delta; greedy: the top-2 gap of its row).  Returns (n_compared,
    token_compared) after asserting whatever was compared."""
    r = verify64(zo, tokens[1:], q, u, mode=mode)
    k = len(tokens) - 1
    if mode == "sample":
        n_ok = all(abs(np.log(max(r.a[i], 1e-300)) - np.log(max(float(u[i]), 1e-300))) >= 2.0 * delta + 1e-6
                   and abs(r.a[i] - float(u[i])) >= 1e-4 for i in range(min(r.n + 1, k)))
        t_ok = n_ok and r.draw_margin >= 4.0 * delta + 1e-9
    else:
        gaps = [float(np.diff(np.sort(np.asarray(zo[i], np.float64))[-2:])[0]) for i in range(min(r.n + 1, k + 1))]
        n_ok = all(g > 2.0 * delta for g in gaps[:min(r.n + 1, k)])
        t_ok = n_ok and gaps[r.n] > 2.0 * delta
    if n_ok:
        assert int(n) == r.n, (int(n), r.n)
    if t_ok:
        assert int(tok) == r.token, (int(tok), r.token)
    return n_ok, t_ok
