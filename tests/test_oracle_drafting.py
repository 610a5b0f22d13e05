"""Pins of the drafter oracle (oracle/drafting.py) and of the speculative
inference loop built from it, independent of the GPU path.

* the inverse-CDF draw, by exact enumeration of its cells and a chi-square
  test of many draws;
* drafter rows: fp64 softmax of the drafter's logits, cross-checked with
  torch, and incremental drafting equal to one forward over the sequence;
* the SI iteration with a real transformer drafter is lossless (exact
  enumeration over V = 6, k = 2, Section 2 / Theorem 1), and a drafter
  identical to the target accepts every draft.
"""
import numpy as np
import pytest
import torch

import dsi_synth as S
from oracle import bruteforce, forward64, softmax64
from oracle.drafting import draft64, draft_q32, draw_inverse_cdf, si_loop64


def test_inverse_cdf_cells_exact():
    q = np.array([0.125, 0.0, 0.25, 0.375, 0.25], np.float32)   # binary fractions: exact sums
    cells = [(0.0, 0.125, 0), (0.125, 0.375, 2), (0.375, 0.75, 3), (0.75, 1.0, 4)]
    for lo, hi, t in cells:
        for u in (lo, 0.5 * (lo + hi), np.nextafter(hi, 0.0)):
            assert draw_inverse_cdf(q, u)[0] == t, (u, t)
    # a zero-probability token is never drawn; boundaries belong to the next cell
    us = np.linspace(0.0, 1.0, 4097)[:-1]
    toks = [draw_inverse_cdf(q, u)[0] for u in us]
    assert 1 not in toks
    counts = np.bincount(toks, minlength=5) / len(us)
    assert np.allclose(counts, q, atol=0.0)      # 4096-point grid hits each cell exactly


def test_inverse_cdf_scale_invariant_and_one_hot():
    rng = np.random.default_rng(3)
    q = rng.random(17).astype(np.float32)
    for u in rng.random(200):
        assert draw_inverse_cdf(q, u)[0] == draw_inverse_cdf(q * np.float32(4.0), u)[0]
    e = np.zeros(9, np.float32)
    e[6] = 1.0
    assert {draw_inverse_cdf(e, u)[0] for u in rng.random(100)} == {6}
    assert draw_inverse_cdf(e, 0.0)[0] == 6


def test_inverse_cdf_statistics():
    rng = np.random.default_rng(5)
    q = draft_q32(rng.standard_normal(40) * 1.5)
    n = 100000
    toks = np.array([draw_inverse_cdf(q, u)[0] for u in rng.random(n)])
    obs = np.bincount(toks, minlength=40)
    exp = q.astype(np.float64) / q.sum() * n
    chi2 = float(((obs - exp) ** 2 / exp).sum())
    assert chi2 < 90.0      # 39 degrees of freedom: p ~ 1e-5 at 90


def test_draft_rows_are_softmax_of_drafter_logits():
    s = S.SHAPES["tiny"]
    get = lambda l, n: S.weight(s, 11, l, n).astype(np.float64)
    prefix = S.prefix_tokens(s, 11, 0, 20)
    _, cache = forward64(s, get, prefix)
    u = np.array([0.1, 0.7, 0.4, 0.95])
    dr = draft64(s, get, cache, [5], 4, u, temperature=0.8)
    assert dr.tokens[0] == 5 and len(dr.tokens) == 5
    full, _ = forward64(s, get, np.concatenate([prefix, dr.tokens[:4]]))
    for i in range(4):
        z = full[20 + i]
        assert np.allclose(dr.logits[i], z, rtol=0, atol=1e-12)
        ref = torch.softmax(torch.tensor(z / 0.8, dtype=torch.float64), 0).numpy().astype(np.float32)
        assert np.array_equal(dr.q[i], ref) or np.abs(dr.q[i] - ref).max() <= 2 ** -24
        assert dr.tokens[i + 1] == draw_inverse_cdf(dr.q[i], u[i])[0]
    # the drafter cache now holds prefix + w0 + d_1..d_3
    assert dr.cache[0][0].shape[0] == 20 + 4


def test_si_iteration_with_transformer_drafter_is_lossless():
    """Target and drafter are both oracle transformers (V = 6); the exact
    distribution of one iteration's emitted tokens equals the target's."""
    st = S.Shape("bf_t", 1, 32, 2, 1, 16, 48, 6, wdtype="f32", kvdtype="f32", gains="random")
    sd = S.Shape("bf_d", 1, 32, 2, 2, 16, 40, 6, wdtype="f32", kvdtype="f32", gains="random")
    tget = lambda l, n: S.weight(st, 3, l, n).astype(np.float64) * (30.0 if n == "lm_head" else 1.0)
    dget = lambda l, n: S.weight(sd, 4, l, n).astype(np.float64) * (20.0 if n == "lm_head" else 1.0)
    ctx = (1, 4, 2)

    def z(pfx):
        return forward64(st, tget, np.array(ctx + tuple(pfx)))[0][-1]

    def q64(pfx):
        return softmax64(forward64(sd, dget, np.array(ctx + tuple(pfx)))[0][-1])

    dist = bruteforce.emitted_distribution(z, q64, 6, 2)
    assert bruteforce.lossless_error(dist, z, 6, 2) < 1e-12
    # drafter and target differ: some draft is rejected with positive probability
    assert sum(p for y, p in dist.items() if len(y) < 3) > 0.05
    # with the stored fp32 rows (used as given, not renormalised) the rule is
    # lossless up to the rounding of q: |sum q - 1| is a few 2^-24
    dist32 = bruteforce.emitted_distribution(z, lambda pfx: draft_q32(
        forward64(sd, dget, np.array(ctx + tuple(pfx)))[0][-1]).astype(np.float64), 6, 2)
    assert bruteforce.lossless_error(dist32, z, 6, 2) < 1e-6


def test_drafter_equal_to_target_accepts_everything():
    s = S.SHAPES["ragged_f32"]
    get = lambda l, n: S.weight(s, 2, l, n).astype(np.float64)
    prefix = S.prefix_tokens(s, 2, 0, 12)
    rng = np.random.default_rng(0)
    iters, k = 3, 3
    res = si_loop64(s, get, s, get, prefix, 7, k, rng.random((iters, k)), rng.random((iters, k + 1)))
    for it, r in enumerate(res):
        if r.accept_margin > 1e-6:
            assert r.n == k, it
        if it:
            assert r.window[0] == res[it - 1].token


def test_si_loop_commits_and_carries_tokens():
    """Iteration bookkeeping: each window starts with the previous emitted
    token, the committed sequence is the concatenation of the emissions, and
    the loop equals one fresh iteration from the committed prefix."""
    st = S.SHAPES["ragged_f32"]
    sd = S.Shape("tiny_v777", 1, 64, 2, 2, 32, 128, 777, wdtype="f32", kvdtype="f32")
    tget = lambda l, n: S.weight(st, 1, l, n).astype(np.float64)
    dget = lambda l, n: S.weight(sd, 9, l, n).astype(np.float64)
    prefix = list(S.prefix_tokens(st, 1, 0, 10))
    rng = np.random.default_rng(4)
    k, iters = 3, 4
    ud, uv = rng.random((iters, k)), rng.random((iters, k + 1))
    res = si_loop64(st, tget, sd, dget, prefix, 3, k, ud, uv)
    committed = list(prefix)
    w0 = 3
    for it, r in enumerate(res):
        assert r.window[0] == w0
        # a fresh single iteration from the committed prefix gives the same result
        one = si_loop64(st, tget, sd, dget, committed, w0, k, ud[it:it + 1], uv[it:it + 1])[0]
        assert (one.n, one.token) == (r.n, r.token)
        assert np.array_equal(one.window, r.window)
        committed += [w0] + [int(t) for t in r.window[1:r.n + 1]]
        w0 = r.token
