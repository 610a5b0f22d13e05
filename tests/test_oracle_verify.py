"""Pins of the fp64 verification oracle (CPU only).

* hand-worked examples (tests/golden/verify_worked_examples.json);
* exact enumeration: sampling mode reproduces the target distribution
  (lossless, Section 2 and Theorem 1) for synthetic and transformer targets;
* greedy mode equals the target's own greedy continuation (Algorithm 1's
  exact-match rule, Theorem 1);
* textbook special cases: k = 0 is an inverse-CDF draw, q = p accepts all,
  a one-hot target in sampling mode behaves as greedy;
* closed forms: P(A_1) = sum_v min(p_v, q_v) when d_1 ~ q_1.
"""
import json
import os

import numpy as np
import pytest

import dsi_synth as S
from oracle import verify64, softmax64, forward64, bruteforce

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "verify_worked_examples.json")


def _case_inputs(c):
    if "p" in c:
        z = np.log(np.asarray(c["p"], dtype=np.float64))
    else:
        z = np.asarray(c["z"], dtype=np.float64)
    q = None
    if c["mode"] == "sample":
        q = np.asarray(c["q"], dtype=np.float64).reshape(len(c["drafts"]), z.shape[1])
    return z, q


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_worked_examples(case):
    z, q = _case_inputs(case)
    res = verify64(z, case["drafts"], q, case.get("u"), mode=case["mode"])
    assert (res.n, res.token) == (case["expect_n"], case["expect_token"])


# --------------------------------------------------------- exact enumeration
def _table_target(V, k, seed):
    """Context-dependent target logits and drafter distributions as lookup
    tables keyed by the draft prefix."""
    rng = np.random.default_rng(seed)
    zt, qt = {}, {}

    def z(pfx):
        if pfx not in zt:
            zt[pfx] = rng.standard_normal(V) * 1.5
        return zt[pfx]

    def q(pfx):
        if pfx not in qt:
            e = np.exp(rng.standard_normal(V))
            qt[pfx] = e / e.sum()
        return qt[pfx]
    return z, q


@pytest.mark.parametrize("V,k,seed", [(2, 1, 0), (3, 2, 1), (4, 3, 2), (5, 2, 3), (4, 1, 4)])
def test_lossless_bruteforce_tables(V, k, seed):
    z, q = _table_target(V, k, seed)
    dist = bruteforce.emitted_distribution(z, q, V, k)
    assert abs(sum(dist.values()) - 1.0) < 1e-12
    assert bruteforce.lossless_error(dist, z, V, k) < 1e-12


def test_lossless_bruteforce_temperature():
    z, q = _table_target(4, 2, 11)
    dist = bruteforce.emitted_distribution(z, q, 4, 2, temperature=0.7)
    assert bruteforce.lossless_error(dist, z, 4, 2, temperature=0.7) < 1e-12


def test_lossless_catches_planted_mistakes():
    """The enumeration must fail for plausible mistakes in the rule."""
    z, q = _table_target(3, 2, 5)
    orig = bruteforce.verify64

    def wrong_residual(zz, d, qq=None, u=None, temperature=1.0, mode="sample"):
        # resample from max(0, q - p) instead of max(0, p - q)
        res = orig(zz, d, qq, u, temperature, mode)
        if res.n < len(d):
            p = softmax64(zz[res.n], temperature)
            r = np.maximum(0.0, np.asarray(qq[res.n]) - p)
            R = r.sum()
            c = np.cumsum(r)
            res.token = int(np.nonzero(c > u[-1] * R)[0][0])
            res.r, res.R = r, R
        return res
    try:
        bruteforce.verify64 = wrong_residual
        dist = bruteforce.emitted_distribution(z, q, 3, 2)
        assert bruteforce.lossless_error(dist, z, 3, 2) > 1e-3
    finally:
        bruteforce.verify64 = orig


def test_lossless_bruteforce_transformer_target():
    """Target p from the oracle transformer itself, shrunk to V = 6."""
    s = S.Shape("bf_tiny", 1, 32, 2, 1, 16, 48, 6, wdtype="f32", kvdtype="f32", gains="random")
    get = lambda l, n: S.weight(s, 3, l, n).astype(np.float64) * (30.0 if n == "lm_head" else 1.0)
    ctx = (1, 4, 2)

    def z(pfx):
        logits, _ = forward64(s, get, np.array(ctx + tuple(pfx)))
        return logits[-1]
    rng = np.random.default_rng(9)
    qt = {}

    def q(pfx):
        if pfx not in qt:
            e = np.exp(rng.standard_normal(6) * 2)
            qt[pfx] = e / e.sum()
        return qt[pfx]
    dist = bruteforce.emitted_distribution(z, q, 6, 2)
    assert bruteforce.lossless_error(dist, z, 6, 2) < 1e-12
    # the scaled head makes the target far from uniform: the check has teeth
    assert softmax64(z(())).max() > 0.4


@pytest.mark.parametrize("V,k,seed", [(3, 2, 0), (4, 3, 1), (5, 2, 2)])
def test_greedy_is_exact_match(V, k, seed):
    rng = np.random.default_rng(seed)
    tab = {}

    def z(pfx):
        if pfx not in tab:
            tab[pfx] = np.round(rng.standard_normal(V), 1)   # rounding creates ties
        return tab[pfx]
    assert bruteforce.greedy_mismatches(z, V, k) == 0


# --------------------------------------------------------- special cases
def test_k0_is_inverse_cdf_draw():
    rng = np.random.default_rng(12)
    z = rng.standard_normal((1, 50))
    p = softmax64(z[0])
    for u in rng.random(200):
        res = verify64(z, [], np.zeros((0, 50)), [u])
        assert res.n == 0
        assert res.token == int(np.searchsorted(np.cumsum(p), u * p.sum(), side="right"))


def test_q_equal_p_accepts_everything():
    rng = np.random.default_rng(13)
    V, k = 40, 6
    z = rng.standard_normal((k + 1, V)) * 2
    q = np.stack([softmax64(z[i]) for i in range(k)])
    for _ in range(100):
        d = rng.integers(0, V, k)
        u = rng.random(k + 1) * (1 - 1e-9)
        assert verify64(z, d, q, u).n == k


def test_one_hot_target_sampling_equals_greedy():
    rng = np.random.default_rng(14)
    V, k = 30, 4
    z = rng.standard_normal((k + 1, V)) * 1e3
    q = np.full((k, V), 1.0 / V)
    for _ in range(100):
        d = np.where(rng.random(k) < 0.7, np.argmax(z[:k], axis=1), rng.integers(0, V, k))
        u = rng.random(k + 1)
        a = verify64(z, d, q, u)
        g = verify64(z, d, mode="greedy")
        assert (a.n, a.token) == (g.n, g.token)


def test_first_acceptance_probability_closed_form():
    """P(A_1 = 1) with d_1 ~ q_1 equals sum_v min(p_v, q_v)."""
    rng = np.random.default_rng(15)
    V = 7
    z = rng.standard_normal((2, V))
    q1 = np.exp(rng.standard_normal(V))
    q1 /= q1.sum()
    p1 = softmax64(z[0])
    tot = 0.0
    for d in range(V):
        a = verify64(z, [d], q1[None], [0.0, 0.5]).a[0]
        tot += q1[d] * min(1.0, a)
    assert abs(tot - np.minimum(p1, q1).sum()) < 1e-14


def test_invalid_draft_inputs_raise():
    z = np.zeros((2, 4))
    with pytest.raises(ValueError):
        verify64(z, [4], np.full((1, 4), 0.25), [0.1, 0.1])
    with pytest.raises(ValueError):
        verify64(z, [1], np.array([[0.5, 0.0, 0.25, 0.25]]), [0.1, 0.1])


def test_accepted_count_bounds_and_tail_independence():
    """1 <= emitted <= k+1 (Section 2) and uniforms after the first rejection
    do not matter (n = min{i: A_i = 0} - 1, Appendix E)."""
    rng = np.random.default_rng(16)
    V, k = 20, 5
    for _ in range(200):
        z = rng.standard_normal((k + 1, V))
        q = rng.random((k, V)) + 0.01
        q /= q.sum(1, keepdims=True)
        d = rng.integers(0, V, k)
        u = rng.random(k + 1)
        r1 = verify64(z, d, q, u)
        assert 0 <= r1.n <= k
        if r1.n < k - 1:
            u2 = u.copy()
            u2[r1.n + 1:k] = rng.random(k - r1.n - 1)
            r2 = verify64(z, d, q, u2)
            assert (r2.n, r2.token) == (r1.n, r1.token)
