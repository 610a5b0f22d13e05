"""Exact enumeration of one verification's output distribution.

Used to pin ``verify64`` against what the paper requires of verification:
  * sampling mode is lossless in expectation -- the emitted tokens follow the
    target's own distribution (Section 2; Theorem 1);
  * greedy mode returns exactly the target's own greedy tokens (Algorithm 1's
    exact-match rule; Theorem 1: the same output as the target alone).

For tiny vocabularies V and lookaheads k every draft sequence d in V^k is
enumerated with weight prod q_i(d_i | d_<i).  Each uniform u_i only matters
through which side of a_i it falls on, and u_{k+1} only through which CDF
cell of the drawn distribution it falls in, so verify64 is evaluated once at
the midpoint of every cell and weighted by the cell length: the result is the
exact output distribution up to fp64 rounding.
"""
from __future__ import annotations

import itertools
from collections import defaultdict

import numpy as np

from .verification import verify64, softmax64


def emitted_distribution(ctx_logits, ctx_q, V: int, k: int, temperature: float = 1.0,
                         probe_tail: bool = True) -> dict:
    """Exact distribution over the emitted token tuples (d_1..d_n, token).

    ctx_logits(prefix) -> target logits [V] after the context extended by the
    tuple `prefix`; ctx_q(prefix) -> drafter distribution [V]."""
    dist = defaultdict(float)
    zcache, qcache = {}, {}

    def zrow(pfx):
        if pfx not in zcache:
            zcache[pfx] = np.asarray(ctx_logits(pfx), dtype=np.float64)
        return zcache[pfx]

    def qrow(pfx):
        if pfx not in qcache:
            qcache[pfx] = np.asarray(ctx_q(pfx), dtype=np.float64)
        return qcache[pfx]

    for d in itertools.product(range(V), repeat=k):
        wd = 1.0
        for i in range(k):
            wd *= qrow(d[:i])[d[i]]
        if wd == 0.0:
            continue
        z = np.stack([zrow(d[:i]) for i in range(k + 1)])
        qm = np.stack([qrow(d[:i]) for i in range(k)]) if k else np.zeros((0, V))
        a = verify64(z, d, qm, np.zeros(k + 1), temperature).a
        acc = np.minimum(a, 1.0)
        for j in range(k + 1):            # j = index of the first rejection (k: none)
            pj = float(np.prod(acc[:j]))
            if j < k:
                pj *= 1.0 - acc[j]
            if pj <= 0.0:
                continue
            u = np.full(k + 1, 0.5)
            u[:j] = acc[:j] / 2.0
            if j < k:
                u[j] = (acc[j] + 1.0) / 2.0
                if probe_tail and j + 1 < k:
                    u[j + 1:k] = 0.0       # later uniforms must not matter
            first = verify64(z, d, qm, u, temperature)
            if first.n != j:
                raise AssertionError(f"cell midpoint gave n={first.n}, expected {j}")
            c = np.cumsum(first.r) / first.R
            lo = 0.0
            for t in range(V):
                hi = c[t]
                if first.r[t] > 0.0 and hi > lo:
                    u[k] = 0.5 * (lo + hi)
                    res = verify64(z, d, qm, u, temperature)
                    if res.n != j or res.token != t:
                        raise AssertionError(f"cell of token {t} drew {res.token}")
                    dist[tuple(d[:j]) + (t,)] += wd * pj * (hi - lo)
                lo = max(lo, hi)
    return dict(dist)


def lossless_error(dist: dict, ctx_logits, V: int, k: int, temperature: float = 1.0) -> float:
    """max over t <= k+1 and emitted prefixes y_<t of
    |P(y_t = v | y_<t, length >= t) - softmax(z(y_<t)/T)(v)|."""
    worst = 0.0
    for t in range(1, k + 2):
        joint = defaultdict(lambda: np.zeros(V))
        for y, pr in dist.items():
            if len(y) >= t:
                joint[y[:t - 1]][y[t - 1]] += pr
        for pfx, row in joint.items():
            tot = row.sum()
            if tot <= 1e-300:
                continue
            p = softmax64(ctx_logits(pfx), temperature)
            worst = max(worst, float(np.max(np.abs(row / tot - p))))
    return worst


def greedy_mismatches(ctx_logits, V: int, k: int) -> int:
    """Count draft sequences where greedy verification differs from the
    target's own greedy continuation (n must be the longest matching prefix,
    the token the target's next greedy token)."""
    target = []
    pfx = ()
    for _ in range(k + 1):
        x = int(np.argmax(np.asarray(ctx_logits(pfx))))
        target.append(x)
        pfx = pfx + (x,)
    bad = 0
    for d in itertools.product(range(V), repeat=k):
        z = np.stack([np.asarray(ctx_logits(d[:i])) for i in range(k + 1)])
        res = verify64(z, d, mode="greedy")
        n = 0
        while n < k and d[n] == target[n]:
            n += 1
        if res.n != n or res.token != target[n]:
            bad += 1
    return bad
