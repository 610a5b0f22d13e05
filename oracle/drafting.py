"""fp64 reference of the drafter side of one speculative-inference iteration,
and of the whole iteration loop on one target server.

Test infrastructure only (see the package header).

Section 2 ("Speculative Inference"): the drafter produces the k lookahead
tokens one at a time, each sampled from the drafter's own next-token
distribution given the context and the drafts before it; the target then
verifies the k+1 prompts in one batch (verification.py) and the iteration
emits d_1..d_n and one more token.  Appendix B treats a language model as a
black box that maps a prompt to logits, sampled through a softmax.

Readings fixed here (the paper is silent on the numerics):
  * q_i = softmax(z_i / T) of the drafter's logits for the row of the i-th
    draft, computed in fp64 and stored in fp32; that stored fp32 row is the
    distribution verification uses as given, so the draft is drawn from it;
  * d_i is drawn by inverse CDF over ascending token ids with the uniform
    u_i: the smallest t with sum_{v <= t} q_v > u_i * sum_v q_v (the sums in
    fp64 of the fp32 values), or, when rounding leaves no such t, the last t
    with q_t > 0 -- the same categorical draw as verification's residual
    draw;
  * the drafter caches its own K/V like the target: it feeds the tokens it
    has not seen yet (the last committed token, and after a fully accepted
    window also the last draft) and then one draft per step, so after k
    steps it holds the context plus d_1..d_{k-1}.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .model import forward64
from .verification import softmax64, verify64


def draft_q32(z, temperature: float = 1.0) -> np.ndarray:
    """The stored drafter distribution: fp64 softmax of z / T, rounded to fp32."""
    return softmax64(z, temperature).astype(np.float32)


def draw_inverse_cdf(q, u: float):
    """Inverse-CDF draw from the (unnormalised) row q with the uniform u.

    Returns (token, margin): margin is the distance of u * sum(q) to the
    nearest CDF boundary divided by sum(q) (how far u is from changing the
    token)."""
    q = np.asarray(q, dtype=np.float64)
    if q.ndim != 1 or not np.all(q >= 0.0):
        raise ValueError("q must be a non-negative vector")
    c = np.cumsum(q)
    total = float(c[-1])
    if not total > 0.0:
        raise ValueError("q has no mass")
    target = float(u) * total
    hit = np.nonzero(c > target)[0]
    token = int(hit[0]) if len(hit) else int(np.nonzero(q > 0.0)[0][-1])
    bounds = np.concatenate([[0.0], c])
    margin = float(np.min(np.abs(bounds - target)) / total)
    return token, margin


@dataclasses.dataclass
class DraftResult:
    tokens: np.ndarray     # [k+1]: the window (w0, d_1..d_k), w0 = last fed token
    q: np.ndarray          # [k][V] fp32 drafter distributions
    logits: np.ndarray     # [k][V] fp64 drafter logits
    margin: np.ndarray     # [k] draw margins
    cache: list            # the drafter's KV after drafting (positions of context + d_1..d_{k-1})


def draft64(s, get, cache, feed, k: int, u, temperature: float = 1.0, forced=None) -> DraftResult:
    """Draft k tokens.

    cache: the drafter's KV (forward64 format) for the tokens it has already
    seen, or None; feed: the tokens it has not seen (at least one; the last
    is w0); u: k uniforms.  forced (optional [k] token ids) replaces each
    draw by a given token while still computing its q row -- for checking a
    drafter's rows against another implementation's draws."""
    feed = [int(t) for t in feed]
    if not feed:
        raise ValueError("feed at least the last committed token")
    V = s.vocab
    q = np.zeros((k, V), np.float32)
    zs = np.zeros((k, V), np.float64)
    margin = np.full(k, np.inf)
    drafts = []
    rows = feed
    for i in range(k):
        z, cache = forward64(s, get, rows, cache)
        zs[i] = z[-1]
        q[i] = draft_q32(z[-1], temperature)
        d, margin[i] = draw_inverse_cdf(q[i], float(u[i]))
        if forced is not None:
            d = int(forced[i])
        drafts.append(d)
        rows = [d]
    tokens = np.array([feed[-1]] + drafts, dtype=np.int64)
    return DraftResult(tokens, q, zs, margin, cache)


@dataclasses.dataclass
class IterationResult:
    window: np.ndarray     # [k+1] (w0, d_1..d_k)
    n: int
    token: int
    accept_margin: float
    draw_margin: float     # min of the drafter's and the verifier's draw margins


def si_loop64(ts, tget, ds, dget, prefix, w0: int, k: int, u_draft, u_verify,
              temperature: float = 1.0):
    """Iterations of speculative inference on one target server (Section 2):
    draft k tokens, verify them with the target, commit d_1..d_n and carry the
    emitted token as the next iteration's w0.

    prefix: committed tokens already in both caches; u_draft [iters][k],
    u_verify [iters][k+1].  Returns the list of IterationResult."""
    prefix = [int(t) for t in prefix]
    _, tcache = forward64(ts, tget, prefix) if prefix else (None, None)
    _, dcache = forward64(ds, dget, prefix) if prefix else (None, None)
    feed = [int(w0)]
    out = []
    for it in range(len(u_draft)):
        dr = draft64(ds, dget, dcache, feed, k, u_draft[it], temperature)
        z, tcache_new = forward64(ts, tget, dr.tokens, tcache)
        r = verify64(z, dr.tokens[1:], dr.q, u_verify[it], temperature)
        n = r.n
        out.append(IterationResult(dr.tokens.copy(), n, r.token, r.accept_margin,
                                   min(r.draw_margin, float(dr.margin.min()) if k else np.inf)))
        # target keeps w0, d_1..d_n
        L = tcache[0][0].shape[0] if tcache is not None else 0
        tcache = [(kk[:L + n + 1], vv[:L + n + 1]) for kk, vv in tcache_new]
        # drafter holds context + w0 + d_1..d_{k-1}; keep w0 + d_1..d_min(n, k-1)
        Ld = L + 1 + min(n, k - 1)
        dcache = [(kk[:Ld], vv[:Ld]) for kk, vv in dr.cache]
        feed = ([int(dr.tokens[k])] if n == k else []) + [int(r.token)]
    return out
