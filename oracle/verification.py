"""fp64 reference of the accept/reject step of one verification window.

Inputs per window: the k+1 target logit rows z_0..z_k of the window rows
(w0, d_1..d_k) -- row i-1 gives the target distribution p_i for draft d_i and
row k the distribution after all drafts -- the drafts d_1..d_k, the drafter
distributions q_1..q_k, and k+1 uniforms u_1..u_{k+1}.

Sampling mode: the lossless rule that the paper adopts from its cited works
(Section 2, "Straightforward algorithms of speculative inference are lossless
in expectation"; Section 3.1, "Acceptance rate"):
  1. p_i = softmax(z_{i-1} / T), max-subtracted, divided by its sum.
  2. a_i = p_i(d_i) / q_i(d_i) with q upcast exactly from fp32;
     A_i = [u_i < a_i].
  3. n = min({i <= k : A_i = 0} u {k+1}) - 1, the accepted-count definition
     in the proof of Theorem 2 (Appendix E), with A_{k+1} unused.
  4. n < k: r = max(0, p_{n+1} - q_{n+1}) elementwise (if its sum is not
     positive, r = p_{n+1}); n = k: r = p_{k+1} (the bonus token).  R = sum r.
  5. token = smallest t with sum_{v<=t} r_v > u_{k+1} R over ascending ids; if
     rounding leaves none, the last t with r_t > 0.
  6. The window emits d_1..d_n then token: between 1 and k+1 tokens, as the
     batched verification of k+1 prompts does (Section 2).

Greedy mode: exact-match verification (Algorithm 1, the terminate and j*
steps): the target's token at each position is argmax z (ties to the lowest
id, the paper's smallest-index choice); A_i = [d_i = g_i]; n as above;
token = g_{n+1}.  q, u and T are ignored.

All arithmetic is fp64; the argmax is taken on the fp32 logits themselves.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass
class VerifyResult:
    n: int                 # accepted drafts, 0..k
    token: int             # correction (n < k) or bonus (n = k) token
    mode: str
    a: np.ndarray          # a_i for i = 1..k (sampling mode), else empty
    accept_margin: float   # min |a_i - u_i| over the decided positions i <= min(n+1, k)
    draw_margin: float     # distance of u_{k+1} R to the nearest CDF boundary, / R
    r: np.ndarray | None   # the distribution the token was drawn from (unnormalised)
    R: float


def softmax64(z, temperature: float = 1.0) -> np.ndarray:
    s = np.asarray(z, dtype=np.float64) / float(temperature)
    e = np.exp(s - s.max())
    return e / e.sum()


def _check_inputs(drafts, q, V):
    for i, d in enumerate(drafts):
        if not (0 <= int(d) < V):
            raise ValueError(f"draft {i} = {d} outside [0, {V})")
        qd = float(q[i][int(d)])
        if not (qd > 0.0) or not np.isfinite(qd):
            raise ValueError(f"q_{i + 1}(d_{i + 1}) = {qd} is not positive")


def verify64(z, drafts, q=None, u=None, temperature: float = 1.0, mode: str = "sample") -> VerifyResult:
    """Verify one window.  z: [k+1, V] logits; drafts: [k]; q: [k, V]; u: [k+1]."""
    z = np.asarray(z)
    drafts = [int(d) for d in np.asarray(drafts).reshape(-1)]
    k = len(drafts)
    V = z.shape[-1]
    if z.shape[0] != k + 1:
        raise ValueError("need k+1 logit rows")
    if mode == "greedy":
        for i, d in enumerate(drafts):
            if not (0 <= d < V):
                raise ValueError(f"draft {i} = {d} outside [0, {V})")
        g = [int(np.argmax(z[i])) for i in range(k + 1)]
        n = k
        for i in range(k):
            if drafts[i] != g[i]:
                n = i
                break
        # margin: gap between the top two logits of every decided row
        gaps = []
        for i in range(min(n + 1, k + 1)):
            srt = np.sort(np.asarray(z[i], dtype=np.float64))
            gaps.append(srt[-1] - srt[-2] if V > 1 else np.inf)
        return VerifyResult(n, g[n], mode, np.zeros(0), float(min(gaps)), np.inf, None, 1.0)
    if mode != "sample":
        raise ValueError(mode)
    q = np.asarray(q)
    u = np.asarray(u, dtype=np.float64).reshape(-1)
    _check_inputs(drafts, q, V)
    p = [softmax64(z[i], temperature) for i in range(k + 1)]
    a = np.array([p[i][drafts[i]] / np.float64(q[i][drafts[i]]) for i in range(k)], dtype=np.float64)
    n = k
    for i in range(k):
        if not (u[i] < a[i]):
            n = i
            break
    decided = range(min(n + 1, k))
    accept_margin = float(min((abs(a[i] - u[i]) for i in decided), default=np.inf))
    if n < k:
        r = np.maximum(0.0, p[n] - np.asarray(q[n], dtype=np.float64))
        R = float(r.sum())
        if not (R > 0.0):
            r = p[n]
            R = float(r.sum())
    else:
        r = p[k]
        R = float(r.sum())
    target = u[k] * R
    c = np.cumsum(r)
    hit = np.nonzero(c > target)[0]
    if len(hit):
        token = int(hit[0])
    else:
        token = int(np.nonzero(r > 0)[0][-1])
    bounds = np.concatenate([[0.0], c])
    draw_margin = float(np.min(np.abs(bounds - target)) / R)
    return VerifyResult(n, token, mode, a, accept_margin, draw_margin, r, R)
