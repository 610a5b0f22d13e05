"""Host side of distributed speculative inference: lookahead selection and
latency simulation of non-SI, SI and DSI (Sections 3.1, 3.2, Appendices D
and F).

DSI's orchestration (Algorithm 1) is task-level host work: it decides when
verification tasks -- the data-parallel step this library runs on the GPU
(dsi_verify) -- are sent to target servers and which threads a rejection
terminates.  This module holds the pieces of it that do not touch a GPU:

* ``lookahead_min`` -- the smallest lookahead for which verification tasks
  never wait for a target server (Equation 1);
* ``simulate_nonsi`` / ``simulate_si`` / ``simulate_dsi`` -- wall time to
  generate N tokens with forward passes replaced by their latencies, the
  paper's offline methodology (Appendix F), for one realisation of the
  acceptance process; ``expected`` averages many realisations;
* ``offline_speedups`` -- the ablation methodology (Appendix F): expected
  speedups of DSI over SI and non-SI on a grid of drafter latencies and
  acceptance rates, SI at its best lookahead and DSI at its best lookahead
  among those Equation 1 allows for the given SP degree.

Acceptance model: every draft is accepted independently with probability a
(the i.i.d. assumption the paper's acceptance-rate estimate rests on,
Appendix F); a verification accepts its drafts up to the first rejection.

DSI timeline (Algorithm 1 with lookahead k, one drafter and SP target
servers, Appendix D).  From a restart point at time T0 (the committed
prefix) the drafter generates drafts back to back, t_d each.  The target
thread started at the restart computes the next token of the committed
prefix and checks the first draft; after every block of k drafts a
verification task for that block is sent, on the prefix extended by all
earlier drafts.  Tasks are processed in order of their drafts: the first
rejected draft (or the first position after the last draft checked) fixes
the committed tokens -- the accepted drafts plus the verifier's own token --
and the drafter restarts from there when that task completes, terminating
everything built on the rejected draft.  A task starts when it is sent or,
if all SP servers are busy, when one frees up; with the lookahead of
Equation 1 no task waits.
"""
from __future__ import annotations

import dataclasses
import heapq
import math

import numpy as np


def lookahead_min(target_latency: float, drafter_latency: float, sp: int) -> int:
    """Smallest lookahead L with ceil(target / (L * drafter)) <= SP (Equation 1)."""
    if not (target_latency > 0 and drafter_latency > 0) or sp < 1:
        raise ValueError("latencies must be positive and SP >= 1")
    L = 1
    while math.ceil(target_latency / (L * drafter_latency) - 1e-12) > sp:
        L += 1
    return L


def servers_needed(target_latency: float, drafter_latency: float, lookahead: int) -> int:
    """Target servers that keep verification tasks from waiting (the left side
    of Equation 1); one more processing unit runs the drafter."""
    return math.ceil(target_latency / (lookahead * drafter_latency) - 1e-12)


class Acceptance:
    """An i.i.d. acceptance process: draws(n) -> booleans, one per draft."""

    def __init__(self, rate: float, rng: np.random.Generator):
        self.rate = float(rate)
        self.rng = rng

    def __call__(self, n: int) -> np.ndarray:
        return self.rng.random(n) < self.rate


def simulate_nonsi(target_latency: float, N: int) -> float:
    """Autoregressive decoding with the target alone: one forward per token."""
    return N * target_latency


def simulate_si(target_latency: float, drafter_latency: float, lookahead: int, N: int,
                accept: Acceptance) -> float:
    """SI (Section 2): each iteration drafts `lookahead` tokens, then one target
    forward verifies them and emits the accepted drafts plus one token."""
    t, made = 0.0, 0
    while made < N:
        ok = accept(lookahead)
        n = int(np.argmin(ok)) if not ok.all() else lookahead
        made += n + 1
        t += lookahead * drafter_latency + target_latency
    return t


@dataclasses.dataclass
class DsiTrace:
    time: float
    tokens: int
    target_forwards: int      # verification tasks started
    waited: float             # total time tasks waited for a free server


def simulate_dsi(target_latency: float, drafter_latency: float, lookahead: int, sp: int, N: int,
                 accept: Acceptance) -> DsiTrace:
    """DSI with one drafter and `sp` target servers (module docstring).

    From a restart at T0 the drafter finishes draft i at T0 + i t_d.  Task j
    (j = 0, 1, ...) is sent when D = j k drafts exist, runs the target on the
    prefix extended by them, and checks every draft not yet checked up to
    draft D + 1 (its last row predicts the token after draft D; draft D + 1
    exists by the time the task ends because the target is slower than the
    drafter, Assumption 2).  The first rejected draft r commits r tokens (the
    r - 1 accepted drafts and the verifier's token) when its task ends, and
    the drafter restarts there."""
    td, tt, k = drafter_latency, target_latency, lookahead
    if not tt > td:
        raise ValueError("the target must be slower than the drafter (Assumption 2)")
    free = [0.0] * sp                 # min-heap of the servers' free times
    T0, made, forwards, waited = 0.0, 0, 0, 0.0
    while made < N:
        checked, j = 0, 0
        while True:
            D = j * k
            send = T0 + D * td
            start = max(send, heapq.heappop(free))
            waited += start - send
            end = start + tt
            heapq.heappush(free, end)
            forwards += 1
            hi = min(D + 1, N - made)   # drafts beyond the N-th token are never needed
            n_new = hi - checked
            ok = accept(n_new)
            if n_new and not ok.all():
                r = checked + 1 + int(np.argmin(ok))
                made, T0 = made + r, end
                break
            checked = hi
            if made + checked >= N:
                made, T0 = N, end
                break
            j += 1
    return DsiTrace(T0, made, forwards, waited)


def expected(fn, runs: int, seed: int = 0, **kw) -> float:
    """Mean wall time of `fn` (simulate_si or simulate_dsi) over independent
    acceptance realisations; `kw` holds its other arguments and `rate`."""
    rate = kw.pop("rate")
    rng = np.random.default_rng(seed)
    vals = []
    for _ in range(runs):
        r = fn(accept=Acceptance(rate, rng), **kw)
        vals.append(r.time if isinstance(r, DsiTrace) else r)
    return float(np.mean(vals))


def prop1_bound(t1: float, t2: float, p: float, N: int) -> float:
    """Proposition 1: expected DSI time is at most t1 p (N-1) + t2 ((1-p)(N-1) + 1)."""
    return t1 * p * (N - 1) + t2 * ((1 - p) * (N - 1) + 1)


def offline_speedups(drafter_fracs, rates, N: int = 100, runs: int = 5, sp: int = 7,
                     max_lookahead: int = 20, seed: int = 0):
    """Expected speedups on a grid (target latency 1, drafter latency f):
    returns (dsi_over_si, dsi_over_nonsi) arrays [len(fracs), len(rates)].
    SI takes its best lookahead in 1..max_lookahead; DSI its best among the
    lookaheads that satisfy Equation 1 for `sp` (at least lookahead_min)."""
    fracs, rates = list(drafter_fracs), list(rates)
    over_si = np.zeros((len(fracs), len(rates)))
    over_nonsi = np.zeros_like(over_si)
    for i, f in enumerate(fracs):
        lmin = lookahead_min(1.0, f, sp)
        for j, a in enumerate(rates):
            si = min(expected(simulate_si, runs, seed, target_latency=1.0, drafter_latency=f,
                              lookahead=L, N=N, rate=a) for L in range(1, max_lookahead + 1))
            dsi = min(expected(simulate_dsi, runs, seed, target_latency=1.0, drafter_latency=f,
                               lookahead=L, sp=sp, N=N, rate=a)
                      for L in range(lmin, max(lmin, max_lookahead) + 1))
            over_si[i, j] = si / dsi
            over_nonsi[i, j] = simulate_nonsi(1.0, N) / dsi
    return over_si, over_nonsi
