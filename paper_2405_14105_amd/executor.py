"""Algorithm 1 (distributed speculative inference) over the library: one
drafter, SP target servers, lookahead k, exact-match verification (the
algorithm's terminate / j* rule: a draft survives iff it equals the target's
own token, here the target's greedy token).

The computations are the library's (dsi_draft, dsi_verify, dsi_prefill,
dsi_kv_rollback on the GPU); the timeline is the one of
``orchestrate.simulate_dsi`` driven by given target and drafter latencies,
so the result reports both the tokens and the wall time DSI would take with
SP real servers.  On one GPU the tasks run one after another; what is
exercised is the orchestration: speculative prefixes, per-server caches,
termination and restart.

Each target server is one window of the target's KV cache -- its own cache
(Section 3.1, "KV cache").  A task on a server first brings that cache to the
task's prefix (roll back what diverges, prefill what is missing: committed
tokens or drafts of the current branch), then verifies the window of tokens
whose next-token predictions the task checks.
"""
from __future__ import annotations

import dataclasses
import heapq

import numpy as np
import torch

from . import dsi


@dataclasses.dataclass
class DsiRun:
    tokens: list          # the N generated tokens (after w0)
    time: float           # simulated wall time with SP servers
    tasks: int            # verification tasks run
    rejections: int


class _Cache:
    """Host record of one window's cached tokens (positions >= the prompt)."""

    def __init__(self, kv: int, window: int, base: int):
        self.kv, self.window, self.base = kv, window, base
        self.toks: list = []

    def sync(self, want: list, model: int, dev) -> None:
        """Make the cached tokens equal `want` (roll back, then prefill)."""
        common = 0
        for a, b in zip(self.toks, want):
            if a != b:
                break
            common += 1
        if common < len(self.toks):
            dsi.dsi_kv_rollback(self.kv, self.window, self.base + common)
            self.toks = self.toks[:common]
        missing = want[common:]
        for off in range(0, len(missing), dsi.DSI_MAX_ROWS):
            part = missing[off:off + dsi.DSI_MAX_ROWS]
            t = torch.tensor(part, dtype=torch.int32, device=dev)
            dsi.dsi_prefill(model, self.kv, self.window, t, len(part), None)
            self.toks += part


def _draft(drafter: int, dcache: _Cache, ctx: list, k: int, V: int, T: float, rng, dev) -> list:
    """k drafts continuing ctx (whose last token the drafter has not cached):
    bring the drafter's cache to ctx[:-1] (roll back what diverges, feed what
    is missing), then dsi_draft."""
    common = 0
    for a, b in zip(dcache.toks, ctx[:-1]):
        if a != b:
            break
        common += 1
    if common < len(dcache.toks):
        dsi.dsi_kv_rollback(dcache.kv, dcache.window, dcache.base + common)
        dcache.toks = dcache.toks[:common]
    feed = ctx[common:]
    while len(feed) > dsi.DSI_MAX_ROWS:              # catch up long gaps first
        dcache.sync(dcache.toks + feed[:dsi.DSI_MAX_ROWS], drafter, dev)
        feed = feed[dsi.DSI_MAX_ROWS:]
    f = torch.tensor(feed, dtype=torch.int32, device=dev)
    u = torch.from_numpy(rng.random(k).astype(np.float32)).to(dev)
    tok = torch.zeros(k + 1, dtype=torch.int32, device=dev)
    q = torch.empty((k, V), dtype=torch.float32, device=dev)
    dsi.dsi_draft(drafter, dcache.kv, dcache.window, f, len(feed), k, u, tok, q, T)
    new = [int(x) for x in tok.cpu().numpy()[1:]]
    dcache.toks += feed + new[:-1]                   # the feed and d_1..d_{k-1} are cached
    return new


class DsiExecutor:
    """target / drafter: dsi_model handles; tkv: the target's cache with >= sp
    windows, dkv: the drafter's cache (window 0).  All hold the same prompt
    of `prompt_len` tokens before generate()."""

    def __init__(self, target: int, tkv: int, drafter: int, dkv: int, vocab: int, k: int, sp: int,
                 prompt_len: int, t_target: float = 1.0, t_drafter: float = 0.1,
                 draft_temperature: float = 1.0, seed: int = 0):
        self.target, self.drafter, self.V, self.k, self.sp = target, drafter, vocab, k, sp
        self.tt, self.td, self.T = t_target, t_drafter, draft_temperature
        self.dev = torch.device("cuda:0")
        self.servers = [_Cache(tkv, s, prompt_len) for s in range(sp)]
        self.dcache = _Cache(dkv, 0, prompt_len)
        self.rng = np.random.default_rng(seed)
        self.n_out = torch.zeros(1, dtype=torch.int32, device=self.dev)
        self.t_out = torch.zeros(1, dtype=torch.int32, device=self.dev)

    def _draft_block(self, committed: list, drafts: list) -> None:
        """Extend `drafts` by k drafts continuing committed + drafts."""
        drafts += _draft(self.drafter, self.dcache, committed + drafts, self.k, self.V, self.T,
                         self.rng, self.dev)

    def generate(self, w0: int, N: int) -> DsiRun:
        k = self.k
        committed = [int(w0)]        # tokens after the prompt; the last one is uncached
        free = [(0.0, s) for s in range(self.sp)]
        heapq.heapify(free)
        T0, tasks, rejections = 0.0, 0, 0
        while len(committed) - 1 < N:
            drafts: list = []
            checked, j = 0, 0
            while True:
                D = j * k
                while len(drafts) < D + 1:
                    self._draft_block(committed, drafts)
                # schedule on the earliest free server
                ft, s = heapq.heappop(free)
                start = max(T0 + D * self.td, ft)
                end = start + self.tt
                heapq.heappush(free, (end, s))
                tasks += 1
                srv = self.servers[s]
                # the task checks drafts checked+1 .. D+1: rows t_checked .. t_D
                seq = committed + drafts                 # t_0 = committed[-1], t_i = drafts[i-1]
                base = len(committed) - 1
                srv.sync(seq[:base + checked], self.target, self.dev)
                window = seq[base + checked:base + D + 1]
                tk = torch.tensor([window], dtype=torch.int32, device=self.dev)
                dsi.dsi_verify(self.target, srv.kv, s, 1, len(window) - 1, tk, None, None,
                               self.n_out, self.t_out, 1.0, dsi.DSI_GREEDY, True)
                n, tok = int(self.n_out.item()), int(self.t_out.item())
                if n < 0:
                    raise RuntimeError("verification reported an input error")
                srv.toks += window[:n + 1]
                # the host's bound on the server's length grew by the window's
                # row count; reading the length (the stream is idle after the
                # reads above) tightens it to the committed L + n + 1
                if dsi.dsi_kv_length(srv.kv, s) != srv.base + len(srv.toks):
                    raise RuntimeError("server cache length disagrees with its committed tokens")
                remaining = N - (len(committed) - 1)
                if n < len(window) - 1:                  # draft checked + 1 + n rejected
                    r = checked + 1 + n
                elif tok != drafts[D]:                   # draft D + 1 rejected
                    r = D + 1
                else:
                    r = None
                if r is not None and r <= remaining:
                    committed += drafts[:r - 1] + [tok]
                    rejections += 1
                    T0 = end
                    break
                checked = D + 1
                if checked >= remaining:                 # N tokens accepted
                    committed += drafts[:remaining]
                    T0 = end
                    break
                j += 1
        return DsiRun(committed[1:N + 1], T0, tasks, rejections)


@dataclasses.dataclass
class TreeRun:
    tokens: list          # the N generated tokens (after w0)
    forwards: int         # target forwards (one tree verification each)
    accepted: list        # drafts accepted by each verification


class TreeExecutor:
    """Algorithm 1's several drafters verified together: every iteration each
    drafter j = 1..m drafts k tokens continuing the committed tokens (one
    thread per drafter on the same prefix); the m chains form one token tree
    rooted at the last committed token (drafter j's chain is numbered after
    drafter j-1's, so children of a node are in drafter order), and one
    target forward verifies the whole tree with exact matching and the j*
    rule (dsi_verify_tree, committed in place).  target / tkv: the target
    and its cache, verifying in `window`; drafters: (model, kv) pairs, each
    cache's window 0 holding the prompt.  1 + m k <= DSI_MAX_ROWS."""

    def __init__(self, target: int, tkv: int, window: int, drafters: list, vocab: int, k: int,
                 prompt_len: int, draft_temperature: float = 1.0, seed: int = 0):
        if not drafters or 1 + len(drafters) * k > dsi.DSI_MAX_ROWS:
            raise ValueError("need 1 + drafters * k <= DSI_MAX_ROWS and at least one drafter")
        self.target, self.tkv, self.window = target, tkv, window
        self.drafters = [(m, _Cache(kv, 0, prompt_len)) for m, kv in drafters]
        self.V, self.k, self.T = vocab, k, draft_temperature
        self.dev = torch.device("cuda:0")
        self.rng = np.random.default_rng(seed)
        m = len(drafters)
        self.R = 1 + m * k
        par = [-1]
        for j in range(m):
            par += [0] + [1 + j * k + i for i in range(k - 1)]
        self.parent = torch.tensor([par], dtype=torch.int32, device=self.dev)
        self.path = torch.zeros((1, self.R), dtype=torch.int32, device=self.dev)
        self.n_out = torch.zeros(1, dtype=torch.int32, device=self.dev)
        self.t_out = torch.zeros(1, dtype=torch.int32, device=self.dev)

    def generate(self, w0: int, N: int) -> TreeRun:
        committed = [int(w0)]        # tokens after the prompt; the last one is uncached
        forwards, accepted = 0, []
        while len(committed) - 1 < N:
            nodes = [committed[-1]]
            for model, cache in self.drafters:
                nodes += _draft(model, cache, committed, self.k, self.V, self.T, self.rng, self.dev)
            tk = torch.tensor([nodes], dtype=torch.int32, device=self.dev)
            dsi.dsi_verify_tree(self.target, self.tkv, self.window, 1, self.R, tk, self.parent, self.path,
                                self.n_out, self.t_out, True)
            n, tok = int(self.n_out.item()), int(self.t_out.item())
            if n < 0:
                raise RuntimeError("token-tree verification reported an input error")
            # the host's bound on the window length grows by the node count per
            # verification; reading the length tightens it to L + n + 1
            dsi.dsi_kv_length(self.tkv, self.window)
            path = self.path.cpu().numpy()[0]
            committed += [nodes[a] for a in path[1:n + 1]] + [tok]
            forwards += 1
            accepted.append(n)
        return TreeRun(committed[1:N + 1], forwards, accepted)
