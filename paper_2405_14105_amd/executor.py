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
        k, V = self.k, self.V
        ctx = committed + drafts                       # the last token is not cached yet
        # the drafter caches ctx[:-1]; feed what it is missing, ending with ctx[-1]
        common = 0
        for a, b in zip(self.dcache.toks, ctx[:-1]):
            if a != b:
                break
            common += 1
        if common < len(self.dcache.toks):
            dsi.dsi_kv_rollback(self.dcache.kv, 0, self.dcache.base + common)
            self.dcache.toks = self.dcache.toks[:common]
        feed = ctx[common:]
        while len(feed) > dsi.DSI_MAX_ROWS:         # catch up long gaps first
            self.dcache.sync(self.dcache.toks + feed[:dsi.DSI_MAX_ROWS], self.drafter, self.dev)
            feed = feed[dsi.DSI_MAX_ROWS:]
        f = torch.tensor(feed, dtype=torch.int32, device=self.dev)
        u = torch.from_numpy(self.rng.random(k).astype(np.float32)).to(self.dev)
        tok = torch.zeros(k + 1, dtype=torch.int32, device=self.dev)
        q = torch.empty((k, V), dtype=torch.float32, device=self.dev)
        dsi.dsi_draft(self.drafter, self.dcache.kv, 0, f, len(feed), k, u, tok, q, self.T)
        new = [int(x) for x in tok.cpu().numpy()[1:]]
        self.dcache.toks += feed + new[:-1]          # the feed and d_1..d_{k-1} are cached
        drafts += new

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
                srv.toks += window[:n + 1]
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
