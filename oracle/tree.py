"""fp64 reference of token-tree verification -- several drafters' branches
verified in one target pass, with Algorithm 1's exact-match and j* rules.

Test infrastructure only (see the package header).

Algorithm 1 starts, after every token, one thread per drafter and one for the
target on the same prefix; the current verifier's token terminates every
thread whose token differs (the terminate step) and, among the threads that
agree, keeps the one of the smallest drafter index j* (the j* step).  With
lookahead, the drafters' proposals form a tree of tokens rooted at the last
committed token w0: node i has a parent p(i) < i (the root has none) and
stands for the prompt "committed prefix, then the tokens on the path from
the root to i".  One target pass computes every node's next-token logits
(each node attends to the prefix and to its own ancestors), and the walk
below is the exact-match verification of all branches at once:

  v = root; repeat: t = the target's greedy token at v (argmax, ties to the
  lowest id); among the children of v whose token is t take the one of
  smallest node index (children are numbered in drafter order: j*); stop
  when no child carries t.

The accepted path root = a_0, a_1, .., a_n gives n accepted drafts and the
next token is the target's greedy token at a_n; the committed cache then
holds the prefix, w0 and the tokens of a_1..a_n.
"""
from __future__ import annotations

import numpy as np

from .model import forward64


def validate_tree(parent) -> None:
    parent = [int(p) for p in parent]
    if not parent or parent[0] != -1:
        raise ValueError("node 0 is the root (parent -1)")
    for i, p in enumerate(parent[1:], 1):
        if not 0 <= p < i:
            raise ValueError(f"node {i}: the parent must be an earlier node")


def ancestors(parent, i: int) -> list:
    """The nodes from the root to i (inclusive)."""
    chain = []
    while i != -1:
        chain.append(i)
        i = int(parent[i])
    return chain[::-1]


def tree_logits64(s, get, cache, tokens, parent) -> np.ndarray:
    """Target logits [R][V] of every node: the forward over the cached prefix
    extended by the tokens on the node's root path (by definition, one
    ordinary causal forward per node)."""
    validate_tree(parent)
    R = len(tokens)
    out = np.zeros((R, s.vocab))
    for i in range(R):
        path = [int(tokens[j]) for j in ancestors(parent, i)]
        z, _ = forward64(s, get, path, cache)
        out[i] = z[-1]
    return out


def greedy64(z) -> int:
    """argmax, ties to the lowest id (np.argmax returns the first maximum)."""
    return int(np.argmax(np.asarray(z)))


def tree_walk(z, tokens, parent):
    """Exact-match verification of a token tree.  Returns (path, token, gap):
    the accepted node path from the root, the next token, and the smallest
    top-2 logit gap among the rows the walk looked at (how far a logit error
    is from changing a decision)."""
    validate_tree(parent)
    z = np.asarray(z, dtype=np.float64)
    children = {}
    for i, p in enumerate(parent):
        children.setdefault(int(p), []).append(i)
    path, v, gap = [0], 0, np.inf
    while True:
        row = z[v]
        t = greedy64(row)
        top2 = np.sort(row)[-2:] if len(row) > 1 else np.array([row[0], -np.inf])
        gap = min(gap, float(top2[1] - top2[0]))
        nxt = [c for c in children.get(v, []) if int(tokens[c]) == t]
        if not nxt:
            return path, t, gap
        v = min(nxt)
        path.append(v)
