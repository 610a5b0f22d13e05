"""Pins of the token-tree oracle (oracle/tree.py): exact-match verification of
several drafters' branches with Algorithm 1's j* rule."""
import numpy as np
import pytest

import dsi_synth as S
from oracle import forward64, verify64
from oracle.tree import ancestors, tree_logits64, tree_walk, validate_tree


def greedy_continuation(s, get, prefix, w0, n):
    out, seq = [], list(prefix) + [int(w0)]
    for _ in range(n):
        z, _ = forward64(s, get, seq)
        t = int(np.argmax(z[-1]))
        out.append(t)
        seq.append(t)
    return out


def random_tree(rng, R, V, greedy=None):
    """A random tree of R nodes; if greedy is given, one branch follows it."""
    parent, tokens = [-1], [int(rng.integers(V))]
    if greedy:
        for i, t in enumerate(greedy):
            parent.append(i)
            tokens.append(int(t))
    while len(parent) < R:
        parent.append(int(rng.integers(len(parent))))
        tokens.append(int(rng.integers(V)))
    return tokens, parent


def test_chain_tree_equals_greedy_verification():
    rng = np.random.default_rng(0)
    for _ in range(50):
        R, V = 6, 7
        z = rng.standard_normal((R, V))
        tokens = [int(rng.integers(V)) for _ in range(R)]
        # make some drafts match the argmax so that acceptance varies
        for i in range(1, R):
            if rng.random() < 0.6:
                tokens[i] = int(np.argmax(z[i - 1]))
        path, tok, _ = tree_walk(z, tokens, [-1] + list(range(R - 1)))
        r = verify64(z, tokens[1:], mode="greedy")
        assert (len(path) - 1, tok) == (r.n, r.token)
        assert path == list(range(len(path)))


def test_jstar_takes_the_smallest_matching_child():
    z = np.zeros((5, 4))
    z[0, 2] = 1.0                  # root's greedy token: 2
    z[2, 3] = 1.0
    z[3, 1] = 1.0
    tokens = [0, 2, 2, 2, 3]
    parent = [-1, 0, 0, 0, 2]      # children 1, 2, 3 of the root all carry 2
    path, tok, _ = tree_walk(z, tokens, parent)
    assert path == [0, 1] and tok == int(np.argmax(z[1]))
    # without node 1 the next smallest (2) is kept and its child 4 follows
    path, tok, _ = tree_walk(z[[0, 2, 3, 4]], [0, 2, 2, 3], [-1, 0, 0, 1])
    assert path == [0, 1, 3] and tok == 0


def test_tree_output_is_the_target_greedy_continuation():
    """Theorem 1 for trees: the accepted tokens and the next token are
    exactly the target's own greedy tokens, for any tree."""
    s = S.SHAPES["ragged_f32"]
    get = lambda l, n: S.weight(s, 5, l, n).astype(np.float64)
    prefix = list(S.prefix_tokens(s, 5, 0, 9))
    _, cache = forward64(s, get, prefix)
    rng = np.random.default_rng(1)
    w0 = 42
    g = greedy_continuation(s, get, prefix, w0, 4)
    for trial in range(6):
        m = trial % 4                                   # a greedy branch of length m
        tokens, parent = random_tree(rng, 9, s.vocab, greedy=g[:m])
        tokens[0] = w0
        z = tree_logits64(s, get, cache, tokens, parent)
        path, tok, _ = tree_walk(z, tokens, parent)
        n = len(path) - 1
        assert n >= m                                   # the greedy branch is accepted
        assert [tokens[a] for a in path[1:]] + [tok] == greedy_continuation(s, get, prefix, w0, n + 1)


def test_node_logits_ignore_other_branches():
    s = S.SHAPES["tiny"]
    get = lambda l, n: S.weight(s, 6, l, n).astype(np.float64)
    prefix = list(S.prefix_tokens(s, 6, 0, 7))
    _, cache = forward64(s, get, prefix)
    tokens, parent = [3, 5, 9, 11, 4], [-1, 0, 0, 1, 2]
    z = tree_logits64(s, get, cache, tokens, parent)
    z2 = tree_logits64(s, get, cache, tokens[:2] + tokens[3:4], [-1, 0, 1])
    assert np.array_equal(z[[0, 1, 3]], z2)
    assert ancestors(parent, 4) == [0, 2, 4]


def test_invalid_trees_raise():
    for bad in ([0, 0], [-1, 1], [-1, 0, 3], []):
        with pytest.raises(ValueError):
            validate_tree(bad)
