"""Token-tree verification (dsi_verify_tree) against the oracle
(oracle/tree.py): several drafters' branches verified in one target pass
with the exact-match and j* rules of Algorithm 1.

Gates:
  * logits: every node's logits within the logit tolerance of the oracle's
    (one causal forward over the prefix and the node's root path);
  * split check: the GPU's path and token equal the oracle walk over the
    GPU's own logits, bit-exactly (argmax over the same fp32 values);
  * end-to-end: equal to the oracle walk over the oracle's logits unless a
    visited row's top-2 gap is within 2 delta;
  * chain tree: bit-identical to dsi_verify greedy on the same window;
  * commit: the compacted cache equals the oracle's cache of the prefix
    extended by the accepted path, and the window verifies on from there;
  * batch invariance and input errors.
"""
import numpy as np
import pytest
import torch

import dsi_synth as S
from oracle import forward64, greedy64, tree_logits64, tree_walk
from paper_2405_14105_amd import dsi

from gpu_rig import Rig
from parity import TOL, getter, tol_of

pytestmark = pytest.mark.gpu

SEED = 0


def greedy_chain(shape, get, cache, w0, n):
    """The oracle's greedy continuation g_1..g_n of prefix + w0."""
    g = []
    for _ in range(n):
        z, _ = forward64(shape, get, [w0] + g, cache)
        g.append(greedy64(z[-1]))
    return g


def branchy_tree(w0, g, V, rng):
    """Eleven nodes in four branches around the greedy chain g: a wrong
    branch first, then two siblings that both carry g_1 (the smaller index
    wins, the j* rule), a wrong and a right child under the winner, and a
    continuation two levels deeper.  Path if the target agrees with g:
    0 -> 3 -> 5 -> 8, next token g_4."""
    def other(t):
        r = int(rng.integers(0, V))
        return r if r != t else (r + 1) % V
    toks = [w0, other(g[0]), other(g[1]), g[0], other(g[1]), g[1], g[0], g[1], g[2], other(g[3]),
            other(g[2])]
    par = [-1, 0, 1, 0, 3, 3, 0, 6, 5, 8, 5]
    return np.array(toks, np.int32), np.array(par, np.int32)


def kv_close(rig, window, shape, cache, n_rows):
    """Exported K/V of a window against an oracle cache (rounding-level)."""
    rel = 2.0 ** -6 if shape.kvdtype == "bf16" else 1e-4
    for layer in range(shape.n_layers):
        kg, vg = rig.export_kv(window, layer, n_rows)
        ko, vo = cache[layer]
        for g, o in ((kg, ko[:n_rows]), (vg, vo[:n_rows])):
            err = float(np.abs(g - o).max())
            assert err <= rel * float(np.abs(o).max()), (layer, err)


# cap: cache capacity (None: just room for the tree); gqa_hd64 with 1600
# positions splits the 1200-key prefix into 5 key chunks of 256, so the tree
# mask meets the chunk partials and their combine; with 11300 positions the
# plan takes 4-wave workgroups and 128-key chunks (10 of them); many_kv with
# 6000 positions and a 2000-key prefix: two chunks of 1280 or 1536 keys
# (three or four query tiles), five or six steps per wave; gqa_hd64 with a
# 500-key prefix and room for the tree only: one key chunk whose waves take
# two or three pipelined steps under the tree mask, normalised in the kernel
@pytest.mark.parametrize("name,L,cap", [("tiny", 40, None), ("ragged_bf16", 33, None),
                                        ("gqa_hd64", 70, None), ("hd96_kvf32", 30, None),
                                        ("f32w_bf16kv", 25, None), ("gqa_hd64", 1200, 1600),
                                        ("gqa_hd64", 1200, 11300), ("many_kv", 2000, 6000),
                                        ("gqa_hd64", 500, None)])
def test_tree_matches_oracle_and_commits(name, L, cap):
    shape = S.SHAPES[name]
    tol = tol_of(shape)
    get = getter(shape, SEED)
    prefix = S.prefix_tokens(shape, SEED, 0, L)
    _, cache = forward64(shape, get, prefix)
    w0 = 11
    g = greedy_chain(shape, get, cache, w0, 4)
    rng = np.random.default_rng(3)
    tokens, parent = branchy_tree(w0, g, shape.vocab, rng)
    R = len(tokens)
    zo = tree_logits64(shape, get, cache, tokens, parent)
    with Rig(shape, SEED, 1, cap or L + 2 * R + 8) as rig:
        rig.prefill(0, prefix)
        out = rig.verify_tree(0, tokens[None], parent[None], commit=True)
        z = out["logits"]
        delta = float(np.abs(z - zo).max())
        print(f"{name}: max|dz| over {R} nodes = {delta:.3g}")
        assert delta <= tol
        n, tok, path = int(out["n"][0]), int(out["token"][0]), out["path"][0]
        # split check: the walk over the GPU's own logits, exactly
        p_own, t_own, _ = tree_walk(z, tokens, parent)
        assert list(path[:n + 1]) == p_own and tok == t_own
        assert (path[n + 1:] == -1).all()
        # end to end, unless a visited row is within the error of a tie
        p_o, t_o, gap = tree_walk(zo, tokens, parent)
        if gap > 2 * delta:
            assert list(path[:n + 1]) == p_o and tok == t_o
            assert p_o == [0, 3, 5, 8] and t_o == g[3]
        # commit: cache = prefix, w0 and the path's tokens, in order
        assert rig.length(0) == L + n + 1
        seq = [int(tokens[a]) for a in path[:n + 1]]
        _, cache2 = forward64(shape, get, seq, cache)
        kv_close(rig, 0, shape, cache2, L + n + 1)
        # and the window verifies on from the committed state
        nxt = [tok, int(rng.integers(0, shape.vocab)), int(rng.integers(0, shape.vocab))]
        v = rig.verify(0, np.array([nxt], np.int32), mode=dsi.DSI_GREEDY, commit=False)
        zo2, _ = forward64(shape, get, nxt, cache2)
        d2 = float(np.abs(v["logits"] - zo2).max())
        print(f"{name}: after commit max|dz| = {d2:.3g}")
        assert d2 <= tol


@pytest.mark.parametrize("name", ["tiny", "ragged_bf16"])
def test_chain_tree_is_bit_identical_to_greedy_verify(name):
    shape = S.SHAPES[name]
    L, k = 29, 6
    prefix = S.prefix_tokens(shape, SEED, 1, L)
    get = getter(shape, SEED)
    _, cache = forward64(shape, get, prefix)
    w0 = 7
    g = greedy_chain(shape, get, cache, w0, 3)
    rng = np.random.default_rng(5)
    tokens = np.array([w0] + g + list(rng.integers(0, shape.vocab, k - 3)), np.int32)
    parent = np.arange(-1, k, dtype=np.int32)
    with Rig(shape, SEED, 2, L + 2 * (k + 1) + 4) as rig:
        rig.prefill(0, prefix)
        rig.prefill(1, prefix)
        a = rig.verify(0, tokens[None], mode=dsi.DSI_GREEDY, commit=True)
        b = rig.verify_tree(1, tokens[None], parent[None], commit=True)
        assert np.array_equal(a["logits"], b["logits"])
        n = int(a["n"][0])
        assert int(b["n"][0]) == n and int(b["token"][0]) == int(a["token"][0])
        assert list(b["path"][0]) == list(range(n + 1)) + [-1] * (k - n)
        assert rig.length(0) == rig.length(1) == L + n + 1
        for layer in range(shape.n_layers):
            ka, va = rig.export_kv(0, layer, L + n + 1)
            kb, vb = rig.export_kv(1, layer, L + n + 1)
            assert np.array_equal(ka, kb) and np.array_equal(va, vb)


def test_single_node_tree():
    """n_nodes = 1: no drafts; the token is the target's greedy token after w0."""
    shape = S.SHAPES["tiny"]
    L = 20
    prefix = S.prefix_tokens(shape, SEED, 2, L)
    get = getter(shape, SEED)
    _, cache = forward64(shape, get, prefix)
    with Rig(shape, SEED, 1, L + 4) as rig:
        rig.prefill(0, prefix)
        out = rig.verify_tree(0, np.array([[9]], np.int32), np.array([[-1]], np.int32))
        assert int(out["n"][0]) == 0 and list(out["path"][0]) == [0]
        z, _ = forward64(shape, get, [9], cache)
        assert np.abs(out["logits"][0] - z[0]).max() <= TOL["f32"]
        assert int(out["token"][0]) == greedy64(out["logits"][0])
        assert rig.length(0) == L + 1


def test_batched_trees_are_batch_invariant():
    """Two windows with different prefixes and trees in one call give the
    same bits as each window alone."""
    shape = S.SHAPES["ragged_bf16"]
    R = 9
    rng = np.random.default_rng(8)
    Ls = [25, 41]
    parents = [np.array([-1, 0, 0, 1, 1, 2, 3, 6, 0], np.int32),
               np.array([-1, 0, 1, 2, 0, 4, 4, 1, 7], np.int32)]
    tokens = [rng.integers(0, shape.vocab, R).astype(np.int32) for _ in range(2)]
    with Rig(shape, SEED, 2, 64) as rig:
        for w in range(2):
            rig.prefill(w, S.prefix_tokens(shape, SEED, w, Ls[w]))
        both = rig.verify_tree(0, np.stack(tokens), np.stack(parents), commit=False)
        for w in range(2):
            one = rig.verify_tree(w, tokens[w][None], parents[w][None], commit=False)
            assert np.array_equal(one["logits"], both["logits"][w * R:(w + 1) * R])
            assert np.array_equal(one["path"][0], both["path"][w])
            assert int(one["n"][0]) == int(both["n"][w])
            assert int(one["token"][0]) == int(both["token"][w])
            p_own, t_own, _ = tree_walk(both["logits"][w * R:(w + 1) * R], tokens[w], parents[w])
            assert list(both["path"][w][:int(both["n"][w]) + 1]) == p_own
            assert int(both["token"][w]) == t_own
            assert rig.length(w) == Ls[w]


def test_tree_input_errors():
    shape = S.SHAPES["tiny"]
    L = 10
    with Rig(shape, SEED, 1, 24) as rig:
        rig.prefill(0, S.prefix_tokens(shape, SEED, 0, L))
        toks = np.array([[3, 4, 5, 6]], np.int32)
        # device-detected: a parent that is not an earlier node, a root with
        # a parent, a token outside [0, V)
        for par, tk in (([-1, 0, 3, 1], toks), ([0, 0, 1, 2], toks),
                        ([-1, 0, 1, 1], np.array([[3, 4, shape.vocab, 6]], np.int32))):
            out = rig.verify_tree(0, tk, np.array([par], np.int32), commit=True)
            assert int(out["n"][0]) == -1 and int(out["token"][0]) == -1
            assert (out["path"][0] == -1).all()
            with pytest.raises(dsi.DsiError) as ei:
                rig.length(0)
            assert ei.value.status == dsi.DSI_EINVAL
            assert rig.length(0) == L
        # host-detected, nothing enqueued
        dev = rig.dev
        t = rig.dev_i32(np.zeros((1, 20), np.int32))
        p = rig.dev_i32(np.arange(-1, 19, dtype=np.int32)[None])
        path = torch.zeros((1, 20), dtype=torch.int32, device=dev)
        n = torch.zeros(1, dtype=torch.int32, device=dev)
        tok = torch.zeros(1, dtype=torch.int32, device=dev)
        with pytest.raises(dsi.DsiError) as ei:        # 10 + 20 > 24
            dsi.dsi_verify_tree(rig.model, rig.kv, 0, 1, 20, t, p, path, n, tok, True)
        assert ei.value.status == dsi.DSI_ECAPACITY
        for args in ((0, 1, 0), (0, 2, 4), (-1, 1, 4), (0, 1, 65)):
            with pytest.raises(dsi.DsiError) as ei:
                dsi.dsi_verify_tree(rig.model, rig.kv, *args, t, p, path, n, tok, True)
            assert ei.value.status == dsi.DSI_EINVAL
        with pytest.raises(dsi.DsiError) as ei:
            dsi.dsi_verify_tree(rig.model, rig.kv, 0, 1, 4, t, None, path, n, tok, True)
        assert ei.value.status == dsi.DSI_EINVAL
        assert rig.length(0) == L


def test_full_64_node_tree():
    """The largest tree (64 nodes: all four row tiles, ancestor bit 63), a
    random shape with long and short branches, against the oracle."""
    shape = S.SHAPES["tiny"]
    L, R = 21, 64
    rng = np.random.default_rng(17)
    parent = np.array([-1] + [int(rng.integers(max(0, i - 6), i)) for i in range(1, R)], np.int32)
    parent[63] = 62                                  # a deep chain ending at node 63
    tokens = rng.integers(0, shape.vocab, R).astype(np.int32)
    get = getter(shape, SEED)
    prefix = S.prefix_tokens(shape, SEED, 3, L)
    _, cache = forward64(shape, get, prefix)
    zo = tree_logits64(shape, get, cache, tokens, parent)
    with Rig(shape, SEED, 1, L + R + 4) as rig:
        rig.prefill(0, prefix)
        out = rig.verify_tree(0, tokens[None], parent[None], commit=True)
        z = out["logits"]
        delta = float(np.abs(z - zo).max())
        print(f"64-node tree: max|dz| = {delta:.3g}")
        assert delta <= TOL["f32"]
        n, tok, path = int(out["n"][0]), int(out["token"][0]), out["path"][0]
        p_own, t_own, _ = tree_walk(z, tokens, parent)
        assert list(path[:n + 1]) == p_own and tok == t_own
        assert rig.length(0) == L + n + 1
