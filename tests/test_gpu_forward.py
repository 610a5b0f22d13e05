"""End-to-end parity of dsi_prefill + dsi_verify against the fp64 oracle on
small models that span several MFMA tiles with ragged tails (vocab, d_ff,
query tiles, key chunks).

Gates:
  * logits: max |z_gpu - z_oracle| <= 1e-4 (fp32 models) or 2e-2 (bf16),
    the contract tolerances, and the regression gate of the shape (about ten
    times the error measured on it, tests/parity.py REG);
  * split check: the GPU's accept/reject on its own logits equals the
    oracle's verification of those same logits (flagged positions excluded);
  * end-to-end: equal to the oracle's verification of the oracle's logits
    except where the logit error delta could flip a decision; the single
    window tests take uniforms settled on the oracle's side (no decision
    within reach of the regression gate) and assert that both checks
    compared the decisions;
  * KV state: committed length L + n + 1, rollback, batch invariance.
"""
import numpy as np
import pytest
import torch

import dsi_synth as S
from oracle import forward64
from paper_2405_14105_amd import dsi

from gpu_rig import Rig
from parity import TOL, e2e_check, getter, oracle_logits, reg_of, settle_u, split_check, tol_of

pytestmark = pytest.mark.gpu

SEED = 0


CASES = [
    ("tiny", 64, 5),
    ("ragged_f32", 37, 4),
    ("ragged_bf16", 45, 6),
    ("gqa_hd64", 50, 3),
    ("mha_hd128", 70, 7),
    ("hd96_kvf32", 41, 5),
    ("f32w_bf16kv", 36, 4),
    # the 1B / 8B attention geometry on a small residual stream: the O
    # projection runs on its ring layout; the 717-position cache is read in
    # one key chunk of three steps per wave (no combine launch)
    ("o_ring_hd64", 700, 5),
    ("o_ring_hd128", 300, 10),
    # a 32-key step whose last key is position len + 1 (row 0's next key:
    # it must take the masked path) and one ending exactly at len (all its
    # keys visible to every row: mask-free); with ~64 keys a wrongly visible
    # key would carry ~1/64 of row 0's attention
    ("o_ring_hd128", 62, 10),
    ("o_ring_hd128", 63, 10),
    # a 9000-wide FFN: 161 gate/up ring workgroups, and the down projection
    # split four ways (the small shapes above split it at most twice)
    ("ring_wide_ff", 200, 6),
]


@pytest.mark.parametrize("name,L,k", CASES)
def test_verify_end_to_end(name, L, k):
    shape = S.SHAPES[name]
    tol, reg = tol_of(shape), reg_of(shape)
    prefix = S.prefix_tokens(shape, SEED, 0, L)
    wi = S.window_inputs(shape, SEED, 1, k)
    tokens, q = wi["tokens"], wi["q"]
    zo, ho = oracle_logits(shape, prefix, tokens[0], return_hidden=True)
    u = settle_u(zo, tokens[0], q[0], wi["u"][0], reg)[None]
    with Rig(shape, SEED, 1, L + 2 * (k + 1) + 5) as rig:
        rig.prefill(0, prefix)
        assert rig.length(0) == L
        out = rig.verify(0, tokens, q, u, commit=True, want_hidden=True)
        per_layer = [float(np.abs(out["hidden"][l] - ho[l]).max()) for l in range(shape.n_layers + 1)]
        delta = float(np.abs(out["logits"] - zo).max())
        print(f"{name}: max|dz| = {delta:.3g} (gate {reg:g}); hidden max err per layer {per_layer}")
        assert delta <= tol and delta <= reg
        assert split_check(out["logits"], tokens[0], q[0], u[0], out["n"][0], out["token"][0]) is not None
        assert e2e_check(zo, delta, tokens[0], q[0], u[0], out["n"][0], out["token"][0]) is not None
        assert 0 <= out["n"][0] <= k
        assert rig.length(0) == L + out["n"][0] + 1
        # greedy on the same window after rolling back: identical logits
        dsi.dsi_kv_rollback(rig.kv, 0, L)
        g = rig.verify(0, tokens, mode=dsi.DSI_GREEDY, commit=False)
        assert np.array_equal(g["logits"], out["logits"])
        assert split_check(g["logits"], tokens[0], None, None, g["n"][0], g["token"][0],
                           mode="greedy") is not None
        assert e2e_check(zo, delta, tokens[0], None, None, g["n"][0], g["token"][0], mode="greedy") is not None
        assert rig.length(0) == L


@pytest.mark.parametrize("name", ["tiny", "ragged_bf16", "hd96_kvf32"])
def test_prefill_last_logits(name):
    shape = S.SHAPES[name]
    L = 150                      # several 64-row prefill chunks plus a ragged one
    with Rig(shape, SEED, 1, L + 8) as rig:
        prefix = S.prefix_tokens(shape, SEED, 0, L)
        z = rig.prefill(0, prefix, want_logits=True)
        zo, _ = forward64(shape, getter(shape), prefix)
        d = float(np.abs(z - zo[-1]).max())
        print(f"{name}: prefill last-row max|dz| = {d:.3g}")
        assert d <= tol_of(shape) and d <= reg_of(shape)
        assert rig.length(0) == L


# Long caches split every (window, KV head) into several key chunks whose
# partials the combine launch folds; the chunk size follows the cache's
# capacity and window count (cdiv(max_len, 512 / (KV heads x query tiles))
# rounded up to whole workgroup steps; when that leaves several 32-key steps
# per wave, cdiv(max_len, 256 / (KV heads x query tiles))):
#   gqa_hd64, 1 x 1600: 8-wave workgroups, 256-key chunks, 6 chunks, the
#     last one 26 keys long;
#   ragged_bf16, 1 x 1600: 5 chunks of 256, 15 query rows in one tile;
#   gqa_hd64, 8 x 4400: many windows -- 4-wave workgroups with 128-key
#     chunks (8 chunks), verified on window 5 of the cache;
#   many_kv, 1 x 6000: 768-key chunks, three 32-key steps per wave, two
#     query tiles;
#   many_kv, 1 x 9000: 1280-key chunks, five steps per wave;
#   tiny (fp32 cache), 8 x 2100: the many-window 4-wave plan on an fp32
#     cache (128-key chunks), window 3;
#   tiny (fp32 cache), 1 x 33000: 768-key chunks, three steps per wave on
#     fp32 keys and values;
#   mha_hd128, 1 x 70000: one query tile with several steps per wave, so the
#     keys and values are streamed with nontemporal loads (768-key chunks,
#     three chunks);
#   o_ring_hd128 (head dim 128) at 8000 positions with k 10: three query
#     tiles whose single 1024-key chunk takes four steps per wave (the
#     kernel normalises its own output); with a 200-key prefix (one partial
#     step, a wave with no key at all); on window 1 of a three-window cache;
#   o_ring_hd64 at 12000 positions: two query tiles (k 7: 768-key chunks of
#     three steps per wave, the prefix spilling into a second chunk) and
#     four (k 15, whose single chunk takes six steps per wave);
#   o_ring_hd128 (k 10) and o_ring_hd64 (k 7) at 30000 positions with a
#     2300-key prefix: up to ten and eight steps per wave (3072- and
#     2048-key chunks) over mostly mask-free prefix steps.
@pytest.mark.parametrize("name,n_windows,max_len,win,L,k", [
    ("gqa_hd64", 1, 1600, 0, 1300, 5),
    ("ragged_bf16", 1, 1600, 0, 1100, 4),
    ("gqa_hd64", 8, 4400, 5, 1000, 5),
    ("many_kv", 1, 6000, 0, 1000, 7),
    ("many_kv", 1, 9000, 0, 2000, 7),
    ("tiny", 8, 2100, 3, 900, 5),
    ("tiny", 1, 33000, 0, 1500, 5),
    ("mha_hd128", 1, 70000, 0, 2000, 5),
    ("o_ring_hd128", 1, 8000, 0, 1000, 10),
    ("o_ring_hd128", 1, 8000, 0, 200, 10),
    ("o_ring_hd128", 3, 8000, 1, 1000, 10),
    ("o_ring_hd64", 1, 12000, 0, 1000, 7),
    ("o_ring_hd64", 1, 12000, 0, 1000, 15),
    ("o_ring_hd128", 1, 30000, 0, 2300, 10),
    ("o_ring_hd64", 1, 30000, 0, 2300, 7),
])
def test_multichunk_attention(name, n_windows, max_len, win, L, k):
    shape = S.SHAPES[name]
    tol, reg = tol_of(shape), reg_of(shape)
    prefix = S.prefix_tokens(shape, SEED, win, L)
    wi = S.window_inputs(shape, SEED, 1, k)
    tokens, q = wi["tokens"], wi["q"]
    zo = oracle_logits(shape, prefix, tokens[0])
    u = settle_u(zo, tokens[0], q[0], wi["u"][0], reg)[None]
    with Rig(shape, SEED, n_windows, max_len) as rig:
        rig.prefill(win, prefix)
        out = rig.verify(win, tokens, q, u, commit=True)
        delta = float(np.abs(out["logits"] - zo).max())
        print(f"{name} {n_windows}x{max_len}: max|dz| = {delta:.3g} (gate {reg:g})")
        assert delta <= tol and delta <= reg
        assert split_check(out["logits"], tokens[0], q[0], u[0], out["n"][0], out["token"][0]) is not None
        assert e2e_check(zo, delta, tokens[0], q[0], u[0], out["n"][0], out["token"][0]) is not None
        assert rig.length(win) == L + out["n"][0] + 1


def test_empty_prefix_and_k0():
    shape = S.SHAPES["ragged_bf16"]
    with Rig(shape, SEED, 1, 16) as rig:
        wi = S.window_inputs(shape, SEED, 1, 3)
        out = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=True)
        zo = oracle_logits(shape, [], wi["tokens"][0])
        delta = float(np.abs(out["logits"] - zo).max())
        assert delta <= TOL["bf16"]
        split_check(out["logits"], wi["tokens"][0], wi["q"][0], wi["u"][0], out["n"][0], out["token"][0])
        L1 = rig.length(0)
        # k = 0: one row, one token drawn from p_1
        t0 = np.array([[int(out["token"][0])]], np.int32)
        u0 = np.array([[0.3]], np.float32)
        o2 = rig.verify(0, t0, np.zeros((1, 0, shape.vocab), np.float32), u0, commit=True)
        assert o2["n"][0] == 0
        split_check(o2["logits"], t0[0], np.zeros((0, shape.vocab)), u0[0], o2["n"][0], o2["token"][0])
        assert rig.length(0) == L1 + 1


# lens, cache capacity: one key chunk; or 256-key chunks over a 1250-key
# prefix, where the 40-key window's later chunks hold no key at all (their
# partials carry max -inf and sum 0) and alone it takes the single-chunk
# path that normalises inside the attention kernel
# ... and with three and four row tiles (48 and 64 rows: four windows of 12
# and of 16 rows), where every GEMM role runs its several-row-tile ring
# kernel, also with fp32 weights and cache (tiny) and bf16 weights over an
# fp32 cache (hd96_kvf32): still bit-identical to each window alone
# ... and three 11-row windows of o_ring_hd128 over a 1200-position cache:
# 72 (window, KV head, query tile) workgroups of five 32-key steps read the
# cache in one key chunk each (no combine launch), as the 7-window 8B batch
# does, with the three-row-tile GEMMs.
@pytest.mark.parametrize("name,lens,cap,k", [("gqa_hd64", [20, 33, 47, 5], 64, 4),
                                             ("gqa_hd64", [300, 1250, 40], 1600, 4),
                                             ("gqa_hd64", [20, 33, 47, 5], 80, 11),
                                             ("o_ring_hd128", [40, 70, 25, 55], 100, 15),
                                             ("tiny", [30, 12, 50, 41], 80, 11),
                                             ("hd96_kvf32", [25, 60, 33, 8], 90, 15),
                                             ("o_ring_hd128", [1000, 1100, 950], 1200, 10)])
def test_batched_windows_ragged_and_batch_invariant(name, lens, cap, k):
    shape = S.SHAPES[name]
    B = len(lens)
    with Rig(shape, SEED, B, cap) as rig:
        prefixes = [S.prefix_tokens(shape, SEED, b, lens[b]) for b in range(B)]
        for b in range(B):
            rig.prefill(b, prefixes[b])
        wi = S.window_inputs(shape, SEED, B, k)
        out = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=False)
        V = shape.vocab
        zz = out["logits"].reshape(B, k + 1, V)
        for b in range(B):
            zo = oracle_logits(shape, prefixes[b], wi["tokens"][b])
            delta = float(np.abs(zz[b] - zo).max())
            assert delta <= tol_of(shape) and delta <= reg_of(shape), (b, delta)
            split_check(zz[b], wi["tokens"][b], wi["q"][b], wi["u"][b], out["n"][b], out["token"][b])
        # each window alone gives bit-identical logits and decisions
        for b in range(B):
            one = rig.verify(b, wi["tokens"][b:b + 1], wi["q"][b:b + 1], wi["u"][b:b + 1], commit=False)
            assert np.array_equal(one["logits"], zz[b])
            assert (one["n"][0], one["token"][0]) == (out["n"][b], out["token"][b])
        # commit the batch: every window advances by its own n + 1
        res = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=True)
        for b in range(B):
            assert rig.length(b) == lens[b] + res["n"][b] + 1


# Models created with DSI_RING=0 keep only the packed weight layout, so every
# GEMM runs the packed kernels (k_gemm_bf16: the two-set pipelined loop for
# one to three row tiles of QKV, O and gate/up, the batch loop otherwise) --
# the path of shapes without a ring layout (the 13B shape).  One, three and
# four row tiles, each window checked against the oracle and against itself
# verified alone.
@pytest.mark.parametrize("name,lens,k", [("o_ring_hd64", [300], 10), ("gqa_hd64", [20, 33, 47, 5], 11),
                                         ("o_ring_hd128", [40, 70, 25, 55], 15)])
def test_packed_kernels_without_ring(monkeypatch, name, lens, k):
    monkeypatch.setenv("DSI_RING", "0")
    shape = S.SHAPES[name]
    B = len(lens)
    with Rig(shape, SEED, B, max(lens) + k + 30) as rig:
        prefixes = [S.prefix_tokens(shape, SEED, b, lens[b]) for b in range(B)]
        for b in range(B):
            rig.prefill(b, prefixes[b])
        wi = S.window_inputs(shape, SEED, B, k)
        out = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=False)
        zz = out["logits"].reshape(B, k + 1, shape.vocab)
        for b in range(B):
            zo = oracle_logits(shape, prefixes[b], wi["tokens"][b])
            delta = float(np.abs(zz[b] - zo).max())
            print(f"{name} packed, window {b}: max|dz| = {delta:.3g}")
            assert delta <= TOL["bf16"] and delta <= reg_of(shape), (b, delta)
            split_check(zz[b], wi["tokens"][b], wi["q"][b], wi["u"][b], out["n"][b], out["token"][b])
            if B > 1:
                one = rig.verify(b, wi["tokens"][b:b + 1], wi["q"][b:b + 1], wi["u"][b:b + 1], commit=False)
                assert np.array_equal(one["logits"], zz[b])


def test_rollback_then_reverify_is_bit_identical():
    shape = S.SHAPES["ragged_bf16"]
    L, k = 30, 5
    with Rig(shape, SEED, 1, 64) as rig:
        rig.prefill(0, S.prefix_tokens(shape, SEED, 0, L))
        wi = S.window_inputs(shape, SEED, 1, k)
        a = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=True)
        # a second window on top of the accepted tokens
        wi2 = S.window_inputs(shape, SEED + 1, 1, k)
        rig.verify(0, wi2["tokens"], wi2["q"], wi2["u"], commit=True)
        dsi.dsi_kv_rollback(rig.kv, 0, L)
        assert rig.length(0) == L
        b = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=True)
        assert np.array_equal(a["logits"], b["logits"])
        assert (a["n"][0], a["token"][0]) == (b["n"][0], b["token"][0])


def test_capacity_and_invalid_inputs_leave_length_unchanged():
    shape = S.SHAPES["ragged_bf16"]
    L, k = 10, 4
    with Rig(shape, SEED, 1, L + k + 1) as rig:
        rig.prefill(0, S.prefix_tokens(shape, SEED, 0, L))
        wi = S.window_inputs(shape, SEED, 1, k)
        toks = wi["tokens"].copy()
        toks[0, 2] = shape.vocab + 5
        out = rig.verify(0, toks, wi["q"], wi["u"], commit=True)
        assert out["n"][0] == -1 and out["token"][0] == -1
        with pytest.raises(dsi.DsiError) as ei:
            rig.length(0)
        assert ei.value.status == dsi.DSI_EINVAL
        assert rig.length(0) == L
        # a full window fits exactly; one more row does not
        rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=False)
        wi5 = S.window_inputs(shape, SEED, 1, k + 1)
        with pytest.raises(dsi.DsiError) as ei:
            rig.verify(0, wi5["tokens"], wi5["q"], wi5["u"], commit=False)
        assert ei.value.status == dsi.DSI_ECAPACITY
        # rollback above the length is rejected on the host
        with pytest.raises(dsi.DsiError):
            dsi.dsi_kv_rollback(rig.kv, 0, L + 3)
        assert rig.length(0) == L


def test_kv_export_matches_oracle_cache():
    shape = S.SHAPES["gqa_hd64"]
    L = 40
    with Rig(shape, SEED, 2, 64) as rig:
        prefix = S.prefix_tokens(shape, SEED, 1, L)
        rig.prefill(1, prefix)
        _, cache = forward64(shape, getter(shape), prefix)
        for layer in range(shape.n_layers):
            kg, vg = rig.export_kv(1, layer, L)
            ko, vo = cache[layer]
            # bf16 storage: equal up to rounding flips.  Layer 0 sees the
            # exact embedding, so only ~0.1% of its entries flip; deeper
            # layers inherit the hidden-state differences those flips cause
            # (the KV rounding cascade), so more entries differ, each by a
            # few ulps at most.  A layout error would show O(1) differences.
            for g, o in ((kg, ko), (vg, vo)):
                diff = np.abs(g - o)
                frac = float(np.mean(diff > 0))
                print(f"layer {layer}: {frac:.4f} of entries differ, max {diff.max():.2e}")
                assert diff.max() <= 2.0 ** -6 * np.abs(o).max()
                if layer == 0:
                    assert frac < 0.005


@pytest.mark.parametrize("name", ["tiny_draft", "ragged_draft"])
def test_many_key_chunks_end_to_end(name):
    """A long prefix for a model with few KV heads splits the keys into more
    than 16 chunks (one KV head group, one query tile: 256-key chunks over
    ~4.4k keys), so the combine kernel folds the chunk partials in two
    batches and rescales between them."""
    shape = S.SHAPES[name]
    tol = TOL[shape.wdtype]
    L, k = 4380, 2
    with Rig(shape, SEED, 1, L + 2 * (k + 1) + 5) as rig:
        prefix = S.prefix_tokens(shape, SEED, 0, L)
        rig.prefill(0, prefix)
        wi = S.window_inputs(shape, SEED, 1, k)
        out = rig.verify(0, wi["tokens"], mode=dsi.DSI_GREEDY, commit=False)
    zo = oracle_logits(shape, prefix, wi["tokens"][0])
    delta = float(np.abs(out["logits"] - zo).max())
    print(f"{name}: L = {L}, max|dz| = {delta:.3g}")
    assert delta <= tol and delta <= reg_of(shape)
    assert split_check(out["logits"], wi["tokens"][0], None, None, out["n"][0], out["token"][0],
                       mode="greedy") is not None


def test_verify_at_the_row_maximum():
    """8 windows x (k = 7) + 1 = 64 rows, the most one call carries (four
    row tiles), ragged prefixes: logits against the oracle per window and
    each window alone bit-identical."""
    shape = S.SHAPES["ragged_f32"]
    B, k = 8, 7
    lens = [5 + 7 * b for b in range(B)]
    with Rig(shape, SEED, B, max(lens) + 2 * (k + 1) + 4) as rig:
        prefixes = [S.prefix_tokens(shape, SEED, b, lens[b]) for b in range(B)]
        for b in range(B):
            rig.prefill(b, prefixes[b])
        wi = S.window_inputs(shape, SEED, B, k)
        out = rig.verify(0, wi["tokens"], wi["q"], wi["u"], commit=False)
        z = out["logits"].reshape(B, k + 1, -1)
        for b in (0, 3, 7):
            one = rig.verify(b, wi["tokens"][b:b + 1], wi["q"][b:b + 1], wi["u"][b:b + 1], commit=False)
            assert np.array_equal(one["logits"], z[b])
    for b in range(B):
        zo = oracle_logits(shape, prefixes[b], wi["tokens"][b])
        assert np.abs(z[b] - zo).max() <= min(TOL["f32"], reg_of(shape)), b
        split_check(z[b], wi["tokens"][b], wi["q"][b], wi["u"][b], out["n"][b], out["token"][b])
