"""The accept/reject kernels alone (dsi_accept) against the fp64 oracle on the
same logits: accepted counts and tokens must be bit-exact except at
positions the oracle flags (|a_i - u_i| < 1e-4, or u_{k+1} R within 1e-9 R of
a CDF boundary).  Vocabularies 1003 (ragged), 32000 and 128256."""
import numpy as np
import pytest
import torch

import dsi_synth as S
from oracle import verify64, softmax64
from paper_2405_14105_amd import dsi

pytestmark = pytest.mark.gpu

ACCEPT_FLAG = 1e-4
DRAW_FLAG = 1e-9


def _inputs(V, k, B, seed, zscale=1.28):
    shape = S.Shape("acc", 1, 32, 1, 1, 32, 32, V)
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((B * (k + 1), V)) * zscale).astype(np.float32)
    wi = S.window_inputs(shape, seed, B, k)
    return z, wi["tokens"], wi["q"], wi["u"]


def run_accept(z, tokens, q, u, mode=dsi.DSI_SAMPLE, T=1.0):
    dev = torch.device("cuda:0")
    B, k1 = tokens.shape
    V = z.shape[1]
    dz = torch.from_numpy(np.ascontiguousarray(z)).to(dev)
    dt = torch.from_numpy(np.ascontiguousarray(tokens, dtype=np.int32)).to(dev)
    dq = torch.from_numpy(np.ascontiguousarray(q, dtype=np.float32)).to(dev) if q is not None else None
    du = torch.from_numpy(np.ascontiguousarray(u, dtype=np.float32)).to(dev) if u is not None else None
    n = torch.full((B,), -7, dtype=torch.int32, device=dev)
    tok = torch.full((B,), -7, dtype=torch.int32, device=dev)
    dsi.dsi_accept(torch.cuda.current_stream().cuda_stream, B, k1 - 1, V, dz, dt, dq, du, n, tok, T, mode)
    torch.cuda.synchronize()
    return n.cpu().numpy(), tok.cpu().numpy()


def compare(z, tokens, q, u, n, tok, mode="sample", T=1.0):
    B, k1 = tokens.shape
    zz = z.reshape(B, k1, -1)
    flagged = 0
    for b in range(B):
        r = verify64(zz[b], tokens[b, 1:], None if q is None else q[b], None if u is None else u[b],
                     T, mode)
        if r.accept_margin < ACCEPT_FLAG or r.draw_margin < DRAW_FLAG:
            flagged += 1
            continue
        assert (int(n[b]), int(tok[b])) == (r.n, r.token), f"window {b}"
    return flagged


@pytest.mark.parametrize("V", [1003, 32000, 128256])
@pytest.mark.parametrize("k,B", [(0, 8), (1, 16), (5, 10), (10, 5)])
def test_sample_matches_oracle(V, k, B):
    z, tokens, q, u = _inputs(V, k, B, seed=V + k)
    n, tok = run_accept(z, tokens, q, u)
    assert compare(z, tokens, q, u, n, tok) <= max(1, B // 10)


@pytest.mark.parametrize("V", [1003, 128256])
@pytest.mark.parametrize("k,B", [(0, 8), (4, 12), (10, 5)])
def test_greedy_matches_oracle(V, k, B):
    z, tokens, _, _ = _inputs(V, k, B, seed=2 * V + k)
    # make some drafts match the target argmax so n > 0 occurs
    zz = z.reshape(B, k + 1, V)
    rng = np.random.default_rng(k)
    for b in range(B):
        for i in range(k):
            if rng.random() < 0.7:
                tokens[b, i + 1] = int(np.argmax(zz[b, i]))
    n, tok = run_accept(z, tokens, None, None, mode=dsi.DSI_GREEDY)
    assert compare(z, tokens, None, None, n, tok, mode="greedy") == 0
    if k > 0:
        assert (n > 0).any()


def test_greedy_ties_go_to_lowest_id():
    V, k, B = 5000, 2, 3
    z = np.zeros((B * (k + 1), V), np.float32)
    z[:, [17, 4097, 4999]] = 3.0          # ties across vocabulary chunks
    tokens = np.array([[0, 17, 17]] * B, np.int32)
    n, tok = run_accept(z, tokens, None, None, mode=dsi.DSI_GREEDY)
    assert (n == 2).all() and (tok == 17).all()


def test_forced_accept_q_equals_p():
    V, k, B = 32000, 6, 8
    z, tokens, _, u = _inputs(V, k, B, seed=5)
    zz = z.reshape(B, k + 1, V)
    q = np.stack([np.stack([softmax64(zz[b, i]) for i in range(k)]) for b in range(B)]).astype(np.float32)
    u = np.minimum(u, np.float32(0.999))
    n, tok = run_accept(z, tokens, q, u)
    assert compare(z, tokens, q, u, n, tok) == 0
    assert (n == k).all()


def test_forced_reject_at_first_draft():
    V, k, B = 32000, 4, 8
    z, tokens, q, u = _inputs(V, k, B, seed=6)
    u[:, 0] = np.float32(1.0 - 2.0 ** -24)
    zz = z.reshape(B, k + 1, V)
    for b in range(B):               # choose d_1 with p < q so a_1 < 1
        p = softmax64(zz[b, 0])
        tokens[b, 1] = int(np.argmax(q[b, 0] - p))
    n, tok = run_accept(z, tokens, q, u)
    assert compare(z, tokens, q, u, n, tok) == 0
    assert (n == 0).all()


def test_temperature():
    V, k, B = 1003, 3, 10
    z, tokens, q, u = _inputs(V, k, B, seed=7)
    n, tok = run_accept(z, tokens, q, u, T=0.6)
    assert compare(z, tokens, q, u, n, tok, T=0.6) <= 1


def test_invalid_inputs_flag_only_their_window():
    V, k, B = 1003, 3, 4
    z, tokens, q, u = _inputs(V, k, B, seed=8)
    tokens[1, 2] = V                  # draft id out of range
    q[2, 0, tokens[2, 1]] = 0.0       # q(d_1) = 0
    n, tok = run_accept(z, tokens, q, u)
    assert n[1] == -1 and tok[1] == -1
    assert n[2] == -1 and tok[2] == -1
    for b in (0, 3):
        r = verify64(z.reshape(B, k + 1, V)[b], tokens[b, 1:], q[b], u[b])
        assert (n[b], tok[b]) == (r.n, r.token)


def test_deterministic_across_runs():
    z, tokens, q, u = _inputs(128256, 10, 5, seed=9)
    a = run_accept(z, tokens, q, u)
    b = run_accept(z, tokens, q, u)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_first_token_is_distributed_as_target():
    """Lossless in expectation (Section 2): with d_1 ~ q_1 the first emitted
    token follows p_1.  64 windows per call share z and q; drafts and
    uniforms differ.  Chi-square over 12800 draws."""
    V, k, B, calls = 12, 1, 32, 400
    rng = np.random.default_rng(10)
    z1 = (rng.standard_normal(V) * 1.2).astype(np.float32)
    z = np.tile(z1, (B * (k + 1), 1))
    q1 = np.exp(rng.standard_normal(V))
    q1 = (q1 / q1.sum()).astype(np.float32)
    q = np.tile(q1, (B, k, 1))
    q64 = q1.astype(np.float64) / q1.astype(np.float64).sum()
    p = softmax64(z1)
    counts = np.zeros(V)
    for _ in range(calls):
        d = rng.choice(V, size=B, p=q64)
        tokens = np.stack([np.zeros(B, np.int32), d.astype(np.int32)], 1)
        u = (rng.integers(0, 1 << 24, size=(B, k + 1)) / float(1 << 24)).astype(np.float32)
        n, tok = run_accept(z, tokens, q, u)
        first = np.where(n >= 1, d, tok)
        np.add.at(counts, first, 1)
    N = counts.sum()
    chi2 = float(((counts - N * p) ** 2 / (N * p)).sum())
    # 11 degrees of freedom: P(chi2 > 40) < 1e-4
    assert chi2 < 40.0, (chi2, counts / N, p)
