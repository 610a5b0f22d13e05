"""fp64 reference of the target forward over a verification window.

Speculative inference sends the k+1 prompts x'_{<=i}, i = 0..k, to the target
as one batch and gets k+1 logit rows back (Section 2, "Speculative Inference").
With a KV cache holding the committed prefix, those k+1 prompts are exactly
the window rows (w0, d_1..d_k) at absolute positions L..L+k, each attending to
the cached prefix and to the window rows before it.  Prompts are the
unpadded suffix of the input (Appendix B), so positions start at 0.

The target LM itself is a black box in the paper (Appendix B: f maps a prompt
to V logits).  This oracle fixes a Llama-style decoder:
  pre-norm RMSNorm  y = x / sqrt(mean(x^2) + eps) * g
  rotate-half RoPE  (x1 + i x2) * exp(i * pos * base^(-2j/hd)), j < hd/2
  causal softmax attention, scale 1/sqrt(hd), query head h reads KV head
  h // (n_heads / n_kv_heads)
  SwiGLU FFN        down(silu(gate h) * up h), silu(x) = x / (1 + e^-x)
  final RMSNorm and an untied LM head; no biases; weights [out, in].

Everything is computed in fp64.  When the KV cache is stored in bf16, K (after
RoPE) and V are rounded to bf16 (round-to-nearest-even) before attention, for
every position, because attention reads them from that cache.

The weights come from a callable get(layer, name) -> array (layer -1 for the
embedding, final norm and LM head), so large models can be streamed layer by
layer.  Nothing here blocks, fuses or reorders beyond the definitions above.
"""
from __future__ import annotations

import numpy as np


def bf16_round64(x) -> np.ndarray:
    """Round to the nearest bf16 value (8 significant bits), ties to even.

    Written from the format's definition: x = m 2^e with 0.5 <= |m| < 1, keep
    8 significant bits of m with round-half-even (np.rint).  bf16 shares the
    fp32 exponent range, so no subnormal or overflow handling is needed for
    the magnitudes a forward produces."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def rmsnorm64(x, g, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, dtype=np.float64)


def rope64(x, pos, base: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [T, H, hd] at absolute positions pos [T].

    Pair j (j < hd/2) is (x[j], x[j + hd/2]) rotated by the angle
    pos * base^(-2j/hd)."""
    x = np.asarray(x, dtype=np.float64)
    hd = x.shape[-1]
    half = hd // 2
    j = np.arange(half, dtype=np.float64)
    inv_freq = np.power(float(base), -2.0 * j / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention64(q, k, v, q_pos, k_pos) -> np.ndarray:
    """Causal multi-head attention with grouped KV heads.

    q [T, Hq, hd], k and v [S, Hkv, hd]; query t sees key s iff
    k_pos[s] <= q_pos[t].  Returns [T, Hq, hd]."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    T, Hq, hd = q.shape
    Hkv = k.shape[1]
    group = Hq // Hkv
    allowed = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]   # [T, S]
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    for h in range(Hq):
        kh = h // group
        sc = (q[:, h, :] @ k[:, kh, :].T) * scale
        sc = np.where(allowed, sc, -np.inf)
        sc = sc - sc.max(axis=1, keepdims=True)
        w = np.exp(sc)
        w = w / w.sum(axis=1, keepdims=True)
        out[:, h, :] = w @ v[:, kh, :]
    return out


def silu64(x) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    with np.errstate(over="ignore"):
        return x / (1.0 + np.exp(-x))


def _w(get, layer, name):
    return np.asarray(get(layer, name), dtype=np.float64)


def embed64(get, tokens) -> np.ndarray:
    """Embedding rows E[w] of the token ids."""
    E = get(-1, "embed")
    return np.asarray(E[np.asarray(tokens, dtype=np.int64)], dtype=np.float64)


def layer64(s, get, l, x, pos, k_prev=None, v_prev=None, kprev_pos=None):
    """One decoder layer over rows x [T, d] at positions pos [T].

    k_prev / v_prev [S, Hkv, hd] are the cached keys/values (already in their
    stored precision) at positions kprev_pos (default 0..S-1).  Returns
    (x_out [T, d], k_new [T, Hkv, hd], v_new [T, Hkv, hd]) where k_new and
    v_new are the rows this layer appends to the cache, rounded to bf16 when
    s.kvdtype == 'bf16'."""
    x = np.asarray(x, dtype=np.float64)
    T = x.shape[0]
    hq, hkv, hd = s.n_heads, s.n_kv_heads, s.head_dim
    pos = np.asarray(pos, dtype=np.int64)
    h = rmsnorm64(x, _w(get, l, "attn_norm"), s.rms_eps)
    q = (h @ _w(get, l, "wq").T).reshape(T, hq, hd)
    kk = (h @ _w(get, l, "wk").T).reshape(T, hkv, hd)
    vv = (h @ _w(get, l, "wv").T).reshape(T, hkv, hd)
    q = rope64(q, pos, s.rope_base)
    kk = rope64(kk, pos, s.rope_base)
    if s.kvdtype == "bf16":
        kk = bf16_round64(kk)
        vv = bf16_round64(vv)
    if k_prev is not None and len(k_prev):
        S = k_prev.shape[0]
        kpos = np.arange(S) if kprev_pos is None else np.asarray(kprev_pos)
        K = np.concatenate([np.asarray(k_prev, dtype=np.float64), kk], axis=0)
        Vv = np.concatenate([np.asarray(v_prev, dtype=np.float64), vv], axis=0)
        kp = np.concatenate([kpos, pos])
    else:
        K, Vv, kp = kk, vv, pos
    o = attention64(q, K, Vv, pos, kp).reshape(T, hq * hd)
    x = x + o @ _w(get, l, "wo").T
    h2 = rmsnorm64(x, _w(get, l, "ffn_norm"), s.rms_eps)
    a = silu64(h2 @ _w(get, l, "w_gate").T) * (h2 @ _w(get, l, "w_up").T)
    x = x + a @ _w(get, l, "w_down").T
    return x, kk, vv


def head64(s, get, x) -> np.ndarray:
    """Final RMSNorm and LM head: logits [T, V]."""
    h = rmsnorm64(x, _w(get, -1, "final_norm"), s.rms_eps)
    return h @ _w(get, -1, "lm_head").T


def forward64(s, get, tokens, cache=None, return_hidden=False):
    """Forward of `tokens` appended after the cached prefix.

    cache: None (empty prefix) or a list over layers of (K, V) arrays
    [S, Hkv, hd] holding positions 0..S-1.  Returns (logits [T, V], new_cache)
    where new_cache holds positions 0..S+T-1; with return_hidden, also the
    residual stream entering each layer and entering the head:
    hidden [n_layers + 1, T, d]."""
    tokens = np.asarray(tokens, dtype=np.int64)
    T = tokens.shape[0]
    S = 0 if cache is None else cache[0][0].shape[0]
    pos = np.arange(S, S + T)
    x = embed64(get, tokens)
    new_cache = []
    hidden = [x]
    for l in range(s.n_layers):
        kp, vp = (None, None) if cache is None else cache[l]
        x, kn, vn = layer64(s, get, l, x, pos, kp, vp)
        if kp is None:
            new_cache.append((kn, vn))
        else:
            new_cache.append((np.concatenate([kp, kn]), np.concatenate([vp, vn])))
        hidden.append(x)
    logits = head64(s, get, x)
    if return_hidden:
        return logits, new_cache, np.stack(hidden)
    return logits, new_cache
