"""Seeded synthetic inputs for the DSI verification step.

This module is shared by the oracle and by the GPU path's tests and bench.
It holds no arithmetic of the verification method itself: it only draws
random-init model weights, prefix token ids, drafter distributions q, draft
tokens sampled from q (the drafter's side of speculative inference), and the
acceptance uniforms u.  Everything is a pure function of (seed, stream, layer,
tensor, window), so the oracle and the GPU path see identical arrays.

Workload shapes follow Llama-style decoders (the paper fixes no architecture:
its target models are off-the-shelf LMs treated as black boxes, Appendix B).
Distributions:
  * weights ~ N(0, 0.02) in fp32, then rounded to bf16 (RNE) for bf16 models;
  * RMSNorm gains = 1 for the named workloads (or 1 + 0.1 N(0,1) on request);
  * prefix ids and w0 uniform on [0, V);
  * drafter logits g ~ N(0,1)^V per position, q = softmax(2 g) in fp64 stored
    as fp32, draft d_i drawn from q_i by inverse CDF with its own uniform;
  * acceptance uniforms u = randint(0, 2^24) / 2^24 (exact in fp32 and fp64).
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

__all__ = [
    "Shape", "Workload", "SHAPES", "WORKLOADS", "LAYER_TENSORS", "GLOBAL_TENSORS",
    "tensor_shape", "weight", "weight_bf16_bits", "f32_to_bf16_bits",
    "prefix_tokens", "window_inputs", "all_weights",
]

# stream identifiers for SeedSequence entropy: keep stable forever
_S_WEIGHT, _S_PREFIX, _S_W0, _S_QLOGIT, _S_DRAFT, _S_U, _S_GAIN = 1, 2, 3, 4, 5, 6, 7


@dataclasses.dataclass(frozen=True)
class Shape:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-5
    wdtype: str = "bf16"     # "bf16" or "f32": storage type of every weight
    kvdtype: str = "bf16"    # "bf16" or "f32": storage type of the KV cache
    gains: str = "ones"      # "ones" or "random": RMSNorm gain vectors

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def n_params(self) -> int:
        d, ff, V = self.d_model, self.d_ff, self.vocab
        per_layer = d * (self.q_dim + 2 * self.kv_dim) + self.q_dim * d + 3 * d * ff + 2 * d
        return self.n_layers * per_layer + 2 * V * d + d


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: Shape
    prefix_lens: tuple      # cached length L_b of each window
    k: int                  # drafts per window
    temperature: float = 1.0

    @property
    def n_windows(self) -> int:
        return len(self.prefix_lens)


SHAPES = {
    # the fp32 tiny decoder: 2 layers, d 128, 4 MHA heads, SwiGLU 512, vocab 1024
    "tiny": Shape("tiny", 2, 128, 4, 4, 32, 512, 1024, wdtype="f32", kvdtype="f32"),
    # Llama-style 1B / 8B / 13B shapes in bf16
    "llama1b": Shape("llama1b", 16, 2048, 32, 8, 64, 8192, 32000),
    "llama8b": Shape("llama8b", 32, 4096, 32, 8, 128, 14336, 128256),
    "llama13b": Shape("llama13b", 40, 5120, 40, 40, 128, 13824, 32000),
    # small ragged shapes for parity tests: several tiles plus ragged tails in
    # every dimension that is not forced to a multiple of 32 (d_ff, vocab)
    "ragged_bf16": Shape("ragged_bf16", 2, 192, 6, 2, 32, 344, 1003, gains="random"),
    "ragged_f32": Shape("ragged_f32", 2, 160, 5, 5, 32, 300, 777, wdtype="f32",
                        kvdtype="f32", gains="random"),
    "gqa_hd64": Shape("gqa_hd64", 3, 256, 8, 2, 64, 688, 2050, gains="random"),
    "mha_hd128": Shape("mha_hd128", 2, 256, 2, 2, 128, 520, 1536, gains="random"),
    # mixed storage types and head_dim 96: bf16 weights over an fp32 cache,
    # fp32 weights over a bf16 cache
    "hd96_kvf32": Shape("hd96_kvf32", 2, 224, 3, 1, 96, 376, 1111, kvdtype="f32", gains="random"),
    "f32w_bf16kv": Shape("f32w_bf16kv", 2, 160, 4, 2, 64, 300, 901, wdtype="f32", gains="random"),
    # many KV heads and query tiles: few key chunks per (window, KV head),
    # so waves take several 32-key steps once the cache is a few thousand long
    "many_kv": Shape("many_kv", 2, 256, 64, 16, 32, 400, 1500, gains="random"),
    # the 1B / 8B attention geometry (32 query heads over 8 KV heads, head
    # dim 64 / 128) on a small residual stream: the O projection takes its
    # ring layout (one n-block per workgroup, 8 / 16 k-blocks per wave), as
    # at the full shapes
    "o_ring_hd64": Shape("o_ring_hd64", 2, 256, 32, 8, 64, 688, 2050, gains="random"),
    "o_ring_hd128": Shape("o_ring_hd128", 2, 256, 32, 8, 128, 344, 1003, gains="random"),
    # a wide FFN on a small residual stream: 1125 gate/up n-blocks in 161
    # ring workgroups of seven, and a four-way K split of the down projection
    "ring_wide_ff": Shape("ring_wide_ff", 2, 256, 8, 2, 64, 9000, 1500, gains="random"),
    # drafters: small models sharing a target's vocabulary
    "tiny_draft": Shape("tiny_draft", 1, 64, 2, 2, 32, 128, 1024, wdtype="f32", kvdtype="f32"),
    "ragged_draft": Shape("ragged_draft", 1, 96, 3, 1, 32, 200, 1003, gains="random"),
    "llama8b_draft": Shape("llama8b_draft", 2, 1024, 16, 4, 64, 2816, 128256),
}
# the drafter paired with each target shape (same vocabulary)
DRAFTERS = {"tiny": "tiny_draft", "ragged_bf16": "ragged_draft", "llama8b": "llama8b_draft"}
DRAFT_SEED_OFFSET = 1000   # drafter weights: seed + this, independent of the target's

WORKLOADS = {
    "tiny_k5": Workload("tiny_k5", SHAPES["tiny"], (64,), 5),
    "llama1b_L512_k5": Workload("llama1b_L512_k5", SHAPES["llama1b"], (512,), 5),
    "llama8b_L2048_k10": Workload("llama8b_L2048_k10", SHAPES["llama8b"], (2048,), 10),
    "llama8b_x7_L1024_k5": Workload("llama8b_x7_L1024_k5", SHAPES["llama8b"],
                                    tuple(1024 + i for i in range(7)), 5),
    "llama13b_L32768_k10": Workload("llama13b_L32768_k10", SHAPES["llama13b"], (32768,), 10),
}

LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
GLOBAL_TENSORS = ("embed", "final_norm", "lm_head")
_TENSOR_ID = {n: i + 1 for i, n in enumerate(GLOBAL_TENSORS + LAYER_TENSORS)}


def tensor_shape(s: Shape, name: str) -> tuple:
    """[out, in] row-major shape of a named tensor (gains are 1-D)."""
    d, ff, V = s.d_model, s.d_ff, s.vocab
    return {
        "embed": (V, d), "lm_head": (V, d), "final_norm": (d,),
        "attn_norm": (d,), "ffn_norm": (d,),
        "wq": (s.q_dim, d), "wk": (s.kv_dim, d), "wv": (s.kv_dim, d), "wo": (d, s.q_dim),
        "w_gate": (ff, d), "w_up": (ff, d), "w_down": (d, ff),
    }[name]


def _rng(*entropy) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(e) for e in entropy]))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round-to-nearest-even); return the uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def _bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


_CHUNK_ELEMS = 1 << 22
_POOL_THREADS = max(1, min(16, os.cpu_count() or 1))


def _normal_rows(seed: int, layer: int, tid: int, shape: tuple, std: float,
                 bf16: bool = False) -> np.ndarray:
    rows = shape[0]
    cols = int(np.prod(shape[1:])) if len(shape) > 1 else 1
    out = np.empty((rows, cols), dtype=np.float32)
    rows_per_chunk = max(1, _CHUNK_ELEMS // cols)
    starts = list(range(0, rows, rows_per_chunk))

    def fill(ci):
        r0 = starts[ci]
        r1 = min(rows, r0 + rows_per_chunk)
        g = _rng(seed, _S_WEIGHT, layer + 1, tid, ci)
        g.standard_normal(out=out[r0:r1], dtype=np.float32)
        out[r0:r1] *= np.float32(std)
        if bf16:
            # round-to-nearest-even to bf16, in place (same result as f32_to_bf16_bits)
            u = out[r0:r1].view(np.uint32)
            u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
            u &= np.uint32(0xFFFF0000)

    if len(starts) == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(min(_POOL_THREADS, len(starts))) as ex:
            list(ex.map(fill, range(len(starts))))
    return out.reshape(shape)


def weight(s: Shape, seed: int, layer: int, name: str) -> np.ndarray:
    """The fp32 values of a tensor; bf16-representable when s.wdtype == 'bf16'.

    layer = -1 for the global tensors (embed, final_norm, lm_head)."""
    shp = tensor_shape(s, name)
    tid = _TENSOR_ID[name]
    if name.endswith("_norm"):
        if s.gains == "ones":
            g = np.ones(shp, dtype=np.float32)
        else:
            g = (1.0 + 0.1 * _rng(seed, _S_GAIN, layer + 1, tid).standard_normal(shp)).astype(np.float32)
        return _bits_to_f32(f32_to_bf16_bits(g)) if s.wdtype == "bf16" else g
    return _normal_rows(seed, layer, tid, shp, 0.02, bf16=(s.wdtype == "bf16"))


def weight_bf16_bits(s: Shape, seed: int, layer: int, name: str) -> np.ndarray:
    """bf16 bit patterns (uint16) of weight(); exact, since the values are bf16."""
    w = weight(s, seed, layer, name)
    if s.wdtype != "bf16":
        return f32_to_bf16_bits(w)
    # the low halves are zero: keep the high 16 bits of each (little-endian) fp32
    flat = w.reshape(-1).view(np.uint16)
    out = np.empty(w.size, dtype=np.uint16)
    step = _CHUNK_ELEMS
    spans = [(i, min(w.size, i + step)) for i in range(0, w.size, step)]

    def cut(span):
        a, b = span
        out[a:b] = flat[2 * a + 1:2 * b:2]

    if len(spans) == 1:
        cut(spans[0])
    else:
        with ThreadPoolExecutor(min(_POOL_THREADS, len(spans))) as ex:
            list(ex.map(cut, spans))
    return out.reshape(w.shape)


def all_weights(s: Shape, seed: int) -> dict:
    """Every tensor of a (small) model as {(layer, name): fp32 array}."""
    out = {(-1, n): weight(s, seed, -1, n) for n in GLOBAL_TENSORS}
    for l in range(s.n_layers):
        for n in LAYER_TENSORS:
            out[(l, n)] = weight(s, seed, l, n)
    return out


def prefix_tokens(s: Shape, seed: int, window: int, length: int) -> np.ndarray:
    """Uniform random prefix ids for one window (int32)."""
    return _rng(seed, _S_PREFIX, window).integers(0, s.vocab, size=length, dtype=np.int64).astype(np.int32)


def window_inputs(s: Shape, seed: int, n_windows: int, k: int, window0: int = 0,
                  q_scale: float = 2.0) -> dict:
    """Per-window verification inputs.

    Returns w0 [B] (the committed-but-uncached token), drafts [B][k],
    tokens [B][k+1] = (w0, d_1..d_k), q [B][k][V] fp32, u [B][k+1] fp32."""
    V = s.vocab
    B = n_windows
    w0 = np.empty(B, np.int32)
    drafts = np.empty((B, k), np.int32)
    q = np.empty((B, k, V), np.float32)
    u = np.empty((B, k + 1), np.float32)
    for b in range(B):
        wid = window0 + b
        w0[b] = _rng(seed, _S_W0, wid).integers(0, V)
        gq = _rng(seed, _S_QLOGIT, wid)
        gd = _rng(seed, _S_DRAFT, wid)
        for i in range(k):
            g = gq.standard_normal(V) * q_scale
            e = np.exp(g - g.max())
            qi = e / e.sum()
            q[b, i] = qi.astype(np.float32)
            c = np.cumsum(q[b, i].astype(np.float64))
            r = gd.random() * c[-1]
            drafts[b, i] = min(int(np.searchsorted(c, r, side="right")), V - 1)
        u[b] = (_rng(seed, _S_U, wid).integers(0, 1 << 24, size=k + 1) / float(1 << 24)).astype(np.float32)
    tokens = np.concatenate([w0[:, None], drafts], axis=1).astype(np.int32)
    return {"w0": w0, "drafts": drafts, "tokens": tokens, "q": q, "u": u}
