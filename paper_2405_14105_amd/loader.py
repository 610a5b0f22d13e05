"""Upload host weight arrays into a dsi_model (marshalling only)."""
from __future__ import annotations

import numpy as np

from . import dsi

LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
GLOBAL_TENSORS = ("embed", "final_norm", "lm_head")


def config_for(shape) -> dsi.dsi_config:
    """dsi_config from any object with the decoder-shape attributes."""
    dt = {"bf16": dsi.DSI_BF16, "f32": dsi.DSI_F32}
    return dsi.make_config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                           shape.head_dim, shape.d_ff, shape.vocab, shape.rope_base, shape.rms_eps,
                           dt[shape.wdtype], dt[shape.kvdtype])


def upload(model: int, shape, tensor_fn) -> None:
    """tensor_fn(layer, name) -> host array in the model's storage format:
    uint16 bf16 bit patterns for bf16 models, float32 for fp32 models."""
    want = np.uint16 if shape.wdtype == "bf16" else np.float32

    def put(layer, name):
        a = np.ascontiguousarray(tensor_fn(layer, name))
        if a.dtype != want:
            raise TypeError(f"{name}: expected {want}, got {a.dtype}")
        dsi.dsi_model_set_tensor(model, layer, dsi.TENSOR_IDS[name], a.ctypes.data, a.nbytes, False)

    for name in GLOBAL_TENSORS:
        put(-1, name)
    for layer in range(shape.n_layers):
        for name in LAYER_TENSORS:
            put(layer, name)
