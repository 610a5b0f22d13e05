"""Upload host weight arrays into a dsi_model (marshalling only)."""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor

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


def upload(model: int, shape, tensor_fn, progress=None) -> None:
    """tensor_fn(layer, name) -> host array in the model's storage format:
    uint16 bf16 bit patterns for bf16 models, float32 for fp32 models.

    The next tensor is produced on a helper thread while the current one
    uploads.  progress(layer) is called after each layer's last tensor."""
    want = np.uint16 if shape.wdtype == "bf16" else np.float32
    names = [(-1, n) for n in GLOBAL_TENSORS] + [(l, n) for l in range(shape.n_layers)
                                                for n in LAYER_TENSORS]
    with ThreadPoolExecutor(1) as ex:
        fut = ex.submit(tensor_fn, *names[0])
        for i, (layer, name) in enumerate(names):
            a = np.ascontiguousarray(fut.result())
            if i + 1 < len(names):
                fut = ex.submit(tensor_fn, *names[i + 1])
            if a.dtype != want:
                raise TypeError(f"{name}: expected {want}, got {a.dtype}")
            dsi.dsi_model_set_tensor(model, layer, dsi.TENSOR_IDS[name], a.ctypes.data, a.nbytes,
                                     False)
            if progress is not None and layer >= 0 and name == LAYER_TENSORS[-1]:
                progress(layer)
