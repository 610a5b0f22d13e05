"""ctypes binding of libdsi.so -- argument marshalling only.

Every function has the name of the C entry point it calls (include/dsi.h)
and raises DsiError on a non-zero status.  Device buffers are passed as
integer addresses or torch tensors (their data_ptr()); torch is used only
for device memory and streams.  Every step of the verification runs in the
library's HIP kernels; there is no fallback: if libdsi.so is missing or was
built for another GPU, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdsi.so")

DSI_OK, DSI_EINVAL, DSI_ENOMEM, DSI_EHIP, DSI_ECAPACITY, DSI_ESTATE = range(6)
DSI_F32, DSI_BF16 = 0, 1
DSI_SAMPLE, DSI_GREEDY = 0, 1
DSI_MAX_ROWS = 64
TENSOR_IDS = {
    "embed": 0, "final_norm": 1, "lm_head": 2, "attn_norm": 3, "wq": 4, "wk": 5, "wv": 6,
    "wo": 7, "ffn_norm": 8, "w_gate": 9, "w_up": 10, "w_down": 11,
}
EXPORTED = (
    "dsi_model_create", "dsi_model_set_tensor", "dsi_model_destroy", "dsi_kv_create",
    "dsi_kv_destroy", "dsi_prefill", "dsi_verify", "dsi_verify_tree", "dsi_draft", "dsi_accept",
    "dsi_accept_noalloc",
    "dsi_kv_rollback", "dsi_kv_poison", "dsi_kv_length", "dsi_sync", "dsi_kv_export", "dsi_kv_import", "dsi_kv_set_length",
    "dsi_profile_begin", "dsi_profile_end", "dsi_profile_kernel", "dsi_profile_stream", "dsi_last_error",
)
DSI_K_QKV, DSI_K_ATTN, DSI_K_OPROJ, DSI_K_GATEUP, DSI_K_DOWN, DSI_K_HEAD, DSI_K_VERIFY = range(1, 8)


class DsiError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"dsi status {status}: {msg}")
        self.status = status


class dsi_config(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float),
        ("wdtype", ctypes.c_int32), ("kvdtype", ctypes.c_int32),
    ]


class dsi_verify_args(ctypes.Structure):
    _fields_ = [
        ("window0", ctypes.c_int32), ("n_windows", ctypes.c_int32), ("k", ctypes.c_int32),
        ("d_tokens", ctypes.c_void_p), ("d_q", ctypes.c_void_p), ("d_u", ctypes.c_void_p),
        ("temperature", ctypes.c_float), ("mode", ctypes.c_int32), ("commit", ctypes.c_int32),
        ("d_logits_out", ctypes.c_void_p), ("d_hidden_out", ctypes.c_void_p),
    ]


class dsi_tree_args(ctypes.Structure):
    _fields_ = [
        ("window0", ctypes.c_int32), ("n_windows", ctypes.c_int32), ("n_nodes", ctypes.c_int32),
        ("d_tokens", ctypes.c_void_p), ("d_parent", ctypes.c_void_p), ("commit", ctypes.c_int32),
        ("d_logits_out", ctypes.c_void_p),
    ]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libdsi.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2405_14105_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, SZ, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t, ctypes.c_float
    PP = ctypes.POINTER(ctypes.c_void_p)
    sig = {
        "dsi_model_create": ([ctypes.POINTER(dsi_config), P, PP], I32),
        "dsi_model_set_tensor": ([P, I32, I32, P, SZ, I32], I32),
        "dsi_model_destroy": ([P], I32),
        "dsi_kv_create": ([P, I32, I32, PP], I32),
        "dsi_kv_destroy": ([P], I32),
        "dsi_prefill": ([P, P, I32, P, I32, P], I32),
        "dsi_verify": ([P, P, ctypes.POINTER(dsi_verify_args), P, P], I32),
        "dsi_verify_tree": ([P, P, ctypes.POINTER(dsi_tree_args), P, P, P], I32),
        "dsi_draft": ([P, P, I32, P, I32, I32, P, F, P, P], I32),
        "dsi_accept": ([P, I32, I32, I32, P, P, P, P, F, I32, P, P], I32),
        "dsi_accept_noalloc": ([P, I32, I32, I32, P, P, P, P, F, I32, P, P], I32),
        "dsi_kv_rollback": ([P, I32, I32], I32),
        "dsi_kv_poison": ([P, I32], I32),
        "dsi_kv_length": ([P, I32, ctypes.POINTER(ctypes.c_int32)], I32),
        "dsi_sync": ([P], I32),
        "dsi_kv_export": ([P, I32, I32, I32, P, P], I32),
        "dsi_kv_import": ([P, I32, I32, I32, P, P], I32),
        "dsi_kv_set_length": ([P, I32, I32], I32),
        "dsi_profile_begin": ([P, I32], I32),
        "dsi_profile_end": ([P, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double)], I32),
        "dsi_profile_kernel": ([P, P, I32, I32, ctypes.POINTER(ctypes.c_int32),
                                ctypes.POINTER(ctypes.c_double)], I32),
        "dsi_profile_stream": ([P, ctypes.c_uint64, I32, I32, I32, I32, P, ctypes.POINTER(ctypes.c_uint64),
                                ctypes.POINTER(ctypes.c_double)], I32),
        "dsi_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _ptr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _check(st: int):
    if st != DSI_OK:
        raise DsiError(st, load().dsi_last_error().decode())


def make_config(n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, rope_base=10000.0,
                rms_eps=1e-5, wdtype=DSI_BF16, kvdtype=DSI_BF16) -> dsi_config:
    return dsi_config(n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, rope_base,
                      rms_eps, wdtype, kvdtype)


def dsi_model_create(cfg: dsi_config, stream: int = 0) -> int:
    out = ctypes.c_void_p()
    _check(load().dsi_model_create(ctypes.byref(cfg), stream or None, ctypes.byref(out)))
    return out.value


def dsi_model_set_tensor(model: int, layer: int, tensor_id: int, src, nbytes: int, src_on_device: bool):
    _check(load().dsi_model_set_tensor(model, layer, tensor_id, src, nbytes, int(src_on_device)))


def dsi_model_destroy(model: int):
    _check(load().dsi_model_destroy(model))


def dsi_kv_create(model: int, n_windows: int, max_len: int) -> int:
    out = ctypes.c_void_p()
    _check(load().dsi_kv_create(model, n_windows, max_len, ctypes.byref(out)))
    return out.value


def dsi_kv_destroy(kv: int):
    _check(load().dsi_kv_destroy(kv))


def dsi_prefill(model: int, kv: int, window: int, d_tokens, n: int, d_last_logits=None):
    _check(load().dsi_prefill(model, kv, window, _ptr(d_tokens), n, _ptr(d_last_logits)))


def dsi_verify(model: int, kv: int, window0: int, n_windows: int, k: int, d_tokens, d_q, d_u,
               d_n_accepted, d_next_token, temperature: float = 1.0, mode: int = DSI_SAMPLE,
               commit: bool = True, d_logits_out=None, d_hidden_out=None):
    a = dsi_verify_args(window0, n_windows, k, _ptr(d_tokens), _ptr(d_q), _ptr(d_u), temperature,
                        mode, int(commit), _ptr(d_logits_out), _ptr(d_hidden_out))
    _check(load().dsi_verify(model, kv, ctypes.byref(a), _ptr(d_n_accepted), _ptr(d_next_token)))


def dsi_verify_tree(model: int, kv: int, window0: int, n_windows: int, n_nodes: int, d_tokens, d_parent,
                    d_path, d_n_accepted, d_next_token, commit: bool = True, d_logits_out=None):
    a = dsi_tree_args(window0, n_windows, n_nodes, _ptr(d_tokens), _ptr(d_parent), int(commit),
                      _ptr(d_logits_out))
    _check(load().dsi_verify_tree(model, kv, ctypes.byref(a), _ptr(d_path), _ptr(d_n_accepted),
                                  _ptr(d_next_token)))


def dsi_draft(model: int, kv: int, window: int, d_feed, n_feed: int, k: int, d_u, d_tokens, d_q,
              temperature: float = 1.0):
    _check(load().dsi_draft(model, kv, window, _ptr(d_feed), n_feed, k, _ptr(d_u), temperature,
                            _ptr(d_tokens), _ptr(d_q)))


def dsi_accept(stream: int, n_windows: int, k: int, vocab: int, d_logits, d_tokens, d_q, d_u,
               d_n_accepted, d_next_token, temperature: float = 1.0, mode: int = DSI_SAMPLE):
    _check(load().dsi_accept(stream or None, n_windows, k, vocab, _ptr(d_logits), _ptr(d_tokens),
                             _ptr(d_q), _ptr(d_u), temperature, mode, _ptr(d_n_accepted),
                             _ptr(d_next_token)))


def dsi_accept_noalloc(stream: int, n_windows: int, k: int, vocab: int, d_logits, d_tokens, d_q, d_u,
                       d_n_accepted, d_next_token, temperature: float = 1.0, mode: int = DSI_SAMPLE):
    _check(load().dsi_accept_noalloc(stream or None, n_windows, k, vocab, _ptr(d_logits), _ptr(d_tokens),
                                     _ptr(d_q), _ptr(d_u), temperature, mode, _ptr(d_n_accepted),
                                     _ptr(d_next_token)))


def dsi_kv_rollback(kv: int, window: int, new_len: int):
    _check(load().dsi_kv_rollback(kv, window, new_len))


def dsi_kv_poison(kv: int, window: int):
    _check(load().dsi_kv_poison(kv, window))


def dsi_kv_length(kv: int, window: int) -> int:
    out = ctypes.c_int32()
    _check(load().dsi_kv_length(kv, window, ctypes.byref(out)))
    return out.value


def dsi_sync(model: int):
    _check(load().dsi_sync(model))


def dsi_kv_export(kv: int, window: int, layer: int, length: int, d_k, d_v):
    _check(load().dsi_kv_export(kv, window, layer, length, _ptr(d_k), _ptr(d_v)))


def dsi_kv_import(kv: int, window: int, layer: int, length: int, d_k, d_v):
    _check(load().dsi_kv_import(kv, window, layer, length, _ptr(d_k), _ptr(d_v)))


def dsi_kv_set_length(kv: int, window: int, length: int):
    _check(load().dsi_kv_set_length(kv, window, length))


def dsi_profile_begin(model: int, kernel_class: int):
    _check(load().dsi_profile_begin(model, kernel_class))


def dsi_profile_end(model: int):
    """Returns (launches, total_ms)."""
    n = ctypes.c_int32()
    t = ctypes.c_double()
    _check(load().dsi_profile_end(model, ctypes.byref(n), ctypes.byref(t)))
    return n.value, t.value


def dsi_profile_kernel(model: int, kv: int, kernel_class: int, rounds: int = 3):
    """Returns (launches, avg_ms) of one GEMM class replayed back to back."""
    n = ctypes.c_int32()
    t = ctypes.c_double()
    _check(load().dsi_profile_kernel(model, kv, kernel_class, rounds, ctypes.byref(n), ctypes.byref(t)))
    return n.value, t.value


def dsi_profile_stream(d_buf, nbytes: int, slices: int, nontemporal: bool, rounds: int, d_sink,
                       workgroups: int = 0):
    """Returns (bytes per launch, avg_ms) of the library's streaming read over
    `slices` slices of the device buffer d_buf, one per launch in turn, with
    `workgroups` workgroups of 8 waves (0: the default 256)."""
    b = ctypes.c_uint64()
    t = ctypes.c_double()
    _check(load().dsi_profile_stream(_ptr(d_buf), nbytes, slices, int(bool(nontemporal)), workgroups, rounds,
                                     _ptr(d_sink), ctypes.byref(b), ctypes.byref(t)))
    return b.value, t.value


def dsi_last_error() -> str:
    return load().dsi_last_error().decode()
