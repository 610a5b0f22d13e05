"""GPU-side helpers for the parity tests and the benchmark: build a model
from the seeded synthetic weights, prefill windows and run verifications
through the C ABI (torch provides device buffers and the stream only)."""
from __future__ import annotations

import numpy as np
import torch

import dsi_synth as S
from paper_2405_14105_amd import dsi, loader


def host_tensor_fn(shape, seed):
    def fn(layer, name):
        if shape.wdtype == "bf16":
            return S.weight_bf16_bits(shape, seed, layer, name)
        return S.weight(shape, seed, layer, name)
    return fn


class Rig:
    def __init__(self, shape, seed: int, n_windows: int, max_len: int, progress=None):
        self.shape = shape
        self.seed = seed
        self.dev = torch.device("cuda:0")
        self.stream = torch.cuda.current_stream().cuda_stream
        self.model = dsi.dsi_model_create(loader.config_for(shape), self.stream)
        loader.upload(self.model, shape, host_tensor_fn(shape, seed), progress)
        self.kv = dsi.dsi_kv_create(self.model, n_windows, max_len)
        self._keep = []

    def close(self):
        torch.cuda.synchronize()
        if self.kv:
            dsi.dsi_kv_destroy(self.kv)
            self.kv = None
        if self.model:
            dsi.dsi_model_destroy(self.model)
            self.model = None

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def dev_i32(self, a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(self.dev)

    def dev_f32(self, a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(self.dev)

    def prefill(self, window: int, tokens, want_logits: bool = False):
        t = self.dev_i32(tokens)
        out = torch.empty(self.shape.vocab, dtype=torch.float32, device=self.dev) if want_logits else None
        dsi.dsi_prefill(self.model, self.kv, window, t, len(tokens), out)
        torch.cuda.synchronize()
        return None if out is None else out.cpu().numpy()

    def verify(self, window0: int, tokens, q=None, u=None, mode=dsi.DSI_SAMPLE, commit=True,
               temperature=1.0, want_logits=True, want_hidden=False):
        tokens = np.asarray(tokens, dtype=np.int32)
        B, k1 = tokens.shape
        k = k1 - 1
        M = B * k1
        t = self.dev_i32(tokens)
        dq = self.dev_f32(q) if q is not None else None
        du = self.dev_f32(u) if u is not None else None
        n = torch.full((B,), -7, dtype=torch.int32, device=self.dev)
        tok = torch.full((B,), -7, dtype=torch.int32, device=self.dev)
        lg = torch.empty((M, self.shape.vocab), dtype=torch.float32, device=self.dev) if want_logits else None
        hid = (torch.empty((self.shape.n_layers + 1, M, self.shape.d_model), dtype=torch.float32,
                           device=self.dev) if want_hidden else None)
        dsi.dsi_verify(self.model, self.kv, window0, B, k, t, dq, du, n, tok, temperature, mode,
                       commit, lg, hid)
        torch.cuda.synchronize()
        out = {"n": n.cpu().numpy(), "token": tok.cpu().numpy()}
        if lg is not None:
            out["logits"] = lg.cpu().numpy()
        if hid is not None:
            out["hidden"] = hid.cpu().numpy()
        return out

    def verify_tree(self, window0: int, tokens, parent, commit=True, want_logits=True):
        tokens = np.asarray(tokens, dtype=np.int32)
        B, R = tokens.shape
        t = self.dev_i32(tokens)
        p = self.dev_i32(parent)
        path = torch.full((B, R), -7, dtype=torch.int32, device=self.dev)
        n = torch.full((B,), -7, dtype=torch.int32, device=self.dev)
        tok = torch.full((B,), -7, dtype=torch.int32, device=self.dev)
        lg = (torch.empty((B * R, self.shape.vocab), dtype=torch.float32, device=self.dev)
              if want_logits else None)
        dsi.dsi_verify_tree(self.model, self.kv, window0, B, R, t, p, path, n, tok, commit, lg)
        torch.cuda.synchronize()
        out = {"path": path.cpu().numpy(), "n": n.cpu().numpy(), "token": tok.cpu().numpy()}
        if lg is not None:
            out["logits"] = lg.cpu().numpy()
        return out

    def length(self, window: int) -> int:
        return dsi.dsi_kv_length(self.kv, window)

    def export_kv(self, window: int, layer: int, length: int):
        s = self.shape
        dt = torch.bfloat16 if s.kvdtype == "bf16" else torch.float32
        k = torch.empty((s.n_kv_heads, length, s.head_dim), dtype=dt, device=self.dev)
        v = torch.empty_like(k)
        dsi.dsi_kv_export(self.kv, window, layer, length, k, v)
        torch.cuda.synchronize()
        # [hkv, len, hd] -> [len, hkv, hd] in fp64
        return (k.float().cpu().numpy().transpose(1, 0, 2).astype(np.float64),
                v.float().cpu().numpy().transpose(1, 0, 2).astype(np.float64))
