"""Device copies of the seeded synthetic inputs (weights, cached KV, batch
inputs) as torch tensors.  Values come from the generator in gen.c, so the
GPU path sees exactly what the oracle sees.  torch is used for device memory
only."""
from __future__ import annotations

import numpy as np
import torch

import workload as wl

LAYER_KINDS = (wl.W_Q, wl.W_K, wl.W_V, wl.W_O, wl.W_G, wl.W_U, wl.W_D,
               wl.N_1, wl.N_2, wl.N_Q, wl.N_K)


def _tdtype(m: wl.ModelShape):
    # bf16 tensors are carried as raw 16-bit patterns (int16 storage)
    return torch.float32 if m.dtype == "f32" else torch.int16


def _to_dev(a: np.ndarray, dev) -> torch.Tensor:
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(dev)


class DeviceWeights:
    """All weights of a seeded model on the GPU: one stacked tensor per
    per-layer kind ([J, out, in]) plus the global tensors."""

    def __init__(self, m: wl.ModelShape, seed: int, gamma: str = "ones", device="cuda"):
        self.m = m
        dt = _tdtype(m)
        self.glob = {k: _to_dev(wl.new_weight(m, seed, -1, k, gamma), device)
                     for k in (wl.EMBED, wl.LM_HEAD, wl.NORM_F)}
        self.layer = {}
        for k in LAYER_KINDS:
            shape = wl.weight_shape(m, k)
            self.layer[k] = torch.empty((m.n_layers,) + shape, dtype=dt, device=device)
        np_dt = np.float32 if m.dtype == "f32" else np.uint16
        for l in range(m.n_layers):
            for k in LAYER_KINDS:
                host = np.empty(wl.weight_shape(m, k), dtype=np_dt)
                wl.fill_weight(m, seed, l, k, host, gamma)
                self.layer[k][l].copy_(torch.from_numpy(host.view(np.int16) if np_dt == np.uint16 else host))

    def ptr(self, kind: int, layer: int = -1) -> int:
        if layer < 0:
            return self.glob[kind].data_ptr()
        t = self.layer[kind]
        return t.data_ptr() + layer * t[0].numel() * t.element_size()


def batch_to_device(b: wl.Batch, device="cuda"):
    """(drafts int32, q fp32, accept_u fp32 or None) on the GPU."""
    drafts = torch.from_numpy(np.ascontiguousarray(b.drafts)).to(device)
    q = torch.from_numpy(np.ascontiguousarray(b.q)).to(device)
    au = None if b.accept_u is None else torch.from_numpy(b.accept_u).to(device)
    return drafts, q, au


def kv_rows(m: wl.ModelShape, seed: int, layer: int, user: int, n: int, device="cuda"):
    """Synthetic cached K and V of positions 0..n-1 as device tensors
    [n][hkv][hd] in the model dtype."""
    np_dt = np.float32 if m.dtype == "f32" else np.uint16
    shape = (n, m.n_kv_heads, m.head_dim)
    k = np.empty(shape, np_dt)
    v = np.empty(shape, np_dt)
    wl.fill_kv(m, seed, layer, user, 0, k)
    wl.fill_kv(m, seed, layer, user, 1, v)
    return _to_dev(k, device), _to_dev(v, device)
