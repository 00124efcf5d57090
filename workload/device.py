"""Device copies of the seeded synthetic inputs (weights, cached KV, batch
inputs) as torch tensors.  Weights and cached keys/values are written on the
GPU by the fill kernels of gen_gpu.hip, which produce the same bits as the
host generator in gen.c (pinned by a GPU test), so the GPU path sees exactly
what the oracle sees.  torch is used for device memory only."""
from __future__ import annotations

import numpy as np
import torch

import workload as wl

LAYER_KINDS = (wl.W_Q, wl.W_K, wl.W_V, wl.W_O, wl.W_G, wl.W_U, wl.W_D,
               wl.N_1, wl.N_2, wl.N_Q, wl.N_K)
NORM_KINDS = (wl.N_1, wl.N_2, wl.N_Q, wl.N_K, wl.NORM_F)


def _tdtype(m: wl.ModelShape):
    # bf16 tensors are carried as raw 16-bit patterns (int16 storage)
    return torch.float32 if m.dtype == "f32" else torch.int16


def _stream_ptr():
    return torch.cuda.current_stream().cuda_stream


def gpu_fill_normal(out: torch.Tensor, seed: int, stream: int, offset: int, std: float):
    bf16 = out.dtype == torch.int16
    rc = wl.glib().wlg_fill_normal(out.data_ptr(), out.numel(), seed, stream, offset, std, int(bf16),
                                   _stream_ptr())
    if rc != 0:
        raise RuntimeError("GPU generator launch failed")


def gpu_fill_uniform(out: torch.Tensor, seed: int, stream: int, offset: int, lo: float, hi: float):
    bf16 = out.dtype == torch.int16
    rc = wl.glib().wlg_fill_uniform(out.data_ptr(), out.numel(), seed, stream, offset, lo, hi,
                                    int(bf16), _stream_ptr())
    if rc != 0:
        raise RuntimeError("GPU generator launch failed")


def fill_weight_gpu(m: wl.ModelShape, seed: int, layer: int, kind: int, out: torch.Tensor,
                    gamma: str = "ones"):
    """GPU twin of workload.fill_weight."""
    s = wl._wstream(layer, kind)
    if kind in NORM_KINDS:
        if gamma == "ones":
            out.fill_(0x3F80 if out.dtype == torch.int16 else 1.0)
        else:
            gpu_fill_uniform(out, seed, s, 0, 0.5, 1.5)
    else:
        gpu_fill_normal(out, seed, s, 0, wl.WEIGHT_STD)


class DeviceWeights:
    """All weights of a seeded model on the GPU: one stacked tensor per
    per-layer kind ([J, out, in]) plus the global tensors."""

    def __init__(self, m: wl.ModelShape, seed: int, gamma: str = "ones", device="cuda"):
        self.m = m
        dt = _tdtype(m)
        self.glob = {}
        for k in (wl.EMBED, wl.LM_HEAD, wl.NORM_F):
            t = torch.empty(wl.weight_shape(m, k), dtype=dt, device=device)
            fill_weight_gpu(m, seed, -1, k, t, gamma)
            self.glob[k] = t
        self.layer = {}
        for k in LAYER_KINDS:
            t = torch.empty((m.n_layers,) + wl.weight_shape(m, k), dtype=dt, device=device)
            for l in range(m.n_layers):
                fill_weight_gpu(m, seed, l, k, t[l], gamma)
            self.layer[k] = t
        torch.cuda.synchronize()

    def ptr(self, kind: int, layer: int = -1) -> int:
        if layer < 0:
            return self.glob[kind].data_ptr()
        t = self.layer[kind]
        return t.data_ptr() + layer * t[0].numel() * t.element_size()

    def nbytes(self) -> int:
        return sum(t.numel() * t.element_size() for t in list(self.glob.values()) + list(self.layer.values()))


def batch_to_device(b: wl.Batch, device="cuda"):
    """(drafts int32, q fp32, accept_u fp32 or None) on the GPU."""
    drafts = torch.from_numpy(np.ascontiguousarray(b.drafts)).to(device)
    q = torch.from_numpy(np.ascontiguousarray(b.q)).to(device)
    au = None if b.accept_u is None else torch.from_numpy(b.accept_u).to(device)
    return drafts, q, au


def kv_rows(m: wl.ModelShape, seed: int, layer: int, user: int, n: int, device="cuda", out=None):
    """Synthetic cached K and V of positions 0..n-1 as device tensors
    [n][hkv][hd] in the model dtype (GPU twin of workload.fill_kv)."""
    shape = (n, m.n_kv_heads, m.head_dim)
    if out is None:
        k = torch.empty(shape, dtype=_tdtype(m), device=device)
        v = torch.empty(shape, dtype=_tdtype(m), device=device)
    else:
        k, v = out[0][:n], out[1][:n]
    gpu_fill_normal(k, seed, wl._kvstream(layer, user, 0), 0, wl.KV_STD)
    gpu_fill_normal(v, seed, wl._kvstream(layer, user, 1), 0, wl.KV_STD)
    return k, v
