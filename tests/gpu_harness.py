"""Shared helpers of the GPU parity tests: build a seeded model on the GPU,
run one verify batch through the C ABI, and run the oracle on the same
inputs.  Not collected by pytest (no test_ prefix)."""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np
import torch

import oracle
import workload as wl
from workload.device import DeviceWeights, batch_to_device, kv_rows
from paper_2604_20919_amd.verifier import Verifier


def layer_ptrs(dw: DeviceWeights):
    names = {"wq": wl.W_Q, "wk": wl.W_K, "wv": wl.W_V, "wo": wl.W_O, "wg": wl.W_G, "wu": wl.W_U,
             "wd": wl.W_D, "norm1": wl.N_1, "norm2": wl.N_2, "qnorm": wl.N_Q, "knorm": wl.N_K}
    return {"embed": dw.ptr(wl.EMBED), "lm_head": dw.ptr(wl.LM_HEAD), "norm_f": dw.ptr(wl.NORM_F),
            "layers": [{f: dw.ptr(k, l) for f, k in names.items()} for l in range(dw.m.n_layers)]}


def make_verifier(w: wl.Workload, dw: DeviceWeights, max_pending: int = 2, extra_ctx: int = 0,
                  max_batch_tokens: Optional[int] = None) -> Verifier:
    m = w.model
    max_ctx = int((w.prefix_len + w.draft_len).max()) + 1 + extra_ctx
    pages = int(sum((p + l + 1 + extra_ctx + 15) // 16 for p, l in zip(w.prefix_len, w.draft_len))) + 8
    T = max_batch_tokens or max(int((w.draft_len[w.assign == n] + 1).sum()) for n in range(w.n_batches))
    B = max(int((w.assign == n).sum()) for n in range(w.n_batches))
    return Verifier(m, layer_ptrs(dw), n_pages=pages, max_users=w.n_users,
                    max_draft=int(w.draft_len.max()), max_batch_users=B, max_batch_tokens=T,
                    max_ctx=max_ctx, max_pending=max_pending)


def load_synthetic_kv(v: Verifier, w: wl.Workload, users=None):
    m = w.model
    users = range(w.n_users) if users is None else users
    pmax = max([int(w.prefix_len[u]) for u in users] + [1])
    dt = torch.float32 if m.dtype == "f32" else torch.int16
    buf = (torch.empty((pmax, m.n_kv_heads, m.head_dim), dtype=dt, device="cuda"),
           torch.empty((pmax, m.n_kv_heads, m.head_dim), dtype=dt, device="cuda"))
    for u in users:
        P = int(w.prefix_len[u])
        v.reset_user(u, P, 0)
        for l in range(m.n_layers):
            if P:
                k, vv = kv_rows(m, w.seed, l, u, P, out=buf)
                v.write_kv(u, l, 0, k, vv)
    torch.cuda.synchronize()


@dataclasses.dataclass
class GpuResult:
    n_acc: np.ndarray
    token: np.ndarray
    logits: Optional[np.ndarray]


def run_gpu(v: Verifier, w: wl.Workload, n: int, b: wl.Batch, mode: str, seed: int = 0,
            round_: int = 0, want_logits: bool = True, commit: bool = False) -> GpuResult:
    for i, u in enumerate(b.users):
        P, _ = v.user_state(int(u))
        v.reset_user(int(u), P, int(b.root[i]))
    drafts, q, au = batch_to_device(b)
    v.verify(n, w.assign, w.draft_len, drafts, q, mode, seed, round_, au)
    lg = v.logits(n, b.T).cpu().numpy() if want_logits else None
    n_acc, tok = v.accept(n, w.n_users, commit)
    torch.cuda.synchronize()
    return GpuResult(n_acc[b.users], tok[b.users], lg)


def run_oracle(w: wl.Workload, b: wl.Batch, mode: str, seed: int = 0, round_: int = 0,
               kv: Optional[oracle.KVSource] = None, weights: Optional[oracle.WeightSource] = None,
               gamma: str = "ones"):
    m = w.model
    ws = weights or oracle.WeightSource(m, w.seed, gamma)
    kvs = kv or oracle.KVSource(m, w.seed, b.users, b.prefix_len)
    logits = oracle.forward(m, ws, kvs, b.prefix_len, b.n_slots, b.slot_tokens())
    res = oracle.sample(mode, b.users, b.draft_len, logits, b.drafts, b.q, b.accept_u, seed, round_)
    return logits, res


def compare_decisions(gpu_acc, gpu_tok, ref, draft_len, window=1e-3, extra=None):
    """Bit-exact comparison of (n_acc, token) with the oracle, except
    borderline cases: a deciding accept with |p/q - u| < window, or a race
    whose two best keys are within `window` (relative).  `extra` widens the
    accept window per user (the end-to-end logit tolerance).  Returns
    (n_mismatch_outside_window, n_borderline)."""
    bad, border = 0, 0
    off = 0
    for b, L in enumerate(draft_len):
        L = int(L)
        r = ref["ratio"][off:off + L]
        u = ref["u"][off:off + L]
        off += L
        if gpu_acc[b] == ref["n_acc"][b] and gpu_tok[b] == ref["token"][b]:
            continue
        wb = window + (0.0 if extra is None else float(extra[b]))
        upto = min(int(max(gpu_acc[b], ref["n_acc"][b])), L - 1)
        near = any(abs(float(r[j]) - float(u[j])) < wb * max(1.0, abs(float(r[j])))
                   for j in range(upto + 1) if np.isfinite(r[j]))
        if gpu_acc[b] == ref["n_acc"][b]:
            near = near or ref["race_gap"][b] < wb
        if near:
            border += 1
        else:
            bad += 1
    return bad, border


def logit_rel_err(gpu: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per row: max |z_gpu - z_ref| / max |z_ref|."""
    return np.max(np.abs(gpu - ref), axis=1) / np.maximum(np.max(np.abs(ref), axis=1), 1e-30)
