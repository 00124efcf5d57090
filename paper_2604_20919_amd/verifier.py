"""Convenience wrapper around the C ABI: owns one library context plus the
device memory torch allocates for it (KV pool, workspace) and marshals
per-batch arguments.  Every step of the verify pass runs in libsdverify.so."""
from __future__ import annotations

import ctypes
from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import sdverify as sv


class Verifier:
    def __init__(self, shape, weight_ptrs: Dict[str, object], *, n_pages: int, max_users: int,
                 max_draft: int, max_batch_users: int, max_batch_tokens: int, max_ctx: int,
                 max_pending: int = 2, logits_out: int = sv.SD_LOGITS_AS_NEEDED, device: str = "cuda"):
        """shape: object with n_layers, d_model, n_q_heads, n_kv_heads,
        head_dim, d_ffn, vocab, qk_norm, dtype ("f32"/"bf16"), rope_base,
        rms_eps.  weight_ptrs: "embed", "lm_head", "norm_f" -> device
        pointer, "layers" -> list of dicts with the sd_layer_weights field
        names -> device pointer.  logits_out: which passes store fp32
        logits (sd_config.logits_out; `logits()` needs them)."""
        dt = sv.SD_BF16 if shape.dtype == "bf16" else sv.SD_F32
        self.cfg = sv.make_config(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads,
                                  shape.head_dim, shape.d_ffn, shape.vocab, shape.qk_norm, dt,
                                  n_pages, max_users, max_draft, max_batch_users, max_batch_tokens,
                                  max_ctx, max_pending, shape.rope_base, shape.rms_eps, logits_out)
        kv_bytes, ws_bytes, wp_bytes = sv.sd_verify_query_sizes(self.cfg)
        self.kv_bytes, self.ws_bytes, self.wp_bytes = kv_bytes, ws_bytes, wp_bytes
        # 256-byte aligned by the caching allocator
        self.kv_pool = torch.empty(kv_bytes, dtype=torch.uint8, device=device)
        self.workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=device)
        self.weight_pack = torch.empty(max(wp_bytes, 256), dtype=torch.uint8, device=device)
        L = shape.n_layers
        self._layers = (sv.sd_layer_weights * L)()
        for l in range(L):
            for f, _ in sv.sd_layer_weights._fields_:
                setattr(self._layers[l], f, int(weight_ptrs["layers"][l].get(f) or 0))
        self._w = sv.sd_weights(int(weight_ptrs["embed"]), int(weight_ptrs["lm_head"]),
                                int(weight_ptrs["norm_f"]), self._layers)
        torch.cuda.synchronize()
        self.ctx = sv.sd_verify_init(self.cfg, self._w, self.kv_pool, self.workspace,
                                     self.weight_pack if wp_bytes else None)
        self.max_users = max_users
        self.vocab = shape.vocab

    def close(self):
        if self.ctx:
            sv.sd_verify_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # --- user state ---
    def reset_user(self, user: int, prefix_len: int, root: int):
        sv.sd_user_reset(self.ctx, user, prefix_len, root)

    def user_state(self, user: int):
        return sv.sd_user_state(self.ctx, user)

    def write_kv(self, user: int, layer: int, pos0: int, k: torch.Tensor, v: torch.Tensor, stream=None):
        sv.sd_kv_write(self.ctx, user, layer, pos0, k.shape[0], k, v, stream)

    def read_kv(self, user: int, layer: int, pos0: int, k: torch.Tensor, v: torch.Tensor, stream=None):
        sv.sd_kv_read(self.ctx, user, layer, pos0, k.shape[0], k, v, stream)

    # --- batches ---
    def verify(self, batch: int, assign: Sequence[int], draft_len: Sequence[int], drafts, q,
               mode="stochastic", seed: int = 0, round_: int = 0, accept_u=None, stream=None,
               graph: bool = False):
        """graph: replay the pass from a HIP graph (sd_verify_batch_graph);
        needs a non-null stream."""
        fn = sv.sd_verify_batch_graph if graph else sv.sd_verify_batch
        fn(self.ctx, batch, assign, draft_len, drafts, q, mode, seed, round_, accept_u, stream)

    def verify_sparse(self, batch: int, assign: Sequence[int], draft_len: Sequence[int], drafts,
                      q_idx, q_val, q_rest, mode="stochastic", seed: int = 0, round_: int = 0,
                      accept_u=None, stream=None):
        """Verification with sparse draft rows (sd_verify_batch_sparse)."""
        sv.sd_verify_batch_sparse(self.ctx, batch, assign, draft_len, drafts, q_idx, q_val, q_rest,
                                  mode, seed, round_, accept_u, stream)

    def draft(self, batch: int, assign: Sequence[int], mode="stochastic", seed: int = 0,
              round_: int = 0, probs=None, probs_row=None, stream=None):
        """One decode step of the users of `batch` (sd_draft_batch); complete
        with accept(batch, n_users, commit=True)."""
        sv.sd_draft_batch(self.ctx, batch, assign, mode, seed, round_, probs, probs_row, stream)

    def sample(self, batch: int, assign, draft_len, drafts, q, logits, mode="stochastic",
               seed: int = 0, round_: int = 0, accept_u=None, stream=None):
        sv.sd_sample_logits(self.ctx, batch, assign, draft_len, drafts, q, logits, mode, seed,
                            round_, accept_u, stream)

    def accept(self, batch: int, n_users: int, commit: bool = False):
        return sv.sd_accept(self.ctx, batch, n_users, commit)

    def wait_limit(self, max_polls: int) -> None:
        """Bound of the split gate/up product's waits (negative: default)."""
        sv.sd_debug_wait_limit(self.ctx, max_polls)

    def logits(self, batch: int, T: int, stream=None) -> torch.Tensor:
        out = torch.empty((T, self.vocab), dtype=torch.float32, device="cuda")
        sv.sd_debug_logits(self.ctx, batch, out, stream)
        return out
