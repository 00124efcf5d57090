"""Python binding of libsdverify.so (the C ABI in include/sd_verify.h).

Argument marshalling only: every step of the verify pass runs in the HIP
kernels of the library.  torch tensors are accepted where the C ABI takes a
device pointer; torch supplies device memory and streams, nothing else.  If
the library has not been built, loading raises -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsdverify.so")

SD_OK, SD_EINVAL, SD_ENOMEM, SD_EHIP, SD_ESTATE, SD_EDEVICE, SD_ENOTIMPL, SD_ENODEV, SD_ELIMIT = (
    0, -1, -2, -3, -4, -5, -6, -7, -8)
SD_NOALLOC_MAX_USERS, SD_NOALLOC_MAX_SLOTS, SD_NOALLOC_MAX_VOCAB = 64, 1024, 1 << 20
SD_F32, SD_BF16 = 0, 1
SD_GREEDY, SD_STOCHASTIC, SD_FORCE = 0, 1, 2
SD_LOGITS_AS_NEEDED, SD_LOGITS_ALL, SD_LOGITS_UNFUSED = 0, 1, 2
MODES = {"greedy": SD_GREEDY, "stochastic": SD_STOCHASTIC, "force": SD_FORCE}

EXPORTS = ("sd_verify_query_sizes", "sd_verify_init", "sd_verify_destroy", "sd_user_reset",
           "sd_user_release", "sd_user_state", "sd_kv_write", "sd_kv_read", "sd_verify_batch",
           "sd_verify_batch_graph", "sd_verify_batch_sparse", "sd_draft_batch", "sd_accept", "sd_sample_logits",
           "sd_sample_logits_noalloc", "sd_debug_logits", "sd_debug_wait_limit", "sd_profile_begin", "sd_profile_end",
           "sd_calib_hbm", "sd_calib_mfma", "sd_status_str")
SD_K_QKV, SD_K_ATTN, SD_K_O, SD_K_GATEUP, SD_K_DOWN, SD_K_LMHEAD, SD_K_SAMPLER, SD_K_SMALL = range(1, 9)


class sd_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_ffn", "vocab", "qk_norm",
        "dtype", "page_tokens", "n_pages", "max_users", "max_draft", "max_batch_users",
        "max_batch_tokens", "max_ctx", "max_pending")] + [("rope_base", ctypes.c_float),
                                                          ("rms_eps", ctypes.c_float),
                                                          ("logits_out", ctypes.c_int32)]


class sd_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "wq", "wk", "wv", "wo", "wg", "wu", "wd", "norm1", "norm2", "qnorm", "knorm")]


class sd_weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
                ("norm_f", ctypes.c_void_p), ("layers", ctypes.POINTER(sd_layer_weights))]


class SdError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: {status_str(status)} ({status})")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64
        P = ctypes.POINTER
        L.sd_status_str.restype = ctypes.c_char_p
        L.sd_status_str.argtypes = [i32]
        L.sd_verify_query_sizes.argtypes = [P(sd_config), P(u64), P(u64), P(u64)]
        L.sd_verify_init.argtypes = [P(sd_config), P(sd_weights), vp, vp, vp, P(vp)]
        L.sd_verify_destroy.argtypes = [vp]
        L.sd_user_reset.argtypes = [vp, i32, i32, i32]
        L.sd_user_release.argtypes = [vp, i32]
        L.sd_user_state.argtypes = [vp, i32, P(i32), P(i32)]
        L.sd_kv_write.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp]
        L.sd_kv_read.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp]
        L.sd_verify_batch.argtypes = [vp, i32, i32, vp, vp, vp, vp, i32, u64, u64, vp, vp]
        L.sd_verify_batch_graph.argtypes = [vp, i32, i32, vp, vp, vp, vp, i32, u64, u64, vp, vp]
        L.sd_draft_batch.argtypes = [vp, i32, i32, vp, i32, u64, u64, vp, vp, vp]
        L.sd_verify_batch_sparse.argtypes = [vp, i32, i32, vp, vp, vp, vp, vp, vp, i32, i32, u64, u64,
                                             vp, vp]
        L.sd_accept.argtypes = [vp, i32, vp, vp, i32]
        L.sd_sample_logits.argtypes = [vp, i32, i32, vp, vp, vp, vp, vp, i32, u64, u64, vp, vp]
        L.sd_sample_logits_noalloc.argtypes = [i32, vp, vp, i32, vp, vp, vp, i32, u64, u64, vp, vp, vp]
        L.sd_debug_logits.argtypes = [vp, i32, vp, vp]
        L.sd_debug_wait_limit.argtypes = [vp, i32]
        L.sd_profile_begin.argtypes = [vp, i32, i32]
        L.sd_profile_end.argtypes = [vp, P(ctypes.c_double), P(i32)]
        L.sd_calib_hbm.argtypes = [vp, ctypes.c_size_t, i32, i32, P(ctypes.c_double), vp]
        L.sd_calib_mfma.argtypes = [vp, i32, P(ctypes.c_double), vp]
        for name in EXPORTS:
            if name != "sd_status_str":
                getattr(L, name).restype = i32
        _lib = L
    return _lib


def status_str(s: int) -> str:
    return lib().sd_status_str(int(s)).decode()


def _check(fn: str, s: int) -> int:
    if s != SD_OK:
        raise SdError(fn, s)
    return s


def _dev(t) -> Optional[int]:
    """Device pointer of a torch tensor (or an int / None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    assert t.is_cuda and t.is_contiguous(), "device arguments must be contiguous GPU tensors"
    return t.data_ptr()


def _host_i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


# ---------------------------------------------------------------------------
# thin wrappers with the C names (raise SdError on a nonzero status)
# ---------------------------------------------------------------------------

def sd_verify_query_sizes(cfg: sd_config):
    """Returns (kv_pool_bytes, workspace_bytes, weight_pack_bytes)."""
    kv, ws, wp = ctypes.c_uint64(), ctypes.c_uint64(), ctypes.c_uint64()
    _check("sd_verify_query_sizes", lib().sd_verify_query_sizes(
        ctypes.byref(cfg), ctypes.byref(kv), ctypes.byref(ws), ctypes.byref(wp)))
    return kv.value, ws.value, wp.value


def sd_verify_init(cfg: sd_config, weights: sd_weights, kv_pool, workspace, weight_pack=None) -> int:
    out = ctypes.c_void_p()
    _check("sd_verify_init", lib().sd_verify_init(ctypes.byref(cfg), ctypes.byref(weights),
                                                  _dev(kv_pool), _dev(workspace), _dev(weight_pack),
                                                  ctypes.byref(out)))
    return out.value


def sd_verify_destroy(ctx: int) -> None:
    _check("sd_verify_destroy", lib().sd_verify_destroy(ctx))


def sd_user_reset(ctx: int, user: int, prefix_len: int, root_token: int) -> None:
    _check("sd_user_reset", lib().sd_user_reset(ctx, user, prefix_len, root_token))


def sd_user_release(ctx: int, user: int) -> None:
    _check("sd_user_release", lib().sd_user_release(ctx, user))


def sd_user_state(ctx: int, user: int):
    p, r = ctypes.c_int32(), ctypes.c_int32()
    _check("sd_user_state", lib().sd_user_state(ctx, user, ctypes.byref(p), ctypes.byref(r)))
    return p.value, r.value


def sd_kv_write(ctx: int, user: int, layer: int, pos0: int, n: int, k, v, stream=None) -> None:
    _check("sd_kv_write", lib().sd_kv_write(ctx, user, layer, pos0, n, _dev(k), _dev(v), _stream(stream)))


def sd_kv_read(ctx: int, user: int, layer: int, pos0: int, n: int, k, v, stream=None) -> None:
    _check("sd_kv_read", lib().sd_kv_read(ctx, user, layer, pos0, n, _dev(k), _dev(v), _stream(stream)))


def sd_verify_batch(ctx: int, batch: int, assign: Sequence[int], draft_len: Sequence[int],
                    draft_tokens, q, mode, seed: int = 0, round_: int = 0, accept_u=None,
                    stream=None) -> None:
    a, L = _host_i32(assign), _host_i32(draft_len)
    mode = MODES[mode] if isinstance(mode, str) else int(mode)
    _check("sd_verify_batch", lib().sd_verify_batch(
        ctx, batch, a.size, a.ctypes.data, L.ctypes.data, _dev(draft_tokens), _dev(q), mode,
        int(seed), int(round_), _dev(accept_u), _stream(stream)))


def sd_verify_batch_graph(ctx: int, batch: int, assign: Sequence[int], draft_len: Sequence[int],
                          draft_tokens, q, mode, seed: int = 0, round_: int = 0, accept_u=None,
                          stream=None) -> None:
    a, L = _host_i32(assign), _host_i32(draft_len)
    mode = MODES[mode] if isinstance(mode, str) else int(mode)
    _check("sd_verify_batch_graph", lib().sd_verify_batch_graph(
        ctx, batch, a.size, a.ctypes.data, L.ctypes.data, _dev(draft_tokens), _dev(q), mode,
        int(seed), int(round_), _dev(accept_u), _stream(stream)))


def sd_verify_batch_sparse(ctx: int, batch: int, assign: Sequence[int], draft_len: Sequence[int],
                           draft_tokens, q_idx, q_val, q_rest, mode, seed: int = 0, round_: int = 0,
                           accept_u=None, stream=None) -> None:
    """q_idx int32 [nd][K], q_val fp32 [nd][K], q_rest fp32 [nd] (device)."""
    a, L = _host_i32(assign), _host_i32(draft_len)
    mode = MODES[mode] if isinstance(mode, str) else int(mode)
    k = int(q_idx.shape[1]) if hasattr(q_idx, "shape") else 0
    _check("sd_verify_batch_sparse", lib().sd_verify_batch_sparse(
        ctx, batch, a.size, a.ctypes.data, L.ctypes.data, _dev(draft_tokens), _dev(q_idx), _dev(q_val),
        _dev(q_rest), k, mode, int(seed), int(round_), _dev(accept_u), _stream(stream)))


def sd_draft_batch(ctx: int, batch: int, assign: Sequence[int], mode, seed: int = 0,
                   round_: int = 0, probs=None, probs_row=None, stream=None) -> None:
    a = _host_i32(assign)
    pr = None if probs_row is None else _host_i32(probs_row)
    mode = MODES[mode] if isinstance(mode, str) else int(mode)
    _check("sd_draft_batch", lib().sd_draft_batch(
        ctx, batch, a.size, a.ctypes.data, mode, int(seed), int(round_), _dev(probs),
        None if pr is None else pr.ctypes.data, _stream(stream)))


def sd_sample_logits(ctx: int, batch: int, assign, draft_len, draft_tokens, q, logits, mode,
                     seed: int = 0, round_: int = 0, accept_u=None, stream=None) -> None:
    a, L = _host_i32(assign), _host_i32(draft_len)
    mode = MODES[mode] if isinstance(mode, str) else int(mode)
    _check("sd_sample_logits", lib().sd_sample_logits(
        ctx, batch, a.size, a.ctypes.data, L.ctypes.data, _dev(draft_tokens), _dev(q), _dev(logits),
        mode, int(seed), int(round_), _dev(accept_u), _stream(stream)))


def sd_sample_logits_noalloc(user_ids, draft_len, vocab: int, draft_tokens, q, logits, mode,
                             result, seed: int = 0, round_: int = 0, accept_u=None,
                             stream=None) -> None:
    """Context-free accept/resample on caller logits; result: device int32
    [2*B + 1] (n_acc, token, flag word), written asynchronously."""
    u, L = _host_i32(user_ids), _host_i32(draft_len)
    if u.size != L.size:
        raise ValueError("user_ids and draft_len differ in length")
    mode = MODES[mode] if isinstance(mode, str) else int(mode)
    _check("sd_sample_logits_noalloc", lib().sd_sample_logits_noalloc(
        u.size, u.ctypes.data, L.ctypes.data, int(vocab), _dev(draft_tokens), _dev(q), _dev(logits),
        mode, int(seed), int(round_), _dev(accept_u), _dev(result), _stream(stream)))


def sd_accept(ctx: int, batch: int, n_users: int, commit: bool = False):
    """Returns (n_accepted[M], out_token[M]); entries of users outside the
    batch are -1."""
    n_acc = np.full(n_users, -1, np.int32)
    tok = np.full(n_users, -1, np.int32)
    _check("sd_accept", lib().sd_accept(ctx, batch, n_acc.ctypes.data, tok.ctypes.data, int(commit)))
    return n_acc, tok


def sd_debug_logits(ctx: int, batch: int, dst, stream=None) -> None:
    _check("sd_debug_logits", lib().sd_debug_logits(ctx, batch, _dev(dst), _stream(stream)))


def sd_debug_wait_limit(ctx: int, max_polls: int) -> None:
    _check("sd_debug_wait_limit", lib().sd_debug_wait_limit(ctx, max_polls))


def sd_profile_begin(ctx: int, kclass: int, max_launches: int = 4096) -> None:
    _check("sd_profile_begin", lib().sd_profile_begin(ctx, kclass, max_launches))


def sd_profile_end(ctx: int):
    """Returns (total_ms, launches) of the profiled kernel class."""
    ms, n = ctypes.c_double(), ctypes.c_int32()
    _check("sd_profile_end", lib().sd_profile_end(ctx, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def sd_calib_hbm(buf_ptr: int, nbytes: int, mode: int, reps: int, stream: int = 0) -> float:
    """Achieved GB/s (bytes read + written) of a copy (mode 0) or read-only
    stream (mode 1) over the caller's device buffer."""
    gbs = ctypes.c_double()
    _check("sd_calib_hbm", lib().sd_calib_hbm(buf_ptr, nbytes, mode, reps, ctypes.byref(gbs), stream))
    return gbs.value


def sd_calib_mfma(sink_ptr: int, iters: int, stream: int = 0) -> float:
    """Achieved dense bf16 MFMA TFLOP/s of a register-only MFMA loop."""
    tf = ctypes.c_double()
    _check("sd_calib_mfma", lib().sd_calib_mfma(sink_ptr, iters, ctypes.byref(tf), stream))
    return tf.value


def make_config(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab, qk_norm, dtype,
                n_pages, max_users, max_draft, max_batch_users, max_batch_tokens, max_ctx,
                max_pending=2, rope_base=1e6, rms_eps=1e-6, logits_out=0) -> sd_config:
    return sd_config(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab, int(qk_norm),
                     int(dtype), 16, n_pages, max_users, max_draft, max_batch_users, max_batch_tokens,
                     max_ctx, max_pending, float(rope_base), float(rms_eps), int(logits_out))
