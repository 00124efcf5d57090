"""CPU oracle for the batched speculative-verify pass -- TEST INFRASTRUCTURE.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the GPU library and
its Python binding) never calls it, and the two share no code: the only
common dependency is the seeded input generator in ``workload``.

The arithmetic lives in ``oracle.c`` (plain C, double accumulation); this
module compiles it, marshals arguments, and feeds it weights and cached
keys/values produced by ``workload``.

Parity status of each function (see the test suite for the pins):
  philox4x64_10    -- pinned to numpy's independent Philox implementation
  sample           -- pinned by exact enumeration of the output law on tiny
                      vocabularies (every draft sequence, accept/reject
                      outcome and resampled token over several rounds, using
                      the oracle's own ratios and race weights: the law of
                      the first n tokens equals the target's to 1e-6), by
                      Monte-Carlo chi^2 tests of the race itself, q = p,
                      greedy longest prefix, and the geometric mean of eq. (1)
  forward          -- pinned by textbook special cases (RMSNorm, RoPE,
                      attention, SwiGLU structure), verify/prefill and
                      autoregressive consistency, and a torch.nn.functional
                      re-implementation on tiny models, with and without the
                      bf16 rounding of the new slots' keys and values
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

import workload as wl

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")

GREEDY, STOCHASTIC, FORCE = 0, 1, 2
MODES = {"greedy": GREEDY, "stochastic": STOCHASTIC, "force": FORCE}


def build(force: bool = True) -> str:
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp"
        # -O2 without fast-math: no reassociation of the double sums
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp,
                               os.path.join(_HERE, "oracle.c"), "-lm"])
        os.replace(tmp, _SO)
    return _SO


class _Model(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_ffn", "vocab",
        "qk_norm", "kv_bf16", "wdtype")] + [("rope_base", ctypes.c_double),
                                             ("rms_eps", ctypes.c_double)]


class _Layer(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "wq", "wk", "wv", "wo", "wg", "wu", "wd", "norm1", "norm2", "qnorm", "knorm")]


_LAYER_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(_Layer))
_KV_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                          ctypes.c_void_p, ctypes.c_void_p)

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        vp, u64, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32
        L.or_philox4x64_10.argtypes = [vp, vp, vp]
        L.or_accept_uniform.restype = ctypes.c_float
        L.or_accept_uniform.argtypes = [u64]
        L.or_race_uniform.restype = ctypes.c_float
        L.or_race_uniform.argtypes = [u64]
        L.or_race_exponential.restype = ctypes.c_float
        L.or_race_exponential.argtypes = [u64]
        L.or_round_bf16.restype = ctypes.c_double
        L.or_round_bf16.argtypes = [ctypes.c_double]
        L.or_rmsnorm.argtypes = [vp, ctypes.c_int, vp, ctypes.c_int, ctypes.c_double, vp]
        L.or_rope.argtypes = [vp, ctypes.c_int, ctypes.c_double, ctypes.c_double]
        L.or_attend.argtypes = [vp, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_long,
                                ctypes.c_double, vp]
        L.or_forward.argtypes = [ctypes.POINTER(_Model), i32, vp, vp, vp, vp, vp, vp,
                                 _LAYER_FN, _KV_FN, vp, vp, vp, vp]
        L.or_sample.argtypes = [i32, i32, vp, vp, ctypes.c_int64, vp, vp, vp, vp, u64, u64,
                                vp, vp, vp, vp, vp, vp]
        L.or_omp_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "arrays passed to the oracle must be contiguous"
    return ctypes.c_void_p(a.ctypes.data)


# ----------------------------------------------------------------------------
# primitives (exposed for the pins)
# ----------------------------------------------------------------------------

def omp_threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return int(lib().or_omp_threads())


def philox4x64_10(ctr, key) -> np.ndarray:
    c = np.asarray(ctr, dtype=np.uint64).copy()
    k = np.asarray(key, dtype=np.uint64).copy()
    out = np.empty(4, dtype=np.uint64)
    lib().or_philox4x64_10(_p(c), _p(k), _p(out))
    return out


def accept_uniform(x: int) -> float:
    return lib().or_accept_uniform(int(x))


def race_uniform(x: int) -> float:
    return lib().or_race_uniform(int(x))


def race_exponential(x: int) -> float:
    return lib().or_race_exponential(int(x))


def round_bf16(x: float) -> float:
    return lib().or_round_bf16(float(x))


def rmsnorm(x, gamma=None, eps=1e-6) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    g = None if gamma is None else np.ascontiguousarray(gamma, dtype=np.float32)
    lib().or_rmsnorm(_p(x), x.size, _p(g), 0, eps, _p(y))
    return y


def rope(v, pos: float, base: float) -> np.ndarray:
    v = np.array(v, dtype=np.float64)
    lib().or_rope(_p(v), v.size, float(pos), float(base))
    return v


def attend(q, k, v, scale: Optional[float] = None) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    n, hd = k.shape
    o = np.empty(hd, dtype=np.float64)
    s = 1.0 / np.sqrt(hd) if scale is None else scale
    lib().or_attend(_p(q), _p(k), _p(v), n, hd, hd, s, _p(o))
    return o


# ----------------------------------------------------------------------------
# forward
# ----------------------------------------------------------------------------

def _model_struct(m: wl.ModelShape, kv_bf16: Optional[bool] = None) -> _Model:
    return _Model(m.n_layers, m.d_model, m.n_q_heads, m.n_kv_heads, m.head_dim, m.d_ffn, m.vocab,
                  int(m.qk_norm), int(m.dtype == "bf16" if kv_bf16 is None else kv_bf16),
                  int(m.dtype == "bf16"), m.rope_base, m.rms_eps)


class WeightSource:
    """Weights of a seeded model, generated per layer on demand."""

    def __init__(self, m: wl.ModelShape, seed: int, gamma: str = "ones"):
        self.m, self.seed, self.gamma = m, seed, gamma
        self._glob = {k: wl.new_weight(m, seed, -1, k, gamma) for k in (wl.EMBED, wl.LM_HEAD, wl.NORM_F)}

    def global_(self, kind):
        return self._glob[kind]

    def layer(self, l: int):
        return {k: wl.new_weight(self.m, self.seed, l, k, self.gamma) for k in (
            wl.W_Q, wl.W_K, wl.W_V, wl.W_O, wl.W_G, wl.W_U, wl.W_D, wl.N_1, wl.N_2, wl.N_Q, wl.N_K)}


class KVSource:
    """Cached keys/values per (layer, batch user): synthetic from the
    generator, or explicit arrays {user: (K[J][P][hkv][hd], V[...])}."""

    def __init__(self, m: wl.ModelShape, seed: int, users, prefix_len, explicit=None):
        self.m, self.seed = m, seed
        self.users = [int(u) for u in users]
        self.prefix_len = [int(p) for p in prefix_len]
        self.explicit = explicit

    def fill(self, layer: int, b: int, kout: np.ndarray, vout: np.ndarray):
        P = self.prefix_len[b]
        n = P * self.m.n_kv_heads * self.m.head_dim
        if self.explicit is not None:
            K, V = self.explicit[self.users[b]]
            kout[:n] = K[layer, :P].reshape(-1)
            vout[:n] = V[layer, :P].reshape(-1)
            return
        if self.m.dtype == "bf16":
            tmp = np.empty(n, np.uint16)
            wl.fill_kv(self.m, self.seed, layer, self.users[b], 0, tmp)
            kout[:n] = wl.bf16_to_f32(tmp)
            wl.fill_kv(self.m, self.seed, layer, self.users[b], 1, tmp)
            vout[:n] = wl.bf16_to_f32(tmp)
        else:
            wl.fill_kv(self.m, self.seed, layer, self.users[b], 0, kout[:n])
            wl.fill_kv(self.m, self.seed, layer, self.users[b], 1, vout[:n])


def forward(m: wl.ModelShape, weights: WeightSource, kv: Optional[KVSource], prefix_len, n_slots,
            tokens, want_kv: bool = False, kv_bf16: Optional[bool] = None):
    """Logits [T][V] (float32) of the verify forward; optionally the new
    slots' K and V [J][T][hkv][hd]."""
    prefix_len = np.ascontiguousarray(prefix_len, dtype=np.int32)
    n_slots = np.ascontiguousarray(n_slots, dtype=np.int32)
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    T = int(n_slots.sum())
    assert tokens.size == T
    assert int(tokens.min(initial=0)) >= 0 and int(tokens.max(initial=0)) < m.vocab
    logits = np.empty((T, m.vocab), dtype=np.float32)
    nk = m.n_kv_heads * m.head_dim
    knew = np.empty((m.n_layers, T, nk), np.float32) if want_kv else None
    vnew = np.empty((m.n_layers, T, nk), np.float32) if want_kv else None
    keep = {}

    def layer_cb(_cb, l, out):
        try:
            w = weights.layer(int(l))
            keep["l"] = w
            o = out.contents
            o.wq, o.wk, o.wv, o.wo = (w[wl.W_Q].ctypes.data, w[wl.W_K].ctypes.data,
                                      w[wl.W_V].ctypes.data, w[wl.W_O].ctypes.data)
            o.wg, o.wu, o.wd = w[wl.W_G].ctypes.data, w[wl.W_U].ctypes.data, w[wl.W_D].ctypes.data
            o.norm1, o.norm2 = w[wl.N_1].ctypes.data, w[wl.N_2].ctypes.data
            o.qnorm, o.knorm = w[wl.N_Q].ctypes.data, w[wl.N_K].ctypes.data
            return 0
        except Exception:  # pragma: no cover - reported as a nonzero status
            import traceback
            traceback.print_exc()
            return -1

    def kv_cb(_cb, l, b, kptr, vptr):
        try:
            P = int(prefix_len[b])
            n = P * nk
            kout = np.ctypeslib.as_array(ctypes.cast(kptr, ctypes.POINTER(ctypes.c_float)), (max(n, 1),))
            vout = np.ctypeslib.as_array(ctypes.cast(vptr, ctypes.POINTER(ctypes.c_float)), (max(n, 1),))
            kv.fill(int(l), int(b), kout, vout)
            return 0
        except Exception:  # pragma: no cover
            import traceback
            traceback.print_exc()
            return -1

    lcb, kcb = _LAYER_FN(layer_cb), _KV_FN(kv_cb)
    ms = _model_struct(m, kv_bf16)
    rc = lib().or_forward(ctypes.byref(ms), len(n_slots), _p(prefix_len), _p(n_slots), _p(tokens),
                          _p(weights.global_(wl.EMBED)), _p(weights.global_(wl.NORM_F)),
                          _p(weights.global_(wl.LM_HEAD)), lcb, kcb, None, _p(logits),
                          _p(knew), _p(vnew))
    if rc != 0:
        raise RuntimeError(f"oracle forward failed ({rc})")
    if want_kv:
        return logits, knew, vnew
    return logits


def prefill(m: wl.ModelShape, weights: WeightSource, tokens, kv_bf16: Optional[bool] = None):
    """Keys/values [J][P][hkv][hd] of a full causal forward over `tokens`."""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    P = tokens.size
    _, K, V = forward(m, weights, None, [0], [P], tokens, want_kv=True, kv_bf16=kv_bf16)
    if m.dtype == "bf16":
        K = wl.bf16_to_f32(wl.f32_to_bf16(K))
        V = wl.bf16_to_f32(wl.f32_to_bf16(V))
    return K, V


# ----------------------------------------------------------------------------
# sampler
# ----------------------------------------------------------------------------

def expand_sparse_q(idx, val, rest, V: int) -> np.ndarray:
    """Dense rows of sparse draft distributions: q_r(k) = val[r][i] where
    k = idx[r][i], else rest[r] (the compact payload of drafted tokens plus a
    little probability information, DiP-SD Sec. II-A).  The accept/resample
    step is defined on these dense rows; nothing else changes."""
    idx = np.asarray(idx)
    q = np.repeat(np.asarray(rest, np.float32)[:, None], V, axis=1)
    rows = np.arange(idx.shape[0])[:, None]
    q[rows, idx] = np.asarray(val, np.float32)
    return q


def sample(mode, users, draft_len, logits, drafts, q, accept_u=None, seed: int = 0,
           round_: int = 0, want_race_w: bool = False):
    """Verify decisions for a batch: returns dict with n_acc, token, and the
    diagnostics ratio (p/q per draft, fp32), u (uniform per draft) and
    race_gap (relative gap of the two best race keys per user); with
    want_race_w also race_w [B][V], the weights of the stop slot's race."""
    mode = MODES[mode] if isinstance(mode, str) else int(mode)
    users = np.ascontiguousarray(users, dtype=np.int32)
    L = np.ascontiguousarray(draft_len, dtype=np.int32)
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    drafts = np.ascontiguousarray(drafts, dtype=np.int32)
    q = np.ascontiguousarray(q, dtype=np.float32)
    V = logits.shape[1]
    nd = int(L.sum())
    assert logits.shape[0] == nd + len(L)
    assert drafts.size == nd
    if mode == STOCHASTIC:
        assert q.shape == (nd, V)
    au = None if accept_u is None else np.ascontiguousarray(accept_u, dtype=np.float32)
    B = len(L)
    n_acc = np.empty(B, np.int32)
    tok = np.empty(B, np.int32)
    ratio = np.empty(max(nd, 1), np.float32)
    uu = np.empty(max(nd, 1), np.float32)
    gap = np.empty(B, np.float64)
    qp = q if q.size else np.zeros((1, V), np.float32)
    rw = np.empty((B, V), np.float32) if want_race_w else None
    lib().or_sample(mode, B, _p(users), _p(L), V, _p(logits), _p(drafts), _p(qp), _p(au),
                    int(seed), int(round_), _p(n_acc), _p(tok), _p(ratio), _p(uu), _p(gap), _p(rw))
    out = {"n_acc": n_acc, "token": tok, "ratio": ratio[:nd], "u": uu[:nd], "race_gap": gap}
    if want_race_w:
        out["race_w"] = rw
    return out
