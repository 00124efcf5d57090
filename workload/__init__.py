"""Seeded synthetic workloads for the speculative-verify pass.

This module holds no arithmetic of the verify method.  It defines the model
shapes and batch recipes, and writes weights, cached keys/values, token ids,
draft distributions and uniforms through the counter-based generator in
``gen.c``.  The CPU oracle and the GPU path both read what it writes.

Shapes follow the Qwen3 models the paper evaluates (DiP-SD, Sec. IV-A and
Table II: a Qwen3-1.7B draft and a Qwen3-32B verifier); weights are random
normal N(0, 0.02) stand-ins because no trained weights are used.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
import subprocess
from typing import Dict, List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libworkload.so")


def build(force: bool = True) -> str:
    """Compile gen.c into libworkload.so (plain gcc, OpenMP)."""
    if force or not os.path.exists(_SO):
        tmp = _SO + ".tmp"
        subprocess.check_call(["gcc", "-O3", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, os.path.join(_HERE, "gen.c"), "-lm"])
        os.replace(tmp, _SO)
    return _SO


_GPU_SO = os.path.join(_HERE, "libworkload_gpu.so")


def build_gpu(force: bool = True) -> str:
    """Compile the bit-identical GPU fill kernels (gen_gpu.hip) for gfx950."""
    if force or not os.path.exists(_GPU_SO):
        tmp = _GPU_SO + ".tmp"
        subprocess.check_call(["hipcc", "--offload-arch=gfx950", "-O3", "-fPIC", "-shared",
                               "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang",
                               "-packed-fp32-ops", "-o", tmp, os.path.join(_HERE, "gen_gpu.hip")],
                              stderr=subprocess.DEVNULL)
        os.replace(tmp, _GPU_SO)
    return _GPU_SO


_glib = None


def glib():
    global _glib
    if _glib is None:
        if not os.path.exists(_GPU_SO):
            raise RuntimeError(f"{_GPU_SO} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(_GPU_SO)
        i64, u64, f32, vp, i32 = ctypes.c_int64, ctypes.c_uint64, ctypes.c_float, ctypes.c_void_p, ctypes.c_int
        L.wlg_fill_normal.argtypes = [vp, i64, u64, u64, i64, f32, i32, vp]
        L.wlg_fill_uniform.argtypes = [vp, i64, u64, u64, i64, f32, f32, i32, vp]
        _glib = L
    return _glib


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        i64, u64, f32 = ctypes.c_int64, ctypes.c_uint64, ctypes.c_float
        vp = ctypes.c_void_p
        L.wl_raw.restype = u64
        L.wl_raw.argtypes = [u64, u64, u64]
        for name in ("wl_fill_normal_f32", "wl_fill_normal_bf16"):
            getattr(L, name).argtypes = [vp, i64, u64, u64, i64, f32]
        for name in ("wl_fill_uniform_f32", "wl_fill_uniform_bf16"):
            getattr(L, name).argtypes = [vp, i64, u64, u64, i64, f32, f32]
        L.wl_fill_int.argtypes = [vp, i64, u64, u64, i64, ctypes.c_int32, ctypes.c_int32]
        L.wl_draft_rows.argtypes = [vp, vp, i64, i64, u64, u64, f32, u64, f32, f32, u64, i64]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    assert a.flags["C_CONTIGUOUS"]
    return ctypes.c_void_p(a.ctypes.data)


# ----------------------------------------------------------------------------
# model shapes
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rope_base: float
    rms_eps: float
    qk_norm: bool
    dtype: str  # "f32" or "bf16": weights, KV cache and GEMM-input precision

    @property
    def wbytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def layer_params(self) -> int:
        d, hd = self.d_model, self.head_dim
        return (d * (self.n_q_heads + 2 * self.n_kv_heads) * hd + self.n_q_heads * hd * d
                + 3 * d * self.d_ffn)

    def kv_bytes_per_token(self) -> int:
        return self.n_layers * 2 * self.n_kv_heads * self.head_dim * self.wbytes


MODELS: Dict[str, ModelShape] = {
    # 2-layer fp32 toy decoder; no QK-norm
    "tiny": ModelShape("tiny", 2, 256, 4, 2, 64, 512, 1024, 1e4, 1e-6, False, "f32"),
    "tiny-qknorm": ModelShape("tiny-qknorm", 2, 256, 4, 2, 64, 512, 1024, 1e4, 1e-6, True, "f32"),
    # bf16 toy decoder with the 32B head layout (hd 128, 8 q per kv head)
    "tiny-bf16": ModelShape("tiny-bf16", 2, 512, 8, 1, 128, 1024, 2048, 1e6, 1e-6, True, "bf16"),
    # the same with a feed-forward width near Qwen3-32B's: 160 gate/up row
    # tiles of 256 rows, more than half and fewer than all of 256 CUs
    "tiny-wide-ffn": ModelShape("tiny-wide-ffn", 2, 512, 8, 1, 128, 20480, 2048, 1e6, 1e-6, True, "bf16"),
    # 96 gate/up row tiles: split over k in two and added by a separate
    # reduction (too wide for the four-wave tiles, too narrow to fill the
    # CUs unsplit)
    "tiny-mid-ffn": ModelShape("tiny-mid-ffn", 2, 512, 8, 1, 128, 12288, 2048, 1e6, 1e-6, True, "bf16"),
    "qwen3-1.7b": ModelShape("qwen3-1.7b", 28, 2048, 16, 8, 128, 6144, 151936, 1e6, 1e-6, True, "bf16"),
    "qwen3-32b": ModelShape("qwen3-32b", 64, 5120, 64, 8, 128, 25600, 151936, 1e6, 1e-6, True, "bf16"),
}

# weight kinds (tensor ids inside a layer); global tensors use layer -1
W_Q, W_K, W_V, W_O, W_G, W_U, W_D, N_1, N_2, N_Q, N_K = range(11)
EMBED, LM_HEAD, NORM_F = 100, 101, 102
WEIGHT_STD = 0.02


def weight_shape(m: ModelShape, kind: int):
    d, hd, F = m.d_model, m.head_dim, m.d_ffn
    return {
        W_Q: (m.n_q_heads * hd, d), W_K: (m.n_kv_heads * hd, d), W_V: (m.n_kv_heads * hd, d),
        W_O: (d, m.n_q_heads * hd), W_G: (F, d), W_U: (F, d), W_D: (d, F),
        N_1: (d,), N_2: (d,), N_Q: (hd,), N_K: (hd,),
        EMBED: (m.vocab, d), LM_HEAD: (m.vocab, d), NORM_F: (d,),
    }[kind]


def _wstream(layer: int, kind: int) -> int:
    return ((layer + 1) << 16) | kind


def fill_weight(m: ModelShape, seed: int, layer: int, kind: int, out: np.ndarray,
                gamma: str = "ones") -> np.ndarray:
    """Write weight `kind` of `layer` into `out` (float32, or uint16 bf16 bits).

    Linear and embedding weights are N(0, 0.02).  Norm gains are 1 ("ones")
    or U(0.5, 1.5) ("uniform", used by tests so that a kernel ignoring a gain
    is caught).
    """
    n = out.size
    is_norm = kind in (N_1, N_2, N_Q, N_K, NORM_F)
    L = lib()
    s = _wstream(layer, kind)
    if is_norm:
        if gamma == "ones":
            if out.dtype == np.uint16:
                out[...] = 0x3F80
            else:
                out[...] = 1.0
        else:
            fn = L.wl_fill_uniform_bf16 if out.dtype == np.uint16 else L.wl_fill_uniform_f32
            fn(_ptr(out), n, seed, s, 0, 0.5, 1.5)
    else:
        fn = L.wl_fill_normal_bf16 if out.dtype == np.uint16 else L.wl_fill_normal_f32
        fn(_ptr(out), n, seed, s, 0, WEIGHT_STD)
    return out


def new_weight(m: ModelShape, seed: int, layer: int, kind: int, gamma: str = "ones") -> np.ndarray:
    dt = np.float32 if m.dtype == "f32" else np.uint16
    out = np.empty(weight_shape(m, kind), dtype=dt)
    return fill_weight(m, seed, layer, kind, out, gamma)


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    return (a.astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 bits (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


# ----------------------------------------------------------------------------
# cached keys / values (synthetic)
# ----------------------------------------------------------------------------

KV_STD = 1.0


def _kvstream(layer: int, user: int, which: int) -> int:
    return (0x4B56 << 48) | (layer << 24) | (user << 1) | which


def fill_kv(m: ModelShape, seed: int, layer: int, user: int, which: int, out: np.ndarray,
            pos0: int = 0) -> np.ndarray:
    """Synthetic cached key (which=0) or value (1) rows of one user at one
    layer: positions pos0.. as [n][n_kv_heads][head_dim], N(0, 1)."""
    per_tok = m.n_kv_heads * m.head_dim
    L = lib()
    fn = L.wl_fill_normal_bf16 if out.dtype == np.uint16 else L.wl_fill_normal_f32
    fn(_ptr(out), out.size, seed, _kvstream(layer, user, which), pos0 * per_tok, KV_STD)
    return out


# ----------------------------------------------------------------------------
# batches
# ----------------------------------------------------------------------------

S_PREFIX_TOK, S_ROOT, S_Q_A, S_Q_B, S_DRAFT_U, S_ACCEPT_U, S_LEN, S_PLEN, S_ASSIGN = (
    0x7001, 0x7002, 0x7003, 0x7004, 0x7005, 0x7006, 0x7007, 0x7008, 0x7009)


@dataclasses.dataclass
class Batch:
    """One verify batch: users (global ids, ascending), their prefix
    lengths i_m, draft lengths l_m, root tokens, drafts and draft
    distributions q (one row per draft), optional accept uniforms."""
    users: np.ndarray          # int32 [B]
    prefix_len: np.ndarray     # int32 [B]
    draft_len: np.ndarray      # int32 [B]
    root: np.ndarray           # int32 [B]
    drafts: np.ndarray         # int32 [sum L]
    q: np.ndarray              # float32 [sum L, V]
    accept_u: Optional[np.ndarray]  # float32 [sum L] or None (in-kernel Philox)

    @property
    def n_slots(self) -> np.ndarray:
        return self.draft_len + 1

    @property
    def T(self) -> int:
        return int(self.n_slots.sum())

    def slot_tokens(self) -> np.ndarray:
        out, o = [], 0
        for b in range(len(self.users)):
            out.append(int(self.root[b]))
            out.extend(int(t) for t in self.drafts[o:o + self.draft_len[b]])
            o += int(self.draft_len[b])
        return np.asarray(out, dtype=np.int32)


@dataclasses.dataclass
class Workload:
    name: str
    model: ModelShape
    n_users: int
    prefix_len: np.ndarray       # int32 [M]
    draft_len: np.ndarray        # int32 [M]
    assign: np.ndarray           # int32 [M] batch index per user
    n_batches: int
    q_sigma: float               # std of the "target-shaped" draft logits
    q_mix: float                 # weight of the target-shaped softmax in q
    q_sigma_b: float             # std of the second softmax component
    accept_u_input: bool         # pass accept uniforms in (else in-kernel Philox)
    kv: str                      # "synthetic" or "prefill"
    seed: int
    modes: tuple = ("stochastic",)

    def batch(self, n: int) -> Batch:
        users = np.nonzero(self.assign == n)[0].astype(np.int32)
        return make_batch(self, users)


def _ints(n: int, seed: int, stream: int, lo: int, hi: int, offset: int = 0) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    lib().wl_fill_int(_ptr(out), n, seed, stream, offset, lo, hi)
    return out


def prefix_tokens(w: Workload, user: int, n: Optional[int] = None) -> np.ndarray:
    n = int(w.prefix_len[user]) if n is None else n
    return _ints(n, w.seed, (S_PREFIX_TOK << 20) | user, 0, w.model.vocab - 1)


def make_batch(w: Workload, users: np.ndarray) -> Batch:
    V = w.model.vocab
    Ls = w.draft_len[users].astype(np.int32)
    nd = int(Ls.sum())
    q = np.empty((nd, V), dtype=np.float32)
    drafts = np.empty(nd, dtype=np.int32)
    o = 0
    for u, Lb in zip(users, Ls):
        lib().wl_draft_rows(_ptr(q[o:o + Lb]), _ptr(drafts[o:o + Lb]), int(Lb), V, w.seed,
                            (S_Q_A << 20) | int(u), w.q_sigma, (S_Q_B << 20) | int(u),
                            w.q_sigma_b, w.q_mix, (S_DRAFT_U << 20) | int(u), 0)
        o += int(Lb)
    root = np.array([_ints(1, w.seed, (S_ROOT << 20) | int(u), 0, V - 1)[0] for u in users],
                    dtype=np.int32)
    acc = None
    if w.accept_u_input:
        acc = np.empty(nd, dtype=np.float32)
        o = 0
        for u, Lb in zip(users, Ls):
            lib().wl_fill_uniform_f32(_ptr(acc[o:o + Lb]), int(Lb), w.seed,
                                      (S_ACCEPT_U << 20) | int(u), 0, 0.0, 1.0)
            o += int(Lb)
    return Batch(users=users.astype(np.int32), prefix_len=w.prefix_len[users].astype(np.int32),
                 draft_len=Ls, root=root, drafts=drafts, q=q, accept_u=acc)


def workload(name: str, seed: Optional[int] = None) -> Workload:
    """The five benchmark workloads plus small test variants."""
    if name == "tiny":
        m, s = MODELS["tiny"], 1 if seed is None else seed
        return Workload(name, m, 4, np.array([64, 96, 112, 128], np.int32),
                        np.array([1, 2, 3, 4], np.int32), np.zeros(4, np.int32), 1,
                        q_sigma=1.0, q_mix=1.0, q_sigma_b=1.0, accept_u_input=True,
                        kv="prefill", seed=s)
    if name == "qwen3-1.7b-b8":
        m, s = MODELS["qwen3-1.7b"], 2 if seed is None else seed
        return Workload(name, m, 8, np.full(8, 512, np.int32), _ints(8, s, S_LEN, 1, 8),
                        np.zeros(8, np.int32), 1, q_sigma=WEIGHT_STD * math.sqrt(m.d_model),
                        q_mix=1.0, q_sigma_b=1.0, accept_u_input=False, kv="synthetic", seed=s)
    if name == "qwen3-32b-b16":
        m, s = MODELS["qwen3-32b"], 3 if seed is None else seed
        return Workload(name, m, 16, np.full(16, 1024, np.int32), np.full(16, 4, np.int32),
                        np.zeros(16, np.int32), 1, q_sigma=WEIGHT_STD * math.sqrt(m.d_model),
                        q_mix=1.0, q_sigma_b=1.0, accept_u_input=False, kv="synthetic", seed=s,
                        modes=("stochastic", "greedy"))
    if name == "qwen3-32b-ragged32":
        m, s = MODELS["qwen3-32b"], 4 if seed is None else seed
        return Workload(name, m, 32, _ints(32, s, S_PLEN, 256, 4096), _ints(32, s, S_LEN, 1, 12),
                        np.zeros(32, np.int32), 1, q_sigma=WEIGHT_STD * math.sqrt(m.d_model),
                        q_mix=0.7, q_sigma_b=1.0, accept_u_input=False, kv="synthetic", seed=s)
    if name == "qwen3-32b-pipe4x16":
        m, s = MODELS["qwen3-32b"], 5 if seed is None else seed
        perm = np.argsort(_ints(64, s, S_ASSIGN, 0, 2**30), kind="stable")
        assign = np.empty(64, np.int32)
        assign[perm] = np.arange(64) // 16
        return Workload(name, m, 64, _ints(64, s, S_PLEN, 1024, 8192), _ints(64, s, S_LEN, 1, 10),
                        assign, 4, q_sigma=WEIGHT_STD * math.sqrt(m.d_model), q_mix=1.0,
                        q_sigma_b=1.0, accept_u_input=False, kv="synthetic", seed=s)
    raise KeyError(name)


WORKLOADS = ("tiny", "qwen3-1.7b-b8", "qwen3-32b-b16", "qwen3-32b-ragged32", "qwen3-32b-pipe4x16")


def custom_workload(model: str, prefix_len: List[int], draft_len: List[int], seed: int = 11,
                    q_sigma: float = 1.0, q_mix: float = 1.0, accept_u_input: bool = False,
                    kv: str = "synthetic", assign: Optional[List[int]] = None) -> Workload:
    """A small workload for tests: explicit per-user prefix and draft lengths."""
    m = MODELS[model]
    n = len(prefix_len)
    a = np.zeros(n, np.int32) if assign is None else np.asarray(assign, np.int32)
    return Workload("custom", m, n, np.asarray(prefix_len, np.int32),
                    np.asarray(draft_len, np.int32), a, int(a.max()) + 1 if n else 1,
                    q_sigma=q_sigma, q_mix=q_mix, q_sigma_b=1.0, accept_u_input=accept_u_input,
                    kv=kv, seed=seed)


S_SPARSE_U = 0x700A  # stream of the uniforms that redraw drafts from sparse rows


@dataclasses.dataclass
class SparseRows:
    idx: np.ndarray    # int32 [nd][K]  listed tokens, distinct
    val: np.ndarray    # fp32 [nd][K]   their probabilities
    rest: np.ndarray   # fp32 [nd]      probability of every other token


def sparsify(b: Batch, K: int, seed: int) -> SparseRows:
    """Input construction for the sparse-payload variant: each dense draft
    row of `b` becomes its K most likely tokens (ties to the lower id) with
    their probabilities plus a uniform remainder (1 - sum) / (V - K), and the
    drafts are redrawn from those sparse rows (inverse CDF on a seeded
    uniform per draft, listed tokens first in increasing id, then the other
    tokens in increasing id), so the drafts follow the distribution the
    verification is given.  `b.drafts` is replaced in place."""
    nd, V = b.q.shape
    assert 1 <= K < V
    idx = np.empty((nd, K), np.int32)
    val = np.empty((nd, K), np.float32)
    rest = np.empty(nd, np.float32)
    u = np.empty(max(nd, 1), np.float32)
    lib().wl_fill_uniform_f32(_ptr(u), int(max(nd, 1)), seed, S_SPARSE_U, 0, 0.0, 1.0)
    for r in range(nd):
        row = b.q[r].astype(np.float64)
        top = np.lexsort((np.arange(V), -row))[:K]
        top = np.sort(top)
        idx[r] = top
        val[r] = b.q[r, top]
        listed = float(np.sum(val[r].astype(np.float64)))
        rest[r] = np.float32(max(1.0 - listed, 0.0) / (V - K))
        # inverse CDF over (listed tokens by id, then the others by id)
        x = float(u[r])
        cum = np.cumsum(val[r].astype(np.float64))
        if x < cum[-1]:
            d = int(top[np.searchsorted(cum, x, side="right")])
        else:
            j = min(int((x - cum[-1]) / max(float(rest[r]), 1e-300)), V - K - 1)
            others = np.setdiff1d(np.arange(V), top, assume_unique=True)
            d = int(others[j])
        b.drafts[r] = d
    return SparseRows(idx, val, rest)
