"""Pins for the oracle's verify forward.

The paper prints no logits, so the forward is pinned by
  * an independent re-implementation built from torch.nn.functional library
    routines (rms_norm, linear, scaled_dot_product_attention with grouped
    query heads, silu) on small models, in float64;
  * properties any correct verify forward has: the verify over
    [root, d_1..d_l] equals the last rows of a full causal forward
    (verify/prefill consistency), one (l+1)-slot verify equals l+1 one-slot
    steps (autoregressive consistency), slots do not see later slots
    (causality), and users are independent (batch permutation);
  * structured weights whose output is known in closed form.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import workload as wl


def _t(a, m):
    a = wl.bf16_to_f32(a) if a.dtype == np.uint16 else a
    return torch.tensor(a, dtype=torch.float64)


def _rope_torch(x, pos, base):
    """rotate-half RoPE written as complex multiplication of (x_a, x_{a+h})"""
    hd = x.shape[-1]
    h = hd // 2
    inv = base ** (-torch.arange(0, hd, 2, dtype=torch.float64) / hd)
    ang = pos[:, None].to(torch.float64) * inv[None]
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]
    c = torch.complex(x[..., :h], x[..., h:]) * rot
    return torch.cat([c.real, c.imag], dim=-1)


def _bf16(x):
    """round through float32 to bfloat16 (nearest-even), back to float64"""
    return x.to(torch.float32).to(torch.bfloat16).to(torch.float64)


def torch_verify(m, ws, kv, prefix_len, n_slots, tokens, kv_bf16=False, round_at="cache"):
    """Verify logits from torch.nn.functional routines in float64.  With
    kv_bf16 the new slots' keys and values are rounded to bfloat16 where a
    bf16 cache stores them: keys after QK-norm and RoPE (round_at="cache"),
    or, for the sensitivity check, before them (round_at="projection")."""
    d, hq, hkv, hd, eps = m.d_model, m.n_q_heads, m.n_kv_heads, m.head_dim, m.rms_eps
    T = int(np.sum(n_slots))
    x = _t(ws.global_(wl.EMBED), m)[torch.tensor(tokens, dtype=torch.long)]
    pos = torch.tensor(np.concatenate([np.arange(n) + p for p, n in zip(prefix_len, n_slots)]))
    off = np.concatenate([[0], np.cumsum(n_slots)])
    for l in range(m.n_layers):
        w = {k: _t(v, m) for k, v in ws.layer(l).items()}
        h = F.rms_norm(x, (d,), w[wl.N_1], eps)
        q = F.linear(h, w[wl.W_Q]).view(T, hq, hd)
        k = F.linear(h, w[wl.W_K]).view(T, hkv, hd)
        v = F.linear(h, w[wl.W_V]).view(T, hkv, hd)
        if kv_bf16 and round_at == "projection":
            k = _bf16(k)
        if m.qk_norm:
            q = F.rms_norm(q, (hd,), w[wl.N_Q], eps)
            k = F.rms_norm(k, (hd,), w[wl.N_K], eps)
        q, k = _rope_torch(q, pos, m.rope_base), _rope_torch(k, pos, m.rope_base)
        if kv_bf16:
            if round_at == "cache":
                k = _bf16(k)
            v = _bf16(v)
        out = torch.empty(T, hq, hd, dtype=torch.float64)
        for b in range(len(n_slots)):
            P, n = int(prefix_len[b]), int(n_slots[b])
            Kc = np.zeros((P, hkv * hd), np.float32)
            Vc = np.zeros((P, hkv * hd), np.float32)
            if P:
                kv.fill(l, b, Kc.reshape(-1), Vc.reshape(-1))
            Kb = torch.cat([torch.tensor(Kc, dtype=torch.float64).view(P, hkv, hd), k[off[b]:off[b + 1]]])
            Vb = torch.cat([torch.tensor(Vc, dtype=torch.float64).view(P, hkv, hd), v[off[b]:off[b + 1]]])
            mask = torch.arange(P + n)[None, :] <= (P + torch.arange(n))[:, None]
            o = F.scaled_dot_product_attention(q[off[b]:off[b + 1]].transpose(0, 1)[None],
                                               Kb.transpose(0, 1)[None], Vb.transpose(0, 1)[None],
                                               attn_mask=mask, enable_gqa=True)
            out[off[b]:off[b + 1]] = o[0].transpose(0, 1)
        x = x + F.linear(out.reshape(T, hq * hd), w[wl.W_O])
        h2 = F.rms_norm(x, (d,), w[wl.N_2], eps)
        x = x + F.linear(F.silu(F.linear(h2, w[wl.W_G])) * F.linear(h2, w[wl.W_U]), w[wl.W_D])
    z = F.rms_norm(x, (d,), _t(ws.global_(wl.NORM_F), m), eps)
    return F.linear(z, _t(ws.global_(wl.LM_HEAD), m)).numpy()


def _rel_err(a, b):
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


@pytest.mark.parametrize("model", ["tiny", "tiny-qknorm", "tiny-bf16"])
def test_forward_matches_torch_functional(model):
    m = wl.MODELS[model]
    ws = oracle.WeightSource(m, seed=21, gamma="uniform")
    prefix, slots = [5, 0, 17, 3], [2, 4, 1, 3]
    users = [0, 1, 2, 3]
    kv = oracle.KVSource(m, 21, users, prefix)
    tokens = np.random.default_rng(0).integers(0, m.vocab, size=sum(slots)).astype(np.int32)
    got = oracle.forward(m, ws, kv, prefix, slots, tokens, kv_bf16=False)
    ref = torch_verify(m, ws, kv, prefix, slots, tokens)
    assert _rel_err(got, ref) < 1e-6  # fp32 storage of the oracle's logits


def _tokens(m, n, seed):
    return np.random.default_rng(seed).integers(0, m.vocab, size=n).astype(np.int32)


@pytest.mark.parametrize("model", ["tiny", "tiny-bf16"])
def test_verify_equals_prefill_rows(model):
    m = wl.MODELS[model]
    ws = oracle.WeightSource(m, seed=22, gamma="uniform")
    P, n = 20, 5
    toks = _tokens(m, P + n, 1)
    full = oracle.forward(m, ws, None, [0], [P + n], toks)
    K, V = oracle.prefill(m, ws, toks[:P])
    kv = oracle.KVSource(m, 22, [0], [P], explicit={0: (K, V)})
    ver = oracle.forward(m, ws, kv, [P], [n], toks[P:])
    tol = 1e-5 if m.dtype == "f32" else 2e-2
    assert _rel_err(ver, full[P:]) < tol


def test_autoregressive_consistency():
    m = wl.MODELS["tiny-qknorm"]
    ws = oracle.WeightSource(m, seed=23, gamma="uniform")
    P, n = 9, 4
    toks = _tokens(m, P + n, 2)
    K, V = oracle.prefill(m, ws, toks[:P])
    one = oracle.forward(m, ws, oracle.KVSource(m, 0, [0], [P], explicit={0: (K, V)}), [P], [n], toks[P:])
    rows = []
    for j in range(n):
        kvj = oracle.KVSource(m, 0, [0], [P + j], explicit={0: (K, V)})
        lg, Kn, Vn = oracle.forward(m, ws, kvj, [P + j], [1], toks[P + j:P + j + 1], want_kv=True)
        rows.append(lg[0])
        K = np.concatenate([K, Kn], axis=1)
        V = np.concatenate([V, Vn], axis=1)
    assert _rel_err(np.stack(rows), one) < 1e-6


def test_causality_and_user_independence():
    m = wl.MODELS["tiny"]
    ws = oracle.WeightSource(m, seed=24)
    prefix, slots = [12, 30, 7], [4, 2, 3]
    kv = oracle.KVSource(m, 24, [5, 6, 7], prefix)
    toks = _tokens(m, sum(slots), 3)
    base = oracle.forward(m, ws, kv, prefix, slots, toks)
    # change the last slot of user 0: its earlier slots and other users are unchanged
    t2 = toks.copy()
    t2[3] = (t2[3] + 1) % m.vocab
    alt = oracle.forward(m, ws, kv, prefix, slots, t2)
    assert np.array_equal(alt[:3], base[:3]) and np.array_equal(alt[4:], base[4:])
    assert not np.array_equal(alt[3], base[3])
    # permute users: rows permute with them
    perm = [2, 0, 1]
    off = np.concatenate([[0], np.cumsum(slots)])
    kvp = oracle.KVSource(m, 24, [[5, 6, 7][i] for i in perm], [prefix[i] for i in perm])
    tp = np.concatenate([toks[off[i]:off[i + 1]] for i in perm])
    pr = oracle.forward(m, ws, kvp, [prefix[i] for i in perm], [slots[i] for i in perm], tp)
    ref = np.concatenate([base[off[i]:off[i + 1]] for i in perm])
    assert np.array_equal(pr, ref)


class _ZeroBlocks(oracle.WeightSource):
    """Attention and FFN output projections set to zero: every block adds
    nothing, so logits = RMSNorm(E[t]) W_lm^T exactly."""

    def layer(self, l):
        w = super().layer(l)
        w[wl.W_O] = np.zeros_like(w[wl.W_O])
        w[wl.W_D] = np.zeros_like(w[wl.W_D])
        return w


def test_structured_weights_closed_form():
    m = wl.MODELS["tiny"]
    ws = _ZeroBlocks(m, seed=25, gamma="uniform")
    toks = _tokens(m, 6, 4)
    got = oracle.forward(m, ws, oracle.KVSource(m, 25, [0], [10]), [10], [6], toks)
    E = ws.global_(wl.EMBED).astype(np.float64)[toks]
    g = ws.global_(wl.NORM_F).astype(np.float64)
    h = E / np.sqrt((E * E).mean(1, keepdims=True) + m.rms_eps) * g
    ref = h @ ws.global_(wl.LM_HEAD).astype(np.float64).T
    assert _rel_err(got, ref) < 1e-6


@pytest.mark.parametrize("model", ["tiny-bf16", "tiny-qknorm"])
def test_bf16_kv_rounding_matches_torch(model):
    """The oracle's bf16 cache reading: the new slots' keys (after QK-norm
    and RoPE) and values are rounded to bf16 before any slot reads them.
    A torch float64 re-implementation that rounds at exactly those points
    agrees to fp32 storage; rounding the keys before QK-norm/RoPE instead
    (a plausible misplacement) is far outside that bound."""
    m = wl.MODELS[model]
    ws = oracle.WeightSource(m, seed=27, gamma="uniform")
    prefix, slots = [9, 0, 21], [3, 4, 2]
    kv = oracle.KVSource(m, 27, [0, 1, 2], prefix)
    tokens = _tokens(m, sum(slots), 6)
    got = oracle.forward(m, ws, kv, prefix, slots, tokens, kv_bf16=True)
    ref = torch_verify(m, ws, kv, prefix, slots, tokens, kv_bf16=True)
    assert _rel_err(got, ref) < 1e-6
    unrounded = torch_verify(m, ws, kv, prefix, slots, tokens, kv_bf16=False)
    misplaced = torch_verify(m, ws, kv, prefix, slots, tokens, kv_bf16=True, round_at="projection")
    assert _rel_err(got, unrounded) > 1e-4
    assert _rel_err(got, misplaced) > 1e-4


def test_bf16_kv_cache_rounding_changes_little():
    """Rounding the new slots' keys and values to bf16 (what a bf16 cache
    stores) moves the logits by bf16-level noise only, and does nothing to
    the first slot of a user with an empty prefix, which sees only itself."""
    m = wl.MODELS["tiny-bf16"]
    ws = oracle.WeightSource(m, seed=26)
    kv = oracle.KVSource(m, 26, [0, 1], [33, 8])
    toks = _tokens(m, 7, 5)
    a = oracle.forward(m, ws, kv, [33, 8], [3, 4], toks, kv_bf16=True)
    b = oracle.forward(m, ws, kv, [33, 8], [3, 4], toks, kv_bf16=False)
    e = _rel_err(a, b)
    assert 1e-6 < e < 2e-2
    # one slot, no prefix: softmax over one key is 1, so o = round(v) vs v;
    # the output projection sees a different input, but the difference is
    # bounded by one bf16 rounding of v
    kv0 = oracle.KVSource(m, 26, [0], [0])
    c = oracle.forward(m, ws, kv0, [0], [1], toks[:1], kv_bf16=True)
    d = oracle.forward(m, ws, kv0, [0], [1], toks[:1], kv_bf16=False)
    assert _rel_err(c, d) < 2e-2
