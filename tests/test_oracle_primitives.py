"""Pins for the oracle's primitives: Philox, uniform conversions, RMSNorm,
RoPE and single-head attention, each checked against something other than
the oracle itself (an independent library, a closed form, an invariant)."""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle


# --------------------------------------------------------------------------
# Philox-4x64-10 against numpy's independent implementation.  numpy
# increments its 256-bit counter before producing a block, so a generator
# started at counter c yields philox(c + 1) first.
# --------------------------------------------------------------------------

def _inc256(c):
    c = list(c)
    for i in range(4):
        c[i] = (c[i] + 1) % 2**64
        if c[i] != 0:
            break
    return c


@pytest.mark.parametrize("key,ctr", [
    ((0, 0), (0, 0, 0, 0)),
    ((1, 2), (0, 0, 0, 0)),
    ((0xDEADBEEFCAFEF00D, 0x0123456789ABCDEF), (7, 3, 2 << 32 | 5, 9)),
    ((2**64 - 1, 2**64 - 1), (2**64 - 2, 2**64 - 1, 2**64 - 1, 2**64 - 1)),
    ((12345, 0), (41, 17, 1 << 32, 0)),
])
def test_philox_matches_numpy(key, ctr):
    ref = np.random.Philox(key=np.array(key, dtype=np.uint64),
                           counter=np.array(ctr, dtype=np.uint64)).random_raw(8)
    c1 = _inc256(ctr)
    got = oracle.philox4x64_10(c1, key)
    assert [int(x) for x in got] == [int(x) for x in ref[:4]]
    got2 = oracle.philox4x64_10(_inc256(c1), key)
    assert [int(x) for x in got2] == [int(x) for x in ref[4:]]


def test_philox_is_a_bijection_sample():
    # distinct counters give distinct blocks (no collisions in a sample)
    seen = set()
    for i in range(2000):
        seen.add(tuple(int(x) for x in oracle.philox4x64_10([i, 0, 0, 0], [5, 6])))
    assert len(seen) == 2000


# --------------------------------------------------------------------------
# uniform conversions
# --------------------------------------------------------------------------

def test_accept_uniform_grid():
    assert oracle.accept_uniform(0) == 0.0
    assert oracle.accept_uniform(2**64 - 1) == 1.0 - 2.0**-24
    x = 0x123456789ABCDEF0
    assert oracle.accept_uniform(x) == (x >> 40) / 2.0**24


def test_race_uniform_is_a_fine_truncation():
    rng = np.random.default_rng(0)
    xs = [int(v) for v in rng.integers(1, 2**63, size=2000, dtype=np.int64)]
    xs += [1, 2, 3, 2**40 - 1, 2**40, 2**64 - 1, 2**63]
    for x in xs:
        v = Fraction(oracle.race_uniform(x))
        exact = Fraction(x, 2**64)
        assert 0 < v <= exact < 1
        assert (exact - v) / exact < Fraction(1, 2**23)  # 24 significant bits at every scale
    assert oracle.race_uniform(0) == 0.0


def test_race_exponential_is_unit_exponential():
    # Kolmogorov-Smirnov against Exp(1) on counter-generated draws
    xs = []
    for i in range(5000):
        xs.extend(int(v) for v in oracle.philox4x64_10([i, 0, 2 << 32, 0], [99, 0]))
    e = np.sort(np.array([oracle.race_exponential(x) for x in xs]))
    cdf = 1.0 - np.exp(-e)
    n = e.size
    ks = max(np.max(np.arange(1, n + 1) / n - cdf), np.max(cdf - np.arange(n) / n))
    assert ks < 1.63 / math.sqrt(n)  # 1% critical value
    assert abs(e.mean() - 1.0) < 4.0 / math.sqrt(n)


def test_round_bf16():
    assert oracle.round_bf16(1.0) == 1.0
    assert oracle.round_bf16(1.0 + 2**-8) == 1.0          # tie -> even
    assert oracle.round_bf16(1.0 + 3 * 2**-8) == 1.0 + 2**-6  # tie -> even (up)
    assert oracle.round_bf16(1.0 + 2**-7) == 1.0 + 2**-7  # representable
    assert oracle.round_bf16(-3.0) == -3.0


# --------------------------------------------------------------------------
# RMSNorm: unit RMS, positive-scale invariance, elementwise gain
# --------------------------------------------------------------------------

def test_rmsnorm_invariants():
    rng = np.random.default_rng(1)
    x = rng.normal(size=257) * 3.7
    y = oracle.rmsnorm(x, eps=0.0)
    assert abs(np.sqrt(np.mean(y * y)) - 1.0) < 1e-14
    assert np.allclose(oracle.rmsnorm(19.0 * x, eps=0.0), y, rtol=0, atol=1e-14)
    assert np.allclose(oracle.rmsnorm(-x, eps=0.0), -y, rtol=0, atol=1e-14)
    g = rng.uniform(0.5, 1.5, size=257).astype(np.float32)
    assert np.allclose(oracle.rmsnorm(x, g, eps=0.0), y * g.astype(np.float64), rtol=1e-15, atol=0)
    # matches torch's library RMSNorm
    t = torch.nn.functional.rms_norm(torch.tensor(x), (257,), torch.tensor(g, dtype=torch.float64), eps=1e-6)
    assert np.allclose(oracle.rmsnorm(x, g, eps=1e-6), t.numpy(), rtol=1e-13, atol=0)


# --------------------------------------------------------------------------
# RoPE: rotation per (a, a + hd/2) pair, identity at 0, relative position
# --------------------------------------------------------------------------

def test_rope_identity_and_norm():
    rng = np.random.default_rng(2)
    v = rng.normal(size=128)
    assert np.array_equal(oracle.rope(v, 0, 1e6), v)
    r = oracle.rope(v, 1234, 1e6)
    h = 64
    assert np.allclose(r[:h] ** 2 + r[h:] ** 2, v[:h] ** 2 + v[h:] ** 2, rtol=1e-12, atol=0)


def test_rope_relative_position():
    rng = np.random.default_rng(3)
    q, k = rng.normal(size=128), rng.normal(size=128)
    for base in (1e4, 1e6):
        a = oracle.rope(q, 1000, base) @ oracle.rope(k, 990, base)
        b = oracle.rope(q, 13, base) @ oracle.rope(k, 3, base)
        assert abs(a - b) < 1e-9 * (1 + abs(a))


def test_rope_complex_form():
    # pair a is the complex number v[a] + i v[a+h] multiplied by
    # exp(i * pos * base^(-2a/hd)): the rotate-half convention
    rng = np.random.default_rng(4)
    hd, h, base, pos = 64, 32, 1e4, 77
    v = rng.normal(size=hd)
    z = (v[:h] + 1j * v[h:]) * np.exp(1j * pos * base ** (-np.arange(0, hd, 2) / hd))
    r = oracle.rope(v, pos, base)
    assert np.allclose(r[:h], z.real, atol=1e-12) and np.allclose(r[h:], z.imag, atol=1e-12)


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------

def test_attend_special_cases():
    rng = np.random.default_rng(5)
    hd = 16
    q = rng.normal(size=hd)
    k = rng.normal(size=(1, hd))
    v = rng.normal(size=(1, hd))
    assert np.allclose(oracle.attend(q, k, v), v[0], atol=1e-15)
    k = np.tile(rng.normal(size=hd), (7, 1))
    v = rng.normal(size=(7, hd))
    assert np.allclose(oracle.attend(q, k, v), v.mean(0), atol=1e-14)
    k = rng.normal(size=(9, hd)) * 0.01
    k[4] = q * 50.0
    v = rng.normal(size=(9, hd))
    assert np.allclose(oracle.attend(q, k, v), v[4], atol=1e-12)


def test_attend_matches_torch_sdpa():
    rng = np.random.default_rng(6)
    n, hd = 37, 64
    q, k, v = rng.normal(size=hd), rng.normal(size=(n, hd)), rng.normal(size=(n, hd))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q)[None, None, None], torch.tensor(k)[None, None], torch.tensor(v)[None, None])
    assert np.allclose(oracle.attend(q, k, v), ref[0, 0, 0].numpy(), rtol=0, atol=1e-13)
