"""Seeded sweep of ragged batch shapes on the bf16 model with the 32B head
layout, each compared with the oracle: 1-12 users, prefixes drawn from
0..1200 with page edges (15, 16, 17, 31, 32, 33) and chunk-sized contexts
mixed in, draft lengths 1-12, all three modes, and users of the context
taken out of the batch (assign != 0).  A second sweep draws up to 60 users
(at most 416 slots, the largest slot class) on the three bf16 toy models,
whose gate/up products take the last-split, split-and-reduce and
stream-K forms.  Logits within the bf16 bar, decisions bit-exact outside
the window the logit error admits."""
import numpy as np
import pytest

import oracle
import workload as wl
from gpu_harness import assert_decisions, compare_decisions, load_synthetic_kv, logit_rel_err, make_verifier, run_gpu, run_oracle
from workload.device import DeviceWeights

pytestmark = pytest.mark.gpu

EDGES = [0, 1, 15, 16, 17, 31, 32, 33, 255, 256, 257, 1023, 1024]


def _shape(seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 13))
    prefix = [int(rng.choice(EDGES)) if rng.random() < 0.4 else int(rng.integers(0, 1201)) for _ in range(n)]
    L = [int(rng.integers(1, 13)) for _ in range(n)]
    # some users of the context sit in another batch of the same context
    assign = [0 if (i == 0 or rng.random() < 0.8) else 1 for i in range(n)]
    mode = ["stochastic", "greedy", "force"][seed % 3]
    return prefix, L, assign, mode


@pytest.mark.parametrize("seed", range(12))
def test_random_ragged_shapes_match_oracle(seed):
    prefix, L, assign, mode = _shape(seed)
    w = wl.custom_workload("tiny-bf16", prefix, L, seed=500 + seed, q_sigma=1.0, assign=assign)
    dw = DeviceWeights(w.model, w.seed, gamma="uniform")
    v = make_verifier(w, dw)
    load_synthetic_kv(v, w)
    b = w.batch(0)
    gpu = run_gpu(v, w, 0, b, mode, seed=seed, round_=seed)
    rl, ref = run_oracle(w, b, mode, seed=seed, round_=seed, weights=oracle.WeightSource(w.model, w.seed, "uniform"))
    err = logit_rel_err(gpu.logits, rl)
    label = f"seed {seed}: users {b.users.tolist()} prefix {b.prefix_len.tolist()} L {b.draft_len.tolist()} {mode}"
    print(f"{label}: logit rel err {err.max():.2e}")
    assert err.max() < 2e-2, label
    chk = compare_decisions(gpu.n_acc, gpu.token, ref, b.draft_len, mode, b.drafts, gpu.logits, rl)
    assert_decisions(chk, label, end_to_end=True)
    if mode == "force":
        assert np.array_equal(gpu.n_acc, b.draft_len)
    v.close()


WIDE_MODELS = ["tiny-bf16", "tiny-mid-ffn", "tiny-wide-ffn"]


def _wide_shape(seed):
    rng = np.random.default_rng(7000 + seed)
    n = int(rng.integers(1, 61))
    prefix = [int(rng.choice(EDGES)) if rng.random() < 0.4 else int(rng.integers(0, 1201)) for _ in range(n)]
    L = [int(rng.integers(1, 13)) for _ in range(n)]
    while sum(l + 1 for l in L) > 416:
        L.pop()
        prefix.pop()
    assign = [0 if (i == 0 or rng.random() < 0.85) else 1 for i in range(len(L))]
    mode = ["stochastic", "greedy", "force"][(seed // 3) % 3]
    return WIDE_MODELS[seed % 3], prefix, L, assign, mode


@pytest.mark.parametrize("seed", range(24))
def test_random_wide_batches_match_oracle(seed):
    model, prefix, L, assign, mode = _wide_shape(seed)
    w = wl.custom_workload(model, prefix, L, seed=900 + seed, q_sigma=1.0, assign=assign)
    dw = DeviceWeights(w.model, w.seed, gamma="uniform")
    v = make_verifier(w, dw)
    load_synthetic_kv(v, w)
    b = w.batch(0)
    gpu = run_gpu(v, w, 0, b, mode, seed=seed, round_=seed)
    rl, ref = run_oracle(w, b, mode, seed=seed, round_=seed, weights=oracle.WeightSource(w.model, w.seed, "uniform"))
    err = logit_rel_err(gpu.logits, rl)
    label = f"seed {seed}: {model} T={b.T} users {len(b.users)} {mode}"
    print(f"{label}: logit rel err {err.max():.2e}")
    assert err.max() < 2e-2, label
    chk = compare_decisions(gpu.n_acc, gpu.token, ref, b.draft_len, mode, b.drafts, gpu.logits, rl)
    assert_decisions(chk, label, end_to_end=True)
    if mode == "force":
        assert np.array_equal(gpu.n_acc, b.draft_len)
    v.close()
