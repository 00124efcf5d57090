"""Sparse draft payloads (sd_verify_batch_sparse) through the C ABI.

A sparse row lists K tokens with their probabilities and gives every other
token one remainder probability.  Verification on it must equal verification
on the equivalent dense row: the GPU's sparse path is compared with its own
dense path on the expanded rows (bit-identical decisions and logits: the
arithmetic is the same, only where q comes from differs), with the oracle
sampler on the GPU's logits, on the tiny model and on the full Qwen3-1.7B
vocabulary (64 race chunks of 2374 tokens each in LDS)."""
import numpy as np
import pytest
import torch

import oracle
import workload as wl
from gpu_harness import load_synthetic_kv, make_verifier
from paper_2604_20919_amd import sdverify as sv
from workload.device import DeviceWeights

pytestmark = pytest.mark.gpu


def _run(v, w, b, sr, sparse, seed=4, round_=2, accept_u=None):
    d = torch.from_numpy(b.drafts).cuda()
    if sparse:
        v.verify_sparse(0, w.assign, w.draft_len, d, torch.from_numpy(sr.idx).cuda(),
                        torch.from_numpy(sr.val).cuda(), torch.from_numpy(sr.rest).cuda(),
                        "stochastic", seed, round_, accept_u)
    else:
        q = torch.from_numpy(oracle.expand_sparse_q(sr.idx, sr.val, sr.rest, w.model.vocab)).cuda()
        v.verify(0, w.assign, w.draft_len, d, q, "stochastic", seed, round_, accept_u)
    lg = v.logits(0, b.T).cpu().numpy()
    n_acc, tok = v.accept(0, w.n_users)
    torch.cuda.synchronize()
    return n_acc[b.users], tok[b.users], lg


def _check(w, b, sr, v, seeds):
    rejected = 0
    for seed in seeds:
        s = _run(v, w, b, sr, True, seed=seed)
        dn = _run(v, w, b, sr, False, seed=seed)
        assert np.array_equal(s[0], dn[0]) and np.array_equal(s[1], dn[1]), seed
        assert np.array_equal(s[2], dn[2])
        # strict level: the oracle sampler on the GPU's logits and the dense rows
        ref = oracle.sample("stochastic", b.users, b.draft_len, s[2], b.drafts,
                            oracle.expand_sparse_q(sr.idx, sr.val, sr.rest, w.model.vocab), None,
                            seed, 2)
        for i in range(len(b.users)):
            if s[0][i] == ref["n_acc"][i] and s[1][i] == ref["token"][i]:
                continue
            assert ref["race_gap"][i] < 1e-3, (seed, i)
        rejected += int((s[0] < b.draft_len).sum())
    return rejected


def test_sparse_rows_match_dense_rows_tiny():
    w = wl.custom_workload("tiny-bf16", [40, 300, 0, 17, 129, 64], [1, 7, 3, 5, 2, 4], seed=61)
    dw = DeviceWeights(w.model, w.seed)
    v = make_verifier(w, dw)
    load_synthetic_kv(v, w)
    b = w.batch(0)
    for i, u in enumerate(b.users):
        v.reset_user(int(u), int(b.prefix_len[i]), int(b.root[i]))
    sr = wl.sparsify(b, 32, seed=61)
    # enough seeds that residual draws at rejected slots are exercised
    assert _check(w, b, sr, v, range(6)) > 0
    v.close()


def test_sparse_rows_match_dense_rows_full_vocab():
    w = wl.workload("qwen3-1.7b-b8")
    dw = DeviceWeights(w.model, w.seed)
    v = make_verifier(w, dw)
    load_synthetic_kv(v, w)
    b = w.batch(0)
    for i, u in enumerate(b.users):
        v.reset_user(int(u), int(b.prefix_len[i]), int(b.root[i]))
    sr = wl.sparsify(b, 64, seed=62)
    assert _check(w, b, sr, v, range(2)) > 0
    v.close()


def test_sparse_argument_errors():
    w = wl.custom_workload("tiny-bf16", [10, 12], [1, 2], seed=63)
    dw = DeviceWeights(w.model, w.seed)
    v = make_verifier(w, dw)
    load_synthetic_kv(v, w)
    b = w.batch(0)
    sr = wl.sparsify(b, 4, seed=63)
    d = torch.from_numpy(b.drafts).cuda()
    idx = torch.from_numpy(sr.idx).cuda()
    val = torch.from_numpy(sr.val).cuda()
    rest = torch.from_numpy(sr.rest).cuda()
    for bad in (idx[:, :0], None):
        with pytest.raises(sv.SdError) as ei:
            v.verify_sparse(0, w.assign, w.draft_len, d, bad if bad is not None else idx, val,
                            rest if bad is not None else None)
        assert ei.value.status == sv.SD_EINVAL
    v.verify_sparse(0, w.assign, w.draft_len, d, idx, val, rest)
    v.accept(0, w.n_users)
    v.close()
