"""Strict parity of the GPU accept/resample kernels with the oracle sampler.

Both sides get the same seeded logits, draft distributions, drafts and
seeds (through sd_sample_logits); decisions and tokens must be bit-exact
except the counted borderline cases (|p/q - u| < 1e-3, or a race whose two
best keys are within 1e-3)."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workload as wl
from gpu_harness import assert_decisions, compare_decisions
from paper_2604_20919_amd.verifier import Verifier

pytestmark = pytest.mark.gpu


def _sampler_verifier(V: int, max_users: int, max_draft: int, Tmax: int):
    m = dataclasses.replace(wl.MODELS["tiny"], vocab=V)
    dummy = torch.zeros(1024, dtype=torch.float32, device="cuda")
    p = dummy.data_ptr()
    lay = {f: p for f in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "norm1", "norm2", "qnorm", "knorm")}
    v = Verifier(m, {"embed": p, "lm_head": p, "norm_f": p, "layers": [lay] * m.n_layers},
                 n_pages=8, max_users=max_users, max_draft=max_draft, max_batch_users=max_users,
                 max_batch_tokens=Tmax, max_ctx=64)
    v._dummy = dummy
    return v


def _softmax(z):
    z = z - z.max(1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(1, keepdims=True)


def _case(V, Ls, mode, seed, with_u, sigma=1.5, user_ids=None):
    rng = np.random.default_rng(seed)
    B = len(Ls)
    T = int(sum(Ls)) + B
    logits = (rng.normal(size=(T, V)) * sigma).astype(np.float32)
    # draft distributions correlated with the target rows so that both
    # acceptances and rejections occur
    q = np.empty((int(sum(Ls)), V), np.float32)
    drafts = np.empty(int(sum(Ls)), np.int32)
    o, t = 0, 0
    for b, L in enumerate(Ls):
        for j in range(L):
            qz = logits[t + j].astype(np.float64) + rng.normal(size=V) * 0.8
            qq = _softmax(qz[None])[0]
            q[o + j] = qq
            if mode == "greedy":
                am = int(logits[t + j].argmax())
                drafts[o + j] = am if rng.random() < 0.7 else int(rng.integers(V))
            else:
                drafts[o + j] = int(rng.choice(V, p=qq / qq.sum()))
        o += L
        t += L + 1
    au = rng.random(int(sum(Ls))).astype(np.float32) if with_u else None
    users = np.arange(B) if user_ids is None else np.asarray(user_ids)
    return logits, q, drafts, au, users


@pytest.mark.parametrize("V,mode,with_u", [
    (1024, "stochastic", False),
    (1024, "stochastic", True),
    (1024, "greedy", False),
    (151936, "stochastic", False),
    (151936, "greedy", False),
    (151936, "force", False),
])
def test_sampler_matches_oracle(V, mode, with_u):
    Ls = [1, 4, 2, 8, 3, 5, 1, 6, 4, 4, 2, 7]
    B = len(Ls)
    v = _sampler_verifier(V, B + 4, 8, sum(Ls) + B)
    total_bad = total_border = 0
    for rep in range(3):
        seed = 100 * rep + V % 97 + (7 if with_u else 0)
        logits, q, drafts, au, users = _case(V, Ls, mode, seed, with_u)
        M = B + 4
        assign = np.full(M, -1, np.int32)
        perm = np.random.default_rng(seed).permutation(M)[:B]
        users = np.sort(perm)
        assign[users] = 0
        dl = np.ones(M, np.int32)
        dl[users] = Ls
        dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
        v.sample(0, assign, dl, dev(drafts), dev(q), dev(logits), mode, seed=seed, round_=rep,
                 accept_u=dev(au))
        n_acc, tok = v.accept(0, M)
        ref = oracle.sample(mode, users, Ls, logits, drafts, q, au, seed, rep)
        chk = compare_decisions(n_acc[users], tok[users], ref, Ls, mode)
        assert_decisions(chk, f"V={V} {mode} u={with_u} rep {rep}", end_to_end=False)
        total_bad += chk.bad
        total_border += chk.border
        if mode == "force":
            assert np.array_equal(n_acc[users], np.asarray(Ls))
    print(f"V={V} mode={mode} accept_u={with_u}: mismatches={total_bad} borderline={total_border}")
    assert total_bad == 0
    v.close()


def test_sampler_q_equals_p_accepts_all():
    """q = softmax(logits) computed on the host: p/q = 1 up to rounding, so
    every draft passes whatever u is (except u within 1e-6 of 1)."""
    V, Ls = 4096, [3, 5, 2]
    B = len(Ls)
    v = _sampler_verifier(V, B, 8, sum(Ls) + B)
    rng = np.random.default_rng(5)
    T = sum(Ls) + B
    logits = rng.normal(size=(T, V)).astype(np.float32)
    rows = []
    t = 0
    for L in Ls:
        rows.extend(range(t, t + L))
        t += L + 1
    q = _softmax(logits[rows].astype(np.float64)).astype(np.float32)
    drafts = np.array([int(rng.choice(V, p=qq / qq.sum())) for qq in q.astype(np.float64)], np.int32)
    au = np.full(sum(Ls), 0.999, np.float32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    v.sample(0, np.zeros(B, np.int32), Ls, dev(drafts), dev(q), dev(logits), "stochastic",
             accept_u=dev(au))
    n_acc, _ = v.accept(0, B)
    assert np.array_equal(n_acc, np.asarray(Ls))
    v.close()
