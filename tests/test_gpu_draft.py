"""Decode steps of a drafting model (sd_draft_batch) through the C ABI.

A decode step is the verify forward with one query slot per user (the root)
followed by the bonus draw of the sampler with l_m = 0; it also writes the
slot's distribution p, which the drafting loop hands to the verification as
q.  Checked against the oracle: p within the bound the logit error implies
(|log p_gpu - log p_ref| <= 2 max|dz|), rows summing to one, and the drawn
token bit-exact with the oracle sampler given the GPU's own logits (except
race near-ties, counted).  End to end: drafts produced by a model and
verified by the same model are all accepted; the drafting loop keeps the
two contexts' user states in step across committed rounds."""
import numpy as np
import pytest
import torch

import oracle
import workload as wl
from gpu_harness import load_synthetic_kv, make_verifier
from paper_2604_20919_amd import sdverify as sv
from paper_2604_20919_amd.draft_loop import DraftLoop, acceptance_mle
from workload.device import DeviceWeights

pytestmark = pytest.mark.gpu


def _ctx(model, prefix, seed, draft_len=None, extra_ctx=64):
    dl = draft_len or [4] * len(prefix)
    w = wl.custom_workload(model, prefix, dl, seed=seed)
    dw = DeviceWeights(w.model, w.seed)
    v = make_verifier(w, dw, extra_ctx=extra_ctx,
                      max_batch_tokens=len(prefix) * (max(dl) + 1))
    load_synthetic_kv(v, w)
    return w, dw, v


@pytest.mark.parametrize("model,mode", [("tiny", "stochastic"), ("tiny-bf16", "stochastic"),
                                        ("tiny-bf16", "greedy")])
def test_draft_step_matches_oracle(model, mode):
    prefix = [0, 17, 64, 129, 300]
    w, dw, v = _ctx(model, prefix, seed=41)
    m = w.model
    B = len(prefix)
    roots = wl._ints(B, 41, 77, 0, m.vocab - 1)
    for u in range(B):
        v.reset_user(u, prefix[u], int(roots[u]))
    probs = torch.full((B, m.vocab), -1.0, dtype=torch.float32, device="cuda")
    assign = np.zeros(B, np.int32)
    v.draft(0, assign, mode, seed=9, round_=3, probs=probs)
    lg = v.logits(0, B).cpu().numpy()
    n_acc, tok = v.accept(0, B, commit=False)
    torch.cuda.synchronize()
    q = probs.cpu().numpy().astype(np.float64)
    assert np.all(n_acc == 0)
    # oracle: one slot per user, the root at position i_m
    ws = oracle.WeightSource(m, w.seed)
    rl = oracle.forward(m, ws, oracle.KVSource(m, w.seed, np.arange(B), prefix), prefix,
                        np.ones(B, np.int32), roots)
    dz = np.abs(lg.astype(np.float64) - rl).max(axis=1)
    ref = np.exp(rl - rl.max(axis=1, keepdims=True))
    ref /= ref.sum(axis=1, keepdims=True)
    bound = np.expm1(2.0 * dz)[:, None] * ref + 1e-6 * ref + 1e-12
    assert np.all(np.abs(q - ref) <= bound), float((np.abs(q - ref) / np.maximum(ref, 1e-30)).max())
    assert np.allclose(q.sum(axis=1), 1.0, atol=1e-5)
    # strict level: the oracle sampler on the GPU's logits with l_m = 0
    res = oracle.sample(mode, np.arange(B), np.zeros(B, np.int32), lg, np.zeros(0, np.int32),
                        np.zeros((0, m.vocab), np.float32), None, 9, 3)
    border = 0
    for b in range(B):
        if tok[b] != res["token"][b]:
            assert res["race_gap"][b] < 1e-3, (b, tok[b], res["token"][b])
            border += 1
        assert q[b, tok[b]] > 0.0
    assert border <= 1
    if mode == "greedy":
        assert np.array_equal(tok, lg.argmax(axis=1))
    v.close()


def test_draft_rows_commit_and_errors():
    prefix = [5, 40, 12]
    w, dw, v = _ctx("tiny-bf16", prefix, seed=43)
    V = w.model.vocab
    B = len(prefix)
    for u in range(B):
        v.reset_user(u, prefix[u], 100 + u)
    a = np.zeros(B, np.int32)
    base = torch.zeros((B, V), dtype=torch.float32, device="cuda")
    v.draft(0, a, "stochastic", seed=1, round_=0, probs=base)
    _, tok0 = v.accept(0, B, commit=False)
    # the same step scattered to rows 5, 1, 3 of a larger array
    big = torch.zeros((6, V), dtype=torch.float32, device="cuda")
    v.draft(0, a, "stochastic", seed=1, round_=0, probs=big, probs_row=[5, 1, 3])
    _, tok1 = v.accept(0, B, commit=True)
    torch.cuda.synchronize()
    assert np.array_equal(tok0, tok1)
    bb, gg = base.cpu().numpy(), big.cpu().numpy()
    for b, r in enumerate([5, 1, 3]):
        assert np.array_equal(gg[r], bb[b])
    for r in (0, 2, 4):
        assert not gg[r].any()
    # commit advanced every user by one position with the drawn token as root
    for u in range(B):
        assert v.user_state(u) == (prefix[u] + 1, int(tok1[u]))
    # errors: force mode, rows without probs, negative rows -- nothing pending after
    for kw, mode in (({}, "force"), ({"probs_row": [0, 1, 2]}, "greedy"),
                     ({"probs": big, "probs_row": [0, -1, 2]}, "greedy")):
        with pytest.raises(sv.SdError) as ei:
            v.draft(0, a, mode, **kw)
        assert ei.value.status == sv.SD_EINVAL
    for u in range(B):
        assert v.user_state(u) == (prefix[u] + 1, int(tok1[u]))
    v.draft(0, a, "greedy")
    v.accept(0, B, commit=False)
    v.close()


@pytest.mark.parametrize("mode", ["stochastic", "greedy"])
def test_drafts_of_the_target_itself_are_accepted(mode):
    """Drafting and target contexts hold the same model: every draft is
    accepted (q equals p up to summation order; with accept uniforms of 0.5
    the stochastic test cannot hit the measure-zero u ~ p/q window), and the
    loop leaves both contexts at the same user state."""
    prefix = [33, 7, 90, 128]
    L = [3, 1, 4, 2]
    w, dw, dv = _ctx("tiny-bf16", prefix, seed=47, draft_len=L)
    tv = make_verifier(w, dw, extra_ctx=64, max_batch_tokens=len(prefix) * 5)
    load_synthetic_kv(tv, w)
    M = len(prefix)
    loop = DraftLoop(dv, tv, M, max(L), w.model.vocab, mode, seed=5)
    roots = wl._ints(M, 47, 78, 0, w.model.vocab - 1)
    for u in range(M):
        loop.start_user(u, prefix[u], int(roots[u]))
    assign = np.zeros(M, np.int32)
    half = torch.full((sum(L),), 0.5, dtype=torch.float32, device="cuda")
    for rnd in range(3):
        # the loop's round, with fixed accept uniforms in the stochastic case
        orig = tv.verify
        tv.verify = lambda *a, **k: orig(*a, **{**k, "accept_u": half if mode == "stochastic" else None})
        r = loop.round(0, assign, L, rnd)
        tv.verify = orig
        assert np.array_equal(r.n_acc, np.asarray(L)), (rnd, r.n_acc)
        for u in range(M):
            assert dv.user_state(u) == tv.user_state(u)
    dv.close()
    tv.close()


def test_loop_with_a_different_target_keeps_states_in_step():
    """A target with other weights rejects most drafts; across committed
    rounds the drafting context follows the target's accepted prefix and
    output token exactly."""
    prefix = [20, 55, 3]
    L = [4, 2, 3]
    wd, dwd, dv = _ctx("tiny-bf16", prefix, seed=51, draft_len=L)
    wt, dwt, tv = _ctx("tiny-bf16", prefix, seed=52, draft_len=L)
    M = len(prefix)
    loop = DraftLoop(dv, tv, M, max(L), wd.model.vocab, "stochastic", seed=8)
    for u in range(M):
        loop.start_user(u, prefix[u], 11 + u)
    assign = np.zeros(M, np.int32)
    acc = []
    for rnd in range(4):
        P0 = [tv.user_state(u)[0] for u in range(M)]
        r = loop.round(0, assign, L, rnd)
        acc.append(r.n_acc)
        for u in range(M):
            assert tv.user_state(u) == (P0[u] + 1 + int(r.n_acc[u]), int(r.token[u]))
            assert dv.user_state(u) == tv.user_state(u)
    alpha = acceptance_mle(np.concatenate(acc), np.tile(L, 4))
    assert 0.0 <= alpha <= 1.0
    dv.close()
    tv.close()
