"""The allocation-free sampler entry point, sd_sample_logits_noalloc,
against sd_sample_logits on the same inputs: identical decisions and tokens
(the same kernels; only where the scratch lives differs), on calls in a row
whose second input is smaller than the first, in all three modes; the error
flag of a bad draft token is reported and cleared again by the next call;
inputs beyond the fixed limits are refused before anything is enqueued."""
import numpy as np
import pytest
import torch

from paper_2604_20919_amd import sdverify as sv
from test_gpu_sampler import _case, _sampler_verifier

pytestmark = pytest.mark.gpu

V = 151936


def _reference(v, users, Ls, M, logits, q, drafts, au, mode, seed, rnd):
    """sd_sample_logits + sd_accept on a context holding the users."""
    assign = np.full(M, -1, np.int32)
    assign[users] = 0
    dl = np.ones(M, np.int32)
    dl[users] = Ls
    dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    v.sample(0, assign, dl, dev(drafts), dev(q), dev(logits), mode, seed=seed, round_=rnd, accept_u=dev(au))
    n_acc, tok = v.accept(0, M)
    return n_acc[users], tok[users]


def _noalloc(users, Ls, logits, q, drafts, au, mode, seed, rnd):
    dev = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    B = len(Ls)
    result = torch.full((2 * B + 1,), -7, dtype=torch.int32, device="cuda")
    lg, qd, dd, ad = dev(logits), dev(q), dev(drafts), dev(au)
    sv.sd_sample_logits_noalloc(users, Ls, logits.shape[1], dd, qd if mode == "stochastic" else None, lg,
                                mode, result, seed=seed, round_=rnd, accept_u=ad)
    torch.cuda.synchronize()
    r = result.cpu().numpy()
    return r[:B], r[B:2 * B], int(r[2 * B])


@pytest.mark.parametrize("mode", ["stochastic", "greedy", "force"])
def test_noalloc_matches_sample_logits_on_calls_in_a_row(mode):
    big = [1, 4, 2, 8, 3, 5, 1, 6, 4, 4, 2, 7, 3, 9, 2, 1, 5, 5, 12, 2]
    small = [3, 1, 6]
    M = 32
    v = _sampler_verifier(V, M, 12, sum(big) + len(big))
    rng = np.random.default_rng(11)
    for k, Ls in enumerate([big, small, big[:7]]):
        seed = 40 + k
        logits, q, drafts, au, _ = _case(V, Ls, mode, seed, with_u=(k == 1))
        users = np.sort(rng.permutation(M)[:len(Ls)]).astype(np.int32)
        ref_acc, ref_tok = _reference(v, users, Ls, M, logits, q, drafts, au, mode, seed, k)
        acc, tok, flags = _noalloc(users, Ls, logits, q, drafts, au, mode, seed, k)
        assert flags == 0
        assert np.array_equal(acc, ref_acc), (k, acc, ref_acc)
        assert np.array_equal(tok, ref_tok), (k, tok, ref_tok)
        if mode == "force":
            assert np.array_equal(acc, np.asarray(Ls))
    v.close()


def test_noalloc_flags_bad_token_then_clears():
    Ls = [2, 3]
    logits, q, drafts, au, _ = _case(1024, Ls, "stochastic", 5, with_u=False)
    bad = drafts.copy()
    bad[3] = 1024  # one past the vocabulary
    users = np.array([0, 1], np.int32)
    _, _, flags = _noalloc(users, Ls, logits, q, bad, au, "stochastic", 5, 0)
    assert flags != 0
    # the next call starts from a cleared flag
    _, _, flags = _noalloc(users, Ls, logits, q, drafts, au, "stochastic", 5, 0)
    assert flags == 0


def test_noalloc_refuses_inputs_beyond_its_limits():
    d = torch.zeros(4096, dtype=torch.int32, device="cuda")
    f = torch.zeros(16, dtype=torch.float32, device="cuda")
    r = torch.zeros(256, dtype=torch.int32, device="cuda")
    too_many_users = np.arange(sv.SD_NOALLOC_MAX_USERS + 1)
    with pytest.raises(sv.SdError) as e:
        sv.sd_sample_logits_noalloc(too_many_users, np.ones(too_many_users.size), 16, d, f, f, "greedy", r)
    assert e.value.status == sv.SD_ELIMIT
    with pytest.raises(sv.SdError) as e:  # 1025 slots
        sv.sd_sample_logits_noalloc([0, 1], [512, 511], 16, d, f, f, "greedy", r)
    assert e.value.status == sv.SD_ELIMIT
    with pytest.raises(sv.SdError) as e:
        sv.sd_sample_logits_noalloc([0], [1], sv.SD_NOALLOC_MAX_VOCAB + 1, d, f, f, "greedy", r)
    assert e.value.status == sv.SD_ELIMIT
    with pytest.raises(sv.SdError) as e:
        sv.sd_sample_logits_noalloc([0], [0], 16, d, f, f, "greedy", r)
    assert e.value.status == sv.SD_EINVAL
    with pytest.raises(sv.SdError) as e:  # stochastic without q
        sv.sd_sample_logits_noalloc([0], [1], 16, d, None, f, "stochastic", r)
    assert e.value.status == sv.SD_EINVAL
