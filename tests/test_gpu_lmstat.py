"""Phase A of the accept step (Sec. II-A step 2) from the lm_head epilogue.

With sd_config.logits_out = SD_LOGITS_AS_NEEDED the lm_head product emits
each slot's softmax statistics (row max, sum of exp, argmax, the logit of
the draft the slot decides) and stores fp32 logits only when the stochastic
race reads them; SD_LOGITS_UNFUSED stores every slot's logits and computes
the statistics from them by separate kernels.  On the Qwen3-1.7B shape
(vocabulary 151936) both contexts, given the same weights and inputs, must
agree bit for bit: accepted counts and tokens in all three modes, at slot
counts of every lm_head tile class (16-slot tiles below 97 slots, 32-slot
tiles of four-wave and eight-wave workgroups, ten and thirteen 32-slot
tiles), and the stored logits wherever both store them."""
import numpy as np
import pytest
import torch

import workload as wl
from gpu_harness import layer_ptrs, load_synthetic_kv
from paper_2604_20919_amd import sdverify as sdv
from paper_2604_20919_amd.verifier import Verifier
from workload.device import DeviceWeights, batch_to_device

pytestmark = pytest.mark.gpu

# (users, draft lengths) per batch; slot counts 40, 100, 225, 300, 400
_BATCHES = [
    [1, 2, 3, 4, 5, 6, 7, 4],
    [4] * 20,
    [(i % 12) + 1 for i in range(31)] + [9],
    [9] * 30,
    [9] * 40,
]


def _workload():
    L = [x for b in _BATCHES for x in b]
    assign = [n for n, b in enumerate(_BATCHES) for _ in b]
    prefix = [int(x) for x in wl._ints(len(L), 61, 0x51, 0, 400)]
    w = wl.custom_workload("qwen3-1.7b", prefix, L, seed=61, assign=assign)
    assert [w.batch(n).T for n in range(len(_BATCHES))] == [40, 100, 225, 300, 400]
    return w


def _verifier(w, dw, logits_out):
    m = w.model
    max_ctx = int((w.prefix_len + w.draft_len).max()) + 1
    pages = int(sum((p + l + 1 + 15) // 16 for p, l in zip(w.prefix_len, w.draft_len))) + 8
    return Verifier(m, layer_ptrs(dw), n_pages=pages, max_users=w.n_users, max_draft=int(w.draft_len.max()),
                    max_batch_users=max(len(b) for b in _BATCHES), max_batch_tokens=400, max_ctx=max_ctx,
                    max_pending=2, logits_out=logits_out)


def _plant_argmax_drafts(v, w, n, b, dev):
    """Drafts of user i follow the target's argmax for its first k_i slots
    (k_i = i mod (l_i + 1)), so greedy passes accept some and reject some;
    found with teacher-forced passes on the context that stores logits."""
    d, q, _ = dev
    k = np.array([i % (int(L) + 1) for i, L in enumerate(b.draft_len)])
    doff = np.concatenate([[0], np.cumsum(b.draft_len)]).astype(np.int64)
    soff = np.concatenate([[0], np.cumsum(b.n_slots)]).astype(np.int64)
    drafts = b.drafts.copy()
    for j in range(int(k.max())):
        d.copy_(torch.from_numpy(drafts))
        v.verify(n, w.assign, w.draft_len, d, q, "force")
        am = v.logits(n, b.T).argmax(dim=1).cpu().numpy()
        v.accept(n, w.n_users)
        for i in range(len(b.users)):
            if j < k[i]:
                drafts[doff[i] + j] = am[soff[i] + j]
    d.copy_(torch.from_numpy(drafts))
    b.drafts = drafts


def test_fused_statistics_match_unfused_path():
    w = _workload()
    dw = DeviceWeights(w.model, w.seed, gamma="uniform")
    vf = _verifier(w, dw, sdv.SD_LOGITS_AS_NEEDED)
    vu = _verifier(w, dw, sdv.SD_LOGITS_UNFUSED)
    load_synthetic_kv(vf, w)
    load_synthetic_kv(vu, w)
    for n in range(len(_BATCHES)):
        b = w.batch(n)
        for i, u in enumerate(b.users):
            for v in (vf, vu):
                v.reset_user(int(u), int(b.prefix_len[i]), int(b.root[i]))
        dev = batch_to_device(b)
        _plant_argmax_drafts(vu, w, n, b, dev)
        d, q, _ = dev
        for mode in ("stochastic", "greedy", "force"):
            res = {}
            for name, v in (("fused", vf), ("unfused", vu)):
                v.verify(n, w.assign, w.draft_len, d, q, mode, seed=7, round_=n)
                lg = v.logits(n, b.T) if (name == "unfused" or mode == "stochastic") else None
                if name == "fused" and mode != "stochastic":
                    # no pass that keeps the logits: the diagnostic copy is refused
                    with pytest.raises(sdv.SdError) as e:
                        v.logits(n, b.T)
                    assert e.value.status == sdv.SD_ESTATE
                n_acc, tok = v.accept(n, w.n_users)
                torch.cuda.synchronize()
                res[name] = (n_acc[b.users].copy(), tok[b.users].copy(), lg)
            (af, tf, lf), (au, tu, lu) = res["fused"], res["unfused"]
            label = f"T={b.T} {mode}"
            print(f"{label}: accepted {int(af.sum())} of {int(b.draft_len.sum())}; "
                  f"differing users {int(np.sum((af != au) | (tf != tu)))}", flush=True)
            assert np.array_equal(af, au), (label, af, au)
            assert np.array_equal(tf, tu), (label, tf, tu)
            if lf is not None:
                assert torch.equal(lf, lu), label
            if mode == "force":
                assert np.array_equal(af, b.draft_len)
            if mode == "greedy":
                assert 0 < int(af.sum()) < int(b.draft_len.sum())
    vf.close()
    vu.close()
