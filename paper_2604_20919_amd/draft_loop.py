"""Speculative decoding with the drafting model on the same GPU.

Each round every user of a batch drafts l_m tokens autoregressively with the
drafting model (one sd_draft_batch decode step per token; Sec. II-A step 1
and eq. 13, where a device runs l_m steps of its small model), each step's
distribution q written straight into the row of the q array that the
verification will read; the target model then verifies the batch
(sd_verify_batch + sd_accept with commit).  Afterwards the drafting model's
cache is rolled back to what the target accepted: sd_user_reset keeps the
first i_m + 1 + a_m cached entries and installs the target's output token as
the next root.  When every draft was accepted the drafting model has not yet
seen its own last draft, so one more decode step (output discarded) caches it
first.

``DraftLoop`` runs this with two library contexts (drafting model and
target).  ``python -m paper_2604_20919_amd.draft_loop`` measures it on the
Qwen3-1.7B-shaped drafting model and the Qwen3-32B-shaped target with
random-init weights: the decode-step latency of the drafting model (a single
user, as on a device, and the batch), the verify latency, the acceptance rate
the two models actually reach, and the loop's token rate.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from dataclasses import dataclass
from typing import List, Sequence

import numpy as np
import torch

from .verifier import Verifier


@dataclass
class RoundResult:
    n_acc: np.ndarray        # accepted drafts per batch user
    token: np.ndarray        # target's output token per batch user
    drafts: np.ndarray       # the drafts of this round, users ascending
    draft_ms: float          # wall time of the drafting steps (host clock)
    verify_ms: float         # wall time of verify + accept


class DraftLoop:
    """Drafting context `dv` and target context `tv` over the same users
    (user ids, prefix lengths and root tokens kept equal by the loop)."""

    def __init__(self, dv: Verifier, tv: Verifier, n_users: int, max_draft: int, vocab: int,
                 mode: str = "stochastic", seed: int = 0):
        assert dv.vocab == tv.vocab == vocab
        self.dv, self.tv = dv, tv
        self.M = n_users
        self.mode = mode
        self.seed = seed
        self.q = torch.empty((n_users * max_draft, vocab), dtype=torch.float32, device="cuda")
        self.drafts = torch.empty(n_users * max_draft, dtype=torch.int32, device="cuda")
        self.stream = torch.cuda.Stream()

    def start_user(self, user: int, prefix_len: int, root: int):
        """Both models begin user `user` at the same cached length and root;
        the caller fills both caches (sd_kv_write) for the prefix."""
        self.dv.reset_user(user, prefix_len, root)
        self.tv.reset_user(user, prefix_len, root)

    def round(self, batch: int, assign: Sequence[int], draft_len: Sequence[int], rnd: int,
              commit: bool = True) -> RoundResult:
        assign = np.asarray(assign, np.int32)
        L = np.asarray(draft_len, np.int32)
        users = np.nonzero(assign == batch)[0]
        doff = np.zeros(len(users) + 1, np.int64)
        doff[1:] = np.cumsum(L[users])
        start = {int(u): self.dv.user_state(int(u)) for u in users}
        drafts = np.zeros(int(doff[-1]), np.int32)
        t0 = time.perf_counter()
        for j in range(int(L[users].max())):
            # users still drafting at step j, each writing row doff + j
            step = np.where((assign == batch) & (L > j), batch, -1).astype(np.int32)
            rows = np.zeros(self.M, np.int32)
            for i, u in enumerate(users):
                rows[u] = doff[i] + j
            self.dv.draft(batch, step, self.mode, seed=self.seed, round_=rnd * 1024 + j, probs=self.q,
                          probs_row=rows, stream=self.stream)
            _, tok = self.dv.accept(batch, self.M, commit=True)
            for i, u in enumerate(users):
                if L[u] > j:
                    drafts[doff[i] + j] = tok[u]
        t1 = time.perf_counter()
        self.drafts[:drafts.size].copy_(torch.from_numpy(drafts))
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        self.tv.verify(batch, assign, L, self.drafts, self.q, self.mode, seed=self.seed, round_=rnd,
                       stream=self.stream)
        n_acc, tok = self.tv.accept(batch, self.M, commit=commit)
        t3 = time.perf_counter()
        # roll the drafting model back to the accepted prefix
        for i, u in enumerate(users):
            u = int(u)
            P0, _ = start[u]
            a = int(n_acc[u])
            if not commit:
                self.dv.reset_user(u, P0, start[u][1])
                continue
            if a == int(L[u]):
                # cache the last draft too (one step; its output is not used)
                solo = np.where(np.arange(self.M) == u, batch, -1).astype(np.int32)
                self.dv.draft(batch, solo, "greedy", stream=self.stream)
                self.dv.accept(batch, self.M, commit=True)
            self.dv.reset_user(u, P0 + 1 + a, int(tok[u]))
        return RoundResult(n_acc[users], tok[users], drafts, 1e3 * (t1 - t0), 1e3 * (t3 - t2))


# ---------------------------------------------------------------------------
# measurement on the Qwen3 shapes
# ---------------------------------------------------------------------------

def _verifier(m, dw, n_users, max_draft, max_ctx):
    import workload as wl
    names = {"wq": wl.W_Q, "wk": wl.W_K, "wv": wl.W_V, "wo": wl.W_O, "wg": wl.W_G, "wu": wl.W_U,
             "wd": wl.W_D, "norm1": wl.N_1, "norm2": wl.N_2, "qnorm": wl.N_Q, "knorm": wl.N_K}
    ptrs = {"embed": dw.ptr(wl.EMBED), "lm_head": dw.ptr(wl.LM_HEAD), "norm_f": dw.ptr(wl.NORM_F),
            "layers": [{f: dw.ptr(k, l) for f, k in names.items()} for l in range(m.n_layers)]}
    pages = n_users * ((max_ctx + 15) // 16) + 16
    return Verifier(m, ptrs, n_pages=pages, max_users=n_users, max_draft=max_draft,
                    max_batch_users=n_users, max_batch_tokens=n_users * (max_draft + 1),
                    max_ctx=max_ctx, max_pending=2)


def acceptance_mle(n_acc: np.ndarray, draft_len: np.ndarray) -> float:
    """Per-draft acceptance probability under i.i.d. acceptance (eq. 1's
    alpha): accepted drafts over accept/reject trials, a trial being every
    accepted draft plus the first rejected one when there is one."""
    n_acc, draft_len = np.asarray(n_acc), np.asarray(draft_len)
    trials = n_acc + (n_acc < draft_len)
    return float(n_acc.sum() / max(trials.sum(), 1))


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--users", type=int, default=6)
    ap.add_argument("--prefix", type=int, default=512)
    ap.add_argument("--draft-len", type=int, default=4)
    ap.add_argument("--rounds", type=int, default=10)
    ap.add_argument("--mode", default="stochastic", choices=["stochastic", "greedy"])
    ap.add_argument("--out", default=None)
    args = ap.parse_args(argv)
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    sys.path.insert(0, root)
    import workload as wl
    from workload.device import DeviceWeights, kv_rows

    torch.cuda.set_device(0)
    M, L, P = args.users, args.draft_len, args.prefix
    max_ctx = P + args.rounds * (L + 2) + 8
    md, mt = wl.MODELS["qwen3-1.7b"], wl.MODELS["qwen3-32b"]
    dwd, dwt = DeviceWeights(md, 2), DeviceWeights(mt, 3)
    dv = _verifier(md, dwd, M, L, max_ctx)
    tv = _verifier(mt, dwt, M, L, max_ctx)
    loop = DraftLoop(dv, tv, M, L, md.vocab, args.mode, seed=7)
    roots = wl._ints(M, 7, 1 << 20, 0, md.vocab - 1)
    for v, m, seed in ((dv, md, 2), (tv, mt, 3)):
        buf = None
        for u in range(M):
            v.reset_user(u, P, int(roots[u]))
            for l in range(m.n_layers):
                k, vv = kv_rows(m, seed, l, u, P, out=buf)
                buf = (k, vv)
                v.write_kv(u, l, 0, k, vv)
    torch.cuda.synchronize()
    assign = np.zeros(M, np.int32)
    draft_len = np.full(M, L, np.int32)

    # decode-step latency of the drafting model: one user (device-like) and the batch
    def step_ms(users, reps=20):
        a = np.where(np.arange(M) < users, 0, -1).astype(np.int32)
        st = loop.stream
        for i in range(3):
            dv.draft(0, a, "greedy", stream=st)
            dv.accept(0, M, commit=False)
        t0 = time.perf_counter()
        for i in range(reps):
            dv.draft(0, a, "greedy", stream=st)
            dv.accept(0, M, commit=False)
        return 1e3 * (time.perf_counter() - t0) / reps

    one = step_ms(1)
    batch_step = step_ms(M)
    log: List[RoundResult] = []
    t0 = time.perf_counter()
    for r in range(args.rounds):
        log.append(loop.round(0, assign, draft_len, r))
    total_s = time.perf_counter() - t0
    acc = np.concatenate([x.n_acc for x in log])
    tokens = int(sum(int((x.n_acc + 1).sum()) for x in log))
    res = {
        "draft_model": md.name, "target_model": mt.name, "users": M, "prefix": P, "draft_len": L,
        "rounds": args.rounds, "mode": args.mode,
        "draft_step_ms_one_user": round(one, 3), "draft_step_ms_batch": round(batch_step, 3),
        "draft_ms_per_round": round(float(np.median([x.draft_ms for x in log])), 3),
        "verify_ms_per_round": round(float(np.median([x.verify_ms for x in log])), 3),
        "mean_accepted_per_user_round": round(float(acc.mean()), 4),
        "acceptance_alpha_mle": round(acceptance_mle(acc, np.full(acc.size, L)), 4),
        "tokens_per_s": round(tokens / total_s, 2),
        "tokens": tokens, "seconds": round(total_s, 3),
    }
    print(json.dumps(res))
    if args.out:
        with open(args.out, "w") as f:
            json.dump(res, f)
    dv.close()
    tv.close()


if __name__ == "__main__":
    main()
