"""Multi-round DiP-SD serving loop: the pipeline of Fig. 2 run for real on
the edge GPU, with the users' drafting simulated as delays.

Each round every user drafts l_m tokens on its device (tau^d_m =
l_m G_m(1, F^d(i_m)), eq. 13) and uploads them (tau^c_m); the edge server
verifies the batches of the assignment x one at a time in a fixed cyclic
order (eq. 14-18): batch n starts when the server is free and every one of
its users' drafts has arrived, and its users begin drafting the next round
as soon as its verification returns.  Verification is the library's
sd_verify_batch + sd_accept with commit, so every user's cache grows by the
accepted tokens plus one and its pages are trimmed to the new length.

In steady state the time per round is S* = max(sum_n t^v_n,
max_n (t^d_n + t^v_n)), the span of eq. 16-18, and the measured throughput
approaches R = U / S (eq. 22) with U the tokens actually emitted.

``run_pipeline`` is the event loop, independent of how a verification is
executed: ``GpuVerify`` runs it on the library with wall-clock waits for the
simulated drafting; a model of t^v and a virtual clock run it on the host.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence


@dataclass
class RoundLog:
    batch: int
    round: int
    start: float          # ms since the loop began
    end: float
    tokens: int           # sum over the batch of (accepted + 1)


@dataclass
class VerifyRecord:
    """One verification of GpuVerify, kept when it records: the batch and
    round, its users, the drafts and draft distributions it was given, and
    what sd_accept returned for each user."""
    batch: int
    round: int
    users: List[int]
    drafts: object        # int32 [sum l_m]
    q: object             # fp32 [sum l_m][V]
    n_acc: List[int]
    token: List[int]


@dataclass
class PipelineResult:
    rounds: int
    total_ms: float
    tokens: int
    log: List[RoundLog] = field(default_factory=list)

    @property
    def tokens_per_s(self) -> float:
        return 1000.0 * self.tokens / self.total_ms

    def period_ms(self, skip: int = 1) -> float:
        """Mean time per round after `skip` warm-up rounds, from the end
        times of the last batch of each round."""
        ends: Dict[int, float] = {}
        for e in self.log:
            ends[e.round] = max(ends.get(e.round, 0.0), e.end)
        rs = sorted(ends)
        if len(rs) <= skip + 1:
            return float("nan")
        return (ends[rs[-1]] - ends[rs[skip]]) / (rs[-1] - rs[skip])


class VirtualClock:
    """Time that advances only when asked to wait (host-side runs)."""

    def __init__(self):
        self.t = 0.0

    def now(self) -> float:
        return self.t

    def wait_until(self, t: float):
        self.t = max(self.t, t)

    def advance(self, dt: float):
        self.t += dt


class WallClock:
    def __init__(self):
        self.t0 = time.perf_counter()

    def now(self) -> float:
        return (time.perf_counter() - self.t0) * 1e3

    def wait_until(self, t: float):
        while True:
            d = t - self.now()
            if d <= 0:
                return
            time.sleep(min(d, 50.0) / 1e3)


def run_pipeline(batches: Sequence[Sequence[int]], draft_ms: Sequence[float], rounds: int,
                 verify: Callable[[int, int], int], clock, verify_ms: Optional[Callable[[int], float]] = None
                 ) -> PipelineResult:
    """The cyclic pipeline for `rounds` rounds.

    batches[n]: users of batch n (the assignment x); draft_ms[m]: tau^d_m +
    tau^c_m of user m per round; verify(n, r): verifies batch n of round r
    and returns the tokens it emitted (the call itself takes real time on a
    wall clock); verify_ms(n): its duration on a virtual clock (the clock is
    advanced by that much), None on a wall clock."""
    M = len(draft_ms)
    ready = [float(draft_ms[m]) for m in range(M)]   # round 0 drafts arrive
    free = 0.0
    res = PipelineResult(rounds, 0.0, 0)
    for r in range(rounds):
        for n, users in enumerate(batches):
            start = max(free, max(ready[m] for m in users))
            clock.wait_until(start)
            start = clock.now()
            tok = verify(n, r)
            if verify_ms is not None:
                clock.advance(verify_ms(n))
            end = clock.now()
            free = end
            for m in users:
                ready[m] = end + float(draft_ms[m])
            res.tokens += tok
            res.log.append(RoundLog(n, r, start, end, tok))
    res.total_ms = free
    return res


class GpuVerify:
    """Verification of the scheduled batches on the library, users' caches
    growing round by round.  Drafts and their distributions are synthetic:
    q a softmax of Gaussian logits with the random-init target's logit
    scale, drafts sampled from q (stochastic accept/resample)."""

    def __init__(self, verifier, assign: Sequence[int], l: Sequence[int], vocab: int,
                 q_sigma: float, seed: int = 0, commit: bool = True, record: bool = False):
        import torch
        self.torch = torch
        self.v = verifier
        self.assign = [int(a) for a in assign]
        self.l = [int(x) for x in l]
        self.vocab = vocab
        self.q_sigma = q_sigma
        self.seed = seed
        self.g = torch.Generator(device="cuda")
        self.g.manual_seed(seed)
        self.commit = commit
        self.accepted: List[int] = []
        self.drafted: List[int] = []
        self.records: Optional[List[VerifyRecord]] = [] if record else None

    def __call__(self, n: int, r: int) -> int:
        torch = self.torch
        users = [m for m, a in enumerate(self.assign) if a == n]
        nd = sum(self.l[m] for m in users)
        logits = torch.randn((nd, self.vocab), generator=self.g, device="cuda") * self.q_sigma
        q = torch.softmax(logits, dim=1)
        d = torch.multinomial(q, 1, generator=self.g).to(torch.int32).reshape(-1)
        self.v.verify(n, self.assign, self.l, d, q, "stochastic", seed=self.seed, round_=r)
        n_acc, tok = self.v.accept(n, len(self.assign), commit=self.commit)
        if self.records is not None:
            self.records.append(VerifyRecord(n, r, users, d.cpu().numpy(), q.cpu().numpy(),
                                             [int(n_acc[m]) for m in users], [int(tok[m]) for m in users]))
        for m in users:
            self.accepted.append(int(n_acc[m]))
            self.drafted.append(self.l[m])
        return int(sum(int(n_acc[m]) + 1 for m in users))

    @property
    def acceptance(self) -> float:
        return sum(self.accepted) / max(sum(self.drafted), 1)


def main():
    """Run the pipeline on the GPU for the Table II setting (M users of
    prefix 512 with the paper's device-side drafting model) with the schedule
    Algorithm 1 picks for this GPU's fitted verify latency; print one JSON
    line with measured and modelled throughput."""
    import argparse
    import json
    import numpy as np
    import torch
    import workload as wl
    from workload.device import DeviceWeights
    from . import scheduler as sch
    from . import sdverify as sv
    from .verifier import Verifier

    ap = argparse.ArgumentParser()
    ap.add_argument("--model", default="qwen3-32b")
    ap.add_argument("--users", type=int, default=6)
    ap.add_argument("--prefix", type=int, default=512)
    ap.add_argument("--rounds", type=int, default=12)
    ap.add_argument("--c-v", type=float, default=2.1687e-12,
                    help="verify latency fit c^v (eq. 6) measured on this GPU")
    ap.add_argument("--beta-v", type=float, default=12.562, help="verify latency fit beta^v (ms)")
    ap.add_argument("--alpha", type=float, default=0.78, help="acceptance rate the schedule assumes")
    ap.add_argument("--seed", type=int, default=5)
    args = ap.parse_args()

    p = sch.paper_defaults(args.users, args.alpha, args.prefix)
    p.c_v, p.beta_v = args.c_v, args.beta_v
    sched = sch.solve(p)
    N = sched.N
    batches = [[m for m in range(p.M) if sched.assign[m] == n] for n in range(N)]
    draft_ms = [sched.l[m] * sch.draft_step_ms(p, m) + p.tau_c[m] for m in range(p.M)]

    assert torch.cuda.is_available(), "the serving loop needs a GPU"
    sv.lib()
    m = wl.MODELS[args.model]
    dw = DeviceWeights(m, args.seed)
    names = {"wq": wl.W_Q, "wk": wl.W_K, "wv": wl.W_V, "wo": wl.W_O, "wg": wl.W_G, "wu": wl.W_U,
             "wd": wl.W_D, "norm1": wl.N_1, "norm2": wl.N_2, "qnorm": wl.N_Q, "knorm": wl.N_K}
    ptrs = {"embed": dw.ptr(wl.EMBED), "lm_head": dw.ptr(wl.LM_HEAD), "norm_f": dw.ptr(wl.NORM_F),
            "layers": [{f: dw.ptr(k, l) for f, k in names.items()} for l in range(m.n_layers)]}
    Lmax = max(sched.l)
    max_ctx = args.prefix + args.rounds * (Lmax + 1) + Lmax + 2
    pages = p.M * ((max_ctx + 15) // 16) + 16
    v = Verifier(m, ptrs, n_pages=pages, max_users=p.M, max_draft=Lmax,
                 max_batch_users=max(len(b) for b in batches),
                 max_batch_tokens=max(sum(sched.l[u] + 1 for u in b) for b in batches),
                 max_ctx=max_ctx, max_pending=1)
    roots = np.random.default_rng(args.seed).integers(0, m.vocab, p.M)
    for u in range(p.M):
        v.reset_user(u, args.prefix, int(roots[u]))
    sigma = 0.02 * (m.d_model ** 0.5)
    # one untimed round without commit (first-launch costs of every call)
    warm = GpuVerify(v, sched.assign, sched.l, m.vocab, q_sigma=sigma, seed=args.seed + 1, commit=False)
    for n in range(N):
        warm(n, 0)
    torch.cuda.synchronize()
    gv = GpuVerify(v, sched.assign, sched.l, m.vocab, q_sigma=sigma, seed=args.seed)
    res = run_pipeline(batches, draft_ms, args.rounds, gv, WallClock())
    # steady state: rounds after the first (whose drafts all start together)
    steady = [e for e in res.log if e.round >= 1]
    end0 = max(e.end for e in res.log if e.round == 0)
    steady_tok = sum(e.tokens for e in steady)
    steady_ms = res.total_ms - end0
    tv = {n: float(np.median([e.end - e.start for e in steady if e.batch == n])) for n in range(N)}
    alpha = gv.acceptance
    U = sum(sch.expected_tokens(alpha, sched.l[u]) for u in range(p.M))
    S_model = max(sum(tv.values()), max(max(draft_ms[u] for u in b) + tv[n] for n, b in enumerate(batches)))
    out = {"model": args.model, "users": p.M, "prefix": args.prefix, "rounds": args.rounds,
           "schedule": {"N": N, "assign": sched.assign, "l": sched.l, "assumed_alpha": args.alpha,
                        "predicted_R_tok_s": round(sched.R, 2), "predicted_S_ms": round(sched.S, 3)},
           "measured": {"tokens": res.tokens, "total_ms": round(res.total_ms, 2),
                        "R_tok_s": round(res.tokens_per_s, 2),
                        "steady_R_tok_s": round(1000.0 * steady_tok / steady_ms, 2),
                        "period_ms": round(res.period_ms(), 3),
                        "verify_ms_per_batch_median": {str(k): round(x, 3) for k, x in tv.items()},
                        "acceptance": round(alpha, 4)},
           "model_at_measured": {"alpha": round(alpha, 4), "S_ms": round(S_model, 3),
                                 "R_tok_s": round(1000.0 * U / S_model, 2)},
           "final_prefix": [int(v.user_state(u)[0]) for u in range(p.M)]}
    v.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
