"""The multi-round serving loop's event order on a virtual clock.

With fixed verify latencies the loop is a cyclic schedule whose time per
round must settle at the pipeline span of eq. 16-18,
S* = max(sum_n t^v_n, max_n (t^d_n + t^v_n)), which the exhaustive
scheduler reference computes independently (oracle/dipsd.py).
"""
import numpy as np
import pytest

from oracle import dipsd as ref
from paper_2604_20919_amd import serve


def _instance(seed, M, N):
    rng = np.random.default_rng(seed)
    sysm = ref.System(alpha=list(rng.uniform(0.5, 0.9, M)), prefix=list(rng.choice([256, 512, 2048], M)),
                      tau_c=list(rng.uniform(1.0, 8.0, M)), c_d=[4.0305e-11] * M,
                      beta_d=list(33.8151 * rng.uniform(0.5, 1.5, M)),
                      beta_v=float(rng.choice([12.6, 95.1])))
    assign = list(rng.permutation(np.arange(M) % N))
    l = [int(x) for x in rng.integers(1, 9, M)]
    batches = [[m for m in range(M) if assign[m] == n] for n in range(N)]
    return sysm, batches, l


@pytest.mark.parametrize("seed", range(8))
def test_steady_round_time_is_the_pipeline_span(seed):
    M, N = 6, 1 + seed % 4
    sysm, batches, l = _instance(seed, M, N)
    draft = [ref.tau_draft(sysm, m, l[m]) + sysm.tau_c[m] for m in range(M)]
    tv = [ref.t_verify(sysm, len(b), max(l[m] for m in b), max(sysm.prefix[m] for m in b)) for b in batches]
    res = serve.run_pipeline(batches, draft, rounds=150, verify=lambda n, r: len(batches[n]),
                             clock=serve.VirtualClock(), verify_ms=lambda n: tv[n])
    ends = {}
    for e in res.log:
        ends[e.round] = max(ends.get(e.round, 0.0), e.end)
    period = (ends[149] - ends[89]) / 60.0
    assert period == pytest.approx(ref.span(sysm, batches, l), rel=1e-9)
    assert res.tokens == 150 * M


def test_batches_start_when_the_server_is_free_and_drafts_have_arrived():
    sysm, batches, l = _instance(3, 5, 3)
    draft = [ref.tau_draft(sysm, m, l[m]) + sysm.tau_c[m] for m in range(5)]
    tv = [7.0, 13.0, 29.0]
    res = serve.run_pipeline(batches, draft, rounds=6, verify=lambda n, r: 1,
                             clock=serve.VirtualClock(), verify_ms=lambda n: tv[n])
    last_end = {}
    free = 0.0
    for e in res.log:
        ready = max((last_end.get(m, 0.0) + draft[m]) for m in batches[e.batch])
        assert e.start == pytest.approx(max(free, ready))
        assert e.end == pytest.approx(e.start + tv[e.batch])
        free = e.end
        for m in batches[e.batch]:
            last_end[m] = e.end
    assert [(e.round, e.batch) for e in res.log] == [(r, n) for r in range(6) for n in range(3)]
