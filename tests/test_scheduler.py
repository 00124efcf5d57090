"""DiP-SD joint scheduler (Algorithm 1) against the exhaustive reference.

The reference (oracle/dipsd.py) is pinned first: to Table II and to the
throughputs and speedups the paper prints for its homogeneous experiments
(Sec. V-B; tests/golden/dipsd_printed_values.json keeps them with their
citations: 74.13 and 117.56 tok/s at alpha = 0.70 / 0.95 with M = 6, 1.59x
between them, 11.25x AD and 1.93x AD with greedy batching at 0.95, about
1.38x AD with greedy batching at 0.78, and 17.89x AD / 1.38x AD with greedy
batching at M = 14), to closed forms, and to its own two independent
searches.  The MILP scheduler is then held to
the reference: each subproblem is solved exactly, so its optimum must equal
the exhaustive optimum of that subproblem on random small instances, and
Algorithm 1 reproduces the paper's numbers.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import dipsd as ref
from paper_2604_20919_amd import scheduler as sch


def _both(alpha, prefix, tau_c, c_d, beta_d, L_ub=20, gamma_max=8.0e10, c_v=1.2077e-11,
          beta_v=95.1074):
    """The same instance for the reference and for the scheduler (built
    separately from plain numbers; the two share no code)."""
    o = ref.System(alpha=list(alpha), prefix=list(prefix), tau_c=list(tau_c), c_d=list(c_d),
                   beta_d=list(beta_d), L_ub=L_ub, gamma_max=gamma_max, c_v=c_v, beta_v=beta_v)
    s = sch.SystemParams(alpha=list(alpha), prefix=list(prefix), tau_c=list(tau_c), c_d=list(c_d),
                         beta_d=list(beta_d), L_ub=L_ub, gamma_max=gamma_max, c_v=c_v,
                         beta_v=beta_v)
    return o, s


def _random_instance(seed, M, L_ub=6):
    rng = np.random.default_rng(seed)
    return _both(alpha=rng.uniform(0.5, 0.95, M).round(3),
                 prefix=rng.choice([256, 512, 1024, 2048], M),
                 tau_c=rng.uniform(1.0, 6.0, M).round(2),
                 c_d=(4.0305e-11 * rng.uniform(0.8, 1.2, M)),
                 beta_d=(33.8151 * rng.uniform(0.7, 1.3, M)),
                 L_ub=L_ub)


# ---- the reference, pinned ----------------------------------------------------

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "dipsd_printed_values.json")))


def test_reference_defaults_are_table_ii():
    """The reference's default system (Table II, as printed)."""
    g = GOLDEN["table_ii_defaults"]
    o = ref.table2()
    assert o.M == g["M"] and set(o.alpha) == {g["alpha"]} and set(o.prefix) == {g["prefix"]}
    assert set(o.tau_c) == {g["tau_c_ms"]} and set(o.c_d) == {g["c_d"]} and set(o.beta_d) == {g["beta_d_ms"]}
    assert [o.draft.J, o.draft.h1, o.draft.h2] == g["draft_model_J_h1_h2"]
    assert [o.verify.J, o.verify.h1, o.verify.h2] == g["verify_model_J_h1_h2"]
    assert (o.c_v, o.beta_v, o.gamma_max, o.L_ub) == (g["c_v"], g["beta_v_ms"], g["gamma_max_bytes"], g["L_ub"])


def test_reference_reproduces_paper_alpha_sweep():
    """Sec. V-B: with M = 6 DiP-SD rises from 74.13 to 117.56 tok/s as alpha
    goes from 0.70 to 0.95 (a 1.59x improvement), which at alpha = 0.95 is
    11.25x vanilla AD and 1.93x AD with greedy batching; at the default
    alpha = 0.78 it is about 1.38x AD with greedy batching."""
    g = GOLDEN["homogeneous_alpha_sweep"]
    r70 = ref.homogeneous_global(ref.table2(g["M"], 0.70))[0]
    s95 = ref.table2(g["M"], 0.95)
    r95 = ref.homogeneous_global(s95)[0]
    assert round(r70, 2) == g["dipsd_tok_s"]["0.70"]
    assert round(r95, 2) == g["dipsd_tok_s"]["0.95"]
    assert round(r95 / r70, 2) == g["improvement_070_to_095"]
    assert round(r95 / ref.autoregressive(s95), 2) == g["speedup_over_ad_at_095"]
    assert round(r95 / ref.ad_greedy_batching(s95)[0], 2) == g["speedup_over_ad_greedy_at_095"]
    s78 = ref.table2(g["M"], 0.78)
    r78 = ref.homogeneous_global(s78)[0]
    assert round(r78 / ref.ad_greedy_batching(s78)[0], 2) == g["speedup_over_ad_greedy_at_078"]


def test_reference_reproduces_paper_peak_speedups():
    """Sec. V-B: at the default alpha = 0.78, DiP-SD's peak over the user
    sweep M in {2..14} (at M = 14) is 17.89x edge-only autoregressive
    decoding and 1.38x AD with greedy batching."""
    g = GOLDEN["homogeneous_user_sweep"]
    sysm = ref.table2(g["M_peak"], g["alpha"])
    r = ref.homogeneous_global(sysm)[0]
    assert round(r / ref.autoregressive(sysm), 2) == g["speedup_over_ad"]
    assert round(r / ref.ad_greedy_batching(sysm)[0], 2) == g["speedup_over_ad_greedy"]


def test_ad_greedy_batching_packs_by_prefix_under_the_memory_bound():
    """Sec. V-A's baseline: users sorted by prefix, longest first, packed
    until the next would break eq. 19-21.  With a cap admitting 2 users of
    prefix 2048 (or 4 of 1024), prefixes {2048, 512, 2048, 1024, 2048} pack
    as [2048, 2048], [2048, 1024], [512] and the rate is M over the summed
    single-token verify latencies."""
    v = ref.Model(64, 5120, 25600)
    params = v.J * (8.0 * v.h1 ** 2 + 4.0 * v.h1 * v.h2)
    cap = params + 4.0 * v.J * v.h1 * 2 * 2048 + 1.0
    prefix = [2048, 512, 2048, 1024, 2048]
    o = ref.System(alpha=[0.8] * 5, prefix=prefix, tau_c=[3.0] * 5, c_d=[4.0305e-11] * 5,
                   beta_d=[33.8151] * 5, gamma_max=cap)
    r, batches = ref.ad_greedy_batching(o)
    assert [[prefix[m] for m in b] for b in batches] == [[2048, 2048], [2048, 1024], [512]]
    ms = ref.t_verify(o, 2, 1, 2048) * 2 + ref.t_verify(o, 1, 1, 512)
    assert r == pytest.approx(5000.0 / ms, rel=1e-12)


def test_autoregressive_baseline_closed_form():
    """One token per G^v(1, F^v(1, 512)) = c^v * 4 J h1 (2 h1 + 513 + h2) +
    beta^v ms, written out with the Table II numbers."""
    ms = 1.2077e-11 * 4 * 64 * 5120 * (2 * 5120 + 512 + 1 + 25600) + 95.1074
    assert ref.autoregressive(ref.table2(6)) == pytest.approx(1000.0 / ms, rel=1e-12)
    assert round(ref.autoregressive(ref.table2(6)), 2) == 10.45


def test_utility_is_the_geometric_series():
    """eq. 1: each of the l drafts is accepted with probability alpha given
    the earlier ones were, plus one bonus token: sum_{j=0}^{l} alpha^j."""
    for a in (0.3, 0.78, 0.95):
        for l in range(0, 12):
            assert ref.utility(a, l) == pytest.approx(sum(a ** j for j in range(l + 1)), rel=1e-12)


def test_reference_searches_agree_on_identical_users():
    """The homogeneous search (one draft length per batch, batch sizes only)
    equals the full search over assignments and per-user lengths."""
    sysm = ref.table2(4, 0.85)
    sysm.L_ub = 6
    for N in (2, 3):
        full = ref.brute_force(sysm, N)[0]
        homo = ref.homogeneous_optimum(sysm, N)[0]
        assert homo == pytest.approx(full, rel=1e-12)


def test_reference_span_matches_explicit_stage_schedule():
    """S* = max(sum t^v, max(t^d + t^v)) is attained by an explicit stage
    schedule (T_n = t^v_n, the slack added to one stage) and no smaller S
    satisfies eq. 16-18."""
    o, _ = _random_instance(3, 4)
    batches, l = [[0, 2], [1, 3]], [2, 5, 3, 1]
    tv = [ref.t_verify(o, len(b), max(l[m] for m in b), max(o.prefix[m] for m in b)) for b in batches]
    td = [max(ref.tau_draft(o, m, l[m]) + o.tau_c[m] for m in b) for b in batches]
    s = ref.span(o, batches, l)
    T = list(tv)
    T[0] += s - sum(tv)
    assert all(t >= v - 1e-9 for t, v in zip(T, tv)) and sum(T) == pytest.approx(s)
    assert all(s >= d + v - 1e-9 for d, v in zip(td, tv))
    assert s == pytest.approx(max(sum(tv), max(d + v for d, v in zip(td, tv))))


# ---- the scheduler against the reference -------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_assignment_subproblem_is_exact(seed):
    o, s = _random_instance(seed, 4)
    rng = np.random.default_rng(100 + seed)
    l = [int(v) for v in rng.integers(1, 7, 4)]
    for N in (2, 3):
        assign, S = sch.solve_assignment(s, N, l)
        S_ref, _ = ref.best_span_for_lengths(o, N, l)
        assert S == pytest.approx(S_ref, rel=1e-9), (N, l, assign)


@pytest.mark.parametrize("seed", range(6))
def test_length_subproblem_is_exact(seed):
    o, s = _random_instance(seed, 4)
    rng = np.random.default_rng(200 + seed)
    for N in (2, 3):
        assign = [int(v) for v in rng.permutation(np.arange(4) % N)]
        batches = [[m for m in range(4) if assign[m] == n] for n in range(N)]
        l, R = sch.solve_lengths(s, N, assign, [3] * 4)
        R_ref, _ = ref.best_lengths_for_batches(o, batches)
        assert R == pytest.approx(R_ref, rel=1e-9), (N, assign, l)
        assert ref.throughput(o, batches, l) == pytest.approx(R_ref, rel=1e-9)


@pytest.mark.parametrize("seed", range(4))
def test_algorithm1_reaches_the_exhaustive_optimum_on_small_instances(seed):
    """Alternating exact subproblems is a local method; on these instances
    it must land within 2% of the exhaustive optimum and never above it."""
    o, s = _random_instance(seed, 4, L_ub=5)
    sched = sch.solve(s)
    best = max(ref.brute_force(o, N)[0] for N in range(2, 5))
    batches = [[m for m in range(4) if sched.assign[m] == n] for n in range(sched.N)]
    assert ref.throughput(o, batches, sched.l) == pytest.approx(sched.R, rel=1e-9)
    assert sched.R <= best * (1 + 1e-9)
    assert sched.R >= 0.98 * best


@pytest.mark.parametrize("M,alpha", [(6, 0.70), (6, 0.95), (14, 0.78)])
def test_algorithm1_reproduces_paper_numbers(M, alpha):
    """Algorithm 1 on the Table II system: the printed 74.13 / 117.56 token/s
    (M = 6), and at M = 14 the exhaustive optimum, which the printed 17.89x
    over AD pins (test_reference_reproduces_paper_peak_speedups)."""
    sched = sch.solve(sch.paper_defaults(M, alpha))
    printed = GOLDEN["homogeneous_alpha_sweep"]["dipsd_tok_s"].get(f"{alpha:.2f}") if M == 6 else None
    if printed is not None:
        assert round(sched.R, 2) == printed
    else:
        assert sched.R == pytest.approx(ref.homogeneous_global(ref.table2(M, alpha))[0], rel=1e-12)
    o = ref.table2(M, alpha)
    batches = [[m for m in range(M) if sched.assign[m] == n] for n in range(sched.N)]
    assert ref.throughput(o, batches, sched.l) == pytest.approx(sched.R, rel=1e-12)


def test_memory_bound_excludes_large_batches():
    """With a memory cap that admits at most two users of prefix 2048 per
    batch, no schedule may batch three of them (eq. 19-21)."""
    v = ref.Model(64, 5120, 25600)
    params = v.J * (8.0 * v.h1 ** 2 + 4.0 * v.h1 * v.h2)
    cap = params + 4.0 * v.J * v.h1 * 2 * 2048 + 1.0
    o, s = _both([0.8] * 5, [2048] * 5, [3.0] * 5, [4.0305e-11] * 5, [33.8151] * 5, L_ub=4,
                 gamma_max=cap)
    sched = sch.solve(s)
    sizes = [sched.assign.count(n) for n in range(sched.N)]
    assert max(sizes) <= 2 and sched.N >= 3
    best = max(ref.brute_force(o, N)[0] for N in range(3, 6))
    assert sched.R <= best * (1 + 1e-9) and sched.R >= 0.98 * best


def test_verify_latency_fit_recovers_affine_model():
    """eq. 6 fitted back from latencies the model itself generates."""
    rng = np.random.default_rng(0)
    samples = []
    for b, L, I in itertools.product((1, 4, 16), (1, 4, 10), (256, 1024, 4096)):
        samples.append((b, L, I, ref.t_verify(ref.table2(1), b, L, I)))
    c, beta = sch.fit_verify_latency(samples, sch.ModelDims(64, 5120, 25600))
    assert c == pytest.approx(1.2077e-11, rel=1e-9)
    assert beta == pytest.approx(95.1074, rel=1e-9)
