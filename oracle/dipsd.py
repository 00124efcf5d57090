"""Exhaustive reference for the DiP-SD joint scheduler -- TEST INFRASTRUCTURE.

Only the test suite may import this module; the scheduler in the package
never calls it and the two share no code.

It evaluates the paper's system model literally and searches every
candidate instead of solving MILPs:

  * utility u_m(l) = (1 - alpha^(l+1)) / (1 - alpha)               (eq. 1, 2)
  * cost terms F^d(i), F^v(L, I)                                    (eq. 3, 4)
  * affine latencies G_m(b, F) = c_m b F + beta_m,
    G^v(b, F) = c^v b F + beta^v                                     (eq. 5, 6)
  * per-user drafting tau^d_m = l_m G_m(1, F^d(i_m))                 (eq. 13)
  * batch draft completion t^d_n = max over the batch of
    tau^d_m + tau^c_m                                                (eq. 14)
  * batch verify t^v_n = G^v(b_n, F^v(L_n, I_n)) with the batch maxima
    L_n, I_n                                                         (eq. 11, 12, 15)
  * stage durations T_n >= t^v_n, span S = sum_n T_n,
    S >= t^d_n + t^v_n                                               (eq. 16-18)
  * memory Gamma_p + 4 J h1 b_n I_n <= Gamma_max                     (eq. 19-21)
  * throughput R = U / S                                             (eq. 22)

For a fixed assignment and fixed draft lengths the smallest feasible span
follows directly from eq. 16-18: the stages must cover the verifications
(S >= sum_n t^v_n) and every batch's precedence (S >= t^d_n + t^v_n), and
stretching stage durations T_n can meet any S above both, so
S* = max(sum_n t^v_n, max_n (t^d_n + t^v_n)).

Searches:
  * ``brute_force``: every assignment of users to N non-empty batches (set
    partitions) and every draft-length vector in {1..L_ub}^M; small M only.
  * ``homogeneous_optimum``: users with identical parameters.  Two facts
    make an exact search small: (a) only the batch sizes matter, so batches
    are integer partitions of M; (b) inside a batch every user may take the
    batch's largest draft length without cost -- L_n, hence t^v_n, and the
    batch's draft completion t^d_n (attained by that user) are unchanged
    while u_m grows -- so one draft length per batch suffices.  Batches of
    equal size are interchangeable, so their lengths are enumerated as
    non-increasing sequences.

Parity status: pinned to the throughputs and speedups the paper prints for
its homogeneous experiments (Sec. V-B, kept with their citations in
tests/golden/dipsd_printed_values.json) and to closed forms (eq. 1's
geometric sum, the autoregressive baseline); see tests/test_scheduler.py.
The heterogeneous experiments (Sec. V-B-2) are not pinned: the per-user
values of their three cases cannot be recovered unambiguously from the
text.
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass, field
from typing import List, Sequence, Tuple


@dataclass
class Model:
    """Decoder blocks and hidden sizes (J, h1, h2) of one model."""
    J: int
    h1: int
    h2: int


@dataclass
class System:
    """Parameters of the DiP-SD system model (Table II defaults)."""
    alpha: List[float]
    prefix: List[int]
    tau_c: List[float]
    c_d: List[float]
    beta_d: List[float]
    draft: Model = field(default_factory=lambda: Model(28, 2048, 6144))
    verify: Model = field(default_factory=lambda: Model(64, 5120, 25600))
    c_v: float = 1.2077e-11
    beta_v: float = 95.1074
    gamma_max: float = 8.0e10
    L_ub: int = 20

    @property
    def M(self) -> int:
        return len(self.alpha)


def table2(M: int = 6, alpha: float = 0.78, prefix: int = 512) -> System:
    """The paper's default parameters (Table II) for M identical users."""
    return System(alpha=[alpha] * M, prefix=[prefix] * M, tau_c=[3.0] * M,
                  c_d=[4.0305e-11] * M, beta_d=[33.8151] * M)


def utility(alpha: float, l: int) -> float:
    """eq. 1: expected tokens of one round with l drafts, bonus included."""
    return (1.0 - alpha ** (l + 1)) / (1.0 - alpha)


def F_d(mdl: Model, i: int) -> float:
    """eq. 3."""
    return 4.0 * mdl.J * mdl.h1 * (2.0 * mdl.h1 + i + 1 + mdl.h2)


def F_v(mdl: Model, L: int, I: int) -> float:
    """eq. 4."""
    return 4.0 * mdl.J * mdl.h1 * L * (2.0 * mdl.h1 + I + L + mdl.h2)


def t_verify(sysm: System, b: int, L: int, I: int) -> float:
    """eq. 6 / 15: verification latency of a batch of b users."""
    return sysm.c_v * b * F_v(sysm.verify, L, I) + sysm.beta_v


def tau_draft(sysm: System, m: int, l: int) -> float:
    """eq. 13: l serial draft steps of G_m(1, F^d(i_m))."""
    return l * (sysm.c_d[m] * F_d(sysm.draft, sysm.prefix[m]) + sysm.beta_d[m])


def memory_ok(sysm: System, b: int, I: int) -> bool:
    """eq. 19-21."""
    v = sysm.verify
    params = v.J * (8.0 * v.h1 * v.h1 + 4.0 * v.h1 * v.h2)
    return params + 4.0 * v.J * v.h1 * b * I <= sysm.gamma_max


def span(sysm: System, batches: Sequence[Sequence[int]], l: Sequence[int]) -> float:
    """Smallest S of eq. 16-18 for the given batches (lists of users) and
    draft lengths; inf when a batch breaks the memory bound."""
    tv_sum, worst = 0.0, 0.0
    for users in batches:
        b = len(users)
        L = max(l[m] for m in users)
        I = max(sysm.prefix[m] for m in users)
        if not memory_ok(sysm, b, I):
            return float("inf")
        tv = t_verify(sysm, b, L, I)
        td = max(tau_draft(sysm, m, l[m]) + sysm.tau_c[m] for m in users)
        tv_sum += tv
        worst = max(worst, td + tv)
    return max(tv_sum, worst)


def throughput(sysm: System, batches: Sequence[Sequence[int]], l: Sequence[int]) -> float:
    """eq. 22 in tokens per second (S is in ms)."""
    U = sum(utility(sysm.alpha[m], l[m]) for m in range(sysm.M))
    return 1000.0 * U / span(sysm, batches, l)


def set_partitions(items: Sequence[int], n: int):
    """Every partition of items into exactly n non-empty unordered blocks."""
    items = list(items)
    if n == 0:
        if not items:
            yield []
        return
    if len(items) < n:
        return
    first, rest = items[0], items[1:]
    # first item alone in a block
    for p in set_partitions(rest, n - 1):
        yield [[first]] + p
    # first item joins one of the blocks of a partition of the rest
    for p in set_partitions(rest, n):
        for k in range(len(p)):
            yield p[:k] + [[first] + p[k]] + p[k + 1:]


def brute_force(sysm: System, N: int) -> Tuple[float, list, list]:
    """Best (R, batches, l) over all assignments into N batches and all
    draft lengths 1..L_ub (exhaustive; small M and L_ub only)."""
    best = (-1.0, None, None)
    M = sysm.M
    for batches in set_partitions(range(M), N):
        for l in itertools.product(range(1, sysm.L_ub + 1), repeat=M):
            r = throughput(sysm, batches, l)
            if r > best[0]:
                best = (r, [list(b) for b in batches], list(l))
    return best


def best_span_for_lengths(sysm: System, N: int, l: Sequence[int]) -> Tuple[float, list]:
    """min over assignments into N batches of S (draft lengths fixed)."""
    best = (float("inf"), None)
    for batches in set_partitions(range(sysm.M), N):
        s = span(sysm, batches, l)
        if s < best[0]:
            best = (s, [list(b) for b in batches])
    return best


def best_lengths_for_batches(sysm: System, batches: Sequence[Sequence[int]]) -> Tuple[float, list]:
    """max over draft lengths 1..L_ub of R (assignment fixed)."""
    best = (-1.0, None)
    for l in itertools.product(range(1, sysm.L_ub + 1), repeat=sysm.M):
        r = throughput(sysm, batches, l)
        if r > best[0]:
            best = (r, list(l))
    return best


def integer_partitions(M: int, N: int, largest: int = None):
    """Non-increasing size tuples of N positive parts summing to M."""
    largest = M if largest is None else largest
    if N == 0:
        if M == 0:
            yield ()
        return
    for s in range(min(M - (N - 1), largest), 0, -1):
        for rest in integer_partitions(M - s, N - 1, s):
            yield (s,) + rest


def homogeneous_optimum(sysm: System, N: int) -> Tuple[float, tuple, tuple]:
    """Best (R, batch sizes, per-batch draft lengths) for identical users
    (see the module docstring for why this search is exact)."""
    a, i = sysm.alpha[0], sysm.prefix[0]
    assert all(x == a for x in sysm.alpha) and all(x == i for x in sysm.prefix)
    best = (-1.0, None, None)
    for sizes in integer_partitions(sysm.M, N):
        groups = [(s, sum(1 for t in sizes if t == s)) for s in sorted(set(sizes), reverse=True)]
        per_group = [list(itertools.combinations_with_replacement(range(sysm.L_ub, 0, -1), cnt))
                     for _, cnt in groups]
        for choice in itertools.product(*per_group):
            lens, szs = [], []
            for (s, _), ls in zip(groups, choice):
                for L in ls:
                    szs.append(s)
                    lens.append(L)
            tv_sum, worst, U, ok = 0.0, 0.0, 0.0, True
            for s, L in zip(szs, lens):
                if not memory_ok(sysm, s, i):
                    ok = False
                    break
                tv = t_verify(sysm, s, L, i)
                td = tau_draft(sysm, 0, L) + sysm.tau_c[0]
                tv_sum += tv
                worst = max(worst, td + tv)
                U += s * utility(a, L)
            if not ok:
                continue
            r = 1000.0 * U / max(tv_sum, worst)
            if r > best[0]:
                best = (r, tuple(szs), tuple(lens))
    return best


def homogeneous_global(sysm: System) -> Tuple[float, int, tuple, tuple]:
    """Best (R, N, sizes, lengths) over N = 2..M for identical users.  A
    batch count is skipped once no solution with that many batches can win:
    every batch verifies in at least beta^v, so R <= U_max / (N beta^v),
    with U_max = M u(L_ub); the bound falls with N, so the scan stops."""
    u_max = sysm.M * utility(sysm.alpha[0], sysm.L_ub)
    best = (-1.0, None, None, None)
    for N in range(2, sysm.M + 1):
        if 1000.0 * u_max / (N * sysm.beta_v) <= best[0]:
            break
        r, sizes, lens = homogeneous_optimum(sysm, N)
        if r > best[0]:
            best = (r, N, sizes, lens)
    return best


def ad_greedy_batching(sysm: System) -> Tuple[float, list]:
    """Sec. V-A's "AD w/ greedy batching" baseline: users sorted by prefix
    length, longest first, are packed into batches in that order, a new
    batch starting whenever the next user would break the memory bound
    (eq. 19-21); every batch then decodes one token per user per forward
    (no drafts: G^v(b, F^v(1, I_n))), the batches one after another.
    Returns (tokens per second, batches)."""
    order = sorted(range(sysm.M), key=lambda m: -sysm.prefix[m])
    batches, cur = [], []
    for m in order:
        if cur and not memory_ok(sysm, len(cur) + 1, max(sysm.prefix[x] for x in cur + [m])):
            batches.append(cur)
            cur = []
        cur.append(m)
    batches.append(cur)
    ms = sum(t_verify(sysm, len(b), 1, max(sysm.prefix[x] for x in b)) for b in batches)
    return 1000.0 * sysm.M / ms, batches


def autoregressive(sysm: System) -> float:
    """Edge-only autoregressive decoding, one user at a time (Sec. V-A's AD
    baseline): one token per G^v(1, F^v(1, i)); tokens per second."""
    return 1000.0 / t_verify(sysm, 1, 1, sysm.prefix[0])
