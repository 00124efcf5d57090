"""DiP-SD joint scheduler: user-to-batch assignment x, draft lengths l and
batch count N that maximise pipelined throughput R = U / S (Sec. III-IV).

The system model (Sec. III): expected tokens per round u_m(l) (eq. 1-2),
cost terms F^d, F^v (eq. 3-4), affine latencies (eq. 5-6), assignment and
batch maxima (eq. 7-12), draft / verify timing and the pipeline span
(eq. 13-18), the edge memory bound (eq. 19-21), throughput (eq. 22).

The solver (Sec. IV, Algorithm 1): for each N = 2..M, alternate
  * the x-subproblem: min S over assignments for the current l (a MILP);
  * the l-subproblem: max U / S over draft lengths for the current x, by
    Dinkelbach's method with one MILP per iteration (eq. 24-29);
until l is unchanged and R changes by less than a tolerance, then keep the
best N (eq. 30).  The MILPs go to HiGHS through scipy.optimize.milp.

Formulation choices where the paper leaves the MILP form open:
  * x-subproblem: t^v_n depends on the product b_n F^v(L_n, I_n); each batch
    picks exactly one configuration (b, L, I) from a one-hot set (b in 1..M,
    L among the current draft lengths, I among the users' prefixes,
    memory-infeasible configurations removed), which makes every constraint
    linear; L_n and I_n then satisfy the epigraph constraints eq. 11-12.
    Batches are interchangeable, so user m may only sit in batches 0..m
    (a labelling by each batch's first user; it removes symmetric copies).
  * l-subproblem: the binary selectors y_mk, z_nk of eq. 23; t^v_n is
    linear in z_nk because b_n and I_n are fixed by x.

Latencies are in ms; throughputs are reported in tokens per second.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


@dataclass
class ModelDims:
    """Decoder blocks and hidden sizes (J, h1, h2)."""
    J: int
    h1: int
    h2: int


@dataclass
class SystemParams:
    """Per-user and edge parameters of the system model."""
    alpha: List[float]          # acceptance rates alpha_m
    prefix: List[int]           # prefix lengths i_m
    tau_c: List[float]          # communication latency tau^c_m (ms)
    c_d: List[float]            # drafting fit c_m (ms per unit of b F)
    beta_d: List[float]         # drafting fit beta_m (ms)
    draft: ModelDims = field(default_factory=lambda: ModelDims(28, 2048, 6144))
    verify: ModelDims = field(default_factory=lambda: ModelDims(64, 5120, 25600))
    c_v: float = 1.2077e-11     # verification fit c^v
    beta_v: float = 95.1074     # verification fit beta^v (ms)
    gamma_max: float = 8.0e10   # edge memory cap (bytes)
    L_ub: int = 20              # draft length upper bound
    T_ub: float = 1e6           # bounds on stage durations and span (ms)
    S_ub: float = 3e6
    l_init: int = 7             # initial draft length

    @property
    def M(self) -> int:
        return len(self.alpha)


def paper_defaults(M: int = 6, alpha: float = 0.78, prefix: int = 512) -> SystemParams:
    """Table II: Qwen3-1.7B drafts on the devices, Qwen3-32B verifies on the
    edge server; M identical users."""
    return SystemParams(alpha=[alpha] * M, prefix=[prefix] * M, tau_c=[3.0] * M,
                        c_d=[4.0305e-11] * M, beta_d=[33.8151] * M)


# ---- system model -----------------------------------------------------------

def expected_tokens(alpha: float, l: int) -> float:
    """u_m(l), eq. 1: accepted drafts plus the bonus token."""
    return (1.0 - alpha ** (l + 1)) / (1.0 - alpha)


def cost_draft(d: ModelDims, i: int) -> float:
    """F^d(i), eq. 3."""
    return 4.0 * d.J * d.h1 * (2.0 * d.h1 + i + 1 + d.h2)


def cost_verify(d: ModelDims, L: int, I: int) -> float:
    """F^v(L, I), eq. 4."""
    return 4.0 * d.J * d.h1 * L * (2.0 * d.h1 + I + L + d.h2)


def verify_ms(p: SystemParams, b: int, L: int, I: int) -> float:
    """t^v = G^v(b, F^v(L, I)), eq. 6 and 15."""
    return p.c_v * b * cost_verify(p.verify, L, I) + p.beta_v


def draft_step_ms(p: SystemParams, m: int) -> float:
    """G_m(1, F^d(i_m)): one draft token on user m's device, eq. 5."""
    return p.c_d[m] * cost_draft(p.draft, p.prefix[m]) + p.beta_d[m]


def memory_fits(p: SystemParams, b: int, I: int) -> bool:
    """Gamma_p + Gamma_kv <= Gamma_max, eq. 19-21."""
    v = p.verify
    return v.J * (8.0 * v.h1 ** 2 + 4.0 * v.h1 * v.h2) + 4.0 * v.J * v.h1 * b * I <= p.gamma_max


def span_ms(p: SystemParams, assign: Sequence[int], l: Sequence[int], N: int) -> float:
    """Smallest pipeline span S for a fixed assignment and draft lengths:
    eq. 16-18 need S >= sum_n t^v_n and S >= t^d_n + t^v_n."""
    tv_sum, worst = 0.0, 0.0
    for n in range(N):
        users = [m for m in range(p.M) if assign[m] == n]
        if not users:
            return float("inf")
        b, L, I = len(users), max(l[m] for m in users), max(p.prefix[m] for m in users)
        if not memory_fits(p, b, I):
            return float("inf")
        tv = verify_ms(p, b, L, I)
        td = max(l[m] * draft_step_ms(p, m) + p.tau_c[m] for m in users)
        tv_sum += tv
        worst = max(worst, td + tv)
    return max(tv_sum, worst)


def throughput(p: SystemParams, assign: Sequence[int], l: Sequence[int], N: int) -> float:
    """R = U / S, eq. 22, in tokens per second."""
    U = sum(expected_tokens(p.alpha[m], l[m]) for m in range(p.M))
    return 1000.0 * U / span_ms(p, assign, l, N)


# ---- MILP plumbing ----------------------------------------------------------

class _Lp:
    """Sparse rows lo <= a x <= hi for scipy.optimize.milp."""

    def __init__(self, nvar: int):
        self.n = nvar
        self.rows: List[Dict[int, float]] = []
        self.lo: List[float] = []
        self.hi: List[float] = []

    def add(self, coefs: Dict[int, float], lo: float, hi: float):
        self.rows.append(coefs)
        self.lo.append(lo)
        self.hi.append(hi)

    def solve(self, c, integrality, lb, ub, time_limit: float):
        from scipy.optimize import Bounds, LinearConstraint, milp
        from scipy.sparse import coo_matrix
        ri, ci, v = [], [], []
        for r, row in enumerate(self.rows):
            for j, a in row.items():
                ri.append(r)
                ci.append(j)
                v.append(a)
        A = coo_matrix((v, (ri, ci)), shape=(len(self.rows), self.n)).tocsr()
        res = milp(np.asarray(c, dtype=float), integrality=np.asarray(integrality),
                   bounds=Bounds(np.asarray(lb, dtype=float), np.asarray(ub, dtype=float)),
                   constraints=LinearConstraint(A, np.asarray(self.lo), np.asarray(self.hi)),
                   options={"time_limit": time_limit, "mip_rel_gap": 1e-9, "disp": False})
        if res.status == 2:      # infeasible
            return None
        if res.x is None:
            raise RuntimeError(f"MILP failed: {res.message}")
        return res.x


# ---- x-subproblem -----------------------------------------------------------

def solve_assignment(p: SystemParams, N: int, l: Sequence[int],
                     time_limit: float = 60.0) -> Tuple[Optional[List[int]], float]:
    """min S over assignments x for fixed draft lengths (Sec. IV-B).
    Returns (batch index per user, S in ms), or (None, inf) when no
    assignment into N batches meets the memory bound."""
    M = p.M
    Lv = sorted(set(int(v) for v in l))
    Iv = sorted(set(int(v) for v in p.prefix))
    cfgs = [(b, L, I) for b in range(1, M + 1) for L in Lv for I in Iv if memory_fits(p, b, I)]
    nx = M * N
    nw = N * len(cfgs)
    iT, itd, iS = nx + nw, nx + nw + N, nx + nw + 2 * N
    nvar = iS + 1
    X = lambda m, n: m * N + n
    W = lambda n, k: nx + n * len(cfgs) + k
    tv = [verify_ms(p, b, L, I) for (b, L, I) in cfgs]
    draw = [l[m] * draft_step_ms(p, m) + p.tau_c[m] for m in range(M)]
    lp = _Lp(nvar)
    for m in range(M):                                  # eq. 8
        lp.add({X(m, n): 1.0 for n in range(N)}, 1.0, 1.0)
    for n in range(N):
        lp.add({W(n, k): 1.0 for k in range(len(cfgs))}, 1.0, 1.0)   # one configuration
        row = {X(m, n): 1.0 for m in range(M)}          # b_n = sum_m x_mn (eq. 10)
        for k, (b, _, _) in enumerate(cfgs):
            row[W(n, k)] = -float(b)
        lp.add(row, 0.0, 0.0)
        for m in range(M):
            rowL = {W(n, k): float(L) for k, (_, L, _) in enumerate(cfgs)}
            rowL[X(m, n)] = -float(l[m])
            lp.add(rowL, 0.0, np.inf)                   # L_n >= l_m x_mn (eq. 11)
            rowI = {W(n, k): float(I) for k, (_, _, I) in enumerate(cfgs)}
            rowI[X(m, n)] = -float(p.prefix[m])
            lp.add(rowI, 0.0, np.inf)                   # I_n >= i_m x_mn (eq. 12)
            lp.add({itd + n: 1.0, X(m, n): -draw[m]}, 0.0, np.inf)   # eq. 14
        rowT = {iT + n: 1.0}
        rowP = {iS: 1.0, itd + n: -1.0}
        for k in range(len(cfgs)):
            rowT[W(n, k)] = -tv[k]
            rowP[W(n, k)] = -tv[k]
        lp.add(rowT, 0.0, np.inf)                       # T_n >= t^v_n (eq. 16)
        lp.add(rowP, 0.0, np.inf)                       # S >= t^d_n + t^v_n (eq. 18)
    row = {iS: 1.0}
    for n in range(N):
        row[iT + n] = -1.0
    lp.add(row, 0.0, 0.0)                               # S = sum_n T_n (eq. 17)
    c = np.zeros(nvar)
    c[iS] = 1.0
    integ = np.zeros(nvar, dtype=int)
    integ[:nx + nw] = 1
    lb = np.zeros(nvar)
    ub = np.full(nvar, np.inf)
    ub[:nx + nw] = 1.0
    for m in range(M):
        for n in range(m + 1, N):
            ub[X(m, n)] = 0.0                           # first-user batch labelling
    ub[iT:iT + N] = p.T_ub
    ub[itd:itd + N] = p.T_ub
    ub[iS] = p.S_ub
    sol = lp.solve(c, integ, lb, ub, time_limit)
    if sol is None:
        return None, float("inf")
    assign = [int(np.argmax([sol[X(m, n)] for n in range(N)])) for m in range(M)]
    return assign, span_ms(p, assign, l, N)


# ---- l-subproblem -----------------------------------------------------------

def solve_lengths(p: SystemParams, N: int, assign: Sequence[int], l0: Sequence[int],
                  eps: float = 1e-9, max_iter: int = 50,
                  time_limit: float = 60.0) -> Tuple[List[int], float]:
    """max U / S over draft lengths for a fixed assignment by Dinkelbach's
    method (Sec. IV-C); starts from l0.  Returns (l, R in tokens/s)."""
    M, K = p.M, p.L_ub
    batches = [[m for m in range(M) if assign[m] == n] for n in range(N)]
    ny, nz = M * K, N * K
    iT, itd, iS = ny + nz, ny + nz + N, ny + nz + 2 * N
    nvar = iS + 1
    Y = lambda m, k: m * K + (k - 1)
    Z = lambda n, k: ny + n * K + (k - 1)
    u = [[expected_tokens(p.alpha[m], k) for k in range(1, K + 1)] for m in range(M)]
    g = [draft_step_ms(p, m) for m in range(M)]
    bI = [(len(bs), max(p.prefix[m] for m in bs)) for bs in batches]
    tvk = [[verify_ms(p, b, k, I) for k in range(1, K + 1)] for (b, I) in bI]
    lp = _Lp(nvar)
    for m in range(M):
        lp.add({Y(m, k): 1.0 for k in range(1, K + 1)}, 1.0, 1.0)    # eq. 23, y
    for n, bs in enumerate(batches):
        lp.add({Z(n, k): 1.0 for k in range(1, K + 1)}, 1.0, 1.0)    # eq. 23, z
        for m in bs:
            row = {Z(n, k): float(k) for k in range(1, K + 1)}
            for k in range(1, K + 1):
                row[Y(m, k)] = -float(k)
            lp.add(row, 0.0, np.inf)                    # L_n >= l_m (eq. 24)
            row = {itd + n: 1.0}
            for k in range(1, K + 1):
                row[Y(m, k)] = -k * g[m]
            lp.add(row, p.tau_c[m], np.inf)             # t^d_n >= tau^d_m + tau^c_m
        rowT = {iT + n: 1.0}
        rowP = {iS: 1.0, itd + n: -1.0}
        for k in range(1, K + 1):
            rowT[Z(n, k)] = -tvk[n][k - 1]
            rowP[Z(n, k)] = -tvk[n][k - 1]
        lp.add(rowT, 0.0, np.inf)
        lp.add(rowP, 0.0, np.inf)
    row = {iS: 1.0}
    for n in range(N):
        row[iT + n] = -1.0
    lp.add(row, 0.0, 0.0)
    integ = np.zeros(nvar, dtype=int)
    integ[:ny + nz] = 1
    lb = np.zeros(nvar)
    ub = np.full(nvar, np.inf)
    ub[:ny + nz] = 1.0
    ub[iT:iT + N] = p.T_ub
    ub[itd:itd + N] = p.T_ub
    ub[iS] = p.S_ub

    l = [int(v) for v in l0]
    U = sum(expected_tokens(p.alpha[m], l[m]) for m in range(M))
    q = U / span_ms(p, assign, l, N)                    # tokens per ms
    for _ in range(max_iter):
        c = np.zeros(nvar)
        for m in range(M):
            for k in range(1, K + 1):
                c[Y(m, k)] = -u[m][k - 1]
        c[iS] = q                                       # min q S - U (eq. 25)
        sol = lp.solve(c, integ, lb, ub, time_limit)
        l_new = [int(np.argmax([sol[Y(m, k)] for k in range(1, K + 1)])) + 1 for m in range(M)]
        U_new = sum(expected_tokens(p.alpha[m], l_new[m]) for m in range(M))
        S_new = span_ms(p, assign, l_new, N)
        gap = U_new - q * S_new                         # eq. 27
        l = l_new
        q_next = U_new / S_new                          # eq. 26
        if abs(gap) <= eps * max(1.0, U_new):
            q = q_next
            break
        q = q_next
    return l, 1000.0 * q


# ---- Algorithm 1 ------------------------------------------------------------

@dataclass
class Schedule:
    N: int
    assign: List[int]           # batch index per user (x_mn = 1 iff assign[m] = n)
    l: List[int]                # draft length per user
    R: float                    # tokens per second
    U: float                    # expected tokens per round
    S: float                    # pipeline span (ms)
    per_N: Dict[int, float]     # converged R*(N) of every scanned N
    iterations: Dict[int, int]  # alternating rounds per N


def solve(p: SystemParams, N_range: Optional[Sequence[int]] = None, tol: float = 1e-9,
          max_rounds: int = 20, time_limit: float = 60.0) -> Schedule:
    """Algorithm 1: scan N, alternate the x and l subproblems, keep the best."""
    N_range = list(N_range) if N_range is not None else list(range(2, p.M + 1))
    best: Optional[Schedule] = None
    per_N, iters = {}, {}
    for N in N_range:
        if N < 1 or N > p.M:
            continue
        l = [p.l_init] * p.M
        R_prev = -1.0
        assign = None
        for r in range(max_rounds):
            assign, _ = solve_assignment(p, N, l, time_limit)
            if assign is None:
                break
            l_new, R = solve_lengths(p, N, assign, l, time_limit=time_limit)
            done = l_new == l and abs(R - R_prev) <= tol * max(1.0, R)
            l, R_prev = l_new, R
            if done:
                break
        iters[N] = r + 1
        if assign is None:       # memory bound: no assignment into N batches
            per_N[N] = 0.0
            continue
        R = throughput(p, assign, l, N)
        per_N[N] = R
        if best is None or R > best.R:
            U = sum(expected_tokens(p.alpha[m], l[m]) for m in range(p.M))
            best = Schedule(N, list(assign), list(l), R, U, span_ms(p, assign, l, N), {}, {})
    if best is None:
        raise ValueError("no feasible batch count")
    best.per_N, best.iterations = per_N, iters
    return best


# ---- the edge server's own verify latency ------------------------------------

def fit_verify_latency(samples: Sequence[Tuple[int, int, int, float]],
                       verify: ModelDims) -> Tuple[float, float]:
    """Least-squares (c^v, beta^v) of eq. 6 from measured verify passes
    (b, L, I, ms): ms ~ c^v b F^v(L, I) + beta^v."""
    xs = np.array([b * cost_verify(verify, L, I) for b, L, I, _ in samples], dtype=float)
    ys = np.array([t for *_, t in samples], dtype=float)
    A = np.stack([xs, np.ones_like(xs)], axis=1)
    (c, beta), *_ = np.linalg.lstsq(A, ys, rcond=None)
    return float(c), float(beta)
