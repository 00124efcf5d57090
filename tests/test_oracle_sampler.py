"""Pins for the oracle's accept/reject/resample step.

What the paper fixes (DiP-SD, Sec. II-A step 2 and eq. (1)): verification
stops at the first rejected draft and always emits one more token, and under
i.i.d. acceptance with rate alpha the expected number of tokens per round is
(1 - alpha^(l+1)) / (1 - alpha).  The accept/resample rule comes from the
speculative-sampling work the paper cites in Sec. I, whose defining property
is that emitted tokens follow the target distribution.  Each test below
checks one of these facts on toy tables where the exact answer is known.
"""
import itertools
import math

import numpy as np
import pytest
from scipy import stats

import oracle


def _tables(rng, L, V, zero_p=None, zero_q=None):
    """Per-slot target p (L+1 rows) and draft q (L rows) distributions."""
    p = rng.dirichlet(np.ones(V), size=L + 1)
    q = rng.dirichlet(np.ones(V), size=L)
    if zero_p is not None:
        p[:, zero_p] = 0.0
        p /= p.sum(1, keepdims=True)
    if zero_q is not None:
        q[:, zero_q] = 0.0
        q /= q.sum(1, keepdims=True)
    return p, q


def _logits(p):
    with np.errstate(divide="ignore"):
        return np.log(p).astype(np.float32)


def _batch(p, q, B, rng, drafts=None):
    """B independent trials of the same per-slot tables; drafts ~ q."""
    L = q.shape[0]
    V = p.shape[1]
    logits = np.tile(_logits(p), (B, 1))
    qq = np.tile(q.astype(np.float32), (B, 1))
    if drafts is None:
        drafts = np.empty((B, L), np.int32)
        for j in range(L):
            drafts[:, j] = rng.choice(V, size=B, p=q[j])
    return logits, qq, drafts.reshape(-1)


def _emitted(res, drafts, L):
    """Emitted sequence per trial: accepted drafts then the final token."""
    out = []
    d = drafts.reshape(-1, L)
    for b in range(d.shape[0]):
        a = int(res["n_acc"][b])
        out.append(list(d[b, :a]) + [int(res["token"][b])])
    return out


def _chi2_ok(counts, probs, alpha=1e-3):
    counts = np.asarray(counts, float)
    probs = np.asarray(probs, float)
    n = counts.sum()
    keep = probs > 0
    assert np.all(counts[~keep] == 0), "a zero-probability token was emitted"
    exp = probs[keep] * n
    chi2 = ((counts[keep] - exp) ** 2 / exp).sum()
    pval = stats.chi2.sf(chi2, keep.sum() - 1)
    return pval > alpha, pval


def test_q_equals_p_accepts_everything():
    rng = np.random.default_rng(10)
    L, V, B = 4, 7, 4000
    p, _ = _tables(rng, L, V)
    q = p[:L].copy()
    logits, qq, drafts = _batch(p, q, B, rng)
    res = oracle.sample("stochastic", np.arange(B), np.full(B, L), logits, drafts, qq, seed=1)
    assert np.all(res["n_acc"] == L)


def test_target_distribution_is_preserved():
    """Each emitted token follows the target row of its position, including
    tokens q never proposes (only the residual can supply them) and never
    tokens p forbids."""
    rng = np.random.default_rng(11)
    L, V, B = 3, 6, 30000
    p, q = _tables(rng, L, V, zero_p=5, zero_q=2)
    logits, qq, drafts = _batch(p, q, B, rng)
    res = oracle.sample("stochastic", np.arange(B), np.full(B, L), logits, drafts, qq, seed=7, round_=3)
    seqs = _emitted(res, drafts, L)
    for k in range(L + 1):
        toks = [s[k] for s in seqs if len(s) > k]
        counts = np.bincount(toks, minlength=V)
        ok, pv = _chi2_ok(counts, p[k])
        assert ok, f"position {k}: chi2 p-value {pv}"


def test_residual_distribution_after_rejection():
    """A rejected draft is replaced by a draw from norm(max(0, p - q))."""
    rng = np.random.default_rng(12)
    V, B = 8, 30000
    p, q = _tables(rng, 1, V)
    d = int(np.argmin(p[0] / q[0]))  # p(d) < q(d), so rejection is possible
    assert p[0, d] / q[0, d] < 0.9
    logits, qq, drafts = _batch(p, q, B, rng, drafts=np.full((B, 1), d, np.int32))
    u = np.full(B, 0.9999, np.float32)  # above r: always reject
    res = oracle.sample("stochastic", np.arange(B), np.ones(B), logits, drafts, qq, accept_u=u, seed=3)
    assert np.all(res["n_acc"] == 0)
    w = np.maximum(0.0, p[0] - q[0])
    ok, pv = _chi2_ok(np.bincount(res["token"], minlength=V), w / w.sum())
    assert ok, pv


def test_bonus_token_follows_last_row():
    rng = np.random.default_rng(13)
    L, V, B = 2, 5, 20000
    p, q = _tables(rng, L, V)
    logits, qq, drafts = _batch(p, q, B, rng)
    u = np.zeros(B * L, np.float32)  # u = 0 < r: always accept
    res = oracle.sample("stochastic", np.arange(B), np.full(B, L), logits, drafts, qq, accept_u=u, seed=4)
    assert np.all(res["n_acc"] == L)
    ok, pv = _chi2_ok(np.bincount(res["token"], minlength=V), p[L])
    assert ok, pv


def test_accept_probability_is_min_one_ratio():
    """With a stratified grid of accept uniforms the accepted fraction is
    min(1, p(d)/q(d)) to the grid resolution, and u == r rejects."""
    rng = np.random.default_rng(14)
    V, G = 6, 4096
    p, q = _tables(rng, 1, V)
    u = ((np.arange(G) + 0.5) / G).astype(np.float32)
    for d in range(V):
        logits, qq, drafts = _batch(p, q, G, rng, drafts=np.full((G, 1), d, np.int32))
        res = oracle.sample("stochastic", np.arange(G), np.ones(G), logits, drafts, qq, accept_u=u)
        frac = res["n_acc"].mean()
        assert abs(frac - min(1.0, p[0, d] / q[0, d])) <= 1.0 / G + 1e-6
        r = res["ratio"][0]
        if r < 1:
            res2 = oracle.sample("stochastic", [0], [1], logits[:2], drafts[:1], qq[:1],
                                 accept_u=np.array([r], np.float32))
            assert res2["n_acc"][0] == 0


@pytest.mark.parametrize("alpha,L", [(0.78, 7), (0.5, 3), (0.95, 12)])
def test_geometric_mean_eq1(alpha, L):
    """q = alpha * p + (1 - alpha) * delta_z with p(z) = 0 gives acceptance
    rate exactly alpha per draft; the mean tokens per round must equal
    (1 - alpha^(L+1)) / (1 - alpha) (eq. 1) and n_acc must follow the
    truncated geometric law."""
    rng = np.random.default_rng(int(alpha * 100) + L)
    V, B = 9, 20000
    z = V - 1
    p = rng.dirichlet(np.ones(V), size=L + 1)
    p[:, z] = 0.0
    p /= p.sum(1, keepdims=True)
    q = alpha * p[:L].copy()
    q[:, z] += 1.0 - alpha
    logits, qq, drafts = _batch(p, q, B, rng)
    res = oracle.sample("stochastic", np.arange(B), np.full(B, L), logits, drafts, qq, seed=5, round_=1)
    tokens = res["n_acc"] + 1
    mean = (1 - alpha ** (L + 1)) / (1 - alpha)
    pk = np.array([alpha ** k * (1 - alpha) for k in range(L)] + [alpha ** L])
    var = float(((np.arange(L + 1) + 1) ** 2 * pk).sum() - mean ** 2)
    assert abs(tokens.mean() - mean) < 4 * math.sqrt(var / B)
    ok, pv = _chi2_ok(np.bincount(res["n_acc"], minlength=L + 1), pk)
    assert ok, pv


def test_greedy_accepts_longest_matching_prefix():
    rng = np.random.default_rng(15)
    L, V, B = 5, 11, 50
    logits = rng.normal(size=(B * (L + 1), V)).astype(np.float32)
    am = logits.argmax(1).reshape(B, L + 1)
    k = rng.integers(0, L + 1, size=B)  # first planted mismatch (L = none)
    drafts = am[:, :L].copy()
    for b in range(B):
        if k[b] < L:
            drafts[b, k[b]] = (am[b, k[b]] + 1 + rng.integers(0, V - 1)) % V
            drafts[b, k[b] + 1:] = rng.integers(0, V, size=L - k[b] - 1)
    res = oracle.sample("greedy", np.arange(B), np.full(B, L), logits, drafts.reshape(-1),
                        np.zeros((0, V), np.float32))
    assert np.array_equal(res["n_acc"], k)
    assert np.array_equal(res["token"], am[np.arange(B), k])


def test_greedy_ties_break_to_lowest_index():
    V = 6
    row = np.array([0.1, 2.0, 0.3, 2.0, -1.0, 2.0], np.float32)
    logits = np.stack([row, row])
    res = oracle.sample("greedy", [0], [1], logits, np.array([3], np.int32), np.zeros((0, V), np.float32))
    assert res["n_acc"][0] == 0 and res["token"][0] == 1
    res = oracle.sample("greedy", [0], [1], logits, np.array([1], np.int32), np.zeros((0, V), np.float32))
    assert res["n_acc"][0] == 1 and res["token"][0] == 1


def test_force_mode_accepts_all():
    rng = np.random.default_rng(16)
    L, V = 3, 9
    logits = rng.normal(size=(L + 1, V)).astype(np.float32)
    res = oracle.sample("force", [0], [L], logits, np.array([1, 2, 3], np.int32), np.zeros((0, V), np.float32))
    assert res["n_acc"][0] == L and res["token"][0] == int(logits[L].argmax())


def test_zero_residual_falls_back_to_target():
    """If max(0, p - q) is zero everywhere the correction is drawn from p."""
    rng = np.random.default_rng(17)
    V, B = 5, 20000
    p = rng.dirichlet(np.ones(V), size=2)
    q = (p[:1] * 1.01).astype(np.float32)  # q >= p elementwise: residual is empty
    logits, qq, drafts = _batch(p, q, B, rng, drafts=np.zeros((B, 1), np.int32))
    res = oracle.sample("stochastic", np.arange(B), np.ones(B), logits, drafts, qq,
                        accept_u=np.full(B, 0.9999, np.float32), seed=9)
    assert np.all(res["n_acc"] == 0)
    ok, pv = _chi2_ok(np.bincount(res["token"], minlength=V), p[0])
    assert ok, pv


def test_zero_draft_probability_edge_cases():
    """p/0 = +inf accepts; 0/0 = NaN rejects (IEEE semantics of r = p/q)."""
    p = np.array([[0.5, 0.5, 0.0], [0.2, 0.3, 0.5]])
    q = np.array([[0.0, 0.0, 1.0]], np.float32)
    logits = _logits(p)
    r1 = oracle.sample("stochastic", [0], [1], logits, np.array([0], np.int32), q,
                       accept_u=np.array([0.999], np.float32))
    assert r1["n_acc"][0] == 1 and np.isinf(r1["ratio"][0])
    q2 = np.array([[0.5, 0.5, 0.0]], np.float32)
    r2 = oracle.sample("stochastic", [0], [1], logits, np.array([2], np.int32), q2,
                       accept_u=np.array([0.0], np.float32))
    assert r2["n_acc"][0] == 0 and np.isnan(r2["ratio"][0])


def test_draws_depend_on_user_not_batch_position():
    """Counter-based draws are keyed by the global user id: permuting the
    batch permutes the results."""
    rng = np.random.default_rng(18)
    L, V, B = 2, 7, 6
    p, q = _tables(rng, L, V)
    logits, qq, drafts = _batch(p, q, B, rng)
    users = np.array([3, 9, 12, 40, 41, 77])
    res = oracle.sample("stochastic", users, np.full(B, L), logits, drafts, qq, seed=2, round_=5)
    perm = np.array([5, 0, 3, 1, 4, 2])
    lg = logits.reshape(B, L + 1, V)[perm].reshape(-1, V)
    qp = qq.reshape(B, L, V)[perm].reshape(-1, V)
    dp = drafts.reshape(B, L)[perm].reshape(-1)
    res2 = oracle.sample("stochastic", users[perm], np.full(B, L), lg, dp, qp, seed=2, round_=5)
    assert np.array_equal(res2["n_acc"], res["n_acc"][perm])
    assert np.array_equal(res2["token"], res["token"][perm])


def test_decode_step_draws_from_p():
    """l_m = 0 (a drafting model's decode step): no accept trial, and the
    emitted token follows p of the single slot; greedy takes its argmax
    (lowest index on ties), zero-probability tokens are never drawn."""
    rng = np.random.default_rng(23)
    V, B = 7, 30000
    p, _ = _tables(rng, 0, V, zero_p=[2])
    logits = np.tile(_logits(p), (B, 1))
    empty_q = np.zeros((0, V), np.float32)
    res = oracle.sample("stochastic", np.arange(B), np.zeros(B), logits, np.zeros(0, np.int32),
                        empty_q, seed=5, round_=1)
    assert np.all(res["n_acc"] == 0)
    ok, pv = _chi2_ok(np.bincount(res["token"], minlength=V), p[0])
    assert ok, pv
    # other rounds and seeds give other draws from the same law
    res2 = oracle.sample("stochastic", np.arange(B), np.zeros(B), logits, np.zeros(0, np.int32),
                         empty_q, seed=5, round_=2)
    assert (res2["token"] != res["token"]).mean() > 0.5
    g = oracle.sample("greedy", np.arange(3), np.zeros(3), logits[:3], np.zeros(0, np.int32), empty_q)
    assert np.all(g["token"] == int(np.argmax(p[0])))


def _sparse_rows(q, K):
    """Top-K of each dense row plus a uniform remainder (test tables)."""
    V = q.shape[1]
    idx = np.argsort(-q, axis=1, kind="stable")[:, :K]
    val = np.take_along_axis(q, idx, axis=1)
    rest = (1.0 - val.sum(1)) / (V - K)
    return idx.astype(np.int32), val.astype(np.float32), rest.astype(np.float32)


def test_sparse_rows_expand_to_their_definition():
    rng = np.random.default_rng(29)
    V, K = 9, 3
    _, q = _tables(rng, 4, V)
    idx, val, rest = _sparse_rows(q, K)
    dense = oracle.expand_sparse_q(idx, val, rest, V)
    for r in range(q.shape[0]):
        for k in range(V):
            hit = np.nonzero(idx[r] == k)[0]
            want = val[r, hit[0]] if hit.size else rest[r]
            assert dense[r, k] == want
        assert abs(dense[r].astype(np.float64).sum() - 1.0) < 1e-6


def test_sparse_draft_rows_keep_the_target_distribution():
    """Drafts drawn from top-K-plus-remainder rows and verified against
    those rows: the first emitted token still follows p (the speculative
    sampling law holds for any draft distribution given exactly)."""
    rng = np.random.default_rng(31)
    L, V, K, B = 2, 8, 3, 30000
    p, q = _tables(rng, L, V)
    idx, val, rest = _sparse_rows(q, K)
    qs = oracle.expand_sparse_q(idx, val, rest, V).astype(np.float64)
    qs /= qs.sum(1, keepdims=True)
    logits, qq, drafts = _batch(p, qs, B, rng)
    # the rows as the verifier receives them (unnormalised float32 values)
    qq = np.tile(oracle.expand_sparse_q(idx, val, rest, V), (B, 1))
    res = oracle.sample("stochastic", np.arange(B), np.full(B, L), logits, drafts, qq, seed=12)
    first = [e[0] for e in _emitted(res, drafts, L)]
    ok, pv = _chi2_ok(np.bincount(first, minlength=V), p[0])
    assert ok, pv


# ----------------------------------------------------------------------------
# exact output law by enumeration
# ----------------------------------------------------------------------------

class _ContextTables:
    """Target p(.|ctx) and draft q(.|ctx) for every context (a tuple of
    tokens), drawn from a seed keyed by the context, with zeros: p forbids a
    token that q may propose, and q never proposes a token p may need (only
    the residual can supply it).  The rows differ from context to context, so
    a sampler reading the wrong slot's row gets a different law."""

    def __init__(self, V, seed):
        self.V, self.seed = V, seed
        self._p, self._q = {}, {}

    def _rng(self, ctx, which):
        return np.random.default_rng([self.seed, which, len(ctx), *ctx])

    def p(self, ctx):
        if ctx not in self._p:
            r = self._rng(ctx, 1).dirichlet(np.full(self.V, 0.7))
            r[(len(ctx) + sum(ctx)) % self.V] = 0.0
            # round-trip through the float32 logits the oracle receives, so
            # the law below is the one the logits define
            z = _logits(r / r.sum())
            e = np.exp(z.astype(np.float64) - z.max())
            self._p[ctx] = (z, e / e.sum())
        return self._p[ctx]

    def q(self, ctx):
        if ctx not in self._q:
            r = self._rng(ctx, 2).dirichlet(np.full(self.V, 0.7))
            r[(len(ctx) + 2 * sum(ctx) + 1) % self.V] = 0.0
            if len(ctx) % 2 == 0:
                r[(sum(ctx) + 3) % self.V] = 0.0
            self._q[ctx] = (r / r.sum()).astype(np.float32)
        return self._q[ctx]


def _round_law(tab, ctx, L, seed):
    """Exact law of one verification round from context ctx: every draft
    sequence weighted by its draft probability, every stop slot a weighted by
    the oracle's own accept ratios (P(accept) = min(1, r) for a uniform u),
    and the emitted token weighted by the oracle's own race weights at the
    stop slot (an exponential race picks k with probability w_k / sum w).
    Returns {emitted tuple: probability}."""
    V = tab.V
    seqs = list(itertools.product(range(V), repeat=L))
    B = len(seqs)
    logits = np.empty((B * (L + 1), V), np.float32)
    q = np.empty((B * L, V), np.float32)
    for b, d in enumerate(seqs):
        for j in range(L + 1):
            logits[b * (L + 1) + j] = tab.p(ctx + d[:j])[0]
        for j in range(L):
            q[b * L + j] = tab.q(ctx + d[:j])
    drafts = np.array(seqs, np.int32).reshape(-1)
    users, lens = np.arange(B), np.full(B, L)
    law = {}
    for a in range(L + 1):
        # uniforms that force the stop at slot a: 0 accepts any r > 0, +inf
        # rejects any finite r (branches they cannot force have probability 0)
        u = np.zeros((B, L), np.float32)
        if a < L:
            u[:, a] = np.inf
        res = oracle.sample("stochastic", users, lens, logits, drafts, q, accept_u=u.reshape(-1),
                            seed=seed, want_race_w=True)
        r = res["ratio"].reshape(B, L).astype(np.float64)
        for b, d in enumerate(seqs):
            pd = float(np.prod([q[b * L + j, d[j]] for j in range(L)], dtype=np.float64))
            if pd == 0.0:
                continue  # a draft q never proposes (its ratio may be 0/0)
            acc = np.minimum(1.0, r[b])
            pa = float(np.prod(acc[:a])) * (1.0 - acc[a] if a < L else 1.0)
            if pa == 0.0:
                continue
            assert res["n_acc"][b] == a
            w = res["race_w"][b].astype(np.float64)
            assert w.sum() > 0
            for k in np.nonzero(w)[0]:
                e = tuple(d[:a]) + (int(k),)
                law[e] = law.get(e, 0.0) + pd * pa * w[k] / w.sum()
    return law


def _first_n_law(tab, ctx, n, L, seed, memo):
    """Exact law of the first n emitted tokens from ctx over as many rounds
    as it takes (each round continues from the tokens it emitted)."""
    if n <= 0:
        return {(): 1.0}
    key = (ctx, n)
    if key in memo:
        return memo[key]
    out = {}
    for e, pe in _round_law(tab, ctx, L, seed).items():
        if len(e) >= n:
            out[e[:n]] = out.get(e[:n], 0.0) + pe
        else:
            for rest, pr in _first_n_law(tab, ctx + e, n - len(e), L, seed, memo).items():
                out[e + rest] = out.get(e + rest, 0.0) + pe * pr
    memo[key] = out
    return out


@pytest.mark.parametrize("V,L,n", [(4, 1, 3), (4, 2, 4), (3, 3, 4), (5, 2, 3)])
def test_output_law_by_enumeration(V, L, n):
    """The tokens emitted by repeated verification rounds follow the target
    model exactly: the law of the first n tokens, summed over every draft
    sequence, accept/reject outcome and resampled token, equals the product
    of the target rows along the sequence (the defining property of the
    speculative-sampling rule of the works cited in Sec. I)."""
    tab = _ContextTables(V, seed=100 * V + 10 * L + n)
    law = _first_n_law(tab, (), n, L, seed=3, memo={})
    worst = 0.0
    total = 0.0
    for y in itertools.product(range(V), repeat=n):
        want = 1.0
        for t in range(n):
            want *= tab.p(y[:t])[1][y[t]]
        got = law.get(y, 0.0)
        total += got
        worst = max(worst, abs(got - want))
        if want == 0.0:
            assert got == 0.0, f"{y} emitted although the target forbids it"
    assert abs(total - 1.0) < 1e-6
    assert worst < 1e-6, f"max |law - target| = {worst}"
