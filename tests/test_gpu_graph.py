"""Graph-replayed verification (sd_verify_batch_graph) against the eager
path, through the C ABI.

The graph path must give bit-identical logits and decisions to
sd_verify_batch: on every replay of an unchanged batch (with eager work and
synchronisations of the program between replays), on several batches in
flight on alternating streams (the pipelined workload's launch pattern), and
across committed rounds, where each round's new prefix lengths force a
re-capture.  The eager path itself is checked against the oracle by the other
GPU tests; one oracle comparison here pins the graph path directly."""
import numpy as np
import pytest
import torch

import workload as wl
from gpu_harness import assert_decisions, compare_decisions, load_synthetic_kv, logit_rel_err, make_verifier, run_oracle
from workload.device import DeviceWeights, batch_to_device

pytestmark = pytest.mark.gpu


def _pass(v, w, n, b, dev, mode, stream, graph, seed=5, round_=0, commit=False):
    d, q, au = dev
    v.verify(n, w.assign, w.draft_len, d, q, mode, seed, round_, au, stream=stream, graph=graph)
    lg = v.logits(n, b.T, stream=stream)
    n_acc, tok = v.accept(n, w.n_users, commit)
    torch.cuda.synchronize()
    return n_acc[b.users].copy(), tok[b.users].copy(), lg.cpu().numpy()


def _setup(prefix, draft, assign, seed, model="tiny-bf16"):
    w = wl.custom_workload(model, prefix, draft, seed=seed, assign=assign)
    dw = DeviceWeights(w.model, w.seed)
    v = make_verifier(w, dw, max_pending=max(2, w.n_batches), extra_ctx=64)
    load_synthetic_kv(v, w)
    batches = [w.batch(n) for n in range(w.n_batches)]
    for b in batches:
        for i, u in enumerate(b.users):
            v.reset_user(int(u), int(b.prefix_len[i]), int(b.root[i]))
    return w, dw, v, batches


@pytest.mark.parametrize("mode", ["stochastic", "greedy"])
def test_graph_replays_match_eager(mode):
    w, dw, v, (b,) = _setup([40, 300, 0, 17, 129], [1, 7, 3, 5, 2], None, 7)
    dev = batch_to_device(b)
    st = torch.cuda.Stream()
    ref = _pass(v, w, 0, b, dev, mode, st, graph=False)
    scratch = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        got = _pass(v, w, 0, b, dev, mode, st, graph=True)
        assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1]), rep
        assert np.array_equal(got[2], ref[2]), f"replay {rep}: logits differ"
        # the program's own eager work between replays
        scratch.mul_(1.0001).add_(0.5)
        eager = _pass(v, w, 0, b, dev, mode, st, graph=False)
        assert np.array_equal(eager[2], ref[2])
        torch.cuda.synchronize()
    # the graph path against the oracle (logits within the bf16 bar, decisions exact
    # outside the window the logit error admits)
    rl, oref = run_oracle(w, b, mode, seed=5)
    err = float(logit_rel_err(ref[2], rl).max())
    assert err < 2e-2, err
    assert_decisions(compare_decisions(ref[0], ref[1], oref, b.draft_len, mode, b.drafts, ref[2], rl),
                     f"graph pass/{mode}", end_to_end=True)
    v.close()


def test_graph_replays_of_the_split_gate_up_product():
    """At 240 slots the 20480-wide gate/up product of the wide-FFN toy model
    is split over one workgroup per CU with per-tile counters that every
    launch must leave at zero; replays of the captured pass (eager passes and
    other work between them) stay bit-identical to the eager pass."""
    prefix = [int(x) for x in np.random.default_rng(3).integers(0, 400, 20)]
    w, dw, v, (b,) = _setup(prefix, [11] * 20, None, 9, model="tiny-wide-ffn")
    assert b.T == 240
    dev = batch_to_device(b)
    st = torch.cuda.Stream()
    ref = _pass(v, w, 0, b, dev, "stochastic", st, graph=False)
    scratch = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        got = _pass(v, w, 0, b, dev, "stochastic", st, graph=True)
        assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1]), rep
        assert np.array_equal(got[2], ref[2]), f"replay {rep}: logits differ"
        scratch.mul_(1.0001).add_(0.5)
        eager = _pass(v, w, 0, b, dev, "stochastic", st, graph=False)
        assert np.array_equal(eager[2], ref[2])
    v.close()


def test_graph_batches_on_alternating_streams():
    """Four batches in flight at once on two streams, each replayed from its
    own slot's graph, as the pipelined workload runs them."""
    prefix = [33, 70, 5, 140, 64, 16, 90, 1]
    draft = [2, 4, 1, 3, 5, 2, 1, 4]
    assign = [0, 1, 2, 3, 3, 2, 1, 0]
    w, dw, v, batches = _setup(prefix, draft, assign, 19)
    devs = [batch_to_device(b) for b in batches]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    refs = [_pass(v, w, n, b, devs[n], "stochastic", streams[n % 2], graph=False)
            for n, b in enumerate(batches)]
    for rep in range(3):
        for n in range(w.n_batches):
            d, q, au = devs[n]
            v.verify(n, w.assign, w.draft_len, d, q, "stochastic", 5, 0, au,
                     stream=streams[n % 2], graph=True)
        for n, b in enumerate(batches):
            lgt = v.logits(n, b.T, stream=streams[n % 2])
            n_acc, tok = v.accept(n, w.n_users)
            torch.cuda.synchronize()
            lg = lgt.cpu().numpy()
            assert np.array_equal(n_acc[b.users], refs[n][0]) and np.array_equal(tok[b.users], refs[n][1])
            assert np.array_equal(lg, refs[n][2]), (rep, n)
    v.close()


@pytest.mark.parametrize("graph", [False, True])
def test_split_gate_up_batches_on_two_streams(graph):
    """Two 240-slot batches of the wide-FFN toy model in flight at once on
    two streams (each pass's split gate/up product uses its own slot's tile
    counters, and its waits end while the other pass shares the CUs), three
    times over, eagerly or from graphs; every pass equals the batch's pass
    run alone."""
    prefix = [int(x) for x in np.random.default_rng(4).integers(0, 400, 40)]
    assign = [i % 2 for i in range(40)]
    w, dw, v, batches = _setup(prefix, [11] * 40, assign, 23, model="tiny-wide-ffn")
    assert [b.T for b in batches] == [240, 240]
    devs = [batch_to_device(b) for b in batches]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    refs = [_pass(v, w, n, b, devs[n], "stochastic", streams[0], graph=False) for n, b in enumerate(batches)]
    for rep in range(3):
        for n in range(2):
            d, q, au = devs[n]
            v.verify(n, w.assign, w.draft_len, d, q, "stochastic", 5, 0, au, stream=streams[n], graph=graph)
        for n, b in enumerate(batches):
            lgt = v.logits(n, b.T, stream=streams[n])
            n_acc, tok = v.accept(n, w.n_users)
            torch.cuda.synchronize()
            assert np.array_equal(n_acc[b.users], refs[n][0]) and np.array_equal(tok[b.users], refs[n][1])
            assert np.array_equal(lgt.cpu().numpy(), refs[n][2]), (rep, n)
    v.close()


def test_graph_recaptures_across_committed_rounds():
    """Two verifiers with identical state, one eager and one on graphs, run
    three committed rounds; every round changes i_m (so the graph is
    re-captured) and the two must agree bit for bit, including the
    committed user state."""
    prefix, draft = [20, 75, 3], [3, 2, 4]
    w, dw, ve, (b,) = _setup(prefix, draft, None, 23)
    vg = make_verifier(w, dw, max_pending=2, extra_ctx=64)
    load_synthetic_kv(vg, w)
    for i, u in enumerate(b.users):
        vg.reset_user(int(u), int(b.prefix_len[i]), int(b.root[i]))
    st = torch.cuda.Stream()
    dev = batch_to_device(b)
    for rnd in range(3):
        e = _pass(ve, w, 0, b, dev, "stochastic", st, graph=False, round_=rnd, commit=True)
        g = _pass(vg, w, 0, b, dev, "stochastic", st, graph=True, round_=rnd, commit=True)
        assert np.array_equal(e[0], g[0]) and np.array_equal(e[1], g[1]), rnd
        assert np.array_equal(e[2], g[2]), rnd
        for u in b.users:
            assert ve.user_state(int(u)) == vg.user_state(int(u))
    ve.close()
    vg.close()


def test_graph_rejects_null_stream():
    from paper_2604_20919_amd import sdverify as sv
    w, dw, v, (b,) = _setup([10, 12], [1, 2], None, 3)
    d, q, au = batch_to_device(b)
    with pytest.raises(sv.SdError) as ei:
        v.verify(0, w.assign, w.draft_len, d, q, "stochastic", 0, 0, au, stream=None, graph=True)
    assert ei.value.status == sv.SD_EINVAL
    # nothing is pending: the eager path still works on the same slot
    v.verify(0, w.assign, w.draft_len, d, q, "stochastic", 0, 0, au)
    v.accept(0, w.n_users)
    v.close()
