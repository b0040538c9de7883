"""The whole step under HIP graph capture: score -> stop -> restart -> OPD gradient captured once
and replayed.  The library allocates, synchronises and memsets nothing, so the captured graph
is the same launches; every replay must equal an eager run bit for bit (all reductions run in
a fixed order), including after the inputs are changed in place between replays, with eager
work and synchronisations between the replays.
"""
import sys

import numpy as np
import pytest

from synth import workloads as W
from tests import harness as H

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available()
    yield
    torch.cuda.synchronize()


OUT = ("logp_t", "logp_s", "kl", "turn_mean", "cum", "stop_unit", "retained", "k_star", "k0",
       "k_max", "flags")


def _snapshot(path, grad, loss):
    h = path.host()
    snap = {k: np.array(h[k]) for k in OUT}
    snap["grad"] = grad.float().cpu().numpy()
    snap["loss"] = loss.cpu().numpy()
    return snap


def _equal(a, b):
    for k in a:
        assert np.array_equal(a[k], b[k], equal_nan=True), k


def test_graph_replay_equals_eager():
    import torch
    import paper_2609_14636_amd as P
    wl = W.make("agentic", seed=1011, scale=dict(R=4, turns=6, tok_lo=40, tok_hi=200, vocab=8192))
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = H.thresholds(wl, sc)
    inp = H.device_inputs(wl)
    ids = inp["ids"]

    def step(path, grad, loss):
        path.run(wl.vocab, inp["teachers"], inp["student"], ids, lam, alpha,
                 start_unit=inp["start"], correct_mask=inp["mask"])
        path.grad(wl.vocab, inp["student"], ids, grad, loss, start_unit=inp["start"],
                  scale=1.0 / wl.n_tokens)

    eager = P.Path(inp["layout"], wl.unit)
    ge, le = torch.empty_like(inp["student"]), torch.empty(wl.n_tokens, device="cuda")
    graphed = P.Path(inp["layout"], wl.unit)
    gg, lg = torch.empty_like(inp["student"]), torch.empty(wl.n_tokens, device="cuda")

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(graphed, gg, lg)  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(graphed, gg, lg)
    torch.cuda.synchronize()

    gen = np.random.default_rng(5)
    for rep in range(4):
        if rep == 3:  # new sampled tokens in place: the graph reads the buffers as they are now
            ids.copy_(torch.from_numpy(gen.integers(0, wl.vocab, size=wl.n_tokens).astype(np.int32)))
        step(eager, ge, le)
        torch.cuda.synchronize()
        want = _snapshot(eager, ge, le)
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(graphed, gg, lg)
        _equal(got, want)
        assert int(got["flags"]) == 0
    say(f"[graph] 4 replays equal to eager; stops {want['stop_unit'].tolist()}")


def test_graph_replay_fused_equals_eager():
    import torch
    import paper_2609_14636_amd as P
    wl = W.make("fused", seed=21, scale=dict(R=2, turns=2, tok=96, vocab=3000, d=256))
    inp = H.device_inputs_fused(wl)

    def step(path):
        path.score_fused(wl.vocab, inp["hidden"], inp["w"], inp["student"], inp["ids"])
        path.stop([-1e30])
        path.restart([-float("inf")])

    eager = P.Path(inp["layout"], wl.unit, fused_vocab=wl.vocab)
    graphed = P.Path(inp["layout"], wl.unit, fused_vocab=wl.vocab)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(graphed)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(graphed)
    torch.cuda.synchronize()
    for rep in range(3):
        step(eager)
        torch.cuda.synchronize()
        want = {k: np.array(v) for k, v in eager.host().items() if v is not None}
        g.replay()
        torch.cuda.synchronize()
        got = {k: np.array(v) for k, v in graphed.host().items() if v is not None}
        for k in want:
            assert np.array_equal(got[k], want[k], equal_nan=True), k
    say("[graph fused] 3 replays equal to eager")


def test_graph_replay_of_the_allocation_free_stop_test():
    """stride_stop_noalloc, the entry point for callers that cannot allocate, captured in a HIP
    graph: every replay equals stride_stop with a caller workspace on the same inputs bit for bit,
    with eager calls between the replays that leave other contents in the shared fixed scratch
    (a smaller layout through stride_stop_noalloc itself) and the values changed in place."""
    import torch
    import paper_2609_14636_amd as P

    g = np.random.default_rng(77)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731

    def layout(sizes):
        R = len(sizes)
        rto = np.arange(R + 1, dtype=np.int32)          # one turn per rollout, token units
        tto = np.zeros(R + 1, np.int64)
        tto[1:] = np.cumsum(sizes)
        return rto, tto

    sizes = np.concatenate([g.integers(1, 3000, size=40), [70000, 2048, 2049]])
    rto, tto = layout(sizes)
    N, R = int(tto[-1]), sizes.size
    dom = g.integers(0, 2, size=R).astype(np.int32)
    lay = P.Layout(dev(rto), dev(tto), N, dev(dom))
    vals = dev((-np.abs(g.normal(0.5, 0.5, size=N))).astype(np.float32))
    start = dev((g.random(R) * sizes * 0.3).astype(np.int32))
    lam = [-150.0, -900.0]
    # a second, smaller layout whose eager calls overwrite the fixed scratch between replays
    sizes2 = g.integers(1, 5000, size=9)
    rto2, tto2 = layout(sizes2)
    lay2 = P.Layout(dev(rto2), dev(tto2), int(tto2[-1]), None)
    vals2 = dev((-np.abs(g.normal(0.3, 0.2, size=int(tto2[-1])))).astype(np.float32))

    def outs(n_units, n_roll):
        return (torch.empty(n_units, dtype=torch.float64, device="cuda"),
                torch.empty(n_roll, dtype=torch.int32, device="cuda"),
                torch.empty(n_roll, dtype=torch.int64, device="cuda"),
                torch.zeros(1, dtype=torch.int32, device="cuda"))

    got, want, other = outs(N, R), outs(N, R), outs(int(tto2[-1]), sizes2.size)
    ws = torch.empty(P.stride_workspace_size(lay, P.STRIDE_UNIT_TOKEN), dtype=torch.uint8, device="cuda")

    def captured():
        P.stride_stop_noalloc(lay, P.STRIDE_UNIT_TOKEN, vals, lam, start, *got)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        captured()  # first call on the device looks up the scratch address, outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        captured()
    torch.cuda.synchronize()

    for rep in range(4):
        if rep == 2:
            vals.mul_(1.5)  # the graph reads the values as they are now
        P.stride_stop_noalloc(lay2, P.STRIDE_UNIT_TOKEN, vals2, [-40.0], None, *other)
        P.stride_stop(lay, P.STRIDE_UNIT_TOKEN, vals, lam, start, *want, ws)
        torch.cuda.synchronize()
        for t in got[:3]:
            t.fill_(-7)
        got[3].zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert int(want[3].item()) == 0 and int(got[3].item()) == 0
        assert np.array_equal(got[0].cpu().numpy().view(np.uint64), want[0].cpu().numpy().view(np.uint64))
        assert np.array_equal(got[1].cpu().numpy(), want[1].cpu().numpy())
        assert np.array_equal(got[2].cpu().numpy(), want[2].cpu().numpy())
    stops = int((want[1] >= 0).sum().item())
    assert 0 < stops < R
    say(f"[graph noalloc] 4 replays equal to stride_stop; {stops}/{R} stops")


def test_two_workloads_on_two_streams_equal_sequential_runs():
    """The calls are asynchronous on the caller's stream and share no state: two different
    workloads (turn units with a prefix offset and a correctness mask, and token units), each
    with its own workspace, launched alternately on two non-default streams so that their kernels
    may overlap, give bit for bit what they give run one after the other on the default stream."""
    import torch
    import paper_2609_14636_amd as P

    w1 = W.make("agentic", seed=3031, scale=dict(R=5, turns=6, tok_lo=40, tok_hi=300, vocab=6000))
    w2 = W.make("reasoning", seed=3032, scale=dict(R=3, tok=5000, vocab=7000))
    runs = []
    for wl in (w1, w2):
        sc = H.oracle_scores(wl, range(wl.n_rollouts), with_student=False)
        lam, alpha = H.thresholds(wl, sc)
        runs.append((wl, lam, alpha, H.device_inputs(wl)))

    def go(path, r, stream):
        wl, lam, alpha, inp = r
        path.run(wl.vocab, inp["teachers"], inp["student"], inp["ids"], lam, alpha,
                 start_unit=inp["start"], correct_mask=inp["mask"], stream=stream)

    seq = [P.Path(r[3]["layout"], r[0].unit) for r in runs]
    for p, r in zip(seq, runs):
        go(p, r, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    want = [{k: np.array(v) for k, v in p.host().items() if v is not None} for p in seq]

    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    conc = [P.Path(r[3]["layout"], r[0].unit) for r in runs]
    torch.cuda.synchronize()
    for rep in range(3):
        for p, r, s in zip(conc, runs, streams):
            go(p, r, s.cuda_stream)
        torch.cuda.synchronize()
        for p, wnt in zip(conc, want):
            got = {k: np.array(v) for k, v in p.host().items() if v is not None}
            for k in wnt:
                assert np.array_equal(got[k], wnt[k], equal_nan=True), (rep, k)
    assert int(want[0]["flags"]) == 0 and int(want[1]["flags"]) == 0
    say(f"[two streams] 3 concurrent runs equal to sequential; stops {want[0]['stop_unit'].tolist()} "
        f"and {want[1]['stop_unit'].tolist()}")


def test_two_host_threads_each_on_its_own_stream():
    """Thread safety of the entry points: two host threads drive two workloads through the
    library at the same time (ctypes releases the interpreter lock during each call), each on its
    own stream with its own workspace; every run equals the sequential one bit for bit."""
    import threading

    import torch
    import paper_2609_14636_amd as P

    w1 = W.make("multi", seed=3041, scale=dict(R=6, turns=3, tok=200, vocab=5000))
    w2 = W.make("agentic", seed=3042, scale=dict(R=4, turns=5, tok_lo=30, tok_hi=250, vocab=4096))
    runs = []
    for wl in (w1, w2):
        sc = H.oracle_scores(wl, range(wl.n_rollouts), with_student=False)
        lam, alpha = H.thresholds(wl, sc)
        runs.append((wl, lam, alpha, H.device_inputs(wl)))

    def go(path, r, stream):
        wl, lam, alpha, inp = r
        path.run(wl.vocab, inp["teachers"], inp["student"], inp["ids"], lam, alpha,
                 start_unit=inp["start"], correct_mask=inp["mask"], stream=stream)

    want = []
    for r in runs:
        p = P.Path(r[3]["layout"], r[0].unit)
        go(p, r, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        want.append({k: np.array(v) for k, v in p.host().items() if v is not None})

    paths = [P.Path(r[3]["layout"], r[0].unit) for r in runs]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    errors = []

    def worker(i):
        try:
            torch.cuda.set_device(0)
            for _ in range(5):
                go(paths[i], runs[i], streams[i].cuda_stream)
                streams[i].synchronize()
                got = {k: np.array(v) for k, v in paths[i].host().items() if v is not None}
                for k in want[i]:
                    if not np.array_equal(got[k], want[i][k], equal_nan=True):
                        errors.append((i, k))
                        return
        except Exception as e:  # noqa: BLE001  (reported below)
            errors.append((i, repr(e)))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads)
    assert not errors, errors
    say("[two threads] 5 runs per thread equal to sequential")
