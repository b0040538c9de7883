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
