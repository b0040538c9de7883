"""Fused projection + log-sum-exp path (stride_score_fused) against the float64 oracle.

The oracle forms z = h W in binary64 from the host-generated bf16 operands (it takes
W as [d, V]; the GPU reads the same values stored as a linear layer's [V, d] weight)
and never sees a GPU value.  Small shapes are compared on every row, including
partial row and vocabulary tiles; the full-size workload on sampled rows and on one
complete turn.
"""
import math
import sys

import numpy as np
import pytest

from synth import workloads as W
from tests import harness as H
from tests import workload_params as WP

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
    torch.cuda.empty_cache()


def _per_rollout(wl, sc):
    out = {}
    for r in range(wl.n_rollouts):
        a, b = wl.rollout_rows(r)
        out[r] = {k: sc[k][a:b] for k in ("logp_t", "logp_s", "kl")}
    return out


@pytest.mark.parametrize("R,turns,tok,vocab,d", [
    (2, 2, 64, 1000, 128),      # vocabulary tile partly filled, one row tile
    (1, 3, 100, 4097, 192),     # 300 rows: a partial row tile; V not a multiple of 128
    (2, 2, 150, 257, 64),       # one K block; last 128-column partial has one column
    (1, 2, 40, 100, 64),        # V < 128: one partial 128-column, the tile's other half empty
    (1, 2, 1, 300, 64),         # two rows in all: one row tile with 254 rows past N
    (1, 2, 33, 256, 320),       # V one whole tile; five K stages, a whole turn of the LDS ring
    (2, 2, 24, 151936, 2048),   # the full hidden size and vocabulary on 96 rows
    (1, 2, 16, 1048581, 64),    # 2^20 + 5 entries: 4,097 vocabulary tiles, 8,193 partials per row
    (1, 2, 5, 1, 128),          # a single vocabulary entry: every log-probability is 0
    (2, 2, 1049, 3000, 128),    # 4,196 rows = 17 row tiles: 16-tile super-rows, the second holding
                                # one ragged tile
    (1, 2, 1152, 700, 64),      # 9 row tiles: 8-tile super-rows, the second holding one
])
def test_fused_parity(R, turns, tok, vocab, d):
    wl = W.make("fused", seed=3 + vocab, scale=dict(R=R, turns=turns, tok=tok, vocab=vocab, d=d))
    say(f"[fused] N={wl.n_tokens} V={vocab} d={d}")
    say(f"[fused] {_fused_vs_oracle(wl)}")


def test_fused_random_shapes():
    """Thirty random small shapes against the oracle: 1 to 1,200 rows (partial row tiles),
    vocabularies of 1 to 5,000 entries (partial 128- and 256-column tiles) and hidden sizes of one
    to eight K stages."""
    g = np.random.default_rng(31337)
    for case in range(30):
        R, turns = int(g.integers(1, 4)), int(g.integers(1, 5))
        if R * turns < 2:  # the threshold needs two turns
            turns = 2
        tok = int(g.integers(1, 101))
        vocab = int(g.choice([1, 2, 127, 128, 129, 255, 256, 257])) if g.random() < 0.5 \
            else int(g.integers(3, 5001))
        d = 64 * int(g.integers(1, 9))
        wl = W.make("fused", seed=900 + case,
                    scale=dict(R=R, turns=turns, tok=tok, vocab=vocab, d=d))
        rep = _fused_vs_oracle(wl)
        if case % 10 == 9:
            say(f"[fused random] case {case}: N={wl.n_tokens} V={vocab} d={d}; {rep}")


def _fused_vs_oracle(wl):
    """Every row of a small fused workload, its turn means, stops and restart picks against the
    oracle."""
    sc, _ = H.oracle_fused_scores(wl, np.arange(wl.n_tokens))
    assert sc["flags"] == 0
    per = _per_rollout(wl, sc)
    tm, _ = H.OP.O.turn_mean(wl.turn_tok_off, sc["logp_t"])
    c = WP.pooled_cum(wl.unit_off(), tm)
    lam, alpha = [WP.midpoint_quantile(c, 0.5)], [-math.inf]
    ora = {r: (per[r], H.oracle_rollout(wl, r, per[r], lam, alpha)) for r in per}
    gpu = H.run_gpu_fused(wl, lam, alpha)
    assert gpu["flags"] == 0, hex(gpu["flags"])
    rep = H.compare(wl, gpu, ora, lam, alpha)
    H.assert_invariants(gpu, wl)
    return rep


def test_fused_full_size():
    """The fused workload at full size (65,536 rows, d = 2048, V = 151,936): one whole rollout
    (4,096 rows, 8 turns) against the oracle -- every row's log-probabilities and KL, its turn
    means, cumulative sums, stop, k*, K0 and K_max -- plus scattered rows of other rollouts and
    tiles, and properties that hold for every rollout."""
    import time
    wl = W.make("fused", 1001)
    lam, alpha = WP.fused_thresholds(wl.vocab, wl.fused_d, wl.hidden_sigma, wl.w_sigma)
    gpu = H.run_gpu_fused(wl, lam, alpha)
    assert gpu["flags"] == 0, hex(gpu["flags"])
    H.assert_invariants(gpu, wl)
    t0 = time.time()
    w_dv = wl.w_dv_host(16)
    r = 3
    a, b = wl.rollout_rows(r)
    sc, _ = H.oracle_fused_scores(wl, np.arange(a, b), w_dv=w_dv, matmul=True)
    assert sc["flags"] == 0
    say(f"[fused full] oracle on rollout {r} ({b - a} rows): {time.time() - t0:.1f} s")
    ora = {r: (sc, H.oracle_rollout(wl, r, sc, lam, alpha))}
    rep = H.compare(wl, gpu, ora, lam, alpha)
    say(f"[fused full] rollout {r}: {rep}")
    assert rep.stop_excused == 0 and rep.restart_excused == 0
    # scattered rows of other rollouts and tiles (the first and last rows, tile edges)
    extra = np.array([0, 1, 255, 256, 4095, 32768, wl.n_tokens - 1])
    sx, _ = H.oracle_fused_scores(wl, extra, w_dv=w_dv)
    for k in ("logp_t", "logp_s"):
        d = np.max(np.abs(gpu[k][extra] - sx[k]))
        assert d <= H.TOL_LOGP, (k, d)
    d = np.max(np.abs(gpu["kl"][extra] - sx["kl"]))
    assert d <= H.TOL_KL, d
    # every turn mean sits near the closed form -(log V + d s_h^2 s_W^2 / 2), and lambda is
    # 5.5 times that value, so every rollout stops on its sixth turn (index 5)
    expect = lam[0] / 5.5
    assert np.all(np.abs(gpu["turn_mean"] - expect) < 0.5), (gpu["turn_mean"].min(), expect)
    assert gpu["stop_unit"].tolist() == [5] * wl.n_rollouts, gpu["stop_unit"]
    assert gpu["k_max"].tolist() == [6] * wl.n_rollouts


def test_fused_partial_band():
    """Bands of super-rows walked one super-column at a time, with a partial last band: 8,300 rows
    are 33 row tiles, three 16-tile super-rows; at d = 8,192 a super-row holds 64 MiB of h, so a
    band is two super-rows and the third forms a band of its own; V = 4,200 is 17 vocabulary tiles,
    two super-columns.  The partial table is filled with NaN before the call, so a tile the grid
    skipped or visited twice shows in the rows it covers.  The first and last row of every row
    tile, each over the whole vocabulary, against the oracle."""
    import torch
    import paper_2609_14636_amd as P
    wl = W.make("fused", seed=77, scale=dict(R=1, turns=2, tok=4150, vocab=4200, d=8192))
    assert wl.n_tokens == 8300
    inp = H.device_inputs_fused(wl)
    path = P.Path(inp["layout"], wl.unit, with_student=True, fused_vocab=wl.vocab)
    path.fused_ws.fill_(0xFF)
    path.score_fused(wl.vocab, inp["hidden"], inp["w"], inp["student"], inp["ids"])
    torch.cuda.synchronize()
    gpu = path.host()
    assert gpu["flags"] == 0, hex(gpu["flags"])
    rows = np.unique(np.minimum(np.concatenate([np.arange(0, wl.n_tokens, 256),
                                                np.arange(255, wl.n_tokens + 255, 256)]),
                                wl.n_tokens - 1))
    sc, _ = H.oracle_fused_scores(wl, rows)
    assert sc["flags"] == 0
    for k in ("logp_t", "logp_s"):
        dmax = np.max(np.abs(gpu[k][rows] - sc[k]))
        assert dmax <= H.TOL_LOGP, (k, dmax)
    say(f"[fused band] {rows.size} rows: max |dlogp_t| = "
        f"{np.max(np.abs(gpu['logp_t'][rows] - sc['logp_t'])):.2e}")


def test_fused_band_order_changes_no_bit():
    """The band of super-rows only orders the tiles: through libstride_debug.so, bands of 1, 2
    (the library's choice at d = 8,192) and 3 super-rows give the same log-probabilities, KL and
    turn means bit for bit, on the partial-band layout (three super-rows, two super-columns)."""
    import torch
    import paper_2609_14636_amd as P
    assert P.library().stride_debug_fused_band(1) == 2  # the product library has no hook
    dbg = P.stride.debug_library()
    wl = W.make("fused", seed=78, scale=dict(R=1, turns=2, tok=4150, vocab=4200, d=8192))
    inp = H.device_inputs_fused(wl)
    path = P.Path(inp["layout"], wl.unit, with_student=True, fused_vocab=wl.vocab)
    out = {}
    try:
        for band in (0, 1, 3):
            assert dbg.stride_debug_fused_band(band) == 0
            path.fused_ws.fill_(0xFF)
            P.stride.stride_score_fused(inp["layout"], wl.vocab, inp["hidden"], inp["w"],
                                        inp["student"], inp["ids"], path.logp_t, path.logp_s,
                                        path.kl, path.turn_mean, path.flags, path.fused_ws,
                                        lib=dbg)
            torch.cuda.synchronize()
            out[band] = {k: getattr(path, k).clone() for k in ("logp_t", "logp_s", "kl", "turn_mean")}
            assert int(path.flags.item()) == 0
    finally:
        dbg.stride_debug_fused_band(0)
    bits = {torch.float32: torch.int32, torch.float64: torch.int64}
    for band in (1, 3):
        for k, v in out[band].items():
            assert torch.equal(v.view(bits[v.dtype]), out[0][k].view(bits[v.dtype])), (band, k)
    say("[fused band] bands 1, 2 and 3: every output equal bit for bit")
