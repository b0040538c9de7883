"""GPU path against the float64 oracle, element by element (needs an MI355X).

Reduced copies of every workload run the oracle on all rollouts; full-size
workloads compare sampled rollouts one by one and check size-independent
properties everywhere.  Every call goes through the C ABI of libstride.so.
"""
import math
import os
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


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_14636_amd  # noqa: F401  (fails loudly without libstride.so)
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _parity(wl, rollouts=None, with_student=True, lam=None, alpha=None):
    say(f"[parity] {wl.name} R={wl.n_rollouts} T={wl.n_turns} N={wl.n_tokens} V={wl.vocab} "
        f"ld={wl.ld} dtype={'bf16' if wl.dtype == W.BF16 else 'f32'} unit={wl.unit}")
    sc = H.oracle_scores(wl, range(wl.n_rollouts) if rollouts is None else rollouts,
                         with_student=with_student)
    if lam is None:
        lam, alpha = H.thresholds(wl, sc)
    ora = {r: (sc[r], H.oracle_rollout(wl, r, sc[r], lam, alpha)) for r in sc}
    gpu = H.run_gpu(wl, lam, alpha, with_student=with_student)
    rep = H.compare(wl, gpu, ora, lam, alpha)
    H.assert_invariants(gpu, wl)
    say(f"[parity] {wl.name}: {rep}")
    return gpu, ora, lam, alpha, rep


# ---------------------------------------------------------------- the generator itself

@pytest.mark.parametrize("name,scale", [("tiny", None),
                                        ("agentic", dict(R=1, turns=2, tok_lo=3, tok_hi=9))])
def test_generator_device_matches_host(name, scale):
    import torch
    wl = W.make(name, seed=7, scale=scale)
    inp = H.device_inputs(wl)
    torch.cuda.synchronize()
    t_host = wl.teacher_rows_host(0, wl.n_tokens)
    s_host = wl.student_rows_host(0, wl.n_tokens)
    view = torch.uint16 if wl.dtype == W.BF16 else torch.float32
    t_dev = inp["teachers"][0].view(torch.int16 if view == torch.uint16 else view).cpu().numpy()
    s_dev = inp["student"].view(torch.int16 if view == torch.uint16 else view).cpu().numpy()
    v = wl.vocab
    assert np.array_equal(t_dev[:, :v].view(t_host.dtype), t_host[:, :v])
    assert np.array_equal(s_dev[:, :v].view(s_host.dtype), s_host[:, :v])


# ---------------------------------------------------------------- the five workloads, reduced

def test_tiny_parity_and_planted_structure():
    wl = W.make("tiny")
    gpu, ora, lam, alpha, rep = _parity(wl)
    # Planted error turn 1 of rollout 0: exactly one stop, on that turn (Eq. 5); it is the first
    # non-correct turn there (Sec. 4.2 step 1), so K_max = 1 and k* = turn 0; rollout 1 runs out.
    assert gpu["stop_unit"].tolist() == [1, -1]
    assert gpu["k_max"].tolist()[0] == 1 and gpu["k_star"].tolist()[0] == 0
    assert gpu["k_max"].tolist()[1] == 3
    assert gpu["k_star"][1] == int(np.argmin(gpu["turn_mean"][3:6]))
    assert rep.stop_excused == 0 and rep.restart_excused == 0


def test_agentic_reduced_parity():
    _parity(W.make("agentic", seed=1002, scale=dict(R=2)))


def test_reasoning_reduced_parity():
    _parity(W.make("reasoning", seed=1003, scale=dict(R=2, tok=4096)))


def test_multi_teacher_reduced_parity():
    wl = W.make("multi", seed=1004, scale=dict(R=4, turns=4, tok=384))
    assert set(wl.domain.tolist()) == {0, 1} or wl.n_rollouts < 2
    _parity(wl)


# ---------------------------------------------------------------- ragged shapes and small vocabularies

def _custom(seed, vocab, dtype, lengths, n_teachers=1, unit=W.UNIT_TURN, start=True, mask=True):
    g = np.random.default_rng(seed)
    rto, tto = W._layout_from_lengths(lengths)
    R, N = rto.size - 1, int(tto[-1])
    ld = vocab + (-vocab) % (8 if dtype == W.BF16 else 4)
    tok = g.integers(0, vocab, size=N).astype(np.int32)
    tb = (4.0 + g.standard_normal(N)).astype(np.float32)
    sb = (4.0 + g.standard_normal(N)).astype(np.float32)
    dom = g.integers(0, n_teachers, size=R).astype(np.int32) if n_teachers > 1 else None
    wl = W.Workload("custom", seed, vocab, ld, dtype, unit, rto, tto, dom, n_teachers, tok,
                    2.0, 2.0, tb, sb)
    n_units = wl.n_units()
    uoff = wl.unit_off()
    if start:
        wl.start = np.array([g.integers(0, max(1, uoff[r + 1] - uoff[r] + 1)) for r in range(R)],
                            np.int32)
    if mask:
        wl.mask = (g.random(n_units) < 0.9).astype(np.uint8)
    return wl


def _custom_thresholds(wl, sc):
    logp = np.concatenate([sc[r]["logp_t"] for r in range(wl.n_rollouts)])
    tm, _ = H.OP.O.turn_mean(wl.turn_tok_off, logp)
    vals = tm if wl.unit == W.UNIT_TURN else logp
    c = WP.pooled_cum(wl.unit_off(), vals)
    nd = wl.n_teachers
    lam = [WP.midpoint_quantile(c, 0.4 + 0.1 * d) for d in range(nd)]
    alpha = [WP.midpoint_quantile(vals, 0.2 + 0.05 * d) for d in range(nd)]
    return lam, alpha


@pytest.mark.parametrize("vocab", [1, 7, 513, 1024, 4097])
@pytest.mark.parametrize("dtype", [W.BF16, W.F32])
def test_small_vocab_ragged_parity(vocab, dtype):
    g = np.random.default_rng(vocab * 10 + dtype)
    lengths = [g.integers(1, 40, size=int(g.integers(0, 6))) for _ in range(7)]
    lengths[1] = np.array([], np.int64)  # an empty rollout
    lengths[2] = np.array([1, 1, 1])     # single-token turns
    wl = _custom(vocab + dtype, vocab, dtype, lengths, n_teachers=2)
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = _custom_thresholds(wl, sc)
    ora = {r: (sc[r], H.oracle_rollout(wl, r, sc[r], lam, alpha)) for r in sc}
    gpu = H.run_gpu(wl, lam, alpha)
    rep = H.compare(wl, gpu, ora, lam, alpha)
    say(f"[ragged V={vocab} dtype={dtype}] {rep}")


@pytest.mark.parametrize("vocab", [1, 7, 9])
@pytest.mark.parametrize("dtype", [W.BF16, W.F32])
def test_small_vocab_on_the_one_wavefront_kernel(vocab, dtype):
    """The small vocabularies above again, in a batch of 8,400 rows (16,800 row items), so the
    one-wavefront kernel's tail handling (a row shorter than one 16-byte word, or one word and a
    ragged tail) is compared with the oracle too."""
    g = np.random.default_rng(vocab * 100 + dtype)
    lengths = [g.integers(200, 500, size=3) for _ in range(7)]
    total = sum(int(l.sum()) for l in lengths)
    lengths.append(np.array([8400 - total]))
    wl = _custom(vocab * 10 + dtype + 7, vocab, dtype, lengths, n_teachers=2)
    assert 2 * wl.n_tokens >= 16384
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = _custom_thresholds(wl, sc)
    ora = {r: (sc[r], H.oracle_rollout(wl, r, sc[r], lam, alpha)) for r in sc}
    gpu = H.run_gpu(wl, lam, alpha)
    rep = H.compare(wl, gpu, ora, lam, alpha)
    say(f"[one-wavefront V={vocab} dtype={dtype}] N={wl.n_tokens} {rep}")


@pytest.mark.parametrize("unit", [W.UNIT_TURN, W.UNIT_TOKEN])
def test_ragged_many_rollouts_token_and_turn_units(unit):
    g = np.random.default_rng(5 + unit)
    lengths = [g.integers(1, 300, size=int(g.integers(1, 9))) for _ in range(40)]
    lengths[3] = np.array([], np.int64)
    wl = _custom(99 + unit, 2048, W.BF16, lengths, n_teachers=3, unit=unit)
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = _custom_thresholds(wl, sc)
    ora = {r: (sc[r], H.oracle_rollout(wl, r, sc[r], lam, alpha)) for r in sc}
    gpu = H.run_gpu(wl, lam, alpha)
    rep = H.compare(wl, gpu, ora, lam, alpha)
    say(f"[ragged many unit={unit}] {rep}")


def test_random_small_layouts():
    """Eighty random small batches, each through the whole path against the oracle: vocabularies
    of 1 to 3,000 entries in bf16 or fp32, one to three teachers, turn or token units, empty
    rollouts, single-token turns, K0 anywhere up to the rollout's end, with and without a mask;
    every other batch takes the paired pass with the exact KL."""
    g = np.random.default_rng(777)
    done = 0
    for case in range(80):
        vocab = int(g.choice([1, 2, 7, 8, 9, 63, 64, 65, 511, 512, 513, 3000]))
        dtype = int(g.choice([W.BF16, W.F32]))
        R = int(g.integers(1, 12))
        lengths = [g.integers(1, int(g.integers(2, 60)), size=int(g.integers(0, 6)))
                   for _ in range(R)]
        if sum(len(l) for l in lengths) < 2:  # the thresholds need two units
            lengths[0] = np.array([1, 1])
        unit = int(g.choice([W.UNIT_TURN, W.UNIT_TOKEN]))
        wl = _custom(5000 + case, vocab, dtype, lengths, n_teachers=int(g.integers(1, 4)),
                     unit=unit, start=bool(g.integers(0, 2)), mask=bool(g.integers(0, 2)))
        exact = case % 2 == 1
        sc = H.oracle_scores(wl, range(wl.n_rollouts), exact_kl=exact)
        lam, alpha = _custom_thresholds(wl, sc)
        ora = {r: (sc[r], H.oracle_rollout(wl, r, sc[r], lam, alpha)) for r in sc}
        gpu = H.run_gpu(wl, lam, alpha, exact_kl=exact)
        assert gpu["flags"] == 0, (case, hex(gpu["flags"]))
        rep = H.compare(wl, gpu, ora, lam, alpha)
        H.assert_invariants(gpu, wl)
        if exact:
            want = np.concatenate([sc[r]["kl_full"] for r in range(wl.n_rollouts)])
            assert np.max(np.abs(gpu["kl_full"] - want), initial=0.0) <= H.TOL_KL, case
        done += 1
        if case % 20 == 19:
            say(f"[random layouts] case {case}: R={R} N={wl.n_tokens} V={vocab} dtype={dtype} "
                f"unit={unit} teachers={wl.n_teachers}; {rep}")
    assert done == 80


# ---------------------------------------------------------------- data errors (forced from the host)

@pytest.mark.parametrize("pad", [0, 8200])
def test_data_error_flags(pad):
    """Non-finite rows and token ids out of range give NaN and flags; with pad, a third rollout of
    valid rows lifts the batch past 16,384 row items, so the one-wavefront kernel handles the same
    bad rows that the shared-row kernel handles without it."""
    import torch
    import paper_2609_14636_amd as P
    vocab = 64
    lengths = [np.array([4, 3]), np.array([5])] + ([np.array([pad])] if pad else [])
    wl = _custom(3, vocab, W.F32, lengths, start=False, mask=False)
    inp = H.device_inputs(wl)
    t = inp["teachers"][0]
    t[0, 5] = float("nan")            # row 0: NaN
    t[1, 0] = float("inf")            # row 1: +inf
    t[2, :] = float("-inf")           # row 2: all -inf
    t[3, 7] = float("-inf")           # row 3: one -inf entry (valid)
    ids = inp["ids"].clone()
    ids[4] = vocab                    # row 4: token id out of range
    ids[5] = -3                       # row 5: negative token id
    inp["ids"] = ids
    path = P.Path(inp["layout"], W.UNIT_TURN)
    path.run(vocab, inp["teachers"], inp["student"], ids, [-50.0], [-50.0])
    torch.cuda.synchronize()
    out = path.host()
    assert np.isnan(out["logp_t"][[0, 1, 2, 4, 5]]).all()
    assert np.isfinite(out["logp_t"][[3, 6, 7, 8]]).all()
    assert np.isnan(out["kl"][[0, 1, 2, 4, 5]]).all()
    assert out["flags"] & P.STRIDE_FLAG_NONFINITE and out["flags"] & P.STRIDE_FLAG_TOKEN_OOB
    with pytest.raises(P.StrideDataError, match="NONFINITE"):
        path.check()
    assert np.isnan(out["turn_mean"][0]) and np.isfinite(out["turn_mean"][2])
    # the oracle agrees on the valid row 3 (the -inf entry only removes mass)
    row3 = wl.teacher_rows_host(3, 1)
    row3[0, 7] = -np.inf
    lp, _, fl = H.OP.O.logp_rows(row3, wl.tok[3:4], vocab)
    assert fl == 0 and abs(lp[0] - out["logp_t"][3]) < H.TOL_LOGP


@pytest.mark.parametrize("pad", [0, 8200])
def test_empty_turn_and_bad_domain_flags(pad):
    """An empty turn and a rollout routed to a teacher that does not exist; with pad, a third
    rollout of valid rows moves the batch onto the one-wavefront kernel."""
    import torch
    import paper_2609_14636_amd as P
    rto = torch.tensor([0, 2, 3] + ([4] if pad else []), dtype=torch.int32, device="cuda")
    tto = torch.tensor([0, 4, 4, 6] + ([6 + pad] if pad else []), dtype=torch.int64,
                       device="cuda")                                   # turn 1 is empty
    dom = torch.tensor([0, 5] + ([0] if pad else []), dtype=torch.int32,
                       device="cuda")                                   # rollout 1: bad domain
    lay = P.Layout(rto, tto, 6 + pad, dom)
    x = torch.zeros((6 + pad, 8), dtype=torch.float32, device="cuda")
    ids = torch.zeros(6 + pad, dtype=torch.int32, device="cuda")
    path = P.Path(lay, W.UNIT_TURN)
    path.run(8, [x, x], x, ids, [-1.0, -1.0], [-5.0, -5.0])
    torch.cuda.synchronize()
    out = path.host()
    assert out["flags"] & P.STRIDE_FLAG_EMPTY_TURN and out["flags"] & P.STRIDE_FLAG_BAD_DOMAIN
    assert np.isnan(out["turn_mean"][1]) and abs(out["turn_mean"][0] + math.log(8)) < 1e-6
    assert np.isnan(out["logp_t"][4:6]).all()  # rows of the badly routed rollout
    if pad:  # the valid rollout is untouched: uniform rows give log(1/8) everywhere
        assert np.allclose(out["logp_t"][6:], -math.log(8), atol=1e-6)
    assert out["stop_unit"][1] == -1 and out["k_star"][1] == -1 and out["k0"][1] == 0


# ---------------------------------------------------------------- scan and restart at scale

def _stop_restart_vs_oracle(g, sizes, lam, alpha, tag):
    """Token-unit stop test and restart pick of one-turn rollouts of the given sizes against the
    oracle; the unit values, K0 offsets, domains and masks are host-made and given to both sides."""
    import torch
    import paper_2609_14636_amd as P
    R = sizes.size
    tto = np.zeros(R + 1, np.int64)
    tto[1:] = np.cumsum(sizes)
    rto = np.arange(R + 1, dtype=np.int32)  # one turn per rollout
    N = int(tto[-1])
    vals = (-np.abs(g.normal(0.5, 0.5, size=N))).astype(np.float32)
    vals[g.random(N) < 0.01] *= 20
    dom = g.integers(0, len(lam), size=R).astype(np.int32)
    start = (g.random(R) * sizes * 0.3).astype(np.int32)
    mask = (g.random(N) < 0.999).astype(np.uint8)
    say(f"[{tag}] R={R} N={N} max rollout {sizes.max()}")
    # oracle
    uoff = tto.copy()
    cum_o, stop_o, ret_o = H.OP.O.stop(uoff, vals.astype(np.float64), np.array(lam)[dom], start,
                                       np.arange(N + 1, dtype=np.int64))
    rec = np.where(stop_o >= 0, stop_o + 1, sizes).astype(np.int32)
    ks_o, k0_o, km_o = H.OP.O.restart(uoff, vals.astype(np.float64), rec, np.array(alpha)[dom], mask)
    # GPU
    dev = lambda a: torch.from_numpy(a).cuda()
    lay = P.Layout(dev(rto), dev(tto), N, dev(dom))
    v = dev(vals)
    ws = torch.empty(P.stride_workspace_size(lay, P.STRIDE_UNIT_TOKEN), dtype=torch.uint8, device="cuda")
    cum = torch.empty(N, dtype=torch.float64, device="cuda")
    stop = torch.empty(R, dtype=torch.int32, device="cuda")
    ret = torch.empty(R, dtype=torch.int64, device="cuda")
    ks = torch.empty(R, dtype=torch.int32, device="cuda")
    k0 = torch.empty_like(ks)
    km = torch.empty_like(ks)
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    P.stride_stop(lay, P.STRIDE_UNIT_TOKEN, v, lam, dev(start), cum, stop, ret, flags, ws)
    P.stride_restart_turn(lay, P.STRIDE_UNIT_TOKEN, v, stop, alpha, dev(mask), ks, k0, km, flags)
    torch.cuda.synchronize()
    assert int(flags.item()) == 0
    c = cum.cpu().numpy()
    rel = np.abs(c - cum_o) / np.maximum(np.abs(cum_o), 1.0)
    assert rel.max() <= H.TOL_CUM_REL, rel.max()
    s = stop.cpu().numpy()
    mism = np.nonzero(s != stop_o)[0]
    for r in mism:  # only inside the band
        a = tto[r]
        hi = sizes[r] if (s[r] < 0 or stop_o[r] < 0) else max(s[r], stop_o[r]) + 1
        assert np.any(np.abs(cum_o[a + start[r]:a + hi] - lam[dom[r]]) <= H.BAND), r
    same = s == stop_o
    assert np.array_equal(ret.cpu().numpy()[same], ret_o[same])
    ok = same
    assert np.array_equal(ks.cpu().numpy()[ok], ks_o[ok])
    assert np.array_equal(km.cpu().numpy()[ok], km_o[ok])
    assert np.array_equal(k0.cpu().numpy()[ok], k0_o[ok])
    say(f"[{tag}] max rel cum err {rel.max():.2e}, stops equal {same.sum()}/{R}, "
        f"stopped {int((s >= 0).sum())}, k* >= 0 {int((ks.cpu().numpy() >= 0).sum())}")
    return s


@pytest.mark.parametrize("seed", [0, 1])
def test_stop_and_restart_many_tiles(seed):
    """Token-unit scan over about a million units: rollouts from 1 to 300k units span many tiles, with K0 and
    per-domain lambda."""
    g = np.random.default_rng(seed)
    sizes = np.concatenate([g.integers(1, 50, size=200), [300000, 2047, 2048, 2049, 250000],
                            g.integers(1000, 40000, size=20)])
    g.shuffle(sizes)
    _stop_restart_vs_oracle(g, sizes, [-40.0, -400.0, -4000.0], [-0.9, -1.5, -np.inf], "scan")


def test_stop_and_restart_with_non_finite_and_extreme_thresholds():
    """lambda = +inf stops at the first unit counted, -inf and NaN never stop (the strict test is
    false), 0 and +-1e-300 sit at the edge of the sums' sign; alpha = +inf and NaN make no unit
    correct (K_max = 0, k* = -1), -inf makes every masked-in unit correct.  Exact against the
    oracle: no value lies within the band of these thresholds."""
    g = np.random.default_rng(77)
    sizes = g.integers(1, 60, size=3000)
    lam = [np.inf, -np.inf, np.nan, 0.0, -1e-300, 1e-300]
    alpha = [np.inf, -np.inf, np.nan, 0.0, -0.5, -1e300]
    s = _stop_restart_vs_oracle(g, sizes, lam, alpha, "extreme thresholds")
    assert (s >= 0).any() and (s < 0).any()


def test_stop_and_restart_a_million_short_rollouts():
    """One million rollouts of one to five units: hundreds of rollout starts in every scan tile,
    a restart launch of a million workgroups, and 64 domains of lambda and alpha."""
    g = np.random.default_rng(1000000)
    sizes = g.integers(1, 6, size=1000000)
    lam = list(-0.4 - 0.04 * np.arange(64))
    alpha = list(-0.3 - 0.01 * np.arange(64))
    s = _stop_restart_vs_oracle(g, sizes, lam, alpha, "short rollouts")
    assert 0 < int((s >= 0).sum()) < s.size


@pytest.mark.parametrize("n_rows,with_student", [(8191, True), (8192, True), (16383, False),
                                                  (16384, False)])
def test_either_side_of_the_shared_row_threshold(n_rows, with_student):
    """Batches of fewer than 16,384 row items (teacher plus student rows) share each row among the
    eight wavefronts of a workgroup; larger ones take one wavefront per row.  Both sides of the
    threshold against the oracle on every row, and the shared form run twice is bit-identical."""
    wl = W.make("reasoning", seed=17, scale=dict(R=1, tok=n_rows, vocab=4099))
    gpu, _, lam, alpha, _ = _parity(wl, with_student=with_student)
    items = n_rows * (2 if with_student else 1)
    if items < 16384:
        again = H.run_gpu(wl, lam, alpha, with_student=with_student)
        for k in ("logp_t", "logp_s", "kl", "turn_mean", "cum", "stop_unit", "k_star"):
            if gpu.get(k) is not None:
                assert np.array_equal(gpu[k].view(np.uint8), again[k].view(np.uint8)), k


@pytest.mark.parametrize("tok", [500, 1100])
def test_fp32_rows_either_side_of_the_shared_row_threshold(tok):
    """fp32 logits (the tiny workload's generator, V = 1024) with 2 rollouts x 4 turns x tok
    tokens: 8,000 row items run the shared-row kernel, 17,600 the one-wavefront kernel; every
    row against the oracle."""
    wl = W.make("tiny", seed=23, scale=dict(R=2, turns=4, tok=tok))
    assert wl.dtype == W.F32
    _parity(wl)


def test_determinism():
    import torch
    wl = W.make("reasoning", seed=5, scale=dict(R=3, tok=3000, vocab=4096))
    inp = H.device_inputs(wl)
    lam, alpha = [-15000.0], [-math.inf]
    a = H.run_gpu(wl, lam, alpha, inp=inp)
    b = H.run_gpu(wl, lam, alpha, inp=inp)
    for k in ("logp_t", "logp_s", "kl", "turn_mean", "cum", "stop_unit", "k_star", "k_max"):
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k
    torch.cuda.synchronize()
