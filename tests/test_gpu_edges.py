"""Edge cases on the GPU: an empty batch through every entry point, data errors in the fused
projection path, a fused hidden size past the full-size workload's, the largest teacher and
domain count, and a vocabulary of about a million entries.

The empty batch has nothing to compare; every call must succeed, raise no flag and write
nothing.  The fused error rows must come back NaN with the right flags while every other row
still matches the float64 oracle.
"""
import math
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


def test_empty_batch_every_entry_point():
    import torch
    import paper_2609_14636_amd as P
    dev = "cuda"
    lay = P.Layout(torch.zeros(1, dtype=torch.int32, device=dev),
                   torch.zeros(1, dtype=torch.int64, device=dev), 0)
    e = torch.empty(0, dtype=torch.float32, device=dev)
    x = torch.empty((0, 64), dtype=torch.bfloat16, device=dev)
    ids = torch.empty(0, dtype=torch.int32, device=dev)
    tm = torch.empty(0, dtype=torch.float64, device=dev)
    i32 = torch.empty(0, dtype=torch.int32, device=dev)
    flags = torch.zeros(1, dtype=torch.int32, device=dev)
    for unit in (P.STRIDE_UNIT_TURN, P.STRIDE_UNIT_TOKEN):
        ws = torch.empty(P.stride_workspace_size(lay, unit), dtype=torch.uint8, device=dev)
        vals = tm if unit == P.STRIDE_UNIT_TURN else e
        P.stride_score(lay, 64, [x], x, ids, e, e, e, tm, flags, ws, kl_full=e)
        P.stride_stop(lay, unit, vals, [-1.0], None, tm, i32, None, flags, ws)
        P.stride_restart_turn(lay, unit, vals, i32, [-1.0], None, i32, i32, i32, flags)
        P.stride_opd_grad(lay, unit, 64, x, ids, e, e, None, i32, 1.0, torch.empty_like(x), e,
                          flags, ws)
        P.stride_stop_step(i32, torch.zeros(1, dtype=torch.int64, device=dev), unit, vals, None,
                           [-1.0], tm, i32, i32, flags)
    fws = torch.empty(P.stride_fused_workspace_size(lay, 64), dtype=torch.uint8, device=dev)
    P.stride_score_fused(lay, 64, torch.empty((0, 64), dtype=torch.bfloat16, device=dev),
                         torch.empty((64, 64), dtype=torch.bfloat16, device=dev), x, ids, e, e, e,
                         tm, flags, fws)
    torch.cuda.synchronize()
    assert int(flags.item()) == 0


def test_fused_data_errors_flag_only_their_rows():
    import torch
    import paper_2609_14636_amd as P
    wl = W.make("fused", seed=77, scale=dict(R=1, turns=2, tok=48, vocab=1000, d=128))
    inp = H.device_inputs_fused(wl)
    ids = inp["ids"].clone()
    ids[3] = wl.vocab        # token id out of range
    ids[7] = -1              # negative token id
    hidden = inp["hidden"].clone()
    hidden[11, 5] = float("inf")   # non-finite hidden state
    N = wl.n_tokens
    lt = torch.empty(N, dtype=torch.float32, device="cuda")
    tm = torch.empty(wl.n_turns, dtype=torch.float64, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(P.stride_fused_workspace_size(inp["layout"], wl.vocab), dtype=torch.uint8,
                     device="cuda")
    P.stride_score_fused(inp["layout"], wl.vocab, hidden, inp["w"], None, ids, lt, None, None, tm,
                         flags, ws)
    torch.cuda.synchronize()
    f = int(flags.item())
    assert f & P.STRIDE_FLAG_TOKEN_OOB and f & P.STRIDE_FLAG_NONFINITE, hex(f)
    got = lt.cpu().numpy()
    bad = [3, 7, 11]
    assert np.isnan(got[bad]).all()
    good = np.setdiff1d(np.arange(N), bad)
    sc, _ = H.oracle_fused_scores(wl, good)
    assert sc["flags"] == 0
    d = np.max(np.abs(got[good] - sc["logp_t"]))
    assert d <= H.TOL_LOGP, d
    say(f"[fused errors] flags {f:#x}, max |d logp_t| on the other {good.size} rows {d:.2e}")


@pytest.mark.parametrize("d", [4096, 65536])
def test_fused_wide_hidden_size(d):
    """d = 4096 (64 LDS stages of the projection) and d = 65,536, the largest hidden size the
    call accepts (1,024 stages), each with a partial row tile and a ragged vocabulary."""
    wl = W.make("fused", seed=d, scale=dict(R=1, turns=2, tok=40, vocab=1000, d=d))
    sc, _ = H.oracle_fused_scores(wl, np.arange(wl.n_tokens))
    assert sc["flags"] == 0
    per = {0: {k: sc[k] for k in ("logp_t", "logp_s", "kl")}}
    lam, alpha = [-math.inf], [-math.inf]
    ora = {0: (per[0], H.oracle_rollout(wl, 0, per[0], lam, alpha))}
    gpu = H.run_gpu_fused(wl, lam, alpha)
    assert gpu["flags"] == 0, hex(gpu["flags"])
    dl = np.max(np.abs(gpu["logp_t"] - sc["logp_t"]))
    assert dl <= H.TOL_LOGP, dl
    rep = H.compare(wl, gpu, ora, lam, alpha)
    say(f"[fused d={wl.fused_d}] max |d logp_t| {dl:.2e}; {rep}")


def test_restart_pick_with_infinite_values_and_long_records():
    """Argmin ties at +inf go to the lowest index, as in the oracle; long token-unit records
    (several 2048-unit chunks of the first pass) keep the exact K_max and k*."""
    import torch
    import paper_2609_14636_amd as P
    g = np.random.default_rng(8)
    sizes = np.array([3, 5000, 1, 9000])
    off = np.zeros(sizes.size + 1, np.int64)
    off[1:] = np.cumsum(sizes)
    vals = -np.abs(g.normal(1.0, 0.5, size=int(off[-1])))
    vals[off[0]:off[1]] = np.inf                      # rollout 0: all +inf
    vals[off[1] + 4321] = -50.0                       # rollout 1: weakest unit deep in the record
    mask = np.ones(vals.size, np.uint8)
    mask[off[3] + 7001] = 0                           # rollout 3: K_max = 7001
    alpha = -np.inf
    vals = vals.astype(np.float32)                    # token units arrive as float32
    ks_o, k0_o, km_o = H.OP.O.restart(off, vals.astype(np.float64), sizes.astype(np.int32),
                                      np.full(sizes.size, alpha), mask)
    rto = torch.arange(sizes.size + 1, dtype=torch.int32, device="cuda")  # one turn per rollout
    tto = torch.from_numpy(off).cuda()
    lay = P.Layout(rto, tto, int(off[-1]))
    ks = torch.empty(sizes.size, dtype=torch.int32, device="cuda")
    k0, km = torch.empty_like(ks), torch.empty_like(ks)
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    P.stride_restart_turn(lay, P.STRIDE_UNIT_TOKEN, torch.from_numpy(vals).cuda(),
                          None, [alpha], torch.from_numpy(mask).cuda(), ks, k0, km, flags)
    torch.cuda.synchronize()
    assert int(flags.item()) == 0
    assert ks.cpu().tolist() == list(ks_o) and k0.cpu().tolist() == list(k0_o)
    assert km.cpu().tolist() == list(km_o)
    assert list(ks_o)[:2] == [0, 4321] and list(km_o)[3] == 7001
    say(f"[restart edges] k* {ks.cpu().tolist()} K_max {km.cpu().tolist()}")


def test_fused_confident_teacher_log_probability_is_at_most_zero():
    """A hidden state aligned with the sampled token's weight row makes the teacher nearly
    certain (p ~ 1): the fused log-probability must stay <= 0 and match the oracle."""
    import torch
    import paper_2609_14636_amd as P
    wl = W.make("fused", seed=99, scale=dict(R=1, turns=1, tok=64, vocab=1000, d=128))
    inp = H.device_inputs_fused(wl)
    ids = inp["ids"]
    w = inp["w"].float()
    # h = 40 * w_y / |w_y|^2 puts z_y near 40 while the other logits stay O(1)
    wy = w[ids.long()]
    h = (40.0 * wy / (wy * wy).sum(1, keepdim=True)).to(torch.bfloat16)
    N = wl.n_tokens
    lt = torch.empty(N, dtype=torch.float32, device="cuda")
    tm = torch.empty(wl.n_turns, dtype=torch.float64, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(P.stride_fused_workspace_size(inp["layout"], wl.vocab), dtype=torch.uint8,
                     device="cuda")
    P.stride_score_fused(inp["layout"], wl.vocab, h, inp["w"], None, ids, lt, None, None, tm,
                         flags, ws)
    torch.cuda.synchronize()
    assert int(flags.item()) == 0
    got = lt.cpu().numpy()
    assert np.all(got <= 0.0), got.max()
    hb = h.cpu().view(torch.int16).numpy().view(np.uint16)
    w_dv = np.ascontiguousarray(inp["w"].cpu().view(torch.int16).numpy().view(np.uint16).T)
    want, _, fl = H.OP.O.fused_logp(hb, w_dv, wl.tok)
    assert fl == 0 and np.max(want) <= 0
    assert np.max(np.abs(got - want)) <= H.TOL_LOGP, np.max(np.abs(got - want))
    say(f"[fused confident] logp in [{got.min():.2e}, {got.max():.2e}], max |d| {np.max(np.abs(got - want)):.2e}")


def test_single_teacher_reads_teacher_zero_whatever_the_domain_ids():
    """With one teacher every row reads teacher 0; the rollouts' domain ids are not used by
    stride_score (they select lambda and alpha in the stop and restart calls, which check them).
    Scoring with domain ids 0..3 gives the same bits as scoring without any, and no flag."""
    import torch
    import paper_2609_14636_amd as P
    wl = W.make("agentic", seed=31, scale=dict(R=4, turns=3, tok_lo=20, tok_hi=70, vocab=1000))
    inp = H.device_inputs(wl)
    lay0 = inp["layout"]
    dom = torch.arange(wl.n_rollouts, dtype=torch.int32, device="cuda")
    lay1 = P.Layout(lay0.rollout_turn_off, lay0.turn_tok_off, wl.n_tokens, dom)
    outs = []
    for lay in (lay0, lay1):
        path = P.Path(lay, wl.unit, with_student=True)
        path.score(wl.vocab, inp["teachers"], inp["student"], inp["ids"])
        torch.cuda.synchronize()
        h = path.host()
        assert h["flags"] == 0, P.flag_names(h["flags"])
        outs.append(h)
    say(f"[single teacher] R={wl.n_rollouts} N={wl.n_tokens}: domain ids 0..{wl.n_rollouts - 1}")
    for k in ("logp_t", "logp_s", "kl", "turn_mean"):
        assert np.array_equal(outs[0][k].view(np.uint8), outs[1][k].view(np.uint8)), k


def test_sixty_four_teachers_and_domains():
    """The largest domain count the ABI accepts (STRIDE_MAX_DOMAINS = 64): 64 teacher matrices,
    each routing one rollout (domain ids a permutation of 0..63), and 64 distinct lambda and alpha
    values chosen from the oracle's own cumulative sums so that rollouts stop at turn 0, at turn 1
    or not at all, and have 0, 1 or 2 correct turns.  Compared with the oracle row by row."""
    import torch
    import paper_2609_14636_amd as P
    from oracle import oracle as O

    D, K, L, V, ld = 64, 2, 12, 257, 260
    R, T, N = D, D * K, D * K * L
    g = np.random.default_rng(6464)
    dom = ((np.arange(R) * 37) % D).astype(np.int32)
    rto = (np.arange(R + 1) * K).astype(np.int32)
    tto = (np.arange(T + 1) * L).astype(np.int64)
    ids = g.integers(0, V, size=N).astype(np.int32)
    teachers = [(2.0 * g.standard_normal((N, ld))).astype(np.float32) for _ in range(D)]
    student = (2.0 * g.standard_normal((N, ld))).astype(np.float32)
    # oracle: each rollout's rows scored with its own teacher
    logp_t = np.empty(N)
    for r in range(R):
        a, b = r * K * L, (r + 1) * K * L
        logp_t[a:b] = O.logp_rows(teachers[dom[r]][a:b], ids[a:b], V)[0]
    logp_s = O.logp_rows(student, ids, V)[0]
    tm, f = O.turn_mean(tto, logp_t)
    assert f == 0
    lam = np.zeros(D)
    alpha = np.zeros(D)
    for r in range(R):
        c0, c1 = tm[2 * r], tm[2 * r] + tm[2 * r + 1]
        lam[dom[r]] = (c0 + 0.5, 0.5 * (c0 + c1), c1 - 0.5)[r % 3]
        hi, lo = max(tm[2 * r], tm[2 * r + 1]), min(tm[2 * r], tm[2 * r + 1])
        alpha[dom[r]] = (hi + 0.5, 0.5 * (hi + lo), lo - 0.5)[r % 4 % 3]
    uoff = rto.astype(np.int64)
    cum, stop, _ = O.stop(uoff, tm, lam[dom])
    rec = np.where(stop >= 0, stop + 1, K).astype(np.int32)
    ks, k0, km = O.restart(uoff, tm, rec, alpha[dom])
    assert set(stop.tolist()) == {-1, 0, 1}

    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    lay = P.Layout(dev(rto), dev(tto), N, dev(dom))
    t_dev = [dev(t) for t in teachers]
    s_dev = dev(student)
    lt = torch.empty(N, dtype=torch.float32, device="cuda")
    ls, kl = torch.empty_like(lt), torch.empty_like(lt)
    tmd = torch.empty(T, dtype=torch.float64, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(P.stride_workspace_size(lay, P.STRIDE_UNIT_TURN), dtype=torch.uint8, device="cuda")
    cumd = torch.empty(T, dtype=torch.float64, device="cuda")
    stopd = torch.empty(R, dtype=torch.int32, device="cuda")
    ksd, k0d, kmd = (torch.empty(R, dtype=torch.int32, device="cuda") for _ in range(3))
    P.stride_score(lay, V, t_dev, s_dev, dev(ids), lt, ls, kl, tmd, flags, ws)
    P.stride_stop(lay, P.STRIDE_UNIT_TURN, tmd, lam.tolist(), None, cumd, stopd, None, flags, ws)
    P.stride_restart_turn(lay, P.STRIDE_UNIT_TURN, tmd, stopd, alpha.tolist(), None, ksd, k0d, kmd,
                          flags)
    torch.cuda.synchronize()
    assert int(flags.item()) == 0, hex(int(flags.item()))
    dlt = np.max(np.abs(lt.cpu().numpy() - logp_t))
    dls = np.max(np.abs(ls.cpu().numpy() - logp_s))
    dkl = np.max(np.abs(kl.cpu().numpy() - (logp_s - logp_t)))
    assert dlt <= H.TOL_LOGP and dls <= H.TOL_LOGP and dkl <= H.TOL_KL, (dlt, dls, dkl)
    assert np.max(np.abs(tmd.cpu().numpy() - tm)) <= H.TOL_LOGP
    # thresholds sit at least a quarter of a turn mean away from every value they are tested
    # against, so stops and picks must match exactly
    assert np.array_equal(stopd.cpu().numpy(), stop)
    assert np.array_equal(ksd.cpu().numpy(), ks)
    assert np.array_equal(k0d.cpu().numpy(), k0)
    assert np.array_equal(kmd.cpu().numpy(), km)
    say(f"[64 domains] |d logp_t| {dlt:.2e} |d logp_s| {dls:.2e}; stops "
        f"{np.bincount(stop + 1).tolist()} (none/0/1), K_max {np.bincount(km).tolist()}")


@pytest.mark.parametrize("dtype", [W.BF16, W.F32])
def test_million_entry_vocabulary(dtype):
    """A vocabulary of 2^20 + 5 entries, about seven times the full-size workloads' and with a
    ragged last 16-byte word: rows of 2 MB (bf16) or 4 MB (fp32), so each lane folds about 2,048
    words into its running (max, sum).  The whole path against the oracle row by row, then the
    exact reverse KL of the paired pass."""
    from tests.test_gpu_parity import _custom, _custom_thresholds

    V = (1 << 20) + 5
    g = np.random.default_rng(2020 + dtype)
    lengths = [g.integers(1, 12, size=3) for _ in range(3)]
    wl = _custom(77 + dtype, V, dtype, lengths)
    say(f"[vocab 2^20+5] dtype={dtype} R={wl.n_rollouts} N={wl.n_tokens} ld={wl.ld}")
    sc = H.oracle_scores(wl, range(wl.n_rollouts), exact_kl=True)
    lam, alpha = _custom_thresholds(wl, sc)
    ora = {r: (sc[r], H.oracle_rollout(wl, r, sc[r], lam, alpha)) for r in sc}
    gpu = H.run_gpu(wl, lam, alpha)
    assert gpu["flags"] == 0, hex(gpu["flags"])
    rep = H.compare(wl, gpu, ora, lam, alpha)
    H.assert_invariants(gpu, wl)
    gk = H.run_gpu(wl, lam, alpha, exact_kl=True)
    assert gk["flags"] == 0, hex(gk["flags"])
    want = np.concatenate([sc[r]["kl_full"] for r in range(wl.n_rollouts)])
    d = np.max(np.abs(gk["kl_full"] - want))
    assert d <= H.TOL_KL, d
    say(f"[vocab 2^20+5] {rep}; exact KL max |d| {d:.2e}")
