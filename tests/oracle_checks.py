"""Pins of the float64 oracle against facts fixed outside it.

Each ``check_*`` function raises AssertionError when the oracle disagrees with
what the paper or the mathematics fixes: brute force in 50-digit decimal
arithmetic, closed forms, invariants, hand-traced cases stored under
``tests/golden/`` and a library matmul.  ``test_oracle_pins.py`` runs every check
on the real oracle; ``test_oracle_mutants.py`` runs them on deliberately broken
builds of ``oracle/oracle.c`` and requires each break to fail at least one.
"""
from __future__ import annotations

import json
import math
import os
from decimal import Decimal, getcontext

import numpy as np

from oracle import oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest-even) and return the bit patterns."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def _bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def _decimal_logp(row, y) -> float:
    """log softmax(row)[y] straight from the definition, 50 significant digits, no max shift."""
    getcontext().prec = 50
    xs = [Decimal(float(v)) for v in row]
    z = sum((x.exp() for x in xs), Decimal(0))
    return float(xs[y] - z.ln())


# ---------------------------------------------------------------- row log-probabilities (Eq. 1)

def check_logp_brute_force():
    """Random tiny rows against 50-digit exp/ln, fp32 and bf16 inputs, padded rows (ld > vocab)."""
    rng = np.random.default_rng(11)
    for vocab in (1, 2, 3, 5, 8, 13, 16):
        n, ld = 6, vocab + 3
        x = rng.normal(0.0, 4.0, size=(n, ld)).astype(np.float32)
        x[:, vocab:] = 1e30  # padding past vocab must never be read
        ids = rng.integers(0, vocab, size=n).astype(np.int32)
        for logits, dense in ((x, x), (_bf16_bits(x), _bf16_to_f32(_bf16_bits(x)))):
            logp, _, flags = O.logp_rows(logits, ids, vocab)
            assert flags == 0
            for i in range(n):
                want = _decimal_logp(dense[i, :vocab], ids[i])
                assert abs(logp[i] - want) <= 1e-13 * max(1.0, abs(want)), (vocab, i, logp[i], want)


def check_logp_uniform_closed_form():
    """Equal logits give every token probability 1/V: logp = -log V, for any common value."""
    for vocab in (1, 2, 3, 7, 1000, 151936):
        for c in (0.0, -3.25, 17.5, 1e30):
            x = np.full((2, vocab), c, np.float32)
            ids = np.array([0, vocab - 1], np.int32)
            logp, lse, flags = O.logp_rows(x, ids)
            assert flags == 0
            want = -math.log(vocab)
            assert np.all(np.abs(logp - want) <= 1e-9 * max(1.0, abs(want))), (vocab, c, logp)


def check_logp_two_way_closed_form():
    """V = 2: log p(0) = -log(1 + e^(b - a))."""
    rng = np.random.default_rng(5)
    ab = rng.normal(0, 6, size=(50, 2)).astype(np.float32)
    logp, _, _ = O.logp_rows(ab, np.zeros(50, np.int32))
    a, b = ab[:, 0].astype(np.float64), ab[:, 1].astype(np.float64)
    want = -np.log1p(np.exp(b - a))
    assert np.allclose(logp, want, rtol=1e-13, atol=1e-14)


def check_logp_shift_invariance_and_sign():
    """log-softmax ignores a common shift, and no log-probability is positive."""
    rng = np.random.default_rng(7)
    x = rng.normal(0, 3, size=(8, 300))
    ids = rng.integers(0, 300, size=8).astype(np.int32)
    lp0, _, _ = O.logp_rows(x, ids)
    lp1, _, _ = O.logp_rows(x + 123.0, ids)
    assert np.allclose(lp0, lp1, rtol=0, atol=1e-11)
    assert np.all(lp0 <= 0.0)


def check_logp_normalises():
    """Enumerating every token of a row, the probabilities sum to one."""
    rng = np.random.default_rng(9)
    vocab = 50
    row = rng.normal(0, 3, size=vocab).astype(np.float32)
    rows = np.repeat(row[None, :], vocab, axis=0)
    logp, _, _ = O.logp_rows(rows, np.arange(vocab, dtype=np.int32))
    assert abs(math.fsum(np.exp(logp)) - 1.0) < 1e-14
    # the probabilities follow the order of the logits
    assert np.all(np.diff(logp[np.argsort(row)]) >= 0)


def check_bf16_decoding():
    """bf16 bit patterns decode exactly: 1.0, -2.0, 0.5 and a 3-way row with a known answer."""
    bits = np.array([[0x3F80, 0xC000, 0x3F00]], np.uint16)  # [1.0, -2.0, 0.5]
    logp, _, _ = O.logp_rows(bits, np.array([0], np.int32))
    want = 1.0 - math.log(math.exp(1.0) + math.exp(-2.0) + math.exp(0.5))
    assert abs(logp[0] - want) < 1e-15


def check_nonfinite_and_oob():
    """Bad rows and token ids give NaN and the matching flag, each on its own; a single -inf entry
    only removes that token's mass."""
    cases = []
    row = np.zeros(4, np.float32); row[2] = np.nan; cases.append((row, 0, O.FLAG_NONFINITE))
    row = np.zeros(4, np.float32); row[0] = np.inf; cases.append((row, 1, O.FLAG_NONFINITE))
    row = np.full(4, -np.inf, np.float32); cases.append((row, 0, O.FLAG_NONFINITE))
    cases.append((np.zeros(4, np.float32), 4, O.FLAG_TOKEN_OOB))
    cases.append((np.zeros(4, np.float32), -1, O.FLAG_TOKEN_OOB))
    for row, y, flag in cases:
        logp, _, flags = O.logp_rows(row[None, :], np.array([y], np.int32))
        assert flags == flag and np.isnan(logp[0]), (row, y, flags, logp)
    row = np.zeros(4, np.float32); row[1] = -np.inf
    logp, _, flags = O.logp_rows(row[None, :], np.array([0], np.int32))
    assert flags == 0 and abs(logp[0] - (-math.log(3.0))) < 1e-15
    logp, _, flags = O.logp_rows(np.zeros((1, 4), np.float32), np.array([3], np.int32))
    assert flags == 0 and abs(logp[0] + math.log(4.0)) < 1e-15


# ---------------------------------------------------------------- token KL (Sec. 3.1-3.2)

def check_token_kl_gibbs():
    """E_{y~pi_S}[log pi_S(y) - log pi_T(y)] equals the full-vocabulary KL, which is >= 0 and
    vanishes exactly when the teacher's logits are the student's plus a constant."""
    rng = np.random.default_rng(13)
    vocab = 12
    for trial in range(4):
        s = rng.normal(0, 2, size=vocab)
        t = s + 2.5 if trial == 0 else rng.normal(0, 2, size=vocab)
        ids = np.arange(vocab, dtype=np.int32)
        lps, _, _ = O.logp_rows(np.repeat(s[None], vocab, 0), ids)
        lpt, _, _ = O.logp_rows(np.repeat(t[None], vocab, 0), ids)
        kl = O.token_kl(lps, lpt)
        assert np.allclose(kl, lps - lpt, rtol=0, atol=0)
        expect = math.fsum(np.exp(lps) * kl)
        exact = O.exact_kl(t[None], s[None])[0]
        assert abs(expect - exact) < 1e-13
        getcontext().prec = 50
        zs = sum((Decimal(float(v)).exp() for v in s), Decimal(0))
        zt = sum((Decimal(float(v)).exp() for v in t), Decimal(0))
        dec = sum(((Decimal(float(a)).exp() / zs) * ((Decimal(float(a)) - zs.ln()) - (Decimal(float(b)) - zt.ln()))
                   for a, b in zip(s, t)), Decimal(0))
        assert abs(exact - float(dec)) < 1e-13
        if trial == 0:
            assert abs(exact) < 1e-14
        else:
            assert exact > 0


# ---------------------------------------------------------------- per-turn mean (Eq. 4)

def check_turn_mean():
    """Dyadic inputs give exact means; random inputs match a correctly rounded sum / n_k;
    an empty turn is NaN and flagged."""
    lp = np.array([-0.5, -0.25, -0.75, -1.0, -2.0, -3.0, -0.125], np.float64)
    off = np.array([0, 4, 5, 7], np.int64)
    m, flags = O.turn_mean(off, lp)
    assert flags == 0
    assert m.tolist() == [-0.625, -2.0, -1.5625]
    rng = np.random.default_rng(17)
    lp = rng.normal(-5, 2, size=1000)
    off = np.array([0, 1, 128, 640, 1000], np.int64)
    m, _ = O.turn_mean(off, lp)
    for k in range(4):
        a, b = off[k], off[k + 1]
        want = math.fsum(lp[a:b]) / (b - a)
        assert abs(m[k] - want) <= 1e-13 * abs(want)
    m, flags = O.turn_mean(np.array([0, 2, 2, 3], np.int64), np.array([-1.0, -2.0, -4.0]))
    assert flags == O.FLAG_EMPTY_TURN and np.isnan(m[1]) and m[0] == -1.5 and m[2] == -4.0


# ---------------------------------------------------------------- early stop (Eq. 5, Sec. 4.1)

def check_stop_closed_form():
    """Constant unit value c < 0 from K0 on: C_u = (u - K0 + 1) c, so the first u with C_u < lambda
    is u = K0 + floor(lambda / c).  When lambda / c is an integer the sum equals lambda exactly one
    unit earlier, which the strict test of Eq. (5) does not count."""
    for c, lam, k0, n in ((-0.5, -1.75, 0, 10), (-0.5, -1.75, 3, 10), (-0.25, -2.0, 2, 20),
                          (-1.0, -0.5, 0, 4), (-0.5, -8.0, 0, 10)):
        vals = np.full(n, c)
        vals[:k0] = -1e9  # units before K0 are context and must not count
        cum, stop, _ = O.stop(np.array([0, n]), vals, np.array([lam]), np.array([k0], np.int32))
        want = k0 + math.floor(lam / c)
        want = want if want < n else -1
        assert stop[0] == want, (c, lam, k0, stop[0], want)
        assert np.all(cum[:k0] == 0.0)
        assert np.allclose(cum[k0:], c * np.arange(1, n - k0 + 1), rtol=0, atol=0)


def check_stop_counting_identity():
    """With non-positive values C is non-increasing, so the stop index equals K0 plus the number of
    units u >= K0 with C_u >= lambda (when that is inside the rollout), and lowering lambda never
    moves the stop earlier."""
    rng = np.random.default_rng(23)
    for _ in range(200):
        n = int(rng.integers(1, 30))
        vals = -np.abs(rng.normal(1.0, 1.0, size=n))
        k0 = int(rng.integers(0, n))
        lam = -float(rng.uniform(0.1, 20.0))
        cum, stop, _ = O.stop(np.array([0, n]), vals, np.array([lam]), np.array([k0], np.int32))
        cnt = int(np.sum(np.cumsum(vals[k0:]) >= lam))
        want = k0 + cnt if k0 + cnt < n else -1
        assert stop[0] == want
        _, stop2, _ = O.stop(np.array([0, n]), vals, np.array([lam - 0.7]), np.array([k0], np.int32))
        assert stop2[0] == -1 or (stop[0] != -1 and stop2[0] >= stop[0])


def check_stop_golden():
    """Hand-traced cases with their citations (tests/golden/stop_cases.json)."""
    with open(os.path.join(GOLDEN, "stop_cases.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        off = np.array(case["unit_off"], np.int64)
        start = np.array(case["start"], np.int32) if case.get("start") is not None else None
        tok = np.array(case["unit_tok_off"], np.int64) if case.get("unit_tok_off") else None
        cum, stop, ret = O.stop(off, np.array(case["values"], np.float64),
                                np.array(case["lambda"], np.float64), start, tok)
        assert stop.tolist() == case["stop"], (case["name"], stop.tolist())
        if "cum" in case:
            assert np.allclose(cum, case["cum"], rtol=0, atol=1e-12), case["name"]
        if "retained" in case:
            assert ret.tolist() == case["retained"], (case["name"], ret.tolist())


def check_thresholds_at_the_extremes():
    """Eq. (5)'s strict test and Sec. 4.2's gate at thresholds that decide every unit alike:
    lambda = +inf stops at the first unit counted (K0), lambda = -inf or NaN never stops (a
    comparison with NaN is false); alpha = +inf or NaN makes no unit correct, so K_max = 0, k* = -1
    and K0 = 0, while alpha = -inf leaves only the mask, so with every unit masked in K_max is the
    whole record and k* its first minimum."""
    rng = np.random.default_rng(31)
    for _ in range(100):
        n = int(rng.integers(1, 20))
        vals = -np.abs(rng.normal(1.0, 1.0, size=n))
        k0 = int(rng.integers(0, n))
        off, st = np.array([0, n]), np.array([k0], np.int32)
        _, stop, _ = O.stop(off, vals, np.array([np.inf]), st)
        assert stop[0] == k0
        for lam in (-np.inf, np.nan):
            _, stop, _ = O.stop(off, vals, np.array([lam]), st)
            assert stop[0] == -1
        rl = np.array([int(rng.integers(0, n + 1))], np.int32)
        for alpha in (np.inf, np.nan):
            ks, k0s, km = O.restart(off, vals, rl, np.array([alpha]), None)
            assert (ks[0], k0s[0], km[0]) == (-1, 0, 0)
        ks, k0s, km = O.restart(off, vals, rl, np.array([-np.inf]), np.ones(n, np.uint8))
        assert km[0] == rl[0]
        want = int(np.argmin(vals[:rl[0]])) if rl[0] > 0 else -1
        assert ks[0] == want and k0s[0] == max(want, 0)


# ---------------------------------------------------------------- restart pick (Sec. 4.2, Eq. 6)

def check_restart_golden():
    """Hand-traced cases with their citations (tests/golden/restart_cases.json)."""
    with open(os.path.join(GOLDEN, "restart_cases.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        vals = np.array(case["values"], np.float64)
        off = np.array(case.get("unit_off", [0, len(vals)]), np.int64)
        rl = np.array(case["record_len"], np.int32) if case.get("record_len") is not None else None
        mask = np.array(case["mask"], np.uint8) if case.get("mask") is not None else None
        alpha = np.array([float(a) for a in case["alpha"]], np.float64)
        ks, k0, km = O.restart(off, vals, rl, alpha, mask)
        assert ks.tolist() == case["k_star"], (case["name"], ks.tolist())
        assert k0.tolist() == case["k0"], (case["name"], k0.tolist())
        assert km.tolist() == case["k_max"], (case["name"], km.tolist())


def check_restart_brute_force():
    """Every mask of up to 7 units with repeated values: K_max from its set definition
    max{K : every k < K is correct}, k* as the lowest index of the minimum over [0, K_max)."""
    rng = np.random.default_rng(29)
    for n in range(1, 8):
        for _ in range(3):
            vals = rng.choice(np.array([-1.5, -1.0, -0.9, -0.8, -0.6, -0.3]), size=n)
            alpha = -0.8 if rng.random() < 0.7 else -np.inf
            for bits in range(1 << n):
                mask = np.array([(bits >> k) & 1 for k in range(n)], np.uint8)
                rl = int(rng.integers(0, n + 1))
                ks, k0, km = O.restart(np.array([0, n]), vals, np.array([rl], np.int32),
                                       np.array([alpha]), mask)
                correct = [bool(mask[k]) and vals[k] > alpha for k in range(rl)]
                kmax = max(K for K in range(rl + 1) if all(correct[:K]))
                if kmax == 0:
                    kst = -1
                else:
                    lo = min(vals[:kmax])
                    kst = min(k for k in range(kmax) if vals[k] == lo)
                assert km[0] == kmax and ks[0] == kst and k0[0] == max(kst, 0), (vals, mask, rl)


# ---------------------------------------------------------------- projected teacher logits

def check_fused_against_matmul():
    """Logits from a hidden state and an lm_head: the oracle's float64 projection must equal a
    library matmul of the decoded bf16 operands, then the same log-softmax."""
    rng = np.random.default_rng(31)
    n, d, vocab = 5, 24, 37  # no two sizes equal, so a transposed operand cannot pass
    h = _bf16_bits(rng.normal(0, 1, size=(n, d)).astype(np.float32))
    w = _bf16_bits(rng.normal(0, 0.3, size=(d, vocab)).astype(np.float32))
    ids = rng.integers(0, vocab, size=n).astype(np.int32)
    z = _bf16_to_f32(h).astype(np.float64) @ _bf16_to_f32(w).astype(np.float64)
    want, want_lse, _ = O.logp_rows(z, ids)
    got, got_lse, flags = O.fused_logp(h, w, ids)
    assert flags == 0
    assert np.allclose(got, want, rtol=0, atol=1e-12)
    assert np.allclose(got_lse, want_lse, rtol=0, atol=1e-12)
    for i in range(n):
        assert abs(got[i] - _decimal_logp(z[i], ids[i])) < 1e-12


def check_fused_matmul_form():
    """fused_logp_matmul (library matmul, then the row log-softmax) equals fused_logp on shapes
    where no two sizes are equal, with W given both as a [d, V] array and as the transposed view
    of its [V, d] storage, across several row blocks; and the 50-digit brute force."""
    rng = np.random.default_rng(41)
    n, d, vocab = 7, 40, 53
    h = _bf16_bits(rng.normal(0, 1, size=(n, d)).astype(np.float32))
    w_vd = _bf16_bits(rng.normal(0, 0.3, size=(vocab, d)).astype(np.float32))
    ids = rng.integers(0, vocab, size=n).astype(np.int32)
    want, want_lse, f0 = O.fused_logp(h, np.ascontiguousarray(w_vd.T), ids)
    assert f0 == 0
    for w in (np.ascontiguousarray(w_vd.T), w_vd.T):
        for block in (1, 3, 256):
            got, got_lse, flags = O.fused_logp_matmul(h, w, ids, rows_per_call=block)
            assert flags == 0
            assert np.allclose(got, want, rtol=0, atol=1e-12)
            assert np.allclose(got_lse, want_lse, rtol=0, atol=1e-12)
    z = _bf16_to_f32(h).astype(np.float64) @ _bf16_to_f32(w_vd).astype(np.float64).T
    got, _, _ = O.fused_logp_matmul(h, w_vd.T, ids)
    for i in range(n):
        assert abs(got[i] - _decimal_logp(z[i], ids[i])) < 1e-12
    bad = ids.copy()
    bad[2] = vocab
    _, _, flags = O.fused_logp_matmul(h, w_vd.T, bad)
    assert flags & O.FLAG_TOKEN_OOB


ALL_CHECKS = [
    check_logp_brute_force,
    check_logp_uniform_closed_form,
    check_logp_two_way_closed_form,
    check_logp_shift_invariance_and_sign,
    check_logp_normalises,
    check_bf16_decoding,
    check_nonfinite_and_oob,
    check_token_kl_gibbs,
    check_turn_mean,
    check_stop_closed_form,
    check_stop_counting_identity,
    check_stop_golden,
    check_restart_golden,
    check_restart_brute_force,
    check_fused_against_matmul,
    check_fused_matmul_form,
]


# ---------------------------------------------------------------- OPD loss gradient (Eq. 2)

def _opd_loss(x, ids, r, mask, scale):
    """L(s) = -scale * sum_t mask_t r_t log pi_S(y_t), evaluated with the oracle's log-softmax."""
    lp, _, _ = O.logp_rows(x, ids)
    return -scale * float(np.sum(mask * r * lp))


def check_opd_grad_finite_differences():
    """The gradient equals central finite differences of the loss of Eq. (2) (with r held
    constant), rows with mask 0 have zero gradient and loss, and every row sums to zero."""
    rng = np.random.default_rng(37)
    n, vocab = 5, 7
    x = rng.normal(0, 2, size=(n, vocab))
    ids = rng.integers(0, vocab, size=n).astype(np.int32)
    r = rng.normal(0, 3, size=n)
    mask = np.array([1, 0, 1, 1, 0], np.uint8)
    scale = 0.37
    g, loss, flags = O.opd_grad(x, ids, r, mask, scale)
    assert flags == 0
    h = 1e-5
    for i in range(n):
        for v in range(vocab):
            xp, xm = x.copy(), x.copy()
            xp[i, v] += h
            xm[i, v] -= h
            fd = (_opd_loss(xp, ids, r, mask, scale) - _opd_loss(xm, ids, r, mask, scale)) / (2 * h)
            assert abs(g[i, v] - fd) < 1e-7, (i, v, g[i, v], fd)
    lp, _, _ = O.logp_rows(x, ids)
    assert np.allclose(loss, -scale * mask * r * lp, rtol=0, atol=1e-14)
    assert np.all(g[mask == 0] == 0.0) and np.all(loss[mask == 0] == 0.0)
    assert np.allclose(g.sum(axis=1), 0.0, atol=1e-14)
    # descent raises the sampled logit when the teacher likes the token more (r > 0)
    for i in np.nonzero(mask)[0]:
        assert np.sign(g[i, ids[i]]) == -np.sign(r[i])


def check_retained_mask():
    """Retained rows: units K0 .. stop inclusive (turn and token units), K0 .. end without a stop."""
    from oracle import pipeline as OP
    lay = OP.Layout(np.array([0, 3, 5], np.int32), np.array([0, 2, 5, 6, 8, 9], np.int64))
    m = OP.retained_mask(lay, OP.UNIT_TURN, np.array([1, 0]), np.array([1, -1]))
    assert m.tolist() == [0, 0, 1, 1, 1, 0, 1, 1, 1]
    m = OP.retained_mask(lay, OP.UNIT_TOKEN, np.array([2, 0]), np.array([3, 1]))
    assert m.tolist() == [0, 0, 1, 1, 0, 0, 1, 1, 0]


ALL_CHECKS += [check_opd_grad_finite_differences, check_retained_mask, check_thresholds_at_the_extremes]
