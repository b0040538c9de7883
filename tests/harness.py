"""Shared helpers of the parity tests: inputs on both sides, the oracle per rollout, comparison.

The GPU side gets its logits from the device generator and runs the library
through its Python binding; the oracle side gets the same rows from the host
generator.  Nothing the GPU computes ever reaches the oracle.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from oracle import pipeline as OP
from synth import workloads as W
from tests import workload_params as WP

# Tolerances: 2e-3 on log-probabilities and turn means, 1e-4 relative on cumulative sums (the
# stated bounds), 4e-3 on the KL estimate, a difference of two log-probabilities
TOL_LOGP = 2e-3     # |d logp_t|, |d logp_s|, |d turn mean|
TOL_KL = 4e-3       # |d kl| (difference of two logps)
TOL_CUM_REL = 1e-4  # |d C| <= TOL_CUM_REL * max(|C|, 1)
BAND = 1e-3         # stop / k* decisions within this distance of lambda / alpha / a tie are excused


# ---------------------------------------------------------------- device inputs

from synth.device import device_inputs, device_inputs_fused  # noqa: E402,F401


def run_gpu_fused(wl: W.Workload, lam, alpha, inp=None):
    import torch
    import paper_2609_14636_amd as P

    inp = inp or device_inputs_fused(wl)
    path = P.Path(inp["layout"], wl.unit, with_student=True, fused_vocab=wl.vocab)
    path.score_fused(wl.vocab, inp["hidden"], inp["w"], inp["student"], inp["ids"])
    path.stop(lam, inp["start"])
    path.restart(alpha, inp["mask"])
    torch.cuda.synchronize()
    return path.host()


def oracle_fused_scores(wl: W.Workload, rows, w_dv=None, threads: int = 16, matmul: bool = False):
    """Oracle teacher/student log-probabilities of the given rows of a fused workload.
    The oracle takes the lm_head as the [d, V] matrix of z = h W, the transpose of the
    [V, d] storage the GPU reads; both come from the host generator.  With ``matmul`` the
    projection is the oracle's library-matmul form (for whole rollouts at full size)."""
    if w_dv is None:
        w_dv = wl.w_dv_host(threads)
    rows = np.asarray(rows, np.int64)
    contiguous = rows.size > 0 and np.array_equal(rows, np.arange(rows[0], rows[0] + rows.size))
    if contiguous:
        h = wl.hidden_host(int(rows[0]), rows.size, threads)
        s = wl.student_rows_host(int(rows[0]), rows.size, threads)
    else:
        h = np.concatenate([wl.hidden_host(int(r), 1, 1) for r in rows]) if rows.size else \
            np.zeros((0, wl.fused_d), np.uint16)
        s = np.concatenate([wl.student_rows_host(int(r), 1, 1) for r in rows])
    ids = wl.tok[rows]
    fused = OP.O.fused_logp_matmul if matmul else OP.O.fused_logp
    lt, _, ft = fused(h, w_dv, ids)
    ls, _, fs = OP.O.logp_rows(s, ids, wl.vocab)
    return {"logp_t": lt, "logp_s": ls, "kl": OP.O.token_kl(ls, lt), "flags": ft | fs}, w_dv


def run_gpu(wl: W.Workload, lam, alpha, inp=None, with_student=True, exact_kl=False):
    import torch
    import paper_2609_14636_amd as P

    inp = inp or device_inputs(wl, with_student)
    path = P.Path(inp["layout"], wl.unit, with_student=inp["student"] is not None,
                  exact_kl=exact_kl)
    path.run(wl.vocab, inp["teachers"], inp["student"], inp["ids"], lam, alpha,
             start_unit=inp["start"], correct_mask=inp["mask"])
    torch.cuda.synchronize()
    return path.host()


# ---------------------------------------------------------------- oracle per rollout

def oracle_scores(wl: W.Workload, rollouts, threads: int = 16, with_student: bool = True,
                  exact_kl: bool = False):
    """Oracle log-probabilities of the rows of the given rollouts: {r: dict(logp_t, logp_s, kl)}
    (and kl_full, the full-vocabulary KL, when exact_kl)."""
    out = {}
    for r in rollouts:
        a, b = wl.rollout_rows(r)
        t = wl.teacher_rows_host(a, b - a, threads)
        s = wl.student_rows_host(a, b - a, threads) if with_student else None
        res = OP.score(t, s, wl.tok[a:b], wl.vocab)
        if exact_kl:
            res["kl_full"] = OP.O.exact_kl(t, s, wl.vocab)
        del t, s
        out[r] = res
    return out


def oracle_rollout(wl: W.Workload, r: int, scores: dict, lam_dom, alpha_dom):
    """Turn means, stop and restart of rollout r from its oracle scores."""
    t0, t1 = int(wl.rollout_turn_off[r]), int(wl.rollout_turn_off[r + 1])
    a = int(wl.turn_tok_off[t0])
    lay = OP.Layout(np.array([0, t1 - t0], np.int32), wl.turn_tok_off[t0:t1 + 1] - a,
                    None if wl.domain is None else wl.domain[r:r + 1])
    if wl.unit == W.UNIT_TURN:
        u0, u1 = t0, t1
    else:
        u0, u1 = a, int(wl.turn_tok_off[t1])
    start = None if wl.start is None else wl.start[r:r + 1]
    mask = None if wl.mask is None else wl.mask[u0:u1]
    res = OP.stop_and_restart(lay, scores["logp_t"], lam_dom, alpha_dom, wl.unit, start, mask)
    res["unit_range"] = (u0, u1)
    return res


def oracle_all(wl: W.Workload, lam, alpha, rollouts=None, threads: int = 16, with_student=True):
    rollouts = range(wl.n_rollouts) if rollouts is None else rollouts
    sc = oracle_scores(wl, rollouts, threads, with_student)
    return {r: (sc[r], oracle_rollout(wl, r, sc[r], lam, alpha)) for r in rollouts}


def thresholds(wl: W.Workload, scores: dict):
    """Workload thresholds from oracle scores of every rollout (reduced workloads)."""
    logp_t = np.concatenate([scores[r]["logp_t"] for r in range(wl.n_rollouts)])
    tm, _ = OP.O.turn_mean(wl.turn_tok_off, logp_t)
    if wl.name == "tiny":
        return WP.tiny_thresholds(tm, wl.rollout_turn_off, wl.planted)
    if wl.name in ("agentic", "multi"):
        return WP.agentic_thresholds(tm, wl.rollout_turn_off, wl.planted, wl.domain, wl.n_teachers)
    if wl.name == "reasoning":
        return WP.reasoning_thresholds(logp_t, wl.unit_off())
    if wl.name == "fused":
        return WP.fused_thresholds(wl.vocab, wl.fused_d, wl.hidden_sigma, wl.w_sigma)
    raise ValueError(wl.name)


# ---------------------------------------------------------------- comparison

@dataclass
class Report:
    max_dlogp_t: float = 0.0
    max_dlogp_s: float = 0.0
    max_dkl: float = 0.0
    max_dturn: float = 0.0
    max_dcum_rel: float = 0.0
    stops: int = 0
    stop_excused: int = 0
    restarts: int = 0
    restart_excused: int = 0

    def __str__(self):
        return (f"dlogp_t={self.max_dlogp_t:.2e} dlogp_s={self.max_dlogp_s:.2e} "
                f"dkl={self.max_dkl:.2e} dturn={self.max_dturn:.2e} dcum_rel={self.max_dcum_rel:.2e} "
                f"stops={self.stops} (excused {self.stop_excused}) restarts={self.restarts} "
                f"(excused {self.restart_excused})")


def _maxabs(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape, (a.shape, b.shape)
    nan_a, nan_b = np.isnan(a), np.isnan(b)
    assert np.array_equal(nan_a, nan_b), "NaN positions differ"
    if (~nan_a).sum() == 0:
        return 0.0
    return float(np.max(np.abs(a[~nan_a] - b[~nan_b])))


def compare(wl: W.Workload, gpu: dict, ora: dict, lam, alpha, rep: Report | None = None) -> Report:
    """Element-wise comparison of the GPU outputs with the oracle on the rollouts in ``ora``."""
    rep = rep or Report()
    dom = np.zeros(wl.n_rollouts, np.int64) if wl.domain is None else wl.domain.astype(np.int64)
    for r, (sc, ro) in ora.items():
        a, b = wl.rollout_rows(r)
        d = _maxabs(gpu["logp_t"][a:b], sc["logp_t"])
        assert d <= TOL_LOGP, f"rollout {r}: |d logp_t| = {d}"
        rep.max_dlogp_t = max(rep.max_dlogp_t, d)
        if "logp_s" in sc and gpu.get("logp_s") is not None:
            d = _maxabs(gpu["logp_s"][a:b], sc["logp_s"])
            assert d <= TOL_LOGP, f"rollout {r}: |d logp_s| = {d}"
            rep.max_dlogp_s = max(rep.max_dlogp_s, d)
            d = _maxabs(gpu["kl"][a:b], sc["kl"])
            assert d <= TOL_KL, f"rollout {r}: |d kl| = {d}"
            rep.max_dkl = max(rep.max_dkl, d)
        t0, t1 = int(wl.rollout_turn_off[r]), int(wl.rollout_turn_off[r + 1])
        d = _maxabs(gpu["turn_mean"][t0:t1], ro["turn_mean"])
        assert d <= TOL_LOGP, f"rollout {r}: |d turn mean| = {d}"
        rep.max_dturn = max(rep.max_dturn, d)
        u0, u1 = ro["unit_range"]
        gc, oc = np.asarray(gpu["cum"][u0:u1]), ro["cum"]
        fin = np.isfinite(oc)
        assert np.array_equal(np.isfinite(gc), fin), f"rollout {r}: non-finite cum positions differ"
        if fin.any():
            rel = np.abs(gc[fin] - oc[fin]) / np.maximum(np.abs(oc[fin]), 1.0)
            assert rel.max() <= TOL_CUM_REL, f"rollout {r}: cum rel err {rel.max()}"
            rep.max_dcum_rel = max(rep.max_dcum_rel, float(rel.max()))
        lam_r, alpha_r = float(lam[dom[r]]), float(alpha[dom[r]])
        # stop: exact unless the oracle's cumulative value passes within BAND of lambda
        gs, os_ = int(gpu["stop_unit"][r]), int(ro["stop"][0])
        rep.stops += 1
        stop_excused = False
        if gs != os_:
            n = u1 - u0
            hi = n if (gs < 0 or os_ < 0) else max(gs, os_) + 1
            k0 = 0 if wl.start is None else int(np.clip(wl.start[r], 0, n))
            near = np.abs(oc[k0:hi] - lam_r) <= BAND
            assert near.any(), f"rollout {r}: stop {gs} != oracle {os_} outside the band"
            rep.stop_excused += 1
            stop_excused = True
        else:
            assert int(gpu["retained"][r]) == int(ro["retained"][0]), f"rollout {r}: retained"
        # restart: exact unless a decision sits within BAND (stop, alpha gate, or a near tie)
        rep.restarts += 1
        gk = (int(gpu["k_star"][r]), int(gpu["k0"][r]), int(gpu["k_max"][r]))
        okk = (int(ro["k_star"][0]), int(ro["k0"][0]), int(ro["k_max"][0]))
        if gk != okk:
            vals = ro["turn_mean"] if wl.unit == W.UNIT_TURN else sc["logp_t"]
            rec = int(ro["record_len"][0])
            near_alpha = np.isfinite(alpha_r) and np.any(np.abs(vals[:rec] - alpha_r) <= BAND)
            km = max(gk[2], okk[2])
            cand = np.sort(vals[:km]) if km > 0 else np.zeros(0)
            near_tie = cand.size >= 2 and (cand[1] - cand[0]) <= BAND
            assert stop_excused or near_alpha or near_tie, \
                f"rollout {r}: restart {gk} != oracle {okk} outside the band"
            rep.restart_excused += 1
    return rep


def assert_invariants(gpu: dict, wl: W.Workload):
    """Properties that hold at any size: logp <= 0 (an output contract: the kernels clamp a
    rounding excess above 0), K0 = max(k*, 0), k* < K_max <= record."""
    lt = gpu["logp_t"]
    assert np.all(lt[np.isfinite(lt)] <= 0.0)
    if gpu.get("logp_s") is not None:
        ls = gpu["logp_s"]
        assert np.all(ls[np.isfinite(ls)] <= 0.0)
        kl = gpu["kl"]
        both = np.isfinite(lt) & np.isfinite(ls)
        assert np.allclose(kl[both], (ls - lt)[both], atol=1e-6, rtol=0)
    ks, k0, km, st = gpu["k_star"], gpu["k0"], gpu["k_max"], gpu["stop_unit"]
    assert np.array_equal(k0, np.maximum(ks, 0))
    assert np.all((ks == -1) == (km == 0))
    assert np.all(ks < np.maximum(km, 1))
    uoff = wl.unit_off()
    n_units = np.diff(uoff)
    rec = np.where(st >= 0, st + 1, n_units)
    assert np.all(km <= rec)
    assert np.all(st < n_units)


def nan_like(x):
    return math.isnan(x) if isinstance(x, float) else np.isnan(x)
