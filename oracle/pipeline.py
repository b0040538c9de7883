"""The whole scoring / early-stop / restart path, composed from the float64 oracle.

TEST INFRASTRUCTURE ONLY (tests, smoke check, CPU-baseline leg of the benchmark).

The steps follow the paper in order: sampled-token log-probabilities of teacher
and student and each token's KL estimate (Eq. 1, Sec. 3.2), the mean teacher
log-probability of each turn (Eq. 4), the early-stop test (Eq. 5, Sec. 4.1; token
units for the single-turn variant of Sec. 5.5), then the prefix-buffer restart
pick over the record of generated units (Sec. 4.2, Eq. 6, Algorithm 1).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import oracle as O

UNIT_TURN, UNIT_TOKEN = 0, 1


@dataclass
class Layout:
    """Flattened student-token stream: rollout r owns turns [rollout_turn_off[r],
    rollout_turn_off[r+1]); turn k owns tokens (rows) [turn_tok_off[k], turn_tok_off[k+1])."""
    rollout_turn_off: np.ndarray  # int32 [R+1]
    turn_tok_off: np.ndarray      # int64 [T+1]
    domain: np.ndarray | None = None  # int32 [R]

    @property
    def n_rollouts(self) -> int:
        return self.rollout_turn_off.size - 1

    @property
    def n_turns(self) -> int:
        return self.turn_tok_off.size - 1

    @property
    def n_tokens(self) -> int:
        return int(self.turn_tok_off[-1])

    def units(self, unit: int):
        """(unit_off [R+1], unit_tok_off [U+1]) for turn or token units."""
        if unit == UNIT_TURN:
            return self.rollout_turn_off.astype(np.int64), self.turn_tok_off.astype(np.int64)
        tok_of_rollout = self.turn_tok_off[self.rollout_turn_off].astype(np.int64)
        return tok_of_rollout, np.arange(self.n_tokens + 1, dtype=np.int64)

    def dom(self) -> np.ndarray:
        return (np.zeros(self.n_rollouts, np.int64) if self.domain is None
                else self.domain.astype(np.int64))


def score(teacher_rows: np.ndarray, student_rows: np.ndarray | None, ids: np.ndarray,
          vocab: int | None = None):
    """Per-token teacher/student log-probabilities and KL estimate.

    ``teacher_rows`` already holds, for every token, the row of the teacher that
    scores its rollout.  Returns dict(logp_t, logp_s, kl, flags)."""
    logp_t, _, ft = O.logp_rows(teacher_rows, ids, vocab)
    out = {"logp_t": logp_t, "flags": ft}
    if student_rows is not None:
        logp_s, _, fs = O.logp_rows(student_rows, ids, vocab)
        out["logp_s"] = logp_s
        out["kl"] = O.token_kl(logp_s, logp_t)
        out["flags"] |= fs
    return out


def stop_and_restart(layout: Layout, logp_t: np.ndarray, lam_dom, alpha_dom, unit: int = UNIT_TURN,
                     start: np.ndarray | None = None, mask: np.ndarray | None = None):
    """Turn means, early stop and restart pick from the teacher log-probabilities."""
    tm, flags = O.turn_mean(layout.turn_tok_off, logp_t)
    unit_off, unit_tok_off = layout.units(unit)
    values = tm if unit == UNIT_TURN else np.asarray(logp_t, np.float64)
    dom = layout.dom()
    lam_r = np.asarray(lam_dom, np.float64)[dom]
    alpha_r = np.asarray(alpha_dom, np.float64)[dom]
    cum, stop, retained = O.stop(unit_off, values, lam_r, start, unit_tok_off)
    n_units = np.diff(unit_off)
    record_len = np.where(stop >= 0, stop + 1, n_units).astype(np.int32)
    k_star, k0, k_max = O.restart(unit_off, values, record_len, alpha_r, mask)
    return {"turn_mean": tm, "cum": cum, "stop": stop, "retained": retained,
            "record_len": record_len, "k_star": k_star, "k0": k0, "k_max": k_max,
            "flags": flags}


def run(layout: Layout, teacher_rows, student_rows, ids, lam_dom, alpha_dom, unit=UNIT_TURN,
        start=None, mask=None, vocab=None):
    """The whole path on routed rows; returns the union of both dicts."""
    s = score(teacher_rows, student_rows, ids, vocab)
    r = stop_and_restart(layout, s["logp_t"], lam_dom, alpha_dom, unit, start, mask)
    flags = s["flags"] | r["flags"]
    s.update(r)
    s["flags"] = flags
    return s


def retained_mask(layout: Layout, unit: int, start, stop) -> np.ndarray:
    """Rows that join the OPD loss: units K0 .. stop of each rollout, or K0 .. last without a stop
    (Sec. 4.1: the triggering unit is kept; Algorithm 1: the loss is on the retained tokens)."""
    mask = np.zeros(layout.n_tokens, np.uint8)
    unit_off, unit_tok_off = layout.units(unit)
    for r in range(layout.n_rollouts):
        first, n = int(unit_off[r]), int(unit_off[r + 1] - unit_off[r])
        k0 = 0 if start is None else min(max(int(start[r]), 0), n)
        s = int(stop[r])
        end = s + 1 if 0 <= s < n else n
        if end > k0:
            mask[int(unit_tok_off[first + k0]):int(unit_tok_off[first + end])] = 1
    return mask
