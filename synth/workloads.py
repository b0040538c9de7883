"""Seeded synthetic workloads shaped like the paper's OPD settings.

This module makes inputs only; it holds none of the method's arithmetic, and it
is the one thing the float64 oracle and the HIP library share.  Per-row
parameters (layout, sampled tokens, boosts, domains, planted error turns,
correctness masks) are drawn on the host with NumPy's Philox counter-based
generator (Salmon et al., SC 2011).  The logits themselves come from
``synth.hip``: ``fill_host`` for the oracle, ``fill_device`` for the GPU,
bit-identical by construction.

The five workloads stand in for the paper's settings (rollouts on tau^2-bench
and AIME scored by Qwen3 models, none of which exist here):

  tiny        2 rollouts x 3 turns x 64 tokens, V = 1024, float32 logits
              sigma 2 with the sampled token boosted by +4; the teacher's boost
              is -6 on turn 1 of rollout 0 (a planted error turn).
  agentic     16 rollouts x 12 turns, turn lengths U{128..768}, V = 151936,
              bf16 sigma 3, boost ~N(5, 2) per row; one planted turn per
              rollout (teacher boost -6) and mask_k = [k < planted turn].
  reasoning   8 rollouts x 1 turn x 16384 tokens, token units, boost falling
              linearly from 6 to 1 along the sequence on both rows.
  multi       32 rollouts x 8 turns x 512 tokens, two teachers, domain
              ~ Bernoulli(1/2); teacher boosts ~N(5, 2) and ~N(3, 2); planted
              turn and mask as in agentic; one student shared by both.
  fused       16 rollouts x 8 turns x 512 tokens; teacher logits z = h W with
              h ~ N(0, 1) [N, 2048] and W ~ N(0, 0.02) [2048, V] (bf16), W held as
              a linear layer stores it ([V, 2048], row v = entry v); student as
              in agentic; no planted turn.

N(mu, s) means mean mu and standard deviation s.  Elements are Irwin-Hall(12)
approximations of a normal draw (``synth.hip``).
"""
from __future__ import annotations

import ctypes
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsynth.so")

BF16, F32 = 0, 1
UNIT_TURN, UNIT_TOKEN = 0, 1
STREAM_STUDENT = 100
STREAM_HIDDEN = 200
STREAM_W = 201
V_FULL = 151936

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run python synth/build.py")
        l = ctypes.CDLL(LIB_PATH)
        i64, i32, u64, vp, f32 = ctypes.c_int64, ctypes.c_int, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_float
        l.synth_fill_host.argtypes = [vp, i32, i64, i64, i64, i64, u64, u64, f32, vp, vp]
        l.synth_fill_host.restype = i32
        l.synth_fill_device.argtypes = [vp, i32, i64, i64, i64, i64, u64, u64, f32, vp, vp, vp]
        l.synth_fill_device.restype = i32
        _lib = l
    return _lib


def teacher_stream(d: int) -> int:
    return d


@dataclass
class Workload:
    name: str
    seed: int
    vocab: int
    ld: int
    dtype: int                    # BF16 or F32
    unit: int                     # UNIT_TURN or UNIT_TOKEN
    rollout_turn_off: np.ndarray  # int32 [R+1]
    turn_tok_off: np.ndarray      # int64 [T+1]
    domain: np.ndarray | None     # int32 [R] or None
    n_teachers: int
    tok: np.ndarray               # int32 [N]
    teacher_sigma: float
    student_sigma: float
    teacher_boost: np.ndarray     # float32 [N], boost of the routed teacher
    student_boost: np.ndarray | None  # float32 [N] or None (no student)
    planted: np.ndarray | None = None  # int32 [R] planted turn (local), -1 = none
    mask: np.ndarray | None = None     # uint8 [U]
    start: np.ndarray | None = None    # int32 [R] K0
    fused_d: int = 0
    hidden_sigma: float = 1.0
    w_sigma: float = 0.02
    notes: dict = field(default_factory=dict)

    # ------------------------------------------------------------------ sizes
    @property
    def n_rollouts(self) -> int:
        return self.rollout_turn_off.size - 1

    @property
    def n_turns(self) -> int:
        return self.turn_tok_off.size - 1

    @property
    def n_tokens(self) -> int:
        return int(self.turn_tok_off[-1])

    @property
    def esize(self) -> int:
        return 2 if self.dtype == BF16 else 4

    def row_domain(self) -> np.ndarray:
        """Teacher index of every row."""
        dom = np.zeros(self.n_rollouts, np.int32) if self.domain is None else self.domain
        turns_per = np.diff(self.rollout_turn_off)
        turn_dom = np.repeat(dom, turns_per)
        return np.repeat(turn_dom, np.diff(self.turn_tok_off)).astype(np.int32)

    def rollout_rows(self, r: int) -> tuple[int, int]:
        a = int(self.turn_tok_off[self.rollout_turn_off[r]])
        b = int(self.turn_tok_off[self.rollout_turn_off[r + 1]])
        return a, b

    def unit_off(self) -> np.ndarray:
        if self.unit == UNIT_TURN:
            return self.rollout_turn_off.astype(np.int64)
        return self.turn_tok_off[self.rollout_turn_off].astype(np.int64)

    def n_units(self) -> int:
        return self.n_turns if self.unit == UNIT_TURN else self.n_tokens

    def logits_bytes(self) -> int:
        return self.n_tokens * self.ld * self.esize

    # ------------------------------------------------------------ host fills
    def _fill_host(self, out: np.ndarray, cols: int, ld: int, dtype: int, row0: int, n: int,
                   stream: int, sigma: float, tok, boost, threads: int):
        l = lib()
        tok = None if tok is None else np.ascontiguousarray(tok, np.int32)
        boost = None if boost is None else np.ascontiguousarray(boost, np.float32)
        esize = 2 if dtype == BF16 else 4
        base = out.ctypes.data
        chunk = max(1, (n + threads - 1) // threads)

        def work(i0):
            k = min(chunk, n - i0)
            tp = None if tok is None else tok[i0:i0 + k].ctypes.data
            bp = None if boost is None else boost[i0:i0 + k].ctypes.data
            rc = l.synth_fill_host(base + i0 * ld * esize, dtype, ld, cols, row0 + i0, k,
                                   self.seed, stream, sigma, tp, bp)
            if rc != 0:
                raise RuntimeError("synth_fill_host failed")

        starts = list(range(0, n, chunk))
        if len(starts) <= 1:
            for s in starts:
                work(s)
        else:
            with ThreadPoolExecutor(len(starts)) as ex:
                list(ex.map(work, starts))

    def teacher_rows_host(self, row0: int, n: int, threads: int = 8) -> np.ndarray:
        """Rows row0..row0+n-1 of the routed teacher (the oracle's teacher input)."""
        out = np.zeros((n, self.ld), np.uint16 if self.dtype == BF16 else np.float32)
        dom = self.row_domain()[row0:row0 + n]
        for d in np.unique(dom):
            idx = np.nonzero(dom == d)[0]
            # runs of consecutive rows of one domain
            splits = np.nonzero(np.diff(idx) != 1)[0] + 1
            for run in np.split(idx, splits):
                a, k = int(run[0]), int(run.size)
                self._fill_host(out[a:a + k], self.vocab, self.ld, self.dtype, row0 + a, k,
                                teacher_stream(int(d)), self.teacher_sigma,
                                self.tok[row0 + a:row0 + a + k],
                                self.teacher_boost[row0 + a:row0 + a + k], threads)
        return out

    def student_rows_host(self, row0: int, n: int, threads: int = 8) -> np.ndarray:
        out = np.zeros((n, self.ld), np.uint16 if self.dtype == BF16 else np.float32)
        self._fill_host(out, self.vocab, self.ld, self.dtype, row0, n, STREAM_STUDENT,
                        self.student_sigma, self.tok[row0:row0 + n],
                        self.student_boost[row0:row0 + n], threads)
        return out

    def hidden_host(self, row0: int, n: int, threads: int = 8) -> np.ndarray:
        d = self.fused_d
        out = np.zeros((n, d), np.uint16)
        self._fill_host(out, d, d, BF16, row0, n, STREAM_HIDDEN, self.hidden_sigma, None, None,
                        threads)
        return out

    def w_host(self, threads: int = 8) -> np.ndarray:
        """lm_head weight as a linear layer stores it: [V, d], row v = vocabulary entry v."""
        d, v = self.fused_d, self.vocab
        out = np.zeros((v, d), np.uint16)
        self._fill_host(out, d, d, BF16, 0, v, STREAM_W, self.w_sigma, None, None, threads)
        return out

    def w_dv_host(self, threads: int = 8) -> np.ndarray:
        """The same lm_head bits as the [d, V] matrix of z = h W (the transpose of w_host),
        copied in blocks of 256 vocabulary rows so that the copy stays cache-friendly."""
        w = self.w_host(threads)
        out = np.empty((w.shape[1], w.shape[0]), np.uint16)
        for i in range(0, w.shape[0], 256):
            out[:, i:i + 256] = w[i:i + 256].T
        return out

    # ---------------------------------------------------------- device fills
    def fill_device(self, ptr: int, cols: int, ld: int, dtype: int, row0: int, n: int, stream: int,
                    sigma: float, tok_dev: int | None, boost_dev: int | None, hip_stream: int):
        rc = lib().synth_fill_device(ptr, dtype, ld, cols, row0, n, self.seed, stream, sigma,
                                     tok_dev, boost_dev, hip_stream)
        if rc != 0:
            raise RuntimeError(f"synth_fill_device failed ({rc})")


def _layout_from_lengths(lengths_per_rollout: list[np.ndarray]):
    turns = np.array([len(l) for l in lengths_per_rollout], np.int64)
    rto = np.zeros(turns.size + 1, np.int32)
    rto[1:] = np.cumsum(turns)
    flat = np.concatenate(lengths_per_rollout).astype(np.int64) if turns.sum() else np.zeros(0, np.int64)
    tto = np.zeros(flat.size + 1, np.int64)
    tto[1:] = np.cumsum(flat)
    return rto, tto


def _rng(seed: int, what: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(key=[seed, what]))


def make(name: str, seed: int = 1001, scale: dict | None = None) -> Workload:
    """Build a workload by name.  ``scale`` overrides sizes for reduced test copies:
    keys R, turns, tok (fixed turn length), tok_lo/tok_hi, vocab, ld, d."""
    s = dict(scale or {})
    if name == "tiny":
        R, K, L = s.get("R", 2), s.get("turns", 3), s.get("tok", 64)
        V = s.get("vocab", 1024)
        ld = s.get("ld", V + (-V) % 4)
        rto, tto = _layout_from_lengths([np.full(K, L)] * R)
        N = int(tto[-1])
        tok = _rng(seed, 1).integers(0, V, size=N).astype(np.int32)
        tb = np.full(N, 4.0, np.float32)
        sb = np.full(N, 4.0, np.float32)
        planted = np.full(R, -1, np.int32)
        planted[0] = 1
        a, b = tto[rto[0] + 1], tto[rto[0] + 2]
        tb[a:b] = -6.0
        return Workload(name, seed, V, ld, F32, UNIT_TURN, rto, tto, None, 1, tok, 2.0, 2.0, tb, sb,
                        planted=planted)
    if name in ("agentic", "multi"):
        multi = name == "multi"
        R = s.get("R", 32 if multi else 16)
        K = s.get("turns", 8 if multi else 12)
        V = s.get("vocab", V_FULL)
        ld = s.get("ld", V + (-V) % 8)
        g = _rng(seed, 2)
        if multi:
            L = s.get("tok", 512)
            lengths = [np.full(K, L)] * R
        else:
            lo, hi = s.get("tok_lo", 128), s.get("tok_hi", 768)
            lengths = [g.integers(lo, hi + 1, size=K) for _ in range(R)]
        rto, tto = _layout_from_lengths(lengths)
        N = int(tto[-1])
        tok = _rng(seed, 1).integers(0, V, size=N).astype(np.int32)
        domain = _rng(seed, 3).integers(0, 2, size=R).astype(np.int32) if multi else None
        mu_t = np.array([5.0, 3.0], np.float32)
        row_dom = np.repeat(np.repeat(domain if multi else np.zeros(R, np.int32), K), np.diff(tto))
        tb = (mu_t[row_dom] + 2.0 * _rng(seed, 4).standard_normal(N)).astype(np.float32)
        sb = (5.0 + 2.0 * _rng(seed, 5).standard_normal(N)).astype(np.float32)
        planted = _rng(seed, 6).integers(0, K, size=R).astype(np.int32)
        mask = np.zeros(R * K, np.uint8)
        for r in range(R):
            t0 = rto[r] + planted[r]
            tb[tto[t0]:tto[t0 + 1]] = -6.0
            mask[rto[r]:rto[r] + planted[r]] = 1
        return Workload(name, seed, V, ld, BF16, UNIT_TURN, rto, tto, domain, 2 if multi else 1,
                        tok, 3.0, 3.0, tb, sb, planted=planted, mask=mask)
    if name == "reasoning":
        R, L = s.get("R", 8), s.get("tok", 16384)
        V = s.get("vocab", V_FULL)
        ld = s.get("ld", V + (-V) % 8)
        rto, tto = _layout_from_lengths([np.array([L])] * R)
        N = int(tto[-1])
        tok = _rng(seed, 1).integers(0, V, size=N).astype(np.int32)
        t = np.arange(L, dtype=np.float64)
        b = (6.0 - 5.0 * t / max(L - 1, 1)).astype(np.float32)
        tb = np.tile(b, R)
        sb = tb.copy()
        return Workload(name, seed, V, ld, BF16, UNIT_TOKEN, rto, tto, None, 1, tok, 3.0, 3.0, tb, sb)
    if name == "fused":
        R, K, L = s.get("R", 16), s.get("turns", 8), s.get("tok", 512)
        V = s.get("vocab", V_FULL)
        ld = s.get("ld", V + (-V) % 8)
        d = s.get("d", 2048)
        rto, tto = _layout_from_lengths([np.full(K, L)] * R)
        N = int(tto[-1])
        tok = _rng(seed, 1).integers(0, V, size=N).astype(np.int32)
        sb = (5.0 + 2.0 * _rng(seed, 5).standard_normal(N)).astype(np.float32)
        tb = np.zeros(N, np.float32)
        return Workload(name, seed, V, ld, BF16, UNIT_TURN, rto, tto, None, 1, tok, 0.0, 3.0, tb, sb,
                        fused_d=d, hidden_sigma=1.0, w_sigma=0.02)
    raise ValueError(f"unknown workload {name!r}")


NAMES = ("tiny", "agentic", "reasoning", "multi", "fused")
