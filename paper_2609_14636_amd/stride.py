"""Python binding of libstride.so: the C entry points under the same names.

Argument marshalling only: tensors become device pointers and sizes, the
caller's current HIP stream is passed through, and a non-OK status raises
``StrideError`` with the library's message.  Every computation runs in the
library's HIP kernels; there is no other code path.  PyTorch provides device
memory and streams.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Sequence

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libstride.so")
# the same library with the stop test's look-back delay hook compiled in (tests only)
DEBUG_LIB_PATH = os.path.join(HERE, "libstride_debug.so")

STRIDE_OK = 0
STRIDE_BF16, STRIDE_F32 = 0, 1
STRIDE_UNIT_TURN, STRIDE_UNIT_TOKEN = 0, 1
STRIDE_FLAG_TOKEN_OOB = 1
STRIDE_FLAG_EMPTY_TURN = 2
STRIDE_FLAG_BAD_OFFSETS = 4
STRIDE_FLAG_NONFINITE = 8
STRIDE_FLAG_BAD_DOMAIN = 16
STRIDE_FLAG_SPIN_LIMIT = 32
STRIDE_MAX_DOMAINS = 64

STATUS_NAMES = {0: "STRIDE_OK", 1: "STRIDE_ERR_INVALID_ARG", 2: "STRIDE_ERR_UNSUPPORTED",
                3: "STRIDE_ERR_WORKSPACE", 4: "STRIDE_ERR_HIP"}


FLAG_NAMES = {STRIDE_FLAG_TOKEN_OOB: "TOKEN_OOB", STRIDE_FLAG_EMPTY_TURN: "EMPTY_TURN",
              STRIDE_FLAG_BAD_OFFSETS: "BAD_OFFSETS", STRIDE_FLAG_NONFINITE: "NONFINITE",
              STRIDE_FLAG_BAD_DOMAIN: "BAD_DOMAIN", STRIDE_FLAG_SPIN_LIMIT: "SPIN_LIMIT"}


def flag_names(flags: int) -> list[str]:
    """Names of the data-error bits set in a device flag word (unknown bits as hex)."""
    names = [n for bit, n in FLAG_NAMES.items() if flags & bit]
    rest = flags & ~sum(FLAG_NAMES)
    if rest:
        names.append(hex(rest))
    return names


class StrideError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class StrideDataError(RuntimeError):
    """Raised by Path.check when the device flag word reports data errors."""

    def __init__(self, flags: int):
        super().__init__("device data errors: " + ", ".join(flag_names(flags)))
        self.flags = flags


class _CLayout(ctypes.Structure):
    _fields_ = [("n_rollouts", ctypes.c_int32), ("n_turns", ctypes.c_int32),
                ("n_tokens", ctypes.c_int64), ("rollout_turn_off", ctypes.c_void_p),
                ("turn_tok_off", ctypes.c_void_p), ("domain", ctypes.c_void_p)]


def _load(path: str = LIB_PATH):
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with "
                          "`python paper_2609_14636_amd/csrc/build.py` (no other code path exists)")
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lp = ctypes.POINTER(_CLayout)
    lib.stride_workspace_size.argtypes = [lp, i32]
    lib.stride_workspace_size.restype = sz
    lib.stride_score.argtypes = [lp, i32, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                 sz, vp]
    lib.stride_score.restype = i32
    lib.stride_score_fused.argtypes = [lp, i32, i32, vp, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp,
                                       sz, vp]
    lib.stride_score_fused.restype = i32
    lib.stride_fused_workspace_size.argtypes = [lp, i32]
    lib.stride_fused_workspace_size.restype = sz
    lib.stride_stop.argtypes = [lp, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.stride_stop.restype = i32
    lib.stride_restart_turn.argtypes = [lp, i32, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp]
    lib.stride_restart_turn.restype = i32
    lib.stride_opd_grad.argtypes = [lp, i32, i32, i64, i32, vp, vp, vp, vp, vp, vp, ctypes.c_float,
                                    vp, vp, vp, vp, sz, vp]
    lib.stride_opd_grad.restype = i32
    lib.stride_stop_noalloc.argtypes = [lp, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp]
    lib.stride_stop_noalloc.restype = i32
    lib.stride_stop_step.argtypes = [i32, vp, vp, i32, vp, vp, vp, i32, vp, vp, vp, vp, vp]
    lib.stride_stop_step.restype = i32
    lib.stride_records_create.argtypes = []
    lib.stride_records_create.restype = vp
    lib.stride_records_destroy.argtypes = [vp]
    lib.stride_records_destroy.restype = None
    lib.stride_records_put.argtypes = [vp, i64, i32, vp, vp]
    lib.stride_records_put.restype = i32
    lib.stride_records_get.argtypes = [vp, i64, i32, vp, vp]
    lib.stride_records_get.restype = i32
    lib.stride_records_size.argtypes = [vp]
    lib.stride_records_size.restype = i64
    lib.stride_records_plan.argtypes = [vp, i32, vp, vp, vp, vp, vp]
    lib.stride_records_plan.restype = i32
    lib.stride_probe_read.argtypes = [vp, vp, i64, i64, i64, vp, vp]
    lib.stride_probe_read.restype = i32
    lib.stride_probe_read_flat.argtypes = [vp, vp, i64, vp, i64, vp]
    lib.stride_probe_read_flat.restype = i32
    lib.stride_probe_copy.argtypes = [vp, vp, vp, i64, i64, i64, vp]
    lib.stride_probe_copy.restype = i32
    lib.stride_debug_scan_delay.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32]
    lib.stride_debug_scan_delay.restype = i32
    lib.stride_debug_scan_spin_limit.argtypes = [ctypes.c_uint32]
    lib.stride_debug_scan_spin_limit.restype = i32
    lib.stride_debug_fused_band.argtypes = [ctypes.c_int32]
    lib.stride_debug_fused_band.restype = i32
    lib.stride_last_error.argtypes = []
    lib.stride_last_error.restype = ctypes.c_char_p
    return lib


_lib = _load()


def library() -> ctypes.CDLL:
    return _lib


def debug_library() -> ctypes.CDLL:
    """libstride_debug.so (the stop test's look-back delay hook and the fused projection's
    band setting compiled in), with the same argument types; for tests and timing probes only."""
    return _load(DEBUG_LIB_PATH)


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _check(status: int):
    if status != STRIDE_OK:
        raise StrideError(status, _lib.stride_last_error().decode())


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Layout:
    """Rollout/turn/token layout: rollout r owns turns [rollout_turn_off[r], rollout_turn_off[r+1]),
    turn k owns rows [turn_tok_off[k], turn_tok_off[k+1]).  Tensors live on the device;
    ``n_tokens`` (N) is passed explicitly so that no device value is read."""

    def __init__(self, rollout_turn_off: torch.Tensor, turn_tok_off: torch.Tensor,
                 n_tokens: int, domain: torch.Tensor | None = None):
        if rollout_turn_off.dtype != torch.int32 or turn_tok_off.dtype != torch.int64:
            raise TypeError("rollout_turn_off must be int32 and turn_tok_off int64")
        if domain is not None and domain.dtype != torch.int32:
            raise TypeError("domain must be int32")
        self.rollout_turn_off = rollout_turn_off.contiguous()
        self.turn_tok_off = turn_tok_off.contiguous()
        self.domain = None if domain is None else domain.contiguous()
        self.n_rollouts = self.rollout_turn_off.numel() - 1
        self.n_turns = self.turn_tok_off.numel() - 1
        self.n_tokens = int(n_tokens)
        self._c = _CLayout(self.n_rollouts, self.n_turns, self.n_tokens,
                           _ptr(self.rollout_turn_off), _ptr(self.turn_tok_off), _ptr(self.domain))

    def c(self):
        return ctypes.byref(self._c)

    def n_units(self, unit: int) -> int:
        return self.n_turns if unit == STRIDE_UNIT_TURN else self.n_tokens


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return STRIDE_BF16
    if t.dtype == torch.float32:
        return STRIDE_F32
    raise TypeError(f"logits must be bfloat16 or float32, got {t.dtype}")


def _doubles(vals: Sequence[float]):
    arr = (ctypes.c_double * len(vals))(*[float(v) for v in vals])
    return arr


def stride_workspace_size(layout: Layout, unit: int) -> int:
    return int(_lib.stride_workspace_size(layout.c(), unit))


def stride_fused_workspace_size(layout: Layout, vocab: int) -> int:
    return int(_lib.stride_fused_workspace_size(layout.c(), int(vocab)))


def stride_score(layout: Layout, vocab: int, teacher_logits: Sequence[torch.Tensor],
                 student_logits: torch.Tensor | None, token_ids: torch.Tensor, logp_t: torch.Tensor,
                 logp_s: torch.Tensor | None, kl: torch.Tensor | None, turn_mean: torch.Tensor,
                 dev_flags: torch.Tensor | None, ws: torch.Tensor | None, stream=None,
                 kl_full: torch.Tensor | None = None) -> None:
    t0 = teacher_logits[0]
    if t0.dim() != 2 or t0.stride(1) != 1:
        raise ValueError("teacher logits must be 2-D with unit column stride")
    for t in list(teacher_logits) + ([student_logits] if student_logits is not None else []):
        if t.dtype != t0.dtype or t.stride() != t0.stride() or t.shape != t0.shape:
            raise ValueError("all logits tensors must share dtype, shape and strides")
    ptrs = (ctypes.c_void_p * len(teacher_logits))(*[t.data_ptr() for t in teacher_logits])
    _check(_lib.stride_score(layout.c(), int(vocab), t0.stride(0), _dtype_code(t0),
                             len(teacher_logits), ctypes.cast(ptrs, ctypes.c_void_p),
                             _ptr(student_logits), _ptr(token_ids), _ptr(logp_t), _ptr(logp_s),
                             _ptr(kl), _ptr(kl_full), _ptr(turn_mean), _ptr(dev_flags), _ptr(ws),
                             0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def stride_score_fused(layout: Layout, vocab: int, hidden_t: torch.Tensor, w_t: torch.Tensor,
                       student_logits: torch.Tensor | None, token_ids: torch.Tensor,
                       logp_t: torch.Tensor, logp_s: torch.Tensor | None, kl: torch.Tensor | None,
                       turn_mean: torch.Tensor, dev_flags: torch.Tensor | None,
                       ws: torch.Tensor | None, stream=None, lib: ctypes.CDLL | None = None) -> None:
    ld = student_logits.stride(0) if student_logits is not None else 0
    _check((lib or _lib).stride_score_fused(layout.c(), int(vocab), hidden_t.shape[1], _ptr(hidden_t),
                                   _ptr(w_t), _ptr(student_logits), ld, _ptr(token_ids),
                                   _ptr(logp_t), _ptr(logp_s), _ptr(kl), _ptr(turn_mean),
                                   _ptr(dev_flags), _ptr(ws),
                                   0 if ws is None else ws.numel() * ws.element_size(),
                                   _stream(stream)))


def stride_stop(layout: Layout, unit: int, values: torch.Tensor, lam: Sequence[float],
                start_unit: torch.Tensor | None, cum: torch.Tensor, stop_unit: torch.Tensor,
                n_retained_tokens: torch.Tensor | None, dev_flags: torch.Tensor | None,
                ws: torch.Tensor, stream=None) -> None:
    lt = _doubles(lam)
    _check(_lib.stride_stop(layout.c(), unit, _ptr(values), ctypes.cast(lt, ctypes.c_void_p),
                            len(lam), _ptr(start_unit), _ptr(cum), _ptr(stop_unit),
                            _ptr(n_retained_tokens), _ptr(dev_flags), _ptr(ws),
                            ws.numel() * ws.element_size(), _stream(stream)))


def stride_stop_noalloc(layout: Layout, unit: int, values: torch.Tensor, lam: Sequence[float],
                        start_unit: torch.Tensor | None, cum: torch.Tensor, stop_unit: torch.Tensor,
                        n_retained_tokens: torch.Tensor | None, dev_flags: torch.Tensor | None,
                        stream=None) -> None:
    """stride_stop with its scratch in the library's fixed per-GPU array (no workspace)."""
    lt = _doubles(lam)
    _check(_lib.stride_stop_noalloc(layout.c(), unit, _ptr(values), ctypes.cast(lt, ctypes.c_void_p),
                                    len(lam), _ptr(start_unit), _ptr(cum), _ptr(stop_unit),
                                    _ptr(n_retained_tokens), _ptr(dev_flags), _stream(stream)))


def stride_stop_step(slot: torch.Tensor, new_off: torch.Tensor, unit: int, values: torch.Tensor,
                     domain: torch.Tensor | None, lam: Sequence[float], state_cum: torch.Tensor,
                     state_units: torch.Tensor, stop_unit: torch.Tensor,
                     dev_flags: torch.Tensor | None, stream=None) -> None:
    lt = _doubles(lam)
    _check(_lib.stride_stop_step(slot.numel(), _ptr(slot), _ptr(new_off), unit, _ptr(values),
                                 _ptr(domain), ctypes.cast(lt, ctypes.c_void_p), len(lam),
                                 _ptr(state_cum), _ptr(state_units), _ptr(stop_unit),
                                 _ptr(dev_flags), _stream(stream)))


def stride_restart_turn(layout: Layout, unit: int, values: torch.Tensor,
                        stop_unit: torch.Tensor | None, alpha: Sequence[float],
                        correct_mask: torch.Tensor | None, k_star: torch.Tensor, k0: torch.Tensor,
                        k_max: torch.Tensor | None, dev_flags: torch.Tensor | None,
                        stream=None) -> None:
    at = _doubles(alpha)
    _check(_lib.stride_restart_turn(layout.c(), unit, _ptr(values), _ptr(stop_unit),
                                    ctypes.cast(at, ctypes.c_void_p), len(alpha),
                                    _ptr(correct_mask), _ptr(k_star), _ptr(k0), _ptr(k_max),
                                    _ptr(dev_flags), _stream(stream)))


def stride_opd_grad(layout: Layout, unit: int, vocab: int, student_logits: torch.Tensor,
                    token_ids: torch.Tensor, logp_t: torch.Tensor, logp_s: torch.Tensor,
                    start_unit: torch.Tensor | None, stop_unit: torch.Tensor | None, scale: float,
                    grad: torch.Tensor, loss: torch.Tensor | None, dev_flags: torch.Tensor | None,
                    ws: torch.Tensor, stream=None) -> None:
    if grad.dtype != student_logits.dtype or grad.stride() != student_logits.stride():
        raise ValueError("grad must match the student logits' dtype and strides")
    _check(_lib.stride_opd_grad(layout.c(), unit, int(vocab), student_logits.stride(0),
                                _dtype_code(student_logits), _ptr(student_logits), _ptr(token_ids),
                                _ptr(logp_t), _ptr(logp_s), _ptr(start_unit), _ptr(stop_unit),
                                float(scale), _ptr(grad), _ptr(loss), _ptr(dev_flags), _ptr(ws),
                                ws.numel() * ws.element_size(), _stream(stream)))


def stride_probe_read(a: torch.Tensor, b: torch.Tensor | None, read_bytes: int,
                      sink: torch.Tensor, stream=None) -> None:
    """Streaming-read reference: reads the first read_bytes of every row of a (and b) with the
    scoring kernel's access pattern and no arithmetic (a measurement aid)."""
    if b is not None and (b.stride() != a.stride() or b.shape != a.shape or b.dtype != a.dtype):
        raise ValueError("a and b must share shape, dtype and strides")
    _check(_lib.stride_probe_read(_ptr(a), _ptr(b), a.shape[0], a.stride(0) * a.element_size(),
                                  int(read_bytes), _ptr(sink), _stream(stream)))


def stride_probe_read_flat(a: torch.Tensor, b: torch.Tensor | None, n_bytes: int,
                           sink: torch.Tensor, stream=None) -> None:
    """Streaming-read reference in grid-stride order over the first n_bytes of a (and b)."""
    _check(_lib.stride_probe_read_flat(_ptr(a), _ptr(b), int(n_bytes), _ptr(sink), sink.numel(),
                                       _stream(stream)))


def stride_probe_copy(src: torch.Tensor, dst: torch.Tensor, row_mask: torch.Tensor | None,
                      copy_bytes: int, stream=None) -> None:
    """Read+write reference: copies the first copy_bytes of every row of src to dst (rows with a
    0 mask byte are zero-filled without a read), the OPD gradient's access pattern."""
    if dst.stride() != src.stride() or dst.shape != src.shape or dst.dtype != src.dtype:
        raise ValueError("src and dst must share shape, dtype and strides")
    _check(_lib.stride_probe_copy(_ptr(src), _ptr(dst), _ptr(row_mask), src.shape[0],
                                  src.stride(0) * src.element_size(), int(copy_bytes),
                                  _stream(stream)))


class Records:
    """Host-side per-task trajectory record H(x) (Algorithm 1) held by libstride.so."""

    def __init__(self):
        self._h = _lib.stride_records_create()
        if not self._h:
            raise MemoryError("stride_records_create failed")

    def close(self):
        if self._h:
            _lib.stride_records_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def __len__(self):
        return int(_lib.stride_records_size(self._h))

    def put(self, task: int, values, mask=None):
        import numpy as np
        v = np.ascontiguousarray(values, dtype=np.float64)
        m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
        st = _lib.stride_records_put(self._h, int(task), v.size, v.ctypes.data,
                                     None if m is None else m.ctypes.data)
        if st != STRIDE_OK:
            raise StrideError(st, "stride_records_put")

    def get(self, task: int):
        import numpy as np
        n = _lib.stride_records_get(self._h, int(task), 0, None, None)
        if n < 0:
            return None
        v = np.empty(n, np.float64)
        m = np.empty(n, np.uint8)
        _lib.stride_records_get(self._h, int(task), n, v.ctypes.data, m.ctypes.data)
        return v, m

    def plan(self, tasks, alpha):
        """(k_star, k0, k_max) per task, 0-based; tasks without a record get (-1, 0, 0)."""
        import numpy as np
        t = np.ascontiguousarray(tasks, dtype=np.int64)
        a = np.ascontiguousarray(np.broadcast_to(np.asarray(alpha, np.float64), t.shape))
        ks, k0, km = (np.empty(t.size, np.int32) for _ in range(3))
        st = _lib.stride_records_plan(self._h, t.size, t.ctypes.data, a.ctypes.data,
                                      ks.ctypes.data, k0.ctypes.data, km.ctypes.data)
        if st != STRIDE_OK:
            raise StrideError(st, "stride_records_plan")
        return ks, k0, km


class Path:
    """Output buffers and workspace for one layout, and the three calls in order.

    ``run`` issues stride_score -> stride_stop -> stride_restart_turn on the
    current stream with no host synchronisation; outputs stay on the device."""

    def __init__(self, layout: Layout, unit: int, with_student: bool = True,
                 device: str | torch.device = "cuda", fused_vocab: int | None = None,
                 exact_kl: bool = False):
        self.layout, self.unit = layout, unit
        n, t, r = layout.n_tokens, layout.n_turns, layout.n_rollouts
        f32 = dict(dtype=torch.float32, device=device)
        self.logp_t = torch.empty(n, **f32)
        self.logp_s = torch.empty(n, **f32) if with_student else None
        self.kl = torch.empty(n, **f32) if with_student else None
        self.kl_full = torch.empty(n, **f32) if (with_student and exact_kl) else None
        self.turn_mean = torch.empty(t, dtype=torch.float64, device=device)
        self.cum = torch.empty(layout.n_units(unit), dtype=torch.float64, device=device)
        i32 = dict(dtype=torch.int32, device=device)
        self.stop_unit = torch.empty(r, **i32)
        self.retained = torch.empty(r, dtype=torch.int64, device=device)
        self.k_star = torch.empty(r, **i32)
        self.k0 = torch.empty(r, **i32)
        self.k_max = torch.empty(r, **i32)
        self.flags = torch.zeros(1, dtype=torch.int32, device=device)
        ws_bytes = max(stride_workspace_size(layout, unit), 256)
        self.ws = torch.empty(ws_bytes, dtype=torch.uint8, device=device)
        self.fused_ws = None
        if fused_vocab is not None:
            self.fused_ws = torch.empty(max(stride_fused_workspace_size(layout, fused_vocab), 256),
                                        dtype=torch.uint8, device=device)

    def values(self) -> torch.Tensor:
        return self.turn_mean if self.unit == STRIDE_UNIT_TURN else self.logp_t

    def score(self, vocab, teachers, student, token_ids, stream=None):
        stride_score(self.layout, vocab, teachers, student, token_ids, self.logp_t, self.logp_s,
                     self.kl, self.turn_mean, self.flags, self.ws, stream, kl_full=self.kl_full)

    def score_fused(self, vocab, hidden, w, student, token_ids, stream=None):
        stride_score_fused(self.layout, vocab, hidden, w, student, token_ids, self.logp_t,
                           self.logp_s, self.kl, self.turn_mean, self.flags, self.fused_ws, stream)

    def stop(self, lam, start_unit=None, stream=None):
        stride_stop(self.layout, self.unit, self.values(), lam, start_unit, self.cum,
                    self.stop_unit, self.retained, self.flags, self.ws, stream)

    def restart(self, alpha, correct_mask=None, stream=None):
        stride_restart_turn(self.layout, self.unit, self.values(), self.stop_unit, alpha,
                            correct_mask, self.k_star, self.k0, self.k_max, self.flags, stream)

    def grad(self, vocab, student, token_ids, grad, loss=None, start_unit=None, scale=1.0,
             stream=None):
        stride_opd_grad(self.layout, self.unit, vocab, student, token_ids, self.logp_t,
                        self.logp_s, start_unit, self.stop_unit, scale, grad, loss, self.flags,
                        self.ws, stream)

    def run(self, vocab, teachers, student, token_ids, lam, alpha, start_unit=None,
            correct_mask=None, stream=None):
        self.score(vocab, teachers, student, token_ids, stream)
        self.stop(lam, start_unit, stream)
        self.restart(alpha, correct_mask, stream)

    def check(self) -> None:
        """Synchronise on the flag word and raise StrideDataError if any data error was
        flagged (bad token ids, empty turns, bad offsets or domains, non-finite rows)."""
        f = int(self.flags.cpu().item()) & 0xFFFFFFFF
        if f:
            raise StrideDataError(f)

    def host(self) -> dict:
        out = {k: getattr(self, k) for k in ("logp_t", "logp_s", "kl", "kl_full", "turn_mean",
                                             "cum", "stop_unit", "retained", "k_star", "k0",
                                             "k_max")}
        res = {k: (None if v is None else v.cpu().numpy()) for k, v in out.items()}
        res["flags"] = int(self.flags.cpu().item()) & 0xFFFFFFFF
        return res


NEG_INF = -math.inf
