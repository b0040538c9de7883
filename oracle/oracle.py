"""NumPy front end of the float64 CPU oracle (liboracle.so, built from oracle.c).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg of
the benchmark use it; the product library never does.  Every function is a thin
marshalling layer over the C function of the same name, which cites the passage
of the STRIDE paper it follows.  bf16 tensors are passed as ``np.uint16`` bit
patterns.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

BF16, F32, F64 = 0, 1, 2
FLAG_TOKEN_OOB, FLAG_EMPTY_TURN, FLAG_NONFINITE = 1, 2, 8

_lib = None


def _bind(path: str):
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run python oracle/build.py")
    l = ctypes.CDLL(path)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
    l.oracle_logp_rows.argtypes = [i64, i64, i64, i32, vp, vp, vp, vp]
    l.oracle_logp_rows.restype = i32
    l.oracle_token_kl.argtypes = [i64, vp, vp, vp]
    l.oracle_token_kl.restype = None
    l.oracle_exact_kl.argtypes = [i64, i64, i64, i32, vp, vp, vp]
    l.oracle_exact_kl.restype = None
    l.oracle_turn_mean.argtypes = [i64, vp, vp, vp]
    l.oracle_turn_mean.restype = i32
    l.oracle_stop.argtypes = [i64, vp, vp, vp, vp, vp, vp, vp, vp]
    l.oracle_stop.restype = None
    l.oracle_restart.argtypes = [i64, vp, vp, vp, vp, vp, vp, vp, vp]
    l.oracle_restart.restype = None
    l.oracle_fused_logp.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp]
    l.oracle_fused_logp.restype = i32
    l.oracle_opd_grad.argtypes = [i64, i64, i64, i32, vp, vp, vp, vp, ctypes.c_double, vp, vp]
    l.oracle_opd_grad.restype = i32
    return l


def use_library(path: str | None):
    """Point this module at another build of oracle.c (the mutation tests use it).

    ``None`` restores the default liboracle.so.  Returns the previous library.
    """
    global _lib
    prev = _lib
    _lib = None if path is None else _bind(path)
    return prev


def lib():
    global _lib
    if _lib is None:
        _lib = _bind(LIB_PATH)
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.uint16:
        return BF16
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.float64:
        return F64
    raise TypeError(f"logits must be uint16 (bf16 bits), float32 or float64, got {a.dtype}")


def logp_rows(logits: np.ndarray, ids: np.ndarray, vocab: int | None = None):
    """Sampled-token log-probabilities of each row (Eq. 1).  Returns (logp, lse, flags)."""
    logits = np.ascontiguousarray(logits)
    if logits.ndim != 2:
        raise ValueError("logits must be 2-D [rows, ld]")
    n, ld = logits.shape
    vocab = ld if vocab is None else int(vocab)
    if not 0 <= vocab <= ld:
        raise ValueError("vocab must lie in [0, ld]")
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    if ids.shape != (n,):
        raise ValueError("ids must have one entry per row")
    logp = np.empty(n, np.float64)
    lse = np.empty(n, np.float64)
    flags = lib().oracle_logp_rows(n, vocab, ld, _dtype_code(logits), _p(logits), _p(ids),
                                   _p(logp), _p(lse))
    return logp, lse, int(flags)


def token_kl(logp_s: np.ndarray, logp_t: np.ndarray) -> np.ndarray:
    """Per-token KL estimate log pi_S - log pi_T = -r_t (Sec. 3.1-3.2)."""
    logp_s = np.ascontiguousarray(logp_s, dtype=np.float64)
    logp_t = np.ascontiguousarray(logp_t, dtype=np.float64)
    if logp_s.shape != logp_t.shape:
        raise ValueError("shape mismatch")
    out = np.empty_like(logp_s)
    lib().oracle_token_kl(logp_s.size, _p(logp_s), _p(logp_t), _p(out))
    return out


def exact_kl(teacher: np.ndarray, student: np.ndarray, vocab: int | None = None) -> np.ndarray:
    """Full-vocabulary KL(pi_S || pi_T) per row."""
    teacher = np.ascontiguousarray(teacher)
    student = np.ascontiguousarray(student)
    if teacher.shape != student.shape or teacher.dtype != student.dtype or teacher.ndim != 2:
        raise ValueError("teacher and student must be 2-D arrays of one shape and dtype")
    n, ld = teacher.shape
    vocab = ld if vocab is None else int(vocab)
    out = np.empty(n, np.float64)
    lib().oracle_exact_kl(n, vocab, ld, _dtype_code(teacher), _p(teacher), _p(student), _p(out))
    return out


def turn_mean(turn_tok_off: np.ndarray, logp_t: np.ndarray):
    """Mean teacher log-probability of each turn, Eq. (4).  Returns (means, flags)."""
    off = np.ascontiguousarray(turn_tok_off, dtype=np.int64)
    logp_t = np.ascontiguousarray(logp_t, dtype=np.float64)
    t = off.size - 1
    if t < 0:
        raise ValueError("offsets need at least one entry")
    if t > 0 and (off.min() < 0 or off.max() > logp_t.size):
        raise ValueError("offsets out of range")
    out = np.empty(t, np.float64)
    flags = lib().oracle_turn_mean(t, _p(off), _p(logp_t), _p(out))
    return out, int(flags)


def stop(unit_off: np.ndarray, values: np.ndarray, lam: np.ndarray, start: np.ndarray | None = None,
         unit_tok_off: np.ndarray | None = None):
    """Early-stop test, Eq. (5) with the prefix offset K0.  Returns (cum, stop, retained)."""
    off = np.ascontiguousarray(unit_off, dtype=np.int64)
    r = off.size - 1
    values = np.ascontiguousarray(values, dtype=np.float64)
    lam = np.ascontiguousarray(np.broadcast_to(np.asarray(lam, np.float64), (r,)))
    if start is not None:
        start = np.ascontiguousarray(start, dtype=np.int32)
    if unit_tok_off is not None:
        unit_tok_off = np.ascontiguousarray(unit_tok_off, dtype=np.int64)
    cum = np.empty(values.size, np.float64)
    stp = np.empty(r, np.int32)
    ret = np.zeros(r, np.int64)
    lib().oracle_stop(r, _p(off), _p(values), _p(lam), _p(start), _p(unit_tok_off), _p(cum),
                      _p(stp), _p(ret) if unit_tok_off is not None else None)
    return cum, stp, (ret if unit_tok_off is not None else None)


def restart(unit_off: np.ndarray, values: np.ndarray, record_len: np.ndarray | None,
            alpha, mask: np.ndarray | None = None):
    """Prefix-buffer pick, Sec. 4.2 / Eq. (6).  Returns (k_star, k0, k_max), 0-based."""
    off = np.ascontiguousarray(unit_off, dtype=np.int64)
    r = off.size - 1
    values = np.ascontiguousarray(values, dtype=np.float64)
    alpha = np.ascontiguousarray(np.broadcast_to(np.asarray(alpha, np.float64), (r,)))
    if record_len is not None:
        record_len = np.ascontiguousarray(record_len, dtype=np.int32)
    if mask is not None:
        mask = np.ascontiguousarray(mask, dtype=np.uint8)
    ks = np.empty(r, np.int32)
    k0 = np.empty(r, np.int32)
    km = np.empty(r, np.int32)
    lib().oracle_restart(r, _p(off), _p(values), _p(record_len), _p(alpha), _p(mask), _p(ks),
                         _p(k0), _p(km))
    return ks, k0, km


def fused_logp(hidden: np.ndarray, w: np.ndarray, ids: np.ndarray):
    """Teacher log-probabilities with logits z = h W formed in float64.  Returns (logp, lse, flags)."""
    hidden = np.ascontiguousarray(hidden, dtype=np.uint16)
    w = np.ascontiguousarray(w, dtype=np.uint16)
    n, d = hidden.shape
    d2, vocab = w.shape
    if d2 != d:
        raise ValueError("hidden is [n, d] and w is [d, vocab]")
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    logp = np.empty(n, np.float64)
    lse = np.empty(n, np.float64)
    flags = lib().oracle_fused_logp(n, d, vocab, _p(hidden), _p(w), _p(ids), _p(logp), _p(lse))
    return logp, lse, int(flags)


def _bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact decode of bf16 bit patterns (each is the top half of a binary32), in float64."""
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def fused_logp_matmul(hidden: np.ndarray, w: np.ndarray, ids: np.ndarray, rows_per_call: int = 256):
    """Teacher log-probabilities of z = h W (Eq. 1 with projected logits) with the projection
    done by a library matmul: both bf16 operands are decoded exactly to float64, z is one
    float64 matrix product per block of rows (rows are independent), and each row of z goes
    through logp_rows, the oracle's row log-softmax.  The same definition as fused_logp, for
    row counts where fused_logp's plain loops are too slow; ``w`` is [d, vocab] (a transposed
    view of a [vocab, d] array is taken as is, without copying).  Returns (logp, lse, flags)."""
    hidden = np.ascontiguousarray(hidden, dtype=np.uint16)
    n, d = hidden.shape
    d2, vocab = w.shape
    if d2 != d or w.dtype != np.uint16:
        raise ValueError("hidden is [n, d] and w is [d, vocab], both bf16 bit patterns")
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    w64 = _bf16_bits_to_f64(w)
    logp = np.empty(n, np.float64)
    lse = np.empty(n, np.float64)
    flags = 0
    for i in range(0, n, rows_per_call):
        j = min(n, i + rows_per_call)
        z = _bf16_bits_to_f64(hidden[i:j]) @ w64
        logp[i:j], lse[i:j], f = logp_rows(z, ids[i:j])
        flags |= f
    return logp, lse, flags


def opd_grad(student: np.ndarray, ids: np.ndarray, r: np.ndarray, mask: np.ndarray, scale: float,
             vocab: int | None = None):
    """Token-level OPD loss and gradient w.r.t. the student logits (Eq. 2).
    Returns (grad [n, vocab] float64, loss [n], flags)."""
    student = np.ascontiguousarray(student)
    n, ld = student.shape
    vocab = ld if vocab is None else int(vocab)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    r = np.ascontiguousarray(r, dtype=np.float64)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    if ids.shape != (n,) or r.shape != (n,) or mask.shape != (n,):
        raise ValueError("ids, r and mask need one entry per row")
    grad = np.empty((n, vocab), np.float64)
    loss = np.empty(n, np.float64)
    flags = lib().oracle_opd_grad(n, vocab, ld, _dtype_code(student), _p(student), _p(ids), _p(r),
                                  _p(mask), float(scale), _p(grad), _p(loss))
    return grad, loss, int(flags)
