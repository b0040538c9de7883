"""The C ABI from plain C: tests/c_client.c (built by tests/c_client_build.py) reads a reduced
workload from files, runs stride_score -> stride_stop -> stride_restart_turn through libstride.so
with device memory from hipMalloc, and writes its outputs; they are compared with the float64
oracle element by element.  Nothing on the client's side of the boundary is Python or torch.
With --graph the client also captures the step into a HIP graph and checks its replays."""
import os
import subprocess
import sys

import numpy as np
import pytest

from synth import workloads as W
from tests import harness as H
from tests import c_client_build as CB

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _write_inputs(wl, lam, alpha, d):
    R, T, N, V = wl.n_rollouts, wl.n_turns, wl.n_tokens, wl.vocab
    U = T if wl.unit == W.UNIT_TURN else N
    with open(os.path.join(d, "meta.txt"), "w") as f:
        f.write(f"{R} {T} {N} {V} {len(lam)} {wl.unit} {int(wl.start is not None)} "
                f"{int(wl.mask is not None)} {int(wl.domain is not None)}\n")
    wl.rollout_turn_off.astype(np.int32).tofile(os.path.join(d, "rto.i32"))
    wl.turn_tok_off.astype(np.int64).tofile(os.path.join(d, "tto.i64"))
    # the routed teacher's rows: with one teacher matrix every row reads its own domain's logits
    np.ascontiguousarray(wl.teacher_rows_host(0, N)[:, :V]).tofile(os.path.join(d, "teacher.bf16"))
    np.ascontiguousarray(wl.student_rows_host(0, N)[:, :V]).tofile(os.path.join(d, "student.bf16"))
    wl.tok.astype(np.int32).tofile(os.path.join(d, "ids.i32"))
    np.asarray(lam, np.float64).tofile(os.path.join(d, "lambda.f64"))
    np.asarray(alpha, np.float64).tofile(os.path.join(d, "alpha.f64"))
    if wl.start is not None:
        wl.start.astype(np.int32).tofile(os.path.join(d, "start.i32"))
    if wl.mask is not None:
        assert wl.mask.size == U
        wl.mask.astype(np.uint8).tofile(os.path.join(d, "mask.u8"))
    if wl.domain is not None:
        wl.domain.astype(np.int32).tofile(os.path.join(d, "domain.i32"))


def _read_outputs(wl, d):
    R, T, N = wl.n_rollouts, wl.n_turns, wl.n_tokens
    U = T if wl.unit == W.UNIT_TURN else N
    rd = lambda name, dt, n: np.fromfile(os.path.join(d, "out_" + name), dtype=dt, count=n)  # noqa: E731
    return {"logp_t": rd("logp_t", np.float32, N), "logp_s": rd("logp_s", np.float32, N),
            "kl": rd("kl", np.float32, N), "turn_mean": rd("turn_mean", np.float64, T),
            "cum": rd("cum", np.float64, U), "stop_unit": rd("stop", np.int32, R),
            "retained": rd("retained", np.int64, R), "k_star": rd("k_star", np.int32, R),
            "k0": rd("k0", np.int32, R), "k_max": rd("k_max", np.int32, R),
            "flags": int(rd("flags", np.uint32, 1)[0])}


@pytest.mark.parametrize("name,seed,scale,start", [
    ("agentic", 2001, dict(R=3, turns=5, tok_lo=20, tok_hi=60, vocab=1000), [1, 0, 2]),
    ("multi", 2002, dict(R=4, turns=3, tok=40, vocab=1003), None),
    ("reasoning", 2003, dict(R=2, tok=700, vocab=999), [0, 150]),
])
def test_c_client_matches_the_oracle(name, seed, scale, start, tmp_path):
    _client_against_the_oracle(name, seed, scale, start, tmp_path, graph=False)


def test_c_client_graph_replay(tmp_path):
    """The client captures score -> stop -> restart into a HIP graph with hipStreamBeginCapture,
    overwrites every output, replays the graph three times and requires each replay to equal its
    eager run bit for bit; the eager outputs are compared with the oracle as above."""
    _client_against_the_oracle("agentic", 2004, dict(R=3, turns=4, tok_lo=10, tok_hi=50, vocab=777),
                               [0, 1, 0], tmp_path, graph=True)


def _client_against_the_oracle(name, seed, scale, start, tmp_path, graph):
    assert os.path.exists(CB.BIN), f"{CB.BIN} is missing: build() compiles it"
    wl = W.make(name, seed=seed, scale=scale)
    if start is not None:
        wl.start = np.array(start, np.int32)
    say(f"[c client] {name}: R={wl.n_rollouts} T={wl.n_turns} N={wl.n_tokens} V={wl.vocab} "
        f"unit={wl.unit}")
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = H.thresholds(wl, sc)
    ora = {r: (sc[r], H.oracle_rollout(wl, r, sc[r], lam, alpha)) for r in sc}
    _write_inputs(wl, lam, alpha, str(tmp_path))
    r = subprocess.run([CB.BIN, str(tmp_path)] + (["--graph"] if graph else []),
                       capture_output=True, text=True, timeout=120)
    say(r.stdout.strip(), r.stderr.strip())
    assert r.returncode == 0, r.stderr
    if graph:
        assert "replayed 3 times" in r.stdout, r.stdout
    out = _read_outputs(wl, str(tmp_path))
    assert out["flags"] == 0, hex(out["flags"])
    rep = H.compare(wl, out, ora, lam, alpha)
    H.assert_invariants(out, wl)
    say(f"[c client] {name}: {rep}")
