"""Full-size workloads on the GPU, in the launch configuration the benchmark times.

At full size (26-120 GB of logits) the oracle cannot score every row within a
test, so: (1) sampled rollouts are compared element by element with the oracle
on host-generated rows; (2) every rollout's turn means, stop, K_max, k* and K0
are compared with the oracle values stored in tests/golden/workload_params.json
(written by tests/golden/make_workload_params.py, which calls only the oracle);
(3) size-independent invariants hold on every row.
"""
import json
import math
import os
import sys

import numpy as np
import pytest

from synth import workloads as W
from tests import harness as H

pytestmark = pytest.mark.gpu
PARAMS = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "workload_params.json")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _params(name, seed=1001):
    with open(PARAMS) as f:
        e = json.load(f)["workloads"][f"{name}:{seed}"]
    lam = [float(x) for x in e["lambda"]]
    alpha = [float(x) for x in e["alpha"]]
    return e, lam, alpha


@pytest.fixture(autouse=True)
def _free():
    import torch
    assert torch.cuda.is_available()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,sample", [("agentic", [0, 15]), ("reasoning", [5]),
                                         ("multi", [0, 31])])
def test_full_size(name, sample):
    e, lam, alpha = _params(name)
    wl = W.make(name, 1001)
    say(f"[full] {name}: R={wl.n_rollouts} T={wl.n_turns} N={wl.n_tokens} "
        f"({2 * wl.logits_bytes() / 1e9:.1f} GB of logits)")
    gpu = H.run_gpu(wl, lam, alpha)
    assert gpu["flags"] == 0, hex(gpu["flags"])
    H.assert_invariants(gpu, wl)
    # every rollout: decisions and turn means against the stored oracle values
    if e.get("oracle_turn_mean") is not None:
        d = np.max(np.abs(gpu["turn_mean"] - np.array(e["oracle_turn_mean"])))
        assert d <= H.TOL_LOGP, d
        say(f"[full] {name}: max |d turn mean| over all {wl.n_turns} turns = {d:.2e}")
    gap = np.array(e["oracle_min_gap_to_lambda"])
    for key, ok in (("stop_unit", "oracle_stop"), ("k_star", "oracle_k_star"),
                    ("k_max", "oracle_k_max"), ("k0", "oracle_k0")):
        want = np.array(e[ok])
        diff = np.nonzero(gpu[key] != want)[0]
        assert np.all(gap[diff] <= H.BAND), (key, diff, gpu[key][diff], want[diff])
    say(f"[full] {name}: stops {gpu['stop_unit'].tolist()}")
    # sampled rollouts element by element
    ora = H.oracle_all(wl, lam, alpha, rollouts=sample)
    rep = H.compare(wl, gpu, ora, lam, alpha)
    say(f"[full] {name}: sampled {sample}: {rep}")
