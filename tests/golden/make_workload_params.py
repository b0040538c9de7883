"""Write tests/golden/workload_params.json: the thresholds of the full-size synthetic workloads.

Calls only the float64 oracle (on host-generated rows; teacher rows suffice, since lambda and
alpha depend on teacher log-probabilities only) and the threshold rules of
tests/workload_params.py.  Run from the repository root:

    python tests/golden/make_workload_params.py [--threads 8]
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import oracle as O  # noqa: E402
from synth import workloads as W  # noqa: E402
from tests import workload_params as WP  # noqa: E402

OUT = os.path.join(ROOT, "tests", "golden", "workload_params.json")


def teacher_logp(wl, threads):
    out = np.empty(wl.n_tokens, np.float64)
    for r in range(wl.n_rollouts):
        a, b = wl.rollout_rows(r)
        step = 2048
        for i in range(a, b, step):
            k = min(step, b - i)
            t = wl.teacher_rows_host(i, k, threads)
            out[i:i + k], _, fl = O.logp_rows(t, wl.tok[i:i + k], wl.vocab)
            assert fl == 0
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=8)
    ap.add_argument("--only", default=None)
    args = ap.parse_args()
    res = {"about": "lambda / alpha per domain of each full-size workload (name:seed), from the "
                    "float64 oracle by the rules in tests/workload_params.py; written by "
                    "tests/golden/make_workload_params.py", "workloads": {}}
    if os.path.exists(OUT):
        with open(OUT) as f:
            res["workloads"].update(json.load(f)["workloads"])
    for name, seed in (("tiny", 1001), ("agentic", 1001), ("reasoning", 1001), ("multi", 1001)):
        if args.only and name != args.only:
            continue
        wl = W.make(name, seed)
        t0 = time.time()
        lp = teacher_logp(wl, args.threads)
        tm, _ = O.turn_mean(wl.turn_tok_off, lp)
        if name == "tiny":
            lam, alpha = WP.tiny_thresholds(tm, wl.rollout_turn_off, wl.planted)
        elif name in ("agentic", "multi"):
            lam, alpha = WP.agentic_thresholds(tm, wl.rollout_turn_off, wl.planted, wl.domain,
                                               wl.n_teachers)
        else:
            lam, alpha = WP.reasoning_thresholds(lp, wl.unit_off())
        dom = np.zeros(wl.n_rollouts, np.int64) if wl.domain is None else wl.domain
        vals = tm if wl.unit == W.UNIT_TURN else lp
        uoff = wl.unit_off()
        cum, stop, _ = O.stop(uoff, vals, np.array(lam)[dom])
        rec = np.where(stop >= 0, stop + 1, np.diff(uoff)).astype(np.int32)
        ks, k0, km = O.restart(uoff, vals, rec, np.array(alpha)[dom], wl.mask)
        # distance of each rollout's cumulative values to its lambda, for the 1e-3 band rule
        gap = [float(np.min(np.abs(cum[uoff[r]:uoff[r + 1]] - lam[dom[r]]))) for r in range(wl.n_rollouts)]
        res["workloads"][f"{name}:{seed}"] = {
            "lambda": lam, "alpha": [a if math.isfinite(a) else "-inf" for a in alpha],
            "oracle_stop": stop.tolist(), "oracle_k_star": ks.tolist(), "oracle_k0": k0.tolist(),
            "oracle_k_max": km.tolist(), "oracle_min_gap_to_lambda": gap,
            "oracle_turn_mean": tm.tolist() if wl.unit == W.UNIT_TURN else None,
            "seconds": round(time.time() - t0, 1)}
        print(name, lam, alpha, stop.tolist(), f"{time.time() - t0:.1f}s", flush=True)
        with open(OUT, "w") as f:
            json.dump(res, f, indent=1)


if __name__ == "__main__":
    main()
