"""The usage example in README.md, run as written and checked against the float64 oracle."""
import re
import sys
from pathlib import Path

import numpy as np
import pytest

from tests import harness as H

pytestmark = pytest.mark.gpu


def _example_source() -> str:
    text = (Path(__file__).resolve().parent.parent / "README.md").read_text()
    sec = text[text.index("## Using it from PyTorch"):]
    return re.search(r"```python\n(.*?)```", sec, re.S).group(1)


def test_readme_example_runs_and_matches_the_oracle():
    import torch
    ns = {}
    exec(compile(_example_source(), "README.md example", "exec"), ns)
    torch.cuda.synchronize()
    path, teacher, student, ids = ns["path"], ns["teacher"], ns["student"], ns["ids"]
    t = teacher.view(torch.int16).cpu().numpy().view(np.uint16)
    s = student.view(torch.int16).cpu().numpy().view(np.uint16)
    y = ids.cpu().numpy()
    lt, _, f1 = H.OP.O.logp_rows(t, y, ns["V"])
    ls, _, f2 = H.OP.O.logp_rows(s, y, ns["V"])
    assert f1 == 0 and f2 == 0
    out = path.host()
    assert out["flags"] == 0
    assert np.max(np.abs(out["logp_t"] - lt)) <= H.TOL_LOGP
    assert np.max(np.abs(out["logp_s"] - ls)) <= H.TOL_LOGP
    tto = np.array([0, 3, 5, 9], np.int64)
    tm, _ = H.OP.O.turn_mean(tto, lt)
    assert np.max(np.abs(out["turn_mean"] - tm)) <= H.TOL_LOGP
    # the stop test and restart pick on the oracle's turn means
    lay = H.OP.Layout(np.array([0, 2, 3], np.int32), tto, None)
    ref = H.OP.stop_and_restart(lay, lt, [-20.0], [-13.0], 0, None, None)
    near = np.abs(ref["cum"] + 20.0) <= H.BAND
    if not near.any():
        assert np.array_equal(out["stop_unit"], ref["stop"])
        assert np.array_equal(out["k_star"], ref["k_star"])
        assert np.array_equal(out["k0"], ref["k0"])
        assert np.array_equal(out["k_max"], ref["k_max"])
    print("[readme example] stop", out["stop_unit"].tolist(), "k*", out["k_star"].tolist(),
          "turn means", np.round(out["turn_mean"], 3).tolist(), flush=True)
    sys.stdout.flush()
