"""Exact full-vocabulary reverse KL per token (stride_score with kl_full) against the oracle.

KL(pi_S || pi_T) = sum_v pi_S(v) log(pi_S(v) / pi_T(v)), the divergence whose sequence-level
form OPD minimises (Sec. 3.1).  The oracle's oracle_exact_kl is pinned by the Gibbs identity
(E_S[log pi_S(y) - log pi_T(y)] = KL, KL >= 0, = 0 iff the logits differ by a constant).
"""
import math
import sys

import numpy as np
import pytest

from synth import workloads as W
from tests import harness as H

pytestmark = pytest.mark.gpu
TOL_KL_FULL = 4e-3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,scale", [
    ("tiny", None),
    ("agentic", dict(R=1, turns=3)),
    ("multi", dict(R=3, turns=2, tok=100)),
    ("reasoning", dict(R=1, tok=700, vocab=4099)),
])
def test_exact_kl_parity(name, scale):
    wl = W.make(name, seed=11, scale=scale)
    sc = H.oracle_scores(wl, range(wl.n_rollouts), exact_kl=True)
    lam, alpha = [-1e9] * wl.n_teachers, [-1e9] * wl.n_teachers  # scores only
    gpu = H.run_gpu(wl, lam, alpha, exact_kl=True)
    assert gpu["flags"] == 0, hex(gpu["flags"])
    want = np.concatenate([sc[r]["kl_full"] for r in range(wl.n_rollouts)])
    d = np.max(np.abs(gpu["kl_full"] - want))
    assert d <= TOL_KL_FULL, d
    # never negative: the kernel clamps a rounding residue below 0 at 0, so this checks the
    # output contract; the arithmetic is checked by the parity bound above and by the zero cases
    assert np.all(gpu["kl_full"] >= 0.0), gpu["kl_full"].min()
    # the paired pass gives the same sampled-token log-probabilities as the row pass
    for k in ("logp_t", "logp_s"):
        o = np.concatenate([sc[r][k] for r in range(wl.n_rollouts)])
        assert np.max(np.abs(gpu[k] - o)) <= H.TOL_LOGP
    say(f"[kl_full {name}] max |d| = {d:.2e}, mean KL = {want.mean():.3f}")


def test_exact_kl_on_the_one_wavefront_kernel():
    """65,600 tokens (the paired pass shares rows among eight wavefronts only below 65,536), with a
    ragged vocabulary of 1,001 entries: the exact KL and both log-probabilities of every token
    against the oracle."""
    wl = W.make("reasoning", seed=13, scale=dict(R=4, tok=16400, vocab=1001))
    assert wl.n_tokens >= 65536
    sc = H.oracle_scores(wl, range(wl.n_rollouts), exact_kl=True)
    lam, alpha = [-1e9], [-1e9]
    gpu = H.run_gpu(wl, lam, alpha, exact_kl=True)
    assert gpu["flags"] == 0, hex(gpu["flags"])
    want = np.concatenate([sc[r]["kl_full"] for r in range(wl.n_rollouts)])
    d = np.max(np.abs(gpu["kl_full"] - want))
    assert d <= TOL_KL_FULL, d
    for k in ("logp_t", "logp_s"):
        o = np.concatenate([sc[r][k] for r in range(wl.n_rollouts)])
        assert np.max(np.abs(gpu[k] - o)) <= H.TOL_LOGP
    say(f"[kl_full one-wavefront] N={wl.n_tokens} V={wl.vocab}: max |d| = {d:.2e}")


def test_exact_kl_zero_for_shifted_teacher_and_inf_entries():
    """Teacher = student + c gives KL = 0; a -inf teacher entry where the student has mass
    gives KL = +inf; a -inf entry in both rows contributes nothing."""
    import torch
    import paper_2609_14636_amd as P
    V, N = 1000, 6
    g = torch.Generator().manual_seed(0)
    s = torch.randn(N, V, generator=g) * 2
    t = s + 3.25
    t[1, 5] = float("-inf")              # student has mass there -> +inf
    t[2, 7] = float("-inf")
    s[2, 7] = float("-inf")              # both -inf -> no contribution
    s_d, t_d = s.cuda(), t.cuda()
    lay = P.Layout(torch.tensor([0, 1], dtype=torch.int32).cuda(),
                   torch.tensor([0, N], dtype=torch.int64).cuda(), N)
    path = P.Path(lay, P.STRIDE_UNIT_TURN, exact_kl=True)
    ids = torch.zeros(N, dtype=torch.int32).cuda()
    path.score(V, [t_d], s_d, ids)
    torch.cuda.synchronize()
    kl = path.kl_full.cpu().numpy()
    assert abs(kl[0]) < 1e-4 and abs(kl[3]) < 1e-4 and abs(kl[2]) < 1e-4, kl
    assert (kl[np.isfinite(kl)] >= 0.0).all(), kl   # the output contract (clamped at 0)
    assert math.isinf(kl[1]) and kl[1] > 0
    want = H.OP.O.exact_kl(t.numpy(), s.numpy())
    assert math.isinf(want[1]) and abs(want[2]) < 1e-12
