"""Algorithm 1 over several training iterations on synthetic tasks (needs a GPU).

Each iteration: plan K0 from the record H(x) (host store), reuse the first K0 units of
the recorded rollout as context, generate the remaining turns with the current
"student", run the early-stop test on the new turns only (stride_stop with
start_unit = K0), record the generated units, then apply a toy training update that
raises the quality of the retained turns.  The per-turn values stand in for the
teacher's turn means.  Checked every iteration: the GPU stop equals the oracle's on
the same values, and the record holds exactly the generated units.  Over the
iterations the restart point K0 moves towards later turns (Sec. 4.2 step 4).
"""
import numpy as np
import pytest

from oracle import oracle as O

pytestmark = pytest.mark.gpu


def test_replay_restart_point_moves_right():
    import torch
    import paper_2609_14636_amd as P
    rng = np.random.default_rng(12)
    X, K = 48, 12
    quality = np.full((X, K), -0.7) + rng.normal(0, 0.05, size=(X, K))
    hard = rng.integers(2, K, size=X)                      # an error-prone turn per task
    quality[np.arange(X), hard] = -2.5
    lam, alpha, eta = [-2.6], [-0.8], 0.35
    rec = P.Records()
    k0_hist = []
    for it in range(8):
        ks, k0, km = rec.plan(np.arange(X), alpha[0])
        k0_hist.append(k0.mean())
        values = np.empty((X, K))
        for x in range(X):
            old = rec.get(x)
            values[x] = quality[x] + rng.normal(0, 0.03, size=K)
            if old is not None:                              # reused prefix: recorded values
                values[x, :k0[x]] = old[0][:k0[x]]
        off = np.arange(X + 1, dtype=np.int64) * K
        flat = values.reshape(-1)
        # X rollouts of K turns (one placeholder row per turn: only turn values are used)
        lay = P.Layout(torch.from_numpy((np.arange(X + 1) * K).astype(np.int32)).cuda(),
                       torch.arange(X * K + 1, dtype=torch.int64).cuda(), X * K)
        v = torch.from_numpy(flat).cuda()
        start = torch.from_numpy(k0.astype(np.int32)).cuda()
        cum = torch.empty(X * K, dtype=torch.float64, device="cuda")
        stop = torch.empty(X, dtype=torch.int32, device="cuda")
        ws = torch.empty(P.stride_workspace_size(lay, P.STRIDE_UNIT_TURN), dtype=torch.uint8,
                         device="cuda")
        P.stride_stop(lay, P.STRIDE_UNIT_TURN, v, lam, start, cum, stop, None, None, ws)
        torch.cuda.synchronize()
        s = stop.cpu().numpy()
        _, s_o, _ = O.stop(off, flat, np.full(X, lam[0]), k0.astype(np.int32))
        assert np.array_equal(s, s_o)
        for x in range(X):
            end = s[x] + 1 if s[x] >= 0 else K
            rec.put(x, values[x, :end])
            assert rec.get(x)[0].size == end
            # toy update: retained new turns improve
            quality[x, k0[x]:end] += eta
    print("mean K0 per iteration:", np.round(k0_hist, 2), flush=True)
    assert k0_hist[-1] > k0_hist[1] + 0.5
