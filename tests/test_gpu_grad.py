"""Token-level OPD loss and gradient (stride_opd_grad) against the float64 oracle.

The oracle's oracle_opd_grad is pinned by central finite differences of the loss of
Eq. (2).  Both sides run the whole path first (score -> stop), each from its own
values; the retained rows follow from each side's own stop decision, and the rows
of a rollout are compared when the two stops agree.
"""
import math
import sys

import numpy as np
import pytest

from synth import workloads as W
from tests import harness as H

pytestmark = pytest.mark.gpu


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


def _run(wl, lam, alpha, scale, sample_rows=None):
    import torch
    import paper_2609_14636_amd as P

    inp = H.device_inputs(wl)
    path = P.Path(inp["layout"], wl.unit)
    path.run(wl.vocab, inp["teachers"], inp["student"], inp["ids"], lam, alpha,
             start_unit=inp["start"], correct_mask=inp["mask"])
    grad = torch.full_like(inp["student"], float("nan"))
    loss = torch.empty(wl.n_tokens, dtype=torch.float32, device="cuda")
    path.grad(wl.vocab, inp["student"], inp["ids"], grad, loss, start_unit=inp["start"],
              scale=scale)
    torch.cuda.synchronize()
    out = path.host()
    rows = np.arange(wl.n_tokens) if sample_rows is None else np.asarray(sample_rows)
    g = grad[torch.from_numpy(rows).cuda()].float().cpu().numpy()[:, :wl.vocab]
    if (wl.ld > wl.vocab):  # padding columns are never written
        pad = grad[torch.from_numpy(rows).cuda()].float().cpu().numpy()[:, wl.vocab:]
        assert np.isnan(pad).all()
    return out, g, loss.cpu().numpy(), rows


def _compare(wl, lam, alpha, scale, sample_rows=None):
    out, g_gpu, loss_gpu, rows = _run(wl, lam, alpha, scale, sample_rows)
    assert out["flags"] == 0, hex(out["flags"])
    ora = H.oracle_all(wl, lam, alpha)
    stop_o = np.array([int(ora[r][1]["stop"][0]) for r in range(wl.n_rollouts)])
    lay = H.OP.Layout(wl.rollout_turn_off, wl.turn_tok_off, wl.domain)
    mask = H.OP.retained_mask(lay, wl.unit, wl.start, stop_o)
    mask_gpu = H.OP.retained_mask(lay, wl.unit, wl.start, out["stop_unit"])
    logp_t = np.concatenate([ora[r][0]["logp_t"] for r in range(wl.n_rollouts)])
    logp_s = np.concatenate([ora[r][0]["logp_s"] for r in range(wl.n_rollouts)])
    same = np.array([out["stop_unit"][r] == stop_o[r] for r in range(wl.n_rollouts)])
    row_rollout = np.repeat(np.repeat(np.arange(wl.n_rollouts), np.diff(wl.rollout_turn_off)),
                            np.diff(wl.turn_tok_off))
    keep = same[row_rollout[rows]]
    rows_k = rows[keep]
    s = wl.student_rows_host(0, wl.n_tokens) if sample_rows is None else \
        np.concatenate([wl.student_rows_host(int(i), 1, 1) for i in rows_k])
    s = s[rows_k] if sample_rows is None else s
    r = (logp_t - logp_s)[rows_k]
    g_o, loss_o, fl = H.OP.O.opd_grad(s, wl.tok[rows_k], r, mask[rows_k], scale, wl.vocab)
    assert fl == 0
    gg = g_gpu[keep]
    c = np.abs(scale * r)[:, None]
    tol = 4e-3 * np.abs(g_o) + 2e-5 * (c + 1.0)
    bad = np.abs(gg - g_o) > tol
    assert not bad.any(), (np.argwhere(bad)[:5], gg[bad][:5], g_o[bad][:5])
    dl = np.abs(loss_gpu[rows_k] - loss_o)
    assert np.all(dl <= 2e-3 * (np.abs(loss_o) + abs(scale))), dl.max()
    assert np.array_equal(mask_gpu[rows_k], mask[rows_k])
    assert np.all(g_gpu[~mask_gpu[rows].astype(bool)] == 0.0)
    say(f"[grad {wl.name}] rows {rows_k.size} (retained {int(mask[rows_k].sum())}), "
        f"max |d g| {np.max(np.abs(gg - g_o)):.2e}, max |d loss| {dl.max():.2e}, "
        f"stops equal {int(same.sum())}/{wl.n_rollouts}")


def test_grad_tiny_fp32():
    wl = W.make("tiny")
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = H.thresholds(wl, sc)
    _compare(wl, lam, alpha, scale=1.0 / 100)


def test_grad_reasoning_token_units():
    wl = W.make("reasoning", seed=21, scale=dict(R=2, tok=900, vocab=4099))
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = H.thresholds(wl, sc)
    _compare(wl, lam, alpha, scale=0.5)


def test_grad_ragged_with_prefix_offsets():
    g = np.random.default_rng(3)
    lengths = [g.integers(1, 30, size=int(g.integers(1, 6))) for _ in range(9)]
    from tests.test_gpu_parity import _custom, _custom_thresholds
    wl = _custom(41, 513, W.BF16, lengths, n_teachers=2)
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = _custom_thresholds(wl, sc)
    _compare(wl, lam, alpha, scale=1.0)


def test_grad_full_vocab_sampled_rows():
    wl = W.make("agentic", seed=1005, scale=dict(R=2))
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = H.thresholds(wl, sc)
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([rng.integers(0, wl.n_tokens, size=24), [0, wl.n_tokens - 1]]))
    _compare(wl, lam, alpha, scale=1.0 / wl.n_tokens, sample_rows=rows)


@pytest.mark.parametrize("dtype", [W.BF16, W.F32])
def test_grad_million_entry_vocabulary(dtype):
    """Gradient rows of 2^20 + 5 entries (a ragged last word, padding columns left unwritten),
    every row and element against the oracle."""
    g = np.random.default_rng(4040 + dtype)
    lengths = [g.integers(1, 10, size=3) for _ in range(3)]
    from tests.test_gpu_parity import _custom, _custom_thresholds
    wl = _custom(91 + dtype, (1 << 20) + 5, dtype, lengths)
    sc = H.oracle_scores(wl, range(wl.n_rollouts))
    lam, alpha = _custom_thresholds(wl, sc)
    _compare(wl, lam, alpha, scale=1.0 / wl.n_tokens)
