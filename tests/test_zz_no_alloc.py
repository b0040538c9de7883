"""stride_stop_noalloc (the stop test with its scratch in the library's fixed per-GPU array)
against stride_stop with a caller workspace: two calls in a row, the second on a smaller layout,
each compared with stride_stop on the same inputs.  The cumulative sums are associated in the
same fixed order by the same kernels, so they must agree bit for bit; stop indices and retained
row counts are integers and must be equal.  Every call goes through the C ABI of libstride.so.
"""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _layout(g, sizes, n_turn_per_rollout):
    """Token rows per rollout split into turns; returns host offsets."""
    R = len(sizes)
    turns = []
    for n in sizes:
        k = min(n_turn_per_rollout, n)
        cuts = np.sort(g.choice(np.arange(1, n), size=k - 1, replace=False)) if k > 1 else []
        edges = np.concatenate([[0], cuts, [n]]).astype(np.int64)
        turns.append(np.diff(edges))
    per_roll = np.array([len(t) for t in turns], np.int32)
    rto = np.zeros(R + 1, np.int32)
    rto[1:] = np.cumsum(per_roll)
    tl = np.concatenate(turns)
    tto = np.zeros(tl.size + 1, np.int64)
    tto[1:] = np.cumsum(tl)
    return rto, tto


def _compare(unit, rto, tto, vals, dom, start, lam):
    import torch
    import paper_2609_14636_amd as P
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    N = int(tto[-1])
    lay = P.Layout(dev(rto), dev(tto), N, dev(dom))
    R = lay.n_rollouts
    U = lay.n_units(unit)
    v = dev(vals)
    st = dev(start)
    ws = torch.empty(max(P.stride_workspace_size(lay, unit), 256), dtype=torch.uint8, device="cuda")
    out = []
    for noalloc in (False, True):
        cum = torch.full((U,), 7.0, dtype=torch.float64, device="cuda")
        stop = torch.full((R,), 99, dtype=torch.int32, device="cuda")
        ret = torch.full((R,), 99, dtype=torch.int64, device="cuda")
        flags = torch.zeros(1, dtype=torch.int32, device="cuda")
        if noalloc:
            P.stride_stop_noalloc(lay, unit, v, lam, st, cum, stop, ret, flags)
        else:
            P.stride_stop(lay, unit, v, lam, st, cum, stop, ret, flags, ws)
        torch.cuda.synchronize()
        out.append((cum.cpu().numpy(), stop.cpu().numpy(), ret.cpu().numpy(), int(flags.item())))
    (c0, s0, r0, f0), (c1, s1, r1, f1) = out
    assert f0 == 0 and f1 == 0, (f0, f1)
    assert np.array_equal(c0.view(np.uint64), c1.view(np.uint64))
    assert np.array_equal(s0, s1)
    assert np.array_equal(r0, r1)
    return int((s1 >= 0).sum()), R


def test_noalloc_stop_matches_workspace_stop_two_calls():
    g = np.random.default_rng(2024)
    # call 1: token units, 400 rollouts, 1.25 M units (about 610 scan tiles) with long rollouts
    # spanning many tiles, ragged tails, K0 offsets and three domains
    sizes = np.concatenate([g.integers(1, 60, size=360), [300000, 2047, 2048, 2049, 250000],
                            g.integers(1000, 40000, size=35)])
    g.shuffle(sizes)
    rto, tto = _layout(g, sizes, 4)
    N = int(tto[-1])
    R = sizes.size
    vals = (-np.abs(g.normal(0.5, 0.5, size=N))).astype(np.float32)
    dom = g.integers(0, 3, size=R).astype(np.int32)
    start = (g.random(R) * sizes * 0.3).astype(np.int32)
    lam = [-40.0, -400.0, -4000.0]
    say(f"[noalloc] call 1: token units, R={R} N={N}")
    stops, _ = _compare(1, rto, tto, vals, dom, start, lam)
    say(f"[noalloc] call 1: {stops}/{R} stops, outputs identical")
    assert stops > 0

    # call 2: turn units on a smaller layout (the scratch still holds call 1's descriptors)
    sizes2 = g.integers(100, 900, size=37)
    rto2, tto2 = _layout(g, sizes2, 12)
    T2 = int(rto2[-1])
    means = -np.abs(g.normal(3.0, 1.0, size=T2))
    dom2 = g.integers(0, 2, size=sizes2.size).astype(np.int32)
    per = np.diff(rto2)
    start2 = (g.random(sizes2.size) * per * 0.5).astype(np.int32)
    lam2 = [-12.0, -20.0]
    say(f"[noalloc] call 2: turn units, R={sizes2.size} T={T2}")
    stops2, R2 = _compare(0, rto2, tto2, means, dom2, start2, lam2)
    say(f"[noalloc] call 2: {stops2}/{R2} stops, outputs identical")
    assert stops2 > 0


def test_noalloc_stop_at_the_largest_layout_it_takes():
    """The largest layout of two-token rollouts whose scratch (256 + 8 (R + 1) + 16 ceil(U / 2048)
    bytes, each part rounded up to 256) fits the fixed 1 MiB array: accepted, and equal to
    stride_stop bit for bit; one more rollout is rejected before any launch."""
    import paper_2609_14636_amd as P
    r256 = lambda x: (x + 255) // 256 * 256  # noqa: E731
    need = lambda R: 256 + r256(8 * (R + 1)) + r256(16 * ((2 * R + 2047) // 2048))  # noqa: E731
    R = 1
    while need(R + 1) <= (1 << 20):
        R += 1
    assert need(R) <= (1 << 20) < need(R + 1)
    g = np.random.default_rng(131)
    rto = np.arange(R + 1, dtype=np.int32)
    tto = (np.arange(R + 1) * 2).astype(np.int64)
    vals = (-np.abs(g.normal(1.0, 0.5, size=2 * R))).astype(np.float32)
    dom = g.integers(0, 2, size=R).astype(np.int32)
    start = g.integers(0, 2, size=R).astype(np.int32)
    say(f"[noalloc] largest layout: R={R}, {2 * R} token units, scratch {need(R)} bytes")
    stops, _ = _compare(1, rto, tto, vals, dom, start, [-1.0, -1.6])
    say(f"[noalloc] largest layout: {stops}/{R} stops, outputs identical")
    assert 0 < stops < R

    import torch
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    R1 = R + 1
    lay = P.Layout(dev(np.arange(R1 + 1, dtype=np.int32)), dev((np.arange(R1 + 1) * 2).astype(np.int64)),
                   2 * R1, None)
    cum = torch.empty(2 * R1, dtype=torch.float64, device="cuda")
    stop = torch.empty(R1, dtype=torch.int32, device="cuda")
    v = torch.zeros(2 * R1, dtype=torch.float32, device="cuda")
    with pytest.raises(P.stride.StrideError) as ei:
        P.stride_stop_noalloc(lay, 1, v, [-1.0], None, cum, stop, None, None)
    assert ei.value.status == 2
