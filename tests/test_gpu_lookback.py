"""Look-back stress test of the stop test's single-pass scan (Eq. 5 over the new units of each
rollout), the only protocol in the library that crosses workgroups.

libstride_debug.so is the library with the scan compiled with a delay hook: scan tiles picked
by a seeded hash sleep a bounded time before publishing their aggregate, so their successors
find unpublished descriptors and must wait in the look-back.  The waits stay far below the
spin limit, so every wave exits normally.  On 1.25 M token units (about 610 tiles, rollouts up
to 300,000 units long) the cumulative sums must equal the undelayed product library's bit for
bit, and the stops and restart picks must equal the float64 oracle's.  Stops at the first
mismatch.  A second test forces the give-up path: a wait bound of one round makes successors of
delayed tiles give up, and the call must flag it and mark exactly the values that lack a carry.
"""
import ctypes
import sys

import numpy as np
import pytest

from tests import harness as H

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _inputs(seed):
    g = np.random.default_rng(seed)
    sizes = np.concatenate([g.integers(1, 50, size=200), [300000, 2047, 2048, 2049, 250000],
                            g.integers(1000, 40000, size=25)])
    g.shuffle(sizes)
    R = sizes.size
    tto = np.zeros(R + 1, np.int64)
    tto[1:] = np.cumsum(sizes)
    rto = np.arange(R + 1, dtype=np.int32)
    N = int(tto[-1])
    vals = (-np.abs(g.normal(0.5, 0.5, size=N))).astype(np.float32)
    vals[g.random(N) < 0.01] *= 20
    dom = g.integers(0, 3, size=R).astype(np.int32)
    start = (g.random(R) * sizes * 0.3).astype(np.int32)
    mask = (g.random(N) < 0.999).astype(np.uint8)
    return sizes, rto, tto, vals, dom, start, mask


def _call(lib, fn, *args):
    st = getattr(lib, fn)(*args)
    assert st == 0, f"{fn}: {lib.stride_last_error().decode()}"


def _run(lib, lay, v, lam, alpha, start, mask, ws):
    """stride_stop then stride_restart_turn through the given library's C ABI."""
    import torch
    import paper_2609_14636_amd as P
    R, N = lay.n_rollouts, lay.n_tokens
    cum = torch.empty(N, dtype=torch.float64, device="cuda")
    stop, ks, k0, km = (torch.empty(R, dtype=torch.int32, device="cuda") for _ in range(4))
    ret = torch.empty(R, dtype=torch.int64, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    lt, at = P.stride._doubles(lam), P.stride._doubles(alpha)
    vp = lambda t: t.data_ptr()
    _call(lib, "stride_stop", lay.c(), P.STRIDE_UNIT_TOKEN, vp(v), ctypes.cast(lt, ctypes.c_void_p),
          len(lam), vp(start), vp(cum), vp(stop), vp(ret), vp(flags), vp(ws),
          ws.numel(), s)
    _call(lib, "stride_restart_turn", lay.c(), P.STRIDE_UNIT_TOKEN, vp(v), vp(stop),
          ctypes.cast(at, ctypes.c_void_p), len(alpha), vp(mask), vp(ks), vp(k0), vp(km),
          vp(flags), s)
    torch.cuda.synchronize()
    return {k: t.cpu().numpy() for k, t in dict(cum=cum, stop=stop, ret=ret, ks=ks, k0=k0,
                                                  km=km, flags=flags).items()}


def test_lookback_under_delayed_publication():
    import torch
    import paper_2609_14636_amd as P
    sizes, rto, tto, vals, dom, start, mask = _inputs(0)
    R, N = sizes.size, int(tto[-1])
    lam = [-40.0, -400.0, -4000.0]
    alpha = [-0.9, -1.5, -np.inf]
    say(f"[lookback] R={R} N={N} tiles={(N + 2047) // 2048} max rollout {sizes.max()}")
    cum_o, stop_o, ret_o = H.OP.O.stop(tto.copy(), vals.astype(np.float64), np.array(lam)[dom],
                                       start, np.arange(N + 1, dtype=np.int64))
    rec = np.where(stop_o >= 0, stop_o + 1, sizes).astype(np.int32)
    ks_o, k0_o, km_o = H.OP.O.restart(tto.copy(), vals.astype(np.float64), rec,
                                      np.array(alpha)[dom], mask)
    dev = lambda a: torch.from_numpy(a).cuda()
    lay = P.Layout(dev(rto), dev(tto), N, dev(dom))
    v, st, mk = dev(vals), dev(start), dev(mask)
    ws = torch.empty(P.stride_workspace_size(lay, P.STRIDE_UNIT_TOKEN), dtype=torch.uint8,
                     device="cuda")
    # the product library has no delay code
    assert P.library().stride_debug_scan_delay(1, 3, 10) == 2
    ref = _run(P.library(), lay, v, lam, alpha, st, mk, ws)
    assert int(ref["flags"][0]) == 0
    # the undelayed reference against the oracle (same bar as the many-tile parity test)
    rel = np.abs(ref["cum"] - cum_o) / np.maximum(np.abs(cum_o), 1.0)
    assert rel.max() <= H.TOL_CUM_REL, rel.max()
    same = ref["stop"] == stop_o
    for r in np.nonzero(~same)[0]:
        a = tto[r]
        hi = sizes[r] if (ref["stop"][r] < 0 or stop_o[r] < 0) else max(ref["stop"][r], stop_o[r]) + 1
        assert np.any(np.abs(cum_o[a + start[r]:a + hi] - lam[dom[r]]) <= H.BAND), r
    say(f"[lookback] undelayed: max rel cum err {rel.max():.2e}, stops equal {same.sum()}/{R}")

    dbg = P.stride.debug_library()
    try:
        assert dbg.stride_debug_scan_delay(0, 0, 0) == 0
        base = _run(dbg, lay, v, lam, alpha, st, mk, ws)
        for k in ref:
            assert np.array_equal(base[k].view(np.uint8), ref[k].view(np.uint8)), k
        assert dbg.stride_debug_scan_delay(5, 1, 0) == 1      # sleeps outside 1..1000
        assert dbg.stride_debug_scan_delay(5, 1, 1001) == 1
        for seed, one_in, sleeps in ((11, 3, 40), (12, 2, 80), (13, 1, 20), (14, 5, 200)):
            assert dbg.stride_debug_scan_delay(seed, one_in, sleeps) == 0
            out = _run(dbg, lay, v, lam, alpha, st, mk, ws)
            say(f"[lookback] seed {seed}: about 1 in {one_in} tiles delayed up to {sleeps} x "
                f"s_sleep(127); flags {int(out['flags'][0])}")
            assert int(out["flags"][0]) == 0, P.flag_names(int(out["flags"][0]))
            assert np.array_equal(out["cum"].view(np.uint64), ref["cum"].view(np.uint64))
            assert np.array_equal(out["stop"], ref["stop"])
            assert np.array_equal(out["ret"], ref["ret"])
            # stops and restart picks against the oracle where the stop is not in the band
            assert np.array_equal(out["stop"][same], stop_o[same])
            assert np.array_equal(out["ret"][same], ret_o[same])
            for k, o in (("ks", ks_o), ("k0", k0_o), ("km", km_o)):
                assert np.array_equal(out[k][same], o[same]), k
    finally:
        dbg.stride_debug_scan_delay(0, 0, 0)


def test_lookback_gives_up_at_a_tiny_spin_limit():
    """The look-back's give-up path, forced from the host: with every tile delayed before it
    publishes and a wait bound of one round of s_sleep(1), successors give up.  The calls still
    complete with STRIDE_FLAG_SPIN_LIMIT, NaN marks exactly the cumulative values that lacked
    their carry, every finite value equals the normal run bit for bit, rollouts inside one tile
    are untouched, and the library's own bound restored gives the normal results again."""
    import torch
    import paper_2609_14636_amd as P
    sizes, rto, tto, vals, dom, start, mask = _inputs(1)
    R, N = sizes.size, int(tto[-1])
    lam = [-40.0, -400.0, -4000.0]
    alpha = [-0.9, -1.5, -np.inf]
    dev = lambda a: torch.from_numpy(a).cuda()
    lay = P.Layout(dev(rto), dev(tto), N, dev(dom))
    v, st, mk = dev(vals), dev(start), dev(mask)
    ws = torch.empty(P.stride_workspace_size(lay, P.STRIDE_UNIT_TOKEN), dtype=torch.uint8,
                     device="cuda")
    assert P.library().stride_debug_scan_spin_limit(1) == 2  # the product library has no hook
    ref = _run(P.library(), lay, v, lam, alpha, st, mk, ws)
    assert int(ref["flags"][0]) == 0

    dbg = P.stride.debug_library()
    try:
        assert dbg.stride_debug_scan_delay(21, 1, 200) == 0
        assert dbg.stride_debug_scan_spin_limit(1) == 0
        out = _run(dbg, lay, v, lam, alpha, st, mk, ws)
        flags = int(out["flags"][0])
        say(f"[give-up] R={R} N={N}: flags {P.flag_names(flags)}, "
            f"{int(np.isnan(out['cum']).sum())} cumulative values NaN")
        assert flags == P.STRIDE_FLAG_SPIN_LIMIT, P.flag_names(flags)
        nan = np.isnan(out["cum"])
        assert nan.any()
        fin = ~nan
        assert np.array_equal(out["cum"][fin].view(np.uint64), ref["cum"][fin].view(np.uint64))
        # a NaN needs a carry from an earlier tile: its rollout starts before the NaN's tile
        unit_r = np.repeat(np.arange(R), sizes)
        first = tto[:-1][unit_r[nan]]
        assert np.all(first < (np.nonzero(nan)[0] // 2048) * 2048)
        # rollouts that start and end in one tile never wait
        one_tile = (tto[:-1] // 2048) == ((tto[1:] - 1) // 2048)
        for r in np.nonzero(one_tile & (sizes > 0))[0]:
            a, b = tto[r], tto[r + 1]
            assert np.array_equal(out["cum"][a:b].view(np.uint64), ref["cum"][a:b].view(np.uint64))
            assert out["stop"][r] == ref["stop"][r]
        # the library's own bound restored: the normal results again, no flag
        assert dbg.stride_debug_scan_spin_limit(0) == 0
        again = _run(dbg, lay, v, lam, alpha, st, mk, ws)
        assert int(again["flags"][0]) == 0
        for k in ref:
            assert np.array_equal(again[k].view(np.uint8), ref[k].view(np.uint8)), k
    finally:
        dbg.stride_debug_scan_spin_limit(0)
        dbg.stride_debug_scan_delay(0, 0, 0)
