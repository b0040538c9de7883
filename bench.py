"""Benchmark of the STRIDE scoring / early-stop / restart path on one MI355X.

One step = stride_score -> stride_stop -> stride_restart_turn over one batch of
synthetic rollouts whose logits are already resident in HBM.  Prints one JSON
line with scored tokens/s, the roofline of the dominant kernel (the row
scoring kernel, timed with HIP events on the stream it runs on) and the
float64 CPU oracle timed on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--workload reasoning|agentic|multi|tiny|fused]

The default workload is the long single-turn reasoning batch (8 rollouts x
16,384 tokens, token units, V = 151,936 bf16): the largest of the
logits-streaming workloads, 79.7 GB of logits per step.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "scored tokens/sec (logp+KL+stop scan) and % of HBM peak, 1 MI355X"
PARAMS = os.path.join(ROOT, "tests", "golden", "workload_params.json")
TRAFFIC = os.path.join(ROOT, "profiles", "traffic.json")
FUSED_SRC = os.path.join(ROOT, "paper_2609_14636_amd", "csrc", "fused.hip")
SCORE_SRC = os.path.join(ROOT, "paper_2609_14636_amd", "csrc", "score.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def stats_ms(pairs):
    """mean, median and min of the elapsed times (ms) of a list of (start, end) events."""
    t = np.array([a.elapsed_time(b) for a, b in pairs], dtype=np.float64)
    return {"mean": float(t.mean()), "median": float(np.median(t)), "min": float(t.min())}


def check_outputs(out: dict, wl) -> None:
    """Properties the timed outputs must have at any size (a guard against timing a broken
    run, not a parity check): finite log-probabilities at most 0, K0 = max(k*, 0),
    k* < K_max <= the recorded units, and stops inside each rollout."""
    for k in ("logp_t", "logp_s"):
        v = out.get(k)
        if v is not None and not (np.all(np.isfinite(v)) and np.all(v <= 0.0)):
            raise SystemExit(f"benchmark outputs: {k} not finite or above 0")
    ks, k0, km, st = out["k_star"], out["k0"], out["k_max"], out["stop_unit"]
    n_units = np.diff(wl.unit_off())
    rec = np.where(st >= 0, st + 1, n_units)
    ok = (np.array_equal(k0, np.maximum(ks, 0)) and np.all((ks == -1) == (km == 0))
          and np.all(ks < np.maximum(km, 1)) and np.all(km <= rec) and np.all(st < n_units))
    if not ok:
        raise SystemExit("benchmark outputs: restart pick or stop outside its bounds")


def workload_params(name: str, seed: int):
    with open(PARAMS) as f:
        p = json.load(f)
    key = f"{name}:{seed}"
    if key not in p["workloads"]:
        raise SystemExit(f"no thresholds for {key} in {PARAMS}")
    e = p["workloads"][key]
    return [float(x) for x in e["lambda"]], [float(x) for x in e["alpha"]]


def source_digest(path: str = None) -> str:
    with open(path or SCORE_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def shape_label(wl) -> str:
    """'R rollouts x K turns' with K per rollout (or its range when rollouts differ)."""
    per = np.diff(np.asarray(wl.rollout_turn_off))
    k = f"{int(per.min())}" if per.min() == per.max() else f"{int(per.min())}-{int(per.max())}"
    return f"{wl.n_rollouts} rollouts x {k} turns ({wl.n_turns} turns)"


def measured_traffic(workload: str, kernel_src: str = None, key: str = "score_hip_sha256_16"):
    """HBM bytes per launch of the dominant kernel from committed rocprofv3 counters, if they
    were taken on the current kernel source; else None.

    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are each scaled by the ratio of known bytes to
    the same counter's reading on a one-dispatch plain copy (torch.neg on float32)."""
    if not os.path.exists(TRAFFIC):
        return None
    with open(TRAFFIC) as f:
        t = json.load(f)
    e = t.get(workload)
    if not e or e.get(key) != source_digest(kernel_src):
        return None
    c = t["copy_calibration"]
    k_fetch = c["bytes"] / (c["fetch_kib"] * 1024.0)
    k_write = c["bytes"] / (c["write_kib"] * 1024.0)
    return e["fetch_kib"] * 1024.0 * k_fetch + e["write_kib"] * 1024.0 * k_write


def measured_mfma_busy():
    """Matrix-core busy fraction of the fused projection kernel from committed rocprofv3
    counters (SQ_VALU_MFMA_BUSY_CYCLES over four SIMDs per CU times GRBM_GUI_ACTIVE per XCD),
    if they were taken on the current fused.hip; else None."""
    if not os.path.exists(TRAFFIC):
        return None
    with open(TRAFFIC) as f:
        e = json.load(f).get("fused_mfma")
    if not e or e.get("fused_hip_sha256_16") != source_digest(FUSED_SRC):
        return None
    return {k: e[k] for k in ("busy_frac", "clock_GHz", "counters")}


def cpu_baseline(wl, lam, alpha, budget_s: float):
    """Float64 oracle on whole rollouts of the workload, in order, until budget_s seconds of
    oracle compute (at least one rollout); compute time only, host input generation excluded."""
    from tests import harness as H

    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    rows, rs = 0, []
    t_gen, t_ora = 0.0, 0.0
    for r in range(wl.n_rollouts):
        if rs and t_ora >= budget_s:
            break
        a, b = wl.rollout_rows(r)
        t0 = time.perf_counter()
        t = wl.teacher_rows_host(a, b - a, threads)
        s = wl.student_rows_host(a, b - a, threads)
        t1 = time.perf_counter()
        sc = H.OP.score(t, s, wl.tok[a:b], wl.vocab)
        H.oracle_rollout(wl, r, sc, lam, alpha)
        t2 = time.perf_counter()
        del t, s
        t_gen += t1 - t0
        t_ora += t2 - t1
        rs.append(r)
        rows += b - a
    return {"value": rows / t_ora, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"rollouts {rs[0]}..{rs[-1]} of {wl.n_rollouts} of the timed workload "
                      f"({rows} tokens = {2 * rows} logit rows of V={wl.vocab}, whole path per "
                      f"rollout); oracle compute {t_ora:.1f} s, host input generation "
                      f"{t_gen:.1f} s not counted"}


def power_under_load(step, seconds: float):
    """Socket power, graphics clocks and hotspot temperature read with amd-smi (read-only
    queries) while `step` runs back to back for `seconds`, after the timed region: nothing here
    is part of the timed numbers.  Samples from the first second of load are dropped."""
    import shutil
    import subprocess
    import threading

    import torch

    exe = shutil.which("amd-smi")
    if exe is None:
        return {"error": "amd-smi not found"}
    samples, stop = [], threading.Event()
    t_start = time.perf_counter()

    def sampler():
        while not stop.is_set():
            t = time.perf_counter() - t_start
            try:
                r = subprocess.run([exe, "metric", "-p", "-c", "-t", "--json"], capture_output=True,
                                   text=True, timeout=20)
                d = json.loads(r.stdout)
                g = (d["gpu_data"] if isinstance(d, dict) else d)[0]
                clk = [v["clk"]["value"] for k, v in g["clock"].items()
                       if k.startswith("gfx_") and isinstance(v, dict)]
                samples.append((t, float(g["power"]["socket_power"]["value"]),
                                sum(clk) / len(clk), float(g["temperature"]["hotspot"]["value"])))
            except (OSError, ValueError, KeyError, IndexError, TypeError, subprocess.SubprocessError):
                pass
            stop.wait(0.2)

    th = threading.Thread(target=sampler, daemon=True)
    th.start()
    n = 0
    while time.perf_counter() - t_start < seconds:
        step()
        n += 1
        if n % 4 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    stop.set()
    th.join(timeout=30)
    keep = [x for x in samples if x[0] >= 1.0]
    if not keep:
        return {"error": "no amd-smi samples under load"}

    def med(i):
        v = sorted(x[i] for x in keep)
        return v[len(v) // 2]

    return {"samples": len(keep), "seconds": seconds, "steps": n,
            "socket_power_W": {"median": med(1), "min": min(x[1] for x in keep),
                               "max": max(x[1] for x in keep)},
            "gfx_clock_MHz_median": med(2), "hotspot_C_max": max(x[3] for x in keep),
            "source": "amd-smi metric -p -c -t (socket power, mean of the gfx clock domains)"}


def cpu_baseline_fused(wl, budget_s: float):
    """Float64 oracle on rows of the fused workload (teacher projection in binary64 plus the
    student row), batches of 16 rows until budget_s seconds of oracle compute."""
    from tests import harness as H

    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    w_dv = wl.w_dv_host(threads)
    rows, t_ora, r0 = 0, 0.0, 0
    while rows == 0 or (t_ora < budget_s and r0 < wl.n_tokens):
        idx = np.arange(r0, min(r0 + 16, wl.n_tokens))
        h = wl.hidden_host(int(idx[0]), idx.size, threads)
        st = wl.student_rows_host(int(idx[0]), idx.size, threads)
        t0 = time.perf_counter()
        H.OP.O.fused_logp(h, w_dv, wl.tok[idx])
        H.OP.O.logp_rows(st, wl.tok[idx], wl.vocab)
        t_ora += time.perf_counter() - t0
        rows += idx.size
        r0 += idx.size
    return {"value": rows / t_ora, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"rows 0..{rows - 1} of the timed workload (teacher logits h W formed in "
                      f"binary64 over d={wl.fused_d}, V={wl.vocab}, plus the student row); "
                      f"oracle compute {t_ora:.1f} s"}


def retained_row_mask(wl, stop, start):
    """1 for the rows the OPD loss keeps (units K0 .. stop of each rollout, to its last unit
    without a stop), 0 elsewhere, on the host from the stop indices (a measurement aid)."""
    from synth import workloads as W
    m = np.zeros(wl.n_tokens, np.uint8)
    for r in range(wl.n_rollouts):
        t0, t1 = int(wl.rollout_turn_off[r]), int(wl.rollout_turn_off[r + 1])
        a = int(wl.turn_tok_off[t0])
        n = (t1 - t0) if wl.unit == W.UNIT_TURN else int(wl.turn_tok_off[t1]) - a
        k0 = 0 if start is None else int(min(max(int(start[r]), 0), n))
        last = int(stop[r]) if 0 <= int(stop[r]) < n else n - 1
        if last < k0:
            continue
        if wl.unit == W.UNIT_TURN:
            m[int(wl.turn_tok_off[t0 + k0]):int(wl.turn_tok_off[t0 + last + 1])] = 1
        else:
            m[a + k0:a + last + 1] = 1
    return m


def bench_read_sweep(args):
    """Read rate against footprint on the buffers of a logits workload: the first n rows of the
    teacher and student matrices, read with the scoring kernel's pattern (stride_probe_read) and
    as two contiguous ranges in grid-stride order (stride_probe_read_flat)."""
    import torch

    import paper_2609_14636_amd as P
    from synth import device as SD
    from synth import workloads as W

    wl = W.make(args.workload, seed=args.seed)
    inp = SD.device_inputs(wl)
    t, st = inp["teachers"][0], inp["student"]
    N = wl.n_tokens
    row_bytes = t.stride(0) * t.element_size()
    stream = torch.cuda.current_stream()
    sink = torch.empty(2 * N, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    reps = max(args.steps // 2, 3)
    for frac in (1 / 6, 1 / 3, 1 / 2, 2 / 3, 5 / 6, 1.0):
        n = int(N * frac)
        nbytes = 2 * n * row_bytes
        out = {"metric": "streaming read rate against footprint", "unit": "GB/s",
               "workload": args.workload, "rows_per_matrix": n, "footprint_GB": nbytes / 1e9}
        for name, call in (
                ("rows", lambda: P.stride_probe_read(t[:n], st[:n], row_bytes, sink)),
                ("flat", lambda: P.stride_probe_read_flat(t[:n], st[:n], n * row_bytes, sink))):
            call()
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(reps)]
            for a, b in ev:
                a.record(stream)
                call()
                b.record(stream)
            torch.cuda.synchronize()
            tm = stats_ms(ev)
            out[name] = {"ms_median": tm["median"], "GBs_median": nbytes / (tm["median"] * 1e-3) / 1e9,
                         "GBs_best": nbytes / (tm["min"] * 1e-3) / 1e9}
        log(f"[sweep] {nbytes / 1e9:.1f} GB: rows {out['rows']['GBs_median']:.0f} GB/s, "
            f"flat {out['flat']['GBs_median']:.0f} GB/s")
        print(json.dumps(out), flush=True)


def bench_fused(args):
    import torch

    import paper_2609_14636_amd as P
    from synth import device as SD
    from synth import workloads as W
    from tests import workload_params as WP

    wl = W.make("fused", seed=args.seed)
    lam, alpha = WP.fused_thresholds(wl.vocab, wl.fused_d, wl.hidden_sigma, wl.w_sigma)
    log(f"[bench] workload fused seed {args.seed}: N={wl.n_tokens} d={wl.fused_d} V={wl.vocab}")
    inp = SD.device_inputs_fused(wl)
    path = P.Path(inp["layout"], wl.unit, with_student=True, fused_vocab=wl.vocab)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    def step():
        path.score_fused(wl.vocab, inp["hidden"], inp["w"], inp["student"], inp["ids"])
        path.stop(lam)
        path.restart(alpha)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    out = path.host()
    if out["flags"] != 0:
        raise SystemExit(f"device flags {out['flags']:#x} on the benchmark workload")
    check_outputs(out, wl)
    # the dominant kernel alone: teacher-only calls (projection + LSE, plus the
    # per-row gather and merge kernels, <1% of the time)
    lt = torch.empty_like(path.logp_t)
    tm = torch.empty_like(path.turn_mean)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(max(args.steps // 2, 3))]
    for a, b in ev:
        a.record(stream)
        P.stride_score_fused(inp["layout"], wl.vocab, inp["hidden"], inp["w"], None, inp["ids"],
                             lt, None, None, tm, path.flags, path.fused_ws)
        b.record(stream)
    torch.cuda.synchronize()
    k_stats = stats_ms(ev)
    k_ms = k_stats["mean"]
    # the student stream alone: the same row-scoring kernel over the student's bf16 rows
    # (scored as the only teacher, so nothing else is read)
    ls = torch.empty_like(path.logp_t)
    ev_s = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(max(args.steps // 2, 3))]
    for a, b in ev_s:
        a.record(stream)
        P.stride_score(inp["layout"], wl.vocab, [inp["student"]], None, inp["ids"], ls, None, None,
                       tm, path.flags, path.ws)
        b.record(stream)
    torch.cuda.synchronize()
    s_stats = stats_ms(ev_s)
    s_bytes = wl.n_tokens * (wl.vocab * 2 + 4 + 4)
    band_ab = bench_fused_band_ab(args, wl, inp, path, lt, tm, stream) if args.band_ab > 0 else None
    power = power_under_load(step, args.power) if args.power > 0 else None
    flops = 2.0 * wl.n_tokens * wl.fused_d * wl.vocab
    achieved = flops / (k_ms * 1e-3) / 1e12
    log(f"[bench] {args.steps} steps: {ms_step:.3f} ms/step; teacher projection {k_ms:.3f} ms "
        f"= {achieved:.0f} TFLOP/s")
    res = {
        "metric": METRIC, "value": wl.n_tokens / (ms_step * 1e-3), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"fused: {shape_label(wl)}, "
                               f"{wl.n_tokens} scored tokens, teacher logits h W on the fly "
                               f"(d={wl.fused_d}, V={wl.vocab}), student logits bf16",
                   "global_batch": wl.n_rollouts, "seq_len": wl.n_tokens // wl.n_rollouts,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / MFMA_BF16_PEAK_TFLOPS,
                     "traffic": measured_traffic("fused", FUSED_SRC, "fused_hip_sha256_16"),
                     "kernel": "fused_lse_kernel (bf16 MFMA 16x16x32); kernel_ms brackets the "
                               "teacher call (projection + per-row gather + merge)",
                     "kernel_ms": k_ms, "kernel_ms_median": k_stats["median"],
                     "kernel_ms_min": k_stats["min"],
                     "mfma_busy": measured_mfma_busy(),
                     "flops_per_launch": flops},
        "student_stream": {"kernel": "score_rows_kernel<bf16> over the student rows alone",
                           "bytes_per_launch": s_bytes, "ms": s_stats["mean"],
                           "ms_median": s_stats["median"], "ms_min": s_stats["min"],
                           "GB/s": s_bytes / (s_stats["mean"] * 1e-3) / 1e9,
                           "frac_of_hbm_peak": s_bytes / (s_stats["mean"] * 1e-3) / 1e9 / HBM_PEAK_GBS},
    }
    if power is not None:
        res["power"] = power
    if band_ab is not None:
        res["band_order"] = band_ab
    if not args.no_cpu:
        log("[bench] timing the float64 oracle on a bounded sample")
        res["cpu_baseline"] = cpu_baseline_fused(wl, args.cpu_seconds)
    print(json.dumps(res), flush=True)


def bench_fused_band_ab(args, wl, inp, path, lt, tm, stream):
    """The teacher call through libstride_debug.so with one super-row per band (each W slab
    read from HBM once per 4,096 rows) against the library's own band, launches alternating on
    one stream; the log-probabilities of the two orders must be equal bit for bit."""
    import torch

    import paper_2609_14636_amd as P

    dbg = P.stride.debug_library()
    lt1 = torch.empty_like(lt)
    ev = {0: [], 1: []}
    try:
        for rep in range(args.band_ab + 1):
            for band in (1, 0):
                if dbg.stride_debug_fused_band(band) != 0:
                    raise SystemExit("libstride_debug.so refused the band setting")
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                P.stride_score_fused(inp["layout"], wl.vocab, inp["hidden"], inp["w"], None,
                                     inp["ids"], lt1 if band == 1 else lt, None, None, tm,
                                     path.flags, path.fused_ws, lib=dbg)
                b.record(stream)
                if rep > 0:  # the first pair warms up
                    ev[band].append((a, b))
        torch.cuda.synchronize()
    finally:
        dbg.stride_debug_fused_band(0)
    if not torch.equal(lt.view(torch.int32), lt1.view(torch.int32)):
        raise SystemExit("the two tile orders gave different log-probabilities")
    one, own = stats_ms(ev[1]), stats_ms(ev[0])
    log(f"[bench] band order: one super-row per band median {one['median']:.3f} ms, "
        f"the library's band median {own['median']:.3f} ms ({args.band_ab} launches each)")
    return {"launches_each": args.band_ab, "one_super_row_ms": one, "library_band_ms": own,
            "speedup_median": one["median"] / own["median"], "outputs_bit_identical": True,
            "library": "libstride_debug.so (stride_debug_fused_band)"}


def bench_online(args):
    """Latency of the online stop test (stride_stop_step): per call, a batch of active rollouts
    appends new units (one turn mean each, or a chunk of token log-probabilities each) and the
    carried state is updated on the device.  lambda is set below every reachable value, so every
    rollout stays active for the whole run."""
    import torch
    import paper_2609_14636_amd as P

    stream = torch.cuda.current_stream()
    lines = []
    for unit, active, per in ((P.STRIDE_UNIT_TURN, 256, 1), (P.STRIDE_UNIT_TOKEN, 64, 512)):
        g = torch.Generator(device="cuda").manual_seed(args.seed)
        dt = torch.float64 if unit == P.STRIDE_UNIT_TURN else torch.float32
        vals = -torch.rand(active * per, generator=g, device="cuda", dtype=torch.float64).to(dt)
        slot = torch.arange(active, dtype=torch.int32, device="cuda")
        off = torch.arange(0, active * per + 1, per, dtype=torch.int64, device="cuda")
        cum = torch.zeros(active, dtype=torch.float64, device="cuda")
        units = torch.zeros(active, dtype=torch.int32, device="cuda")
        stop = torch.full((active,), -1, dtype=torch.int32, device="cuda")
        flags = torch.zeros(1, dtype=torch.int32, device="cuda")
        lam = [-1e300]

        def call():
            P.stride_stop_step(slot, off, unit, vals, None, lam, cum, units, stop, flags)

        for _ in range(args.warmup):
            call()
        torch.cuda.synchronize()
        calls = max(args.steps, 1) * 10
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(calls):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / calls
        t0 = time.perf_counter()
        for _ in range(calls):
            call()
            torch.cuda.synchronize()
        rt = (time.perf_counter() - t0) * 1e6 / calls
        if int(flags.item()) != 0 or int((stop >= 0).sum().item()) != 0:
            raise SystemExit("online stop test: unexpected flags or stops")
        name = "turn" if unit == P.STRIDE_UNIT_TURN else "token"
        lines.append({
            "metric": "online stop test latency (stride_stop_step), 1 MI355X", "value": us,
            "unit": "us/call", "n_gpus": 1, "steps": calls, "warmup": args.warmup,
            "ms_per_step": us * 1e-3, "higher_is_better": False, "scaling": "weak",
            "vs_baseline": None, "dtype": "f64" if unit == P.STRIDE_UNIT_TURN else "f32",
            "data": "synthetic",
            "config": {"workload": f"online {name} units: {active} active rollouts x {per} new "
                                   f"unit(s) per call", "global_batch": active, "seq_len": per,
                       "parallelism": "single GPU"},
            "host_round_trip_us": rt})
    for line in lines:
        print(json.dumps(line), flush=True)


def bench_graph(args):
    """Eager calls against HIP-graph replay of the same step (score -> stop -> restart) on small
    batches, where the step is six short kernels and their launches dominate: the library
    allocates, synchronises and memsets nothing, so the step is captured once and replayed with
    one launch.  A measurement aid; the headline step is timed with eager calls."""
    import torch

    import paper_2609_14636_amd as P
    from synth import device as SD
    from synth import workloads as W

    stream = torch.cuda.current_stream()
    calls = max(args.steps, 1) * 10
    lines = []
    for R, tok in ((8, 8), (16, 64), (64, 256)):
        wl = W.make("reasoning", seed=args.seed, scale=dict(R=R, tok=tok))
        inp = SD.device_inputs(wl)
        lam, alpha = [-0.5 * tok * math.log(wl.vocab)], [-math.inf]
        paths = [P.Path(inp["layout"], wl.unit) for _ in range(2)]

        def step(path):
            path.run(wl.vocab, inp["teachers"], inp["student"], inp["ids"], lam, alpha,
                     start_unit=inp["start"], correct_mask=inp["mask"])

        eager, graphed = paths
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step(graphed)  # warm-up outside the capture
        stream.wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step(graphed)
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            step(eager)
            g.replay()
        torch.cuda.synchronize()
        times, issue = {}, {}
        for name, fn in (("eager", lambda: step(eager)), ("graph", g.replay)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            t0 = time.perf_counter()
            for _ in range(calls):
                fn()
            issue[name] = (time.perf_counter() - t0) * 1e6 / calls  # host time to issue a step
            e1.record(stream)
            torch.cuda.synchronize()
            times[name] = e0.elapsed_time(e1) * 1e3 / calls
        a, b = eager.host(), graphed.host()
        if a["flags"] or b["flags"]:
            raise SystemExit(f"device flags {a['flags']:#x} / {b['flags']:#x}")
        for k in a:
            if a[k] is not None and not np.array_equal(np.asarray(a[k]), np.asarray(b[k])):
                raise SystemExit(f"graph replay differs from eager calls in {k}")
        check_outputs(a, wl)
        log(f"[bench] graph R={R} tok={tok}: eager {times['eager']:.1f} us/step "
            f"(host issue {issue['eager']:.1f}), graph {times['graph']:.1f} us/step "
            f"(host issue {issue['graph']:.1f})")
        lines.append({
            "metric": "step latency with HIP graph replay (score+stop+restart), 1 MI355X",
            "value": times["graph"], "unit": "us/step", "n_gpus": 1, "steps": calls,
            "warmup": args.warmup, "ms_per_step": times["graph"] * 1e-3,
            "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic",
            "config": {"workload": f"reasoning-shaped: {R} rollouts x {tok} tokens "
                                   f"({wl.n_tokens} rows, V={wl.vocab}), token units",
                       "global_batch": R, "seq_len": tok, "parallelism": "single GPU"},
            "eager_us_per_step": times["eager"],
            "host_issue_us_per_step": {"eager": issue["eager"], "graph": issue["graph"]},
            "graph_speedup": times["eager"] / times["graph"]})
    for line in lines:
        print(json.dumps(line), flush=True)


def bench_gemm_reference(args):
    """The unfused alternative to the fused projection, for scale: the vendor library's bf16 GEMM
    (torch.matmul -> hipBLASLt) writing the [N, V] teacher logits, then torch.logsumexp over them,
    on the fused workload's operands.  A measurement aid only: nothing here is part of the path."""
    import torch

    from synth import device as SD
    from synth import workloads as W

    wl = W.make("fused", seed=args.seed)
    inp = SD.device_inputs_fused(wl)
    h, w_vd = inp["hidden"], inp["w"]
    w_dv = w_vd.t().contiguous()  # [d, V], contiguous: no transposed view reaches the GEMM
    del inp
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    reps = max(args.steps // 4, 3)
    z = torch.matmul(h, w_dv)
    torch.logsumexp(z, dim=1)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps)]
    for e in ev:
        e[0].record(stream)
        z = torch.matmul(h, w_dv)
        e[1].record(stream)
        lse = torch.logsumexp(z, dim=1)
        e[2].record(stream)
    torch.cuda.synchronize()
    mm = stats_ms([(e[0], e[1]) for e in ev])
    ls = stats_ms([(e[1], e[2]) for e in ev])
    flops = 2.0 * wl.n_tokens * wl.fused_d * wl.vocab
    print(json.dumps({
        "metric": "unfused reference: bf16 GEMM writing the logits, then logsumexp (torch / hipBLASLt)",
        "value": flops / (mm["mean"] * 1e-3) / 1e12, "unit": "TFLOP/s (GEMM alone)", "n_gpus": 1,
        "steps": reps, "warmup": 1, "ms_per_step": mm["mean"] + ls["mean"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"fused operands: h [{wl.n_tokens}, {wl.fused_d}] x W [{wl.fused_d}, "
                               f"{wl.vocab}] bf16, logits [{wl.n_tokens}, {wl.vocab}] bf16 in HBM",
                   "global_batch": wl.n_rollouts, "seq_len": wl.n_tokens // wl.n_rollouts,
                   "parallelism": "single GPU"},
        "gemm_ms": mm, "logsumexp_ms": ls, "lse_sample": float(lse[0].float().item())}), flush=True)


def bench_records(args):
    """Host trajectory record H(x): put a record per task, then plan every task's restart point
    in one call (Sec. 4.2 on the host)."""
    import paper_2609_14636_amd as P

    rng = np.random.default_rng(args.seed)
    n_tasks, turns = 100_000, 12
    vals = -np.abs(rng.normal(0.7, 0.3, size=(n_tasks, turns)))
    mask = (rng.random((n_tasks, turns)) < 0.9).astype(np.uint8)
    rec = P.Records()
    t0 = time.perf_counter()
    for t in range(n_tasks):
        rec.put(t, vals[t], mask[t])
    put_s = time.perf_counter() - t0
    tasks = np.arange(n_tasks, dtype=np.int64)
    t0 = time.perf_counter()
    ks, k0, km = rec.plan(tasks, -0.8)
    plan_s = time.perf_counter() - t0
    assert len(rec) == n_tasks and (k0 >= 0).all() and (km <= turns).all()
    print(json.dumps({
        "metric": "trajectory record plan throughput (stride_records_plan), host", "value":
        n_tasks / plan_s, "unit": "tasks/s", "n_gpus": 0, "steps": 1, "warmup": 0,
        "ms_per_step": plan_s * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"records: {n_tasks} tasks x {turns} turns", "global_batch": n_tasks,
                   "seq_len": turns, "parallelism": "host, one thread"},
        "put_tasks_per_s_with_binding": n_tasks / put_s}), flush=True)


def build_parser() -> argparse.ArgumentParser:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="reasoning",
                    choices=["tiny", "agentic", "reasoning", "multi", "fused"])
    ap.add_argument("--seed", type=int, default=1001)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="bound on the oracle sample: whole rollouts are added until the oracle "
                         "has computed this long (at least one rollout)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--power", type=float, default=0.0, metavar="SECONDS",
                    help="after the timed steps, run the step back to back for SECONDS while "
                         "sampling socket power, clocks and temperature with amd-smi")
    ap.add_argument("--band-ab", type=int, default=0, metavar="N",
                    help="with --workload fused: also time the teacher call with one super-row "
                         "per band against the library's band, N launches each, alternating")
    ap.add_argument("--exact-kl", action="store_true",
                    help="also compute the exact full-vocabulary KL per token (paired kernel)")
    ap.add_argument("--opd-grad", action="store_true",
                    help="also run the OPD loss gradient (stride_opd_grad) in each step")
    ap.add_argument("--online", action="store_true",
                    help="only time the online stop test (stride_stop_step) per call")
    ap.add_argument("--graph", action="store_true",
                    help="only time small steps as eager calls against HIP graph replay")
    ap.add_argument("--records", action="store_true",
                    help="only time the host trajectory record (put / plan)")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="only time the unfused alternative to the fused projection on its operands: "
                         "torch.matmul (hipBLASLt) writing the logits, then torch.logsumexp")
    ap.add_argument("--read-sweep", action="store_true",
                    help="only measure the streaming read rate against footprint on the "
                         "workload's logits buffers (row pattern and grid-stride order)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain elementwise copy (torch.neg on float32) reading and "
                         "writing BYTES each per dispatch, to calibrate the HBM byte counters; keep "
                         "BYTES <= 1 GiB so that torch issues one dispatch per copy")
    return ap


def main():
    args = build_parser().parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} is not supported "
              "(the path shards by whole rollouts with no exchange between GPUs)", file=sys.stderr)
        sys.exit(2)

    if args.band_ab and args.workload != "fused":
        print("--band-ab times the fused projection's tile order: use it with --workload fused",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        if args.copy_calibration > 1 << 30:
            raise SystemExit("--copy-calibration above 1 GiB is split into several dispatches")
        n = args.copy_calibration // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": 4 * n, "launches": 3}), flush=True)
        return

    if args.records:
        return bench_records(args)

    import paper_2609_14636_amd as P
    from synth import device as SD
    from synth import workloads as W

    torch.cuda.set_device(0)
    if args.online:
        return bench_online(args)
    if args.graph:
        return bench_graph(args)
    if args.read_sweep:
        return bench_read_sweep(args)
    if args.gemm_reference:
        return bench_gemm_reference(args)
    if args.workload == "fused":
        return bench_fused(args)
    wl = W.make(args.workload, seed=args.seed)
    lam, alpha = workload_params(args.workload, args.seed)
    log(f"[bench] workload {args.workload} seed {args.seed}: R={wl.n_rollouts} T={wl.n_turns} "
        f"N={wl.n_tokens} V={wl.vocab}; generating {2 * wl.logits_bytes() / 1e9:.1f} GB on device")
    inp = SD.device_inputs(wl)
    path = P.Path(inp["layout"], wl.unit, with_student=True, exact_kl=args.exact_kl)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    grad = torch.empty_like(inp["student"]) if args.opd_grad else None
    loss = torch.empty(wl.n_tokens, dtype=torch.float32, device="cuda") if args.opd_grad else None
    gev = []

    def step():
        path.score(wl.vocab, inp["teachers"], inp["student"], inp["ids"])
        path.stop(lam, inp["start"])
        path.restart(alpha, inp["mask"])
        if args.opd_grad:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            path.grad(wl.vocab, inp["student"], inp["ids"], grad, loss, inp["start"],
                      scale=1.0 / wl.n_tokens)
            e1.record(stream)
            gev.append((e0, e1))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({args.warmup} steps)")

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    sev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    gev.clear()
    for i in range(args.steps):
        ev[i][0].record(stream)
        path.score(wl.vocab, inp["teachers"], inp["student"], inp["ids"])
        ev[i][1].record(stream)
        path.stop(lam, inp["start"])
        path.restart(alpha, inp["mask"])
        sev[i].record(stream)
        if args.opd_grad:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            path.grad(wl.vocab, inp["student"], inp["ids"], grad, loss, inp["start"],
                      scale=1.0 / wl.n_tokens)
            e1.record(stream)
            gev.append((e0, e1))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    k_stats = stats_ms(ev)
    step_stats = stats_ms([(ev[i][0], sev[i]) for i in range(args.steps)])
    score_ms = k_stats["mean"]
    out = path.host()
    if out["flags"] != 0:
        raise SystemExit(f"device flags {out['flags']:#x} on the benchmark workload")
    check_outputs(out, wl)
    log(f"[bench] {args.steps} steps: {ms_step:.3f} ms/step (device: median "
        f"{step_stats['median']:.3f}, min {step_stats['min']:.3f}), scoring mean {score_ms:.3f} "
        f"median {k_stats['median']:.3f} min {k_stats['min']:.3f} ms; "
        f"stops {int((out['stop_unit'] >= 0).sum())}/{wl.n_rollouts}")

    n_tok = wl.n_tokens
    per_token = 2 * wl.vocab * wl.esize + 4 + 8  # two logit rows in, token id in, two logps out
    bytes_alg = per_token * n_tok
    achieved = bytes_alg / (score_ms * 1e-3) / 1e9
    traffic = None if args.exact_kl else measured_traffic(args.workload)
    dt = "bf16" if wl.dtype == W.BF16 else "f32"
    # streaming-read reference: the same rows read with the same access pattern, no arithmetic
    sink = torch.empty(2 * n_tok, dtype=torch.int32, device="cuda")
    read_bytes = (wl.vocab * wl.esize) // 16 * 16
    pev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(max(args.steps // 2, 3))]
    P.stride_probe_read(inp["teachers"][0], inp["student"], read_bytes, sink)
    for a, b in pev:
        a.record(stream)
        P.stride_probe_read(inp["teachers"][0], inp["student"], read_bytes, sink)
        b.record(stream)
    torch.cuda.synchronize()
    probe_ms = sum(a.elapsed_time(b) for a, b in pev) / len(pev)
    ceiling = 2 * n_tok * read_bytes / (probe_ms * 1e-3) / 1e9
    log(f"[bench] streaming-read reference on the same rows: {probe_ms:.3f} ms = {ceiling:.0f} GB/s; "
        f"scoring reaches {100 * achieved / ceiling:.1f}% of it")
    res = {
        "metric": METRIC,
        "value": n_tok / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "step_ms": step_stats,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == W.BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {shape_label(wl)}, "
                               f"{n_tok} scored tokens, V={wl.vocab}, teacher+student logits",
                   "global_batch": wl.n_rollouts, "seq_len": int(n_tok // max(wl.n_rollouts, 1)),
                   "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": (f"score_pairs_kernel<{dt}> (with exact KL)" if args.exact_kl
                                else f"score_rows_kernel<{dt}>"), "kernel_ms": score_ms,
                     "kernel_ms_median": k_stats["median"], "kernel_ms_min": k_stats["min"],
                     "bytes_per_launch": bytes_alg,
                     "read_ceiling": {"achieved": ceiling, "unit": "GB/s", "frac": achieved / ceiling,
                                      "kernel": "probe_read_kernel: the same rows, same loads, "
                                                "no arithmetic"}},
    }
    if args.opd_grad:
        g = stats_ms(gev)
        g_ms = g["mean"]
        kept = int(out["retained"].sum())
        gbytes = kept * 2 * wl.vocab * wl.esize + (n_tok - kept) * wl.vocab * wl.esize + 13 * n_tok
        # read+write reference on the same rows: retained rows copied from the student logits,
        # the others zero-filled without a read, one wavefront per row (the gradient's pattern)
        rmask = torch.from_numpy(retained_row_mask(wl, out["stop_unit"], wl.start)).cuda()
        assert int(rmask.sum().item()) == kept
        row_bytes = (wl.vocab * wl.esize) // 16 * 16
        cev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(max(args.steps // 2, 3))]
        P.stride_probe_copy(inp["student"], grad, rmask, row_bytes)
        for a, b in cev:
            a.record(stream)
            P.stride_probe_copy(inp["student"], grad, rmask, row_bytes)
            b.record(stream)
        torch.cuda.synchronize()
        c_ms = stats_ms(cev)["mean"]
        cbytes = kept * 2 * row_bytes + (n_tok - kept) * row_bytes
        copy_gbs = cbytes / (c_ms * 1e-3) / 1e9
        res["opd_grad"] = {"kernel_ms": g_ms, "kernel_ms_median": g["median"],
                           "kernel_ms_min": g["min"], "retained_rows": kept,
                           "bytes_per_launch": gbytes, "achieved_GBs": gbytes / (g_ms * 1e-3) / 1e9,
                           "frac": gbytes / (g_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                           "copy_ceiling": {"achieved_GBs": copy_gbs, "kernel_ms": c_ms,
                                            "frac": gbytes / (g_ms * 1e-3) / 1e9 / copy_gbs,
                                            "kernel": "probe_copy_kernel: the same rows moved with "
                                                      "the same loads and stores, no arithmetic"}}
        log(f"[bench] OPD gradient {g_ms:.3f} ms, {kept}/{n_tok} rows retained, "
            f"{res['opd_grad']['achieved_GBs']:.0f} GB/s; read+write reference {c_ms:.3f} ms = "
            f"{copy_gbs:.0f} GB/s")
    if args.power > 0:
        res["power"] = power_under_load(step, args.power)
    if not args.no_cpu:
        log("[bench] timing the float64 oracle on a bounded sample")
        res["cpu_baseline"] = cpu_baseline(wl, lam, alpha, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
