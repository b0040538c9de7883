"""The C ABI on the CPU: the library loads, exports what include/stride.h declares, and rejects
bad arguments on the host before launching anything (no call here reaches a kernel)."""
import ctypes
import os
import re

import pytest
import torch

import paper_2609_14636_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = []
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names += re.findall(r"\b(stride_[a-z_]+)\s*\(", text)
    return sorted(set(names))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert {"stride_score", "stride_stop", "stride_restart_turn", "stride_score_fused",
            "stride_workspace_size", "stride_last_error"} <= set(names)
    lib = ctypes.CDLL(P.stride.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} is declared but not exported"


def test_header_compiles_as_c():
    import subprocess
    src = '#include "stride.h"\nint main(void){ return (int)sizeof(stride_layout); }\n'
    r = subprocess.run(["gcc", "-std=c99", "-fsyntax-only", "-I", os.path.join(ROOT, "include"),
                        "-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__", "-x", "c", "-"],
                       input=src, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def _layout(R=2, T=3, N=10):
    rto = torch.tensor([0, 2, 3][:R + 1], dtype=torch.int32)
    tto = torch.tensor([0, 4, 7, N][:T + 1], dtype=torch.int64)
    return P.Layout(rto, tto, N)


def test_workspace_size():
    lay = _layout()
    a = P.stride_workspace_size(lay, P.STRIDE_UNIT_TURN)
    b = P.stride_workspace_size(lay, P.STRIDE_UNIT_TOKEN)
    assert a > 0 and b >= a and a % 256 == 0
    big = P.Layout(torch.zeros(9, dtype=torch.int32), torch.zeros(2, dtype=torch.int64), 10**6)
    assert P.stride_workspace_size(big, P.STRIDE_UNIT_TOKEN) >= 10**6


def _fake(n):
    """A CPU tensor standing in for a device buffer; only calls that fail validation use it."""
    return torch.zeros(n, dtype=torch.float32)


@pytest.mark.parametrize("case,code", [
    ("vocab0", 1), ("ld_small", 1), ("bad_unit", 1), ("ws_small", 3), ("n_dom0", 2),
    ("kl_without_student", 1), ("student_without_logp_s", 1), ("kl_without_logp_s", 1),
    ("kl_full_without_logp_s", 1), ("fused_student_without_logp_s", 1),
    ("fused_kl_without_logp_s", 1), ("fused_ws_small", 3), ("ws_unaligned", 3),
    ("n_teachers_65", 2), ("n_dom_65", 2), ("grad_bad_unit", 1),
])
def test_argument_errors_raise_before_launch(case, code):
    """Each bad argument returns its status (1 invalid argument, 2 unsupported, 3 workspace)
    before anything is launched: the buffers here are host memory, which no kernel could read."""
    status = P.stride.StrideError
    lay = _layout()
    x = torch.zeros((10, 16), dtype=torch.float32)
    ids = torch.zeros(10, dtype=torch.int32)
    out = _fake(10)
    tm = torch.zeros(3, dtype=torch.float64)
    ws = torch.zeros(P.stride_workspace_size(lay, P.STRIDE_UNIT_TOKEN), dtype=torch.uint8)
    with pytest.raises(status) as ei:
        if case == "vocab0":
            P.stride_score(lay, 0, [x], x, ids, out, out, out, tm, None, ws, stream=0)
        elif case == "ld_small":
            P.stride_score(lay, 17, [x], x, ids, out, out, out, tm, None, ws, stream=0)
        elif case == "bad_unit":
            P.stride_stop(lay, 9, tm, [-1.0], None, tm, ids, None, None, ws, stream=0)
        elif case == "ws_small":
            P.stride_stop(lay, P.STRIDE_UNIT_TOKEN, out, [-1.0], None, tm, ids, None, None,
                          ws[:100], stream=0)
        elif case == "n_dom0":
            P.stride_restart_turn(lay, P.STRIDE_UNIT_TURN, tm, None, [], None, ids, ids, None,
                                  None, stream=0)
        elif case == "kl_without_student":
            P.stride_score(lay, 16, [x], None, ids, out, None, out, tm, None, ws, stream=0)
        elif case == "student_without_logp_s":
            # the student rows' log-probabilities would be written through logp_s
            P.stride_score(lay, 16, [x], x, ids, out, None, None, tm, None, ws, stream=0)
        elif case == "kl_without_logp_s":
            P.stride_score(lay, 16, [x], x, ids, out, None, out, tm, None, ws, stream=0)
        elif case == "kl_full_without_logp_s":
            P.stride_score(lay, 16, [x], x, ids, out, None, None, tm, None, ws, stream=0,
                           kl_full=out)
        elif case in ("fused_student_without_logp_s", "fused_kl_without_logp_s"):
            h = torch.zeros((10, 64), dtype=torch.bfloat16)
            w = torch.zeros((16, 64), dtype=torch.bfloat16)
            xs = torch.zeros((10, 16), dtype=torch.bfloat16)
            kl = out if case == "fused_kl_without_logp_s" else None
            P.stride_score_fused(lay, 16, h, w, xs, ids, out, None, kl, tm, None, ws, stream=0)
        elif case == "fused_ws_small":
            # 256-byte aligned, so the size check (not the alignment check) is what fails
            h = torch.zeros((10, 64), dtype=torch.bfloat16)
            w = torch.zeros((16, 64), dtype=torch.bfloat16)
            need = P.stride_fused_workspace_size(lay, 16)
            buf = torch.zeros(need + 256, dtype=torch.uint8)
            off = (-buf.data_ptr()) % 256
            small = buf[off:off + need - 8]
            assert small.data_ptr() % 256 == 0
            P.stride_score_fused(lay, 16, h, w, None, ids, out, None, None, tm, None, small,
                                 stream=0)
        elif case == "ws_unaligned":
            P.stride_stop(lay, P.STRIDE_UNIT_TOKEN, out, [-1.0], None, tm, ids, None, None,
                          ws[1:], stream=0)
        elif case == "n_teachers_65":
            P.stride_score(lay, 16, [x] * 65, x, ids, out, out, out, tm, None, ws, stream=0)
        elif case == "n_dom_65":
            P.stride_stop(lay, P.STRIDE_UNIT_TOKEN, out, [-1.0] * 65, None, tm, ids, None, None,
                          ws, stream=0)
        elif case == "grad_bad_unit":
            P.stride_opd_grad(lay, 7, 16, x, ids, out, out, None, ids, 1.0, x, out, None, ws,
                              stream=0)
    assert ei.value.status == code, P.library().stride_last_error().decode()
    if case == "fused_ws_small":
        assert "need" in P.library().stride_last_error().decode()
    assert P.library().stride_last_error().decode()


def test_unaligned_row_stride_is_unsupported():
    lay = _layout()
    x = torch.zeros((10, 15), dtype=torch.bfloat16)  # 30-byte rows
    ids = torch.zeros(10, dtype=torch.int32)
    with pytest.raises(P.StrideError) as ei:
        P.stride_score(lay, 15, [x], None, ids, _fake(10), None, None,
                       torch.zeros(3, dtype=torch.float64), None, None, stream=0)
    assert ei.value.status == 2


@pytest.mark.parametrize("d", [32, 96, 65536 + 64])
def test_fused_hidden_size_outside_the_supported_range_is_rejected(d):
    """The fused projection takes d in multiples of 64 up to 65,536 (one operand tile must fit
    a 32-bit buffer range); anything else returns STRIDE_ERR_UNSUPPORTED before any launch."""
    lay = _layout()
    h = torch.zeros((10, d), dtype=torch.bfloat16)
    w = torch.zeros((16, d), dtype=torch.bfloat16)
    ids = torch.zeros(10, dtype=torch.int32)
    with pytest.raises(P.StrideError) as ei:
        P.stride_score_fused(lay, 16, h, w, None, ids, _fake(10), None, None,
                             torch.zeros(3, dtype=torch.float64), None, None, stream=0)
    assert ei.value.status == 2
    assert "hidden size" in P.library().stride_last_error().decode()


@pytest.mark.parametrize("case", ["read_past_row", "misaligned_stride", "null_sink"])
def test_probe_read_argument_errors(case):
    a = torch.zeros((4, 64), dtype=torch.bfloat16)
    sink = torch.zeros(8, dtype=torch.int32)
    with pytest.raises(P.StrideError) as ei:
        if case == "read_past_row":
            P.stride_probe_read(a, None, 129 * 2, sink, stream=0)
        elif case == "misaligned_stride":
            P.stride_probe_read(torch.zeros((4, 60), dtype=torch.bfloat16), None, 64, sink,
                                stream=0)  # 120-byte rows
        else:
            P.stride_probe_read(a, None, 64, None, stream=0)
    assert ei.value.status == (2 if case == "misaligned_stride" else 1)


def test_flag_word_decoding():
    assert P.flag_names(0) == []
    assert P.flag_names(P.STRIDE_FLAG_TOKEN_OOB | P.STRIDE_FLAG_NONFINITE) == ["TOKEN_OOB", "NONFINITE"]
    assert P.flag_names(1 << 20) == [hex(1 << 20)]
    err = P.StrideDataError(P.STRIDE_FLAG_EMPTY_TURN | P.STRIDE_FLAG_SPIN_LIMIT)
    assert "EMPTY_TURN" in str(err) and "SPIN_LIMIT" in str(err) and err.flags == 34


def test_noalloc_stop_rejects_layouts_past_its_fixed_scratch():
    """stride_stop_noalloc keeps its scratch in a fixed per-GPU array; a layout whose tile
    counter, unit offsets and scan descriptors do not fit returns STRIDE_ERR_UNSUPPORTED on the
    host, before the array is looked up or anything is launched."""
    R = 200_000  # 8 (R + 1) bytes of unit offsets alone exceed the array
    lay = P.Layout(torch.zeros(R + 1, dtype=torch.int32), torch.zeros(2, dtype=torch.int64), 10)
    tm = torch.zeros(1, dtype=torch.float64)
    stop = torch.zeros(R, dtype=torch.int32)
    with pytest.raises(P.StrideError) as ei:
        P.stride_stop_noalloc(lay, P.STRIDE_UNIT_TURN, tm, [-1.0], None, tm, stop, None, None,
                              stream=0)
    assert ei.value.status == 2
    assert "scratch" in P.library().stride_last_error().decode()


def test_last_error_is_per_thread():
    """Argument errors raised concurrently on several host threads each leave their own message:
    the library keeps the last error per thread, so a caller never reads another thread's."""
    import threading

    lay = _layout()
    x = torch.zeros((10, 16), dtype=torch.float32)
    ids = torch.zeros(10, dtype=torch.int32)
    out = _fake(10)
    tm = torch.zeros(3, dtype=torch.float64)
    ws = torch.zeros(P.stride_workspace_size(lay, P.STRIDE_UNIT_TOKEN), dtype=torch.uint8)
    failures = []

    def worker(kind):
        for _ in range(300):
            try:
                if kind == "vocab":
                    P.stride_score(lay, 0, [x], x, ids, out, out, out, tm, None, ws, stream=0)
                else:
                    P.stride_score(lay, 17, [x], x, ids, out, out, out, tm, None, ws, stream=0)
            except P.stride.StrideError as e:
                msg = str(e)
                want = "vocab = 0" if kind == "vocab" else "ld = 16 < vocab = 17"
                if want not in msg:
                    failures.append((kind, msg))
                    return
            else:
                failures.append((kind, "no error"))
                return

    threads = [threading.Thread(target=worker, args=(k,)) for k in ("vocab", "ld") * 4]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not failures, failures[:3]


def test_c_client_compiles_against_the_header():
    """The plain C caller (tests/c_client.c) compiles as C11 against include/stride.h alone."""
    import subprocess
    src = os.path.join(ROOT, "tests", "c_client.c")
    r = subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-fsyntax-only",
                        "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                        "-D__HIP_PLATFORM_AMD__", src], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_fused_band_hook():
    """The fused projection's band setting exists only in the test library: the product library
    returns STRIDE_ERR_UNSUPPORTED, the test library rejects a negative band and takes 0 (the
    library's own choice); setting it launches nothing."""
    assert P.library().stride_debug_fused_band(2) == 2
    dbg = P.stride.debug_library()
    assert dbg.stride_debug_fused_band(-1) == 1
    assert dbg.stride_debug_fused_band(0) == 0
