"""Build libstride.so for gfx950 from the HIP sources in this directory.

Each source is compiled by hipcc in parallel, then linked into
``paper_2609_14636_amd/libstride.so``.  Packed-FP32 instruction selection is
switched off for all device code.  A second library for testing,
``libstride_debug.so``, links the same objects except that the stop test's scan
is compiled with its look-back delay hook (STRIDE_SCAN_DELAY_HOOK) and the fused
projection with a settable tile-band size (STRIDE_FUSED_BAND_HOOK).
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libstride.so")
DEBUG_LIB = os.path.join(PKG, "libstride_debug.so")
BUILD = os.path.join(ROOT, "_build")

SOURCES = ["stride_abi.cpp", "record.cpp", "score.hip", "turn.hip", "scan.hip", "restart.hip", "fused.hip", "grad.hip", "probe.hip"]
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]


def _compile(src: str, verbose: bool, defines=(), suffix: str = "") -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + suffix + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    cmd = ["hipcc", *FLAGS, *[f"-D{d}" for d in defines], *lang, "-c", os.path.join(HERE, src),
           "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{msg}")
    if msg.strip() and verbose:
        print(msg)
    return obj


def _link(objs, out: str, verbose: bool) -> None:
    tmp = out + ".tmp"
    cmd = ["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    hooks = {"scan.hip": "STRIDE_SCAN_DELAY_HOOK", "fused.hip": "STRIDE_FUSED_BAND_HOOK"}
    jobs = [(s, (), "") for s in SOURCES] + [(s, (d,), "_debug") for s, d in hooks.items()]
    with ThreadPoolExecutor(min(8, len(jobs))) as ex:
        objs = list(ex.map(lambda j: _compile(j[0], verbose, j[1], j[2]), jobs))
    product = objs[:len(SOURCES)]
    debug = dict(zip(hooks, objs[len(SOURCES):]))
    _link(product, LIB, verbose)
    _link([debug.get(SOURCES[i], o) for i, o in enumerate(product)], DEBUG_LIB, verbose)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
