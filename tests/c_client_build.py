"""Builds tests/c_client.bin, the plain C caller of libstride.so used by test_gpu_c_client.py
(gcc, host code only; linked against libstride.so and the HIP runtime, found at run time
relative to the binary and under /opt/rocm/lib)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "c_client.c")
BIN = os.path.join(HERE, "c_client.bin")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           SRC, "-o", BIN + ".tmp",
           "-L", os.path.join(ROOT, "paper_2609_14636_amd"), "-lstride",
           "-Wl,-rpath,$ORIGIN/../paper_2609_14636_amd",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"gcc failed on c_client.c:\n{r.stdout}{r.stderr}")
    os.replace(BIN + ".tmp", BIN)
    return BIN


if __name__ == "__main__":
    print(build(verbose=True))
