"""Build the gfx950 XAttention library in-tree: paper_2503_16428_amd/lib/libxattn.so,
the benchmark's measurement probe: paper_2503_16428_amd/lib/libxattn_probe.so,
and a plain C client of the library used by a GPU test:
paper_2503_16428_amd/lib/xattn_c_client (tests/c_client.c, host code only).

Every source is compiled by hipcc for gfx950 only. Packed-fp32 instructions
are disabled (-packed-fp32-ops): hipcc otherwise forms v_pk_* fp32 ops from
ordinary float code.
"""
from __future__ import annotations

import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "lib")
LIB = os.path.join(OUT_DIR, "libxattn.so")
PROBE_LIB = os.path.join(OUT_DIR, "libxattn_probe.so")
C_CLIENT = os.path.join(OUT_DIR, "xattn_c_client")
SOURCES = ["score.hip", "select.hip", "attn.hip", "error.hip", "noalloc.hip", "api.cpp",
           "threshold.cpp"]
PROBE_SOURCES = ["probe.hip"]
ARCH = "gfx950"

COMMON_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-Wall", "-Wno-unused-function",
]


def _hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    p = os.path.join(rocm, "bin", "hipcc")
    return p if os.path.exists(p) else "hipcc"


def build(verbose: bool = False, extra_flags: tuple = ()) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    obj_dir = os.path.join(OUT_DIR, "obj")
    os.makedirs(obj_dir, exist_ok=True)
    hipcc = _hipcc()

    def compile_one(src):
        obj = os.path.join(obj_dir, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"]
        cmd = [hipcc, *lang, *COMMON_FLAGS, *extra_flags, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
        if verbose and r.stderr.strip():
            print(r.stderr, flush=True)
        return obj

    with ThreadPoolExecutor(min(8, len(SOURCES) + len(PROBE_SOURCES))) as ex:
        objs = list(ex.map(compile_one, SOURCES + PROBE_SOURCES))
    for lib, lib_objs in ((LIB, objs[:len(SOURCES)]), (PROBE_LIB, objs[len(SOURCES):])):
        cmd = [hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *lib_objs, "-o", lib + ".tmp"]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(lib + ".tmp", lib)
    build_c_client(verbose)
    return LIB


def c_client_command(src: str, out: str, lib_dir: str = OUT_DIR) -> list:
    """gcc line of the C client: C11 host code against include/xattn.h and the
    HIP runtime API, linked to libxattn.so (found next to the binary)."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
            "-I", os.path.join(rocm, "include"), "-I", os.path.join(ROOT, "include"), src,
            "-L", lib_dir, "-lxattn", "-L", os.path.join(rocm, "lib"), "-lamdhip64", "-lm",
            "-Wl,-rpath,$ORIGIN", "-Wl,-rpath," + os.path.join(rocm, "lib"), "-o", out]


def build_c_client(verbose: bool = False) -> str:
    cmd = c_client_command(os.path.join(ROOT, "tests", "c_client.c"), C_CLIENT + ".tmp")
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"gcc failed on tests/c_client.c:\n{r.stdout}\n{r.stderr}")
    os.replace(C_CLIENT + ".tmp", C_CLIENT)
    return C_CLIENT


if __name__ == "__main__":
    print(build(verbose=True))
