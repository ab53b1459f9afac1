"""Build libnestquant.so (the HIP kernels and the C ABI) for gfx950 with hipcc, in-tree.

Usage: python -m paper_2502_09720_amd.build
"""

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libnestquant.so")

SOURCES = ["nq_api.cpp", "nq_encode.hip", "nq_decode.hip", "nq_matmul.hip", "nq_gemm.hip",
           "nq_fused.hip", "nq_rotate.hip", "nq_beta.hip", "nq_host.cpp",
           "nq_static.hip"]

# -ffp-contract=off: the exact-sign logic needs every product and sum rounded separately.
# -packed-fp32-ops off: no v_pk_*_f32 in the generated code.
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    log = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + log)
    return log


def build(verbose=False):
    """Compile every source to an object in parallel (a temporary directory), then link."""
    import concurrent.futures
    import tempfile
    with tempfile.TemporaryDirectory(prefix="nq_build_") as tmpdir:
        objs, cmds = [], []
        for src in SOURCES:
            obj = os.path.join(tmpdir, src + ".o")
            objs.append(obj)
            cmds.append([hipcc(), *[f for f in FLAGS if f != "-shared"], "-c", "-I", INCLUDE,
                         "-o", obj, os.path.join(CSRC, src)])
        workers = max(1, min(len(cmds), os.cpu_count() or 1))
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            logs = list(ex.map(_run, cmds))
        tmp = LIB + ".tmp"
        logs.append(_run([hipcc(), *FLAGS, "-o", tmp] + objs))
    if verbose:
        for log in logs:
            if log.strip():
                print(log)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
