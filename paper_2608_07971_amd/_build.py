"""Build step of the HIP library: compiles csrc/*.hip for gfx950 with hipcc
(one object per source, in parallel) and links paper_2608_07971_amd/libesp.so
(in-tree)."""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libesp.so")
# measurement kernel (streaming ceiling of the table layout), a library of its own
CALIB_LIB = os.path.join(HERE, "libesp_calib.so")
CALIB_SOURCES = ["esp_calib.hip"]
# the fused kernels' instances are split by R over esp_inst_*.hip
SOURCES = ["esp_api.hip", "esp_kernels.hip", "esp_extras.hip",
           "esp_inst_dense12.hip", "esp_inst_dense34.hip", "esp_inst_dense56.hip", "esp_inst_dense78.hip",
           "esp_inst_csr1234.hip", "esp_inst_csr5678.hip"]
ARCH = "gfx950"

COMPILE_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # binary64 scores must match the CPU oracle bit for bit: no contraction
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]
FLAGS = COMPILE_FLAGS + ["-shared"]     # one-step form (kept for tools that compile a single file)


def hipcc() -> str:
    for p in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if p and (os.path.sep not in p or os.path.exists(p)):
            return p
    return "hipcc"


def _jobs() -> int:
    n = int(os.environ.get("MAX_JOBS", "0") or 0) or (os.cpu_count() or 4)
    return max(1, min(n, 16, len(SOURCES) + len(CALIB_SOURCES)))


def build(verbose: bool = False) -> str:
    """Build libesp.so and libesp_calib.so; returns the path of libesp.so."""
    tmpdir = tempfile.mkdtemp(prefix="espbuild", dir=HERE)
    try:
        targets = [(LIB, SOURCES), (CALIB_LIB, CALIB_SOURCES)]
        cmds, objs_of = [], []
        for _, srcs in targets:
            objs = [os.path.join(tmpdir, os.path.splitext(s)[0] + ".o") for s in srcs]
            cmds += [[hipcc(), *COMPILE_FLAGS, "-c", "-o", o, os.path.join(CSRC, s)] for s, o in zip(srcs, objs)]
            objs_of.append(objs)
        if verbose:
            for c in cmds:
                print(" ".join(c), flush=True)
        with cf.ThreadPoolExecutor(max_workers=_jobs()) as ex:
            for f in [ex.submit(subprocess.run, c, check=True) for c in cmds]:
                f.result()
        for (lib, _), objs in zip(targets, objs_of):
            tmp = lib + f".tmp{os.getpid()}"
            link = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
            if verbose:
                print(" ".join(link), flush=True)
            subprocess.run(link, check=True)
            os.replace(tmp, lib)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
