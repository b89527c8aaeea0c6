"""Build libdps.so (HIP kernels + C ABI) and libdps_probe.so (the ceiling
probes the benchmark measures against) for gfx950 with hipcc.

Usage: python -m paper_2609_34380_amd.csrc.build  (or build() from Python).
Objects go to paper_2609_34380_amd/_build/, the libraries to
paper_2609_34380_amd/.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libdps.so")
PROBE_LIB = os.path.join(PKG, "libdps_probe.so")
PROBE_SOURCES = ["dps_probe.hip"]
SOURCES = ["dps_elementwise.hip", "dps_skinny.hip", "dps_gemv.hip", "dps_rows.hip", "dps_gemm.hip",
           "dps_restore.hip", "dps_api.hip", "dps_sum.cpp", "dps_vmm.hip",
           "dps_worker.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH, "-fvisibility=hidden",
    "-Wall", "-Wno-unused-function",
    # no packed-fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", HERE,
]


# Kernel sources whose kernels must not use scratch: a spill or a stack array
# in a streaming or matrix-core kernel adds memory traffic beside the weight
# stream and costs time with no error, so the build fails on it instead.
NO_SCRATCH = {"dps_elementwise.hip", "dps_skinny.hip", "dps_gemv.hip", "dps_rows.hip",
              "dps_gemm.hip", "dps_probe.hip"}


def _scratch_users(report):
    """Kernels with non-zero scratch in a -Rpass-analysis=kernel-resource-usage
    report."""
    users, name = [], None
    for line in report.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split("[")[0].strip()
        elif "ScratchSize [bytes/lane]:" in line and name:
            size = int(line.split("ScratchSize [bytes/lane]:")[1].split("[")[0])
            if size:
                users.append((name, size))
    return users


def _compile(src):
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    extra = ["-Rpass-analysis=kernel-resource-usage"] if src in NO_SCRATCH else []
    cmd = [HIPCC, *CFLAGS, *extra, "-c", os.path.join(HERE, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = r.stdout + r.stderr
    rc = r.returncode
    if rc == 0 and src in NO_SCRATCH:
        users = _scratch_users(out)
        if users:
            out = "kernels of %s use scratch: %s\n" % (src, users)
            rc = 1
        else:
            out = ""
    return src, obj, rc, out, cmd


def _link(objs, lib, verbose):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=" + ARCH, *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)


def build(verbose=False, jobs=None):
    os.makedirs(BUILD_DIR, exist_ok=True)
    every = SOURCES + PROBE_SOURCES
    jobs = jobs or min(len(every), max(1, (os.cpu_count() or 2) // 2))
    objs = {}
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        for src, obj, rc, out, cmd in ex.map(_compile, every):
            if verbose:
                print(" ".join(cmd), flush=True)
            if rc != 0:
                sys.stderr.write(out)
                raise RuntimeError("hipcc failed on %s" % src)
            if out.strip() and verbose:
                sys.stderr.write(out)
            objs[src] = obj
    _link([objs[s] for s in SOURCES], LIB, verbose)
    _link([objs[s] for s in PROBE_SOURCES], PROBE_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
