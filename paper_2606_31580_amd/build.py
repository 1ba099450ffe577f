"""Builds liblaser.so for gfx950 in-tree (paper_2606_31580_amd/lib/liblaser.so).

Every call recompiles: the HIP sources with hipcc --offload-arch=gfx950 (packed fp32
instructions disabled), the C controller with gcc, then links one shared library; and the
stand-alone design-probe program (lib/design_probes, run by bench.py --design-probes).
Usage: python -m paper_2606_31580_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJ = os.path.join(PKG, "_build")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "liblaser.so")
# measurement program behind the kernel structure (bench.py --design-probes); not part of the library
PROBES_SRC = os.path.join(PKG, "probes", "design_probes.hip")
PROBES = os.path.join(LIBDIR, "design_probes")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
HIP_SOURCES = ["gemm.hip", "attn.hip", "misc.hip", "runtime.cpp", "pages.cpp"]
C_SOURCES = ["controller.c", "sim.c"]
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-result",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]
C_FLAGS = ["-O2", "-fPIC", "-std=c99", "-Wall", "-ffp-contract=off", f"-I{INCLUDE}", f"-I{CSRC}"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    return r.returncode, out


def _compile(src):
    path = os.path.join(CSRC, src)
    obj = os.path.join(OBJ, src + ".o")
    if src.endswith(".c"):
        cmd = ["gcc", *C_FLAGS, "-c", path, "-o", obj]
    else:
        cmd = [HIPCC, *HIP_FLAGS, "-x", "hip", "-c", path, "-o", obj]
    rc, out = _run(cmd)
    return src, obj, rc, out, cmd


def build(verbose: bool = False) -> str:
    os.makedirs(OBJ, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    jobs = min(8, max(1, len(os.sched_getaffinity(0))))
    objs, failed = [], []
    probe_cmd = [HIPCC, *HIP_FLAGS, "-o", PROBES + ".tmp", PROBES_SRC]
    with cf.ThreadPoolExecutor(jobs) as ex:
        probe_job = ex.submit(_run, probe_cmd)
        for src, obj, rc, out, cmd in ex.map(_compile, HIP_SOURCES + C_SOURCES):
            if rc != 0:
                failed.append((src, out, cmd))
            elif verbose and out.strip():
                print(f"[{src}]\n{out}")
            objs.append(obj)
        rc, out = probe_job.result()
        if rc != 0:
            failed.append(("probes/design_probes.hip", out, probe_cmd))
        else:
            os.replace(PROBES + ".tmp", PROBES)
    if failed:
        msg = "\n".join(f"--- {s} ---\n{' '.join(c)}\n{o}" for s, o, c in failed)
        raise RuntimeError("liblaser build failed:\n" + msg)
    tmp = LIB + ".tmp"
    rc, out = _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    if rc != 0:
        raise RuntimeError("liblaser link failed:\n" + out)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
