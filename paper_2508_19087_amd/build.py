"""Builds libapt.so, the gfx950 HIP library behind include/apt.h, in-tree.

Each source in csrc/ is compiled to an object with hipcc in parallel, then the
objects are linked into paper_2508_19087_amd/libapt.so.  A source named
*_inst.hip instantiates kernels for one weight bit width and is compiled once
per width with -DAPT_INST_P=1..8.  The measurement probes in probes/ (not part
of the library) are linked into a library of their own, libapt_probe.so, which
only bench.py loads.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
PROBES = os.path.join(HERE, "probes")
PROBE_LIB = os.path.join(HERE, "libapt_probe.so")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libapt.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
    # packed fp32 VALU ops stay off (plain float code only)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def units(directory=CSRC):
    """(source, extra flags, object name) of every compilation unit."""
    out = []
    for f in sorted(os.listdir(directory)):
        if not f.endswith(".hip"):
            continue
        src = os.path.join(directory, f)
        if f.endswith("_inst.hip"):
            for p in range(1, 9):
                out.append((src, ["-DAPT_INST_P=%d" % p], f[:-4] + "_p%d.o" % p))
        else:
            out.append((src, [], f[:-4] + ".o"))
    return out


def _compile(unit) -> str:
    src, extra, name = unit
    obj = os.path.join(BUILD, name)
    cmd = [HIPCC] + CFLAGS + extra + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, r.stdout, r.stderr))
    return obj


def _link(objs, lib):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC"] + objs + ["-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (r.stdout, r.stderr))
    os.replace(tmp, lib)


def build(jobs: int | None = None, verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    todo = units()
    probes = [(src, extra, "probe_" + name) for src, extra, name in units(PROBES)]
    jobs = jobs or min(len(todo), max(1, min(16, os.cpu_count() or 1)))
    # longest units first
    todo.sort(key=lambda u: -os.path.getsize(u[0]) - (10 ** 6 if u[1] else 0))
    with concurrent.futures.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, todo + probes))
    _link(objs[:len(todo)], LIB)
    if probes:
        _link(objs[len(todo):], PROBE_LIB)
    if verbose:
        print("built", LIB, "and", PROBE_LIB if probes else "")
    return LIB


def clean():
    shutil.rmtree(BUILD, ignore_errors=True)
    for lib in (LIB, PROBE_LIB):
        if os.path.exists(lib):
            os.remove(lib)


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
