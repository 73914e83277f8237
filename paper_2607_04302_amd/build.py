"""Build libhifa4.so (gfx950) in-tree with hipcc.

Usage: python -m paper_2607_04302_amd.build   (or call build()).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libhifa4.so")
SOURCES = ["hifa4_api.cpp", "hifa4_quant.hip", "hifa4_attn.hip", "hifa4_decode.hip"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 into paper_2607_04302_amd/libhifa4.so.
    Packed-FP32 instructions are disabled on purpose: some of their forms have
    given wrong results intermittently on gfx950 without any error."""
    objs = []
    builddir = os.path.join(HERE, "_build")
    os.makedirs(builddir, exist_ok=True)
    common = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
              "-Wno-unused-result", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
              "-I", os.path.join(HERE, "..", "include")]
    procs = []
    for src in SOURCES:
        obj = os.path.join(builddir, src + ".o")
        lang = ["-x", "hip"]
        cmd = [hipcc(), *common, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
        procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
    failed = False
    for cmd, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        text = "\n".join(l for l in text.splitlines() if "is not a recognized feature" not in l
                         and "unused during compilation" not in l)
        if p.returncode != 0:
            failed = True
            sys.stderr.write(" ".join(cmd) + "\n" + text + "\n")
        elif verbose and text.strip():
            sys.stderr.write(text + "\n")
    if failed:
        raise RuntimeError("libhifa4 compilation failed")
    tmp = LIB + ".tmp"
    subprocess.check_call([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    # the instruction issue-cost probe behind bench.py --issue-probe (not part of the library)
    probe = os.path.join(HERE, "issue_probe")
    subprocess.check_call([hipcc(), "--offload-arch=gfx950", "-O3", "-Xclang", "-target-feature", "-Xclang",
                           "-packed-fp32-ops", os.path.join(CSRC, "issue_probe.hip"), "-o", probe + ".tmp"],
                          stderr=subprocess.DEVNULL)
    os.replace(probe + ".tmp", probe)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
