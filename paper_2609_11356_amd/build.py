"""Build libdg.so (HIP for gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libdg.so")
SOURCES = ["dg_api.cpp", "dg_gemm.hip", "dg_panel.hip", "dg_rowsum.hip", "dg_attn.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# -ffp-contract=off: no multiply-add is fused unless the source spells it out.
# -packed-fp32-ops off: packed fp32 VALU forms are kept out of the code.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-ffp-contract=off", "-fno-fast-math",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-command-line-argument",
         "-Rpass-analysis=kernel-resource-usage"]


def spilling_kernels(remarks: str) -> list[str]:
    """Kernels whose resource-usage remark reports spilled VGPRs.

    No kernel here is meant to spill: the spill code of a kernel that did was
    seen to drop part of a spilled 16-byte register, so a spill fails the build.
    """
    bad, name = [], None
    for line in remarks.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split()[0]
        elif "VGPRs Spill:" in line and name is not None:
            n = int(line.split("VGPRs Spill:")[1].split()[0])
            if n:
                bad.append("%s (%d VGPRs)" % (name, n))
    return bad


def _compile(src: str, obj: str) -> tuple[int, str]:
    flags = [f for f in FLAGS if f != "-shared"]
    r = subprocess.run([HIPCC] + flags + ["-c", "-o", obj, src], capture_output=True, text=True)
    return r.returncode, r.stdout + r.stderr


def build(verbose: bool = False) -> str:
    """Compile every source to an object in parallel, then link them."""
    from concurrent.futures import ThreadPoolExecutor
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = [os.path.join(objdir, os.path.basename(s) + ".%d.o" % os.getpid()) for s in srcs]
    with ThreadPoolExecutor(max_workers=min(len(srcs), os.cpu_count() or 1)) as ex:
        results = list(ex.map(lambda so: _compile(*so), zip(srcs, objs)))
    text = "\n".join(t for _, t in results)
    tmp = LIB + ".tmp%d" % os.getpid()
    rc = max(r for r, _ in results)
    if rc == 0:
        r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs,
                           capture_output=True, text=True)
        rc, text = r.returncode, text + r.stdout + r.stderr
    for o in objs:
        if os.path.exists(o):
            os.unlink(o)
    # the resource remarks (and their source-context lines) are read, not shown
    out = "\n".join(l for l in text.splitlines()
                    if "packed-fp32-ops" not in l and "kernel-resource-usage" not in l
                    and not re.match(r"^\s*\d*\s*\|", l) and l.strip())
    if rc != 0:
        raise RuntimeError("hipcc failed:\n" + out)
    spills = spilling_kernels(text)
    if spills:
        os.unlink(tmp)
        raise RuntimeError("kernels spill registers: " + ", ".join(spills))
    # a kernel template whose host-side stub was not emitted links silently
    # and fails only when the library is loaded
    nm = subprocess.run(["nm", "--undefined-only", tmp], capture_output=True, text=True)
    stubs = [l.split()[-1] for l in nm.stdout.splitlines() if "__device_stub__" in l]
    if nm.returncode == 0 and stubs:
        os.unlink(tmp)
        raise RuntimeError("kernel stubs missing from the library: " + ", ".join(stubs[:4]))
    if verbose and out:
        print(out, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
