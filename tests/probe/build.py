"""Build the probe kernels (test infrastructure) with hipcc: raw MFMAs, and
the library's device exp / SiLU over ranges of binary32 inputs."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libmfma_probe.so")
MATH_LIB = os.path.join(HERE, "libmath_probe.so")
CHECK_LIB = os.path.join(os.path.dirname(HERE), "checker", "libcheck_fixtures.so")


def _hipcc(src, lib, extra=()):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [os.environ.get("HIPCC", "/opt/rocm/bin/hipcc"), "--offload-arch=gfx950", "-O2", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *extra,
           "-o", tmp, os.path.join(HERE, src)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError(r.stdout + r.stderr)
    os.replace(tmp, lib)
    return lib


def build():
    # the math probe is compiled as the library is (no contraction, no fast math)
    _hipcc("math_probe.hip", MATH_LIB, ("-O3", "-ffp-contract=off", "-fno-fast-math"))
    # the order checker's fixtures, with the flags the checker compiles them with
    _hipcc(os.path.join("..", "checker", "launch.hip"), CHECK_LIB, ("-O3", "-std=c++17", "-ffp-contract=off",
                                                                     "-fno-fast-math"))
    return _hipcc("mfma_probe.hip", LIB)
