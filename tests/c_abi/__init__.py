"""Build of the plain-C client of the library (abi_check.c): gcc, the HIP runtime's C API,
libsnnlif.so, and the test-side oracle and input generator libraries.  The binary finds the
libraries next to the repository through its run path, so it runs from any directory."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
BIN = os.path.join(HERE, "abi_check")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    """Always recompiles; the libraries it links must be built first."""
    libdirs = [os.path.join(ROOT, d) for d in ("paper_2408_00280_amd", "oracle", "synth")]
    rpath = ":".join("$ORIGIN/" + os.path.relpath(d, HERE) for d in libdirs)
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "oracle"),
           os.path.join(HERE, "abi_check.c"), "-o", BIN + ".tmp",
           *[f"-L{d}" for d in libdirs], "-lsnnlif", "-loracle", "-lsynth",
           f"-L{os.path.join(ROCM, 'lib')}", "-lamdhip64", "-lm", f"-Wl,-rpath,{rpath}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("building the C client failed:\n" + r.stdout + r.stderr)
    os.replace(BIN + ".tmp", BIN)
    return BIN
