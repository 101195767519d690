"""Compile the HIP library libsnnlif.so for gfx950 (in-tree, next to this file).

The kernel variants are split over several translation units (one per forward I/O dtype and
spike format, one per backward I/O dtype, the same for the gain-fed layer and for the
stack fused across depth, the gain kernels, the serial baseline, the C ABI) that compile in
parallel and link into one shared library.
"""
from __future__ import annotations

import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libsnnlif.so")
OBJ_DIR = os.path.join(HERE, "_build")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # the membrane update must be one IEEE multiply and one IEEE add, never a fused FMA
    "-ffp-contract=off",
    # no packed-fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]

# (object name, source, defines)
UNITS = (
    [(f"fwd_io{io}_spk{spk}", "lif_forward.hip", [f"-DSNNLIF_IO={io}", f"-DSNNLIF_SPK={spk}"])
     for io in (0, 1) for spk in (0, 1, 2)]
    + [(f"fwdgain_io{io}_spk{spk}", "lif_forward.hip", [f"-DSNNLIF_IO={io}", f"-DSNNLIF_SPK={spk}", "-DSNNLIF_GAIN=1"])
       for io in (0, 1) for spk in (0, 1, 2)]
    + [(f"bwd_io{io}", "lif_backward.hip", [f"-DSNNLIF_IO={io}"]) for io in (0, 1)]
    + [(f"bwdgain_io{io}_spk{spk}", "lif_backward.hip", [f"-DSNNLIF_IO={io}", f"-DSNNLIF_SPK={spk}", "-DSNNLIF_GAIN=1"])
       for io in (0, 1) for spk in (0, 1, 2)]
    + [(f"stackf_io{io}_spk{spk}", "lif_stack.hip", [f"-DSNNLIF_IO={io}", f"-DSNNLIF_SPK={spk}"])
       for io in (0, 1) for spk in (0, 1, 2)]
    + [(f"stackb_io{io}", "lif_stack.hip", [f"-DSNNLIF_IO={io}", "-DSNNLIF_STACK_BWD=1"]) for io in (0, 1)]
    + [("glue", "lif_glue.hip", []), ("serial", "lif_serial.hip", []), ("api", "snn_lif_api.hip", [])]
)


def _compile(unit, extra):
    name, src, defs = unit
    obj = os.path.join(OBJ_DIR, name + ".o")
    cmd = ["hipcc", *HIPCC_FLAGS, *extra, *defs, "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "'-packed-fp32-ops' is not a recognized feature for this target (ignoring feature)"
    msgs = "\n".join(ln for ln in (r.stdout + r.stderr).splitlines() if noise not in ln)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {name}:\n{msgs}")
    return obj


def build(out: str = OUT, extra=(), jobs: int | None = None) -> str:
    """Always recompiles every translation unit, then links."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    jobs = jobs or min(len(UNITS), os.cpu_count() or 4)
    with ThreadPoolExecutor(max_workers=jobs) as pool:
        objs = list(pool.map(lambda u: _compile(u, list(extra)), UNITS))
    subprocess.run(["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", out + ".tmp"], check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build())
