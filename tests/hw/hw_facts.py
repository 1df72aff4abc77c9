"""Build and run the gfx950 hardware-fact probe (`hw_facts.hip` beside this file).

    python tests/hw/hw_facts.py --build     # hipcc for gfx950, writes tests/hw/hw_facts (no GPU needed)
    python tests/hw/hw_facts.py             # every rate as a markdown table, then the two checks
    python tests/hw/hw_facts.py --checks    # the two correctness checks only

The rates are measurements of the chip, not of the YOSO kernels; the two checks (fp16 subnormal
products in MFMA, the lane layout of the transposing LDS read) are facts the backward kernels rely on.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "hw_facts.hip")
EXE = os.path.join(HERE, "hw_facts")


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def build() -> str:
    """Compile the probe executable in place; always rebuilds."""
    tmp = EXE + ".tmp"
    cmd = [_hipcc(), "--offload-arch=gfx950", "-O3", "-std=c++17", "-munsafe-fp-atomics",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-o", tmp, SRC]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for hw_facts.hip:\n{res.stderr}")
    os.replace(tmp, EXE)
    return EXE


def run(checks_only: bool, timeout: float = 120.0) -> subprocess.CompletedProcess:
    if not os.path.exists(EXE):
        raise RuntimeError(f"{EXE} is not built (python tests/hw/hw_facts.py --build)")
    args = [EXE] + (["--checks"] if checks_only else [])
    return subprocess.run(args, capture_output=True, text=True, timeout=timeout)


if __name__ == "__main__":
    if "--build" in sys.argv:
        print(build())
        sys.exit(0)
    res = run("--checks" in sys.argv)
    sys.stdout.write(res.stdout)
    sys.stderr.write(res.stderr)
    sys.exit(res.returncode)
