"""Build libamk.so (the decode megakernel and its C ABI) in-tree for gfx950.

    python -m paper_2606_09682_amd.build      # or build() from Python
"""
from __future__ import annotations

import os
import re
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libamk.so")

ARCH = "gfx950"
# Packed fp32 VALU forms are disabled on purpose: hipcc would otherwise
# generate them from ordinary float code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", os.path.join(ROOT, "include"),
          "-Wall", "-Wno-unused-command-line-argument"]

SOURCES = ["megakernel.hip", "schedule.cpp", "api.cpp"]
# per-kernel register / scratch report of the device code, parsed from the
# compiler's resource-usage remarks
RESOURCES = os.path.join(BUILD, "resource_usage.txt")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    extra = ["-Rpass-analysis=kernel-resource-usage"] if src.endswith(".hip") else []
    cmd = [hipcc()] + COMMON + DEVICE_FLAGS + extra + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if extra:
        _write_resources(r.stderr)
    return obj


def _write_resources(remarks: str) -> None:
    """One line per kernel: name, VGPRs, scratch bytes per lane, spilled VGPRs."""
    rows, cur = [], None
    for line in remarks.splitlines():
        m = re.search(r"remark:\s+(Function Name|VGPRs|ScratchSize \[bytes/lane\]|VGPRs Spill):\s+(\S+)", line)
        if not m:
            continue
        key, val = m.group(1), m.group(2)
        if key == "Function Name":
            cur = {"name": val}
            rows.append(cur)
        elif cur is not None:
            cur[key] = val
    with open(RESOURCES, "w") as f:
        for r in rows:
            f.write(f"{r['name']} vgprs={r.get('VGPRs')} scratch={r.get('ScratchSize [bytes/lane]')} "
                    f"vgpr_spill={r.get('VGPRs Spill')}\n")


def build(verbose: bool = False) -> str:
    """Compile every source and link libamk.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
