"""Build libecmoe.so (the HIP library behind include/ec_moe.h) in-tree for gfx950.

Usage: python -m paper_2604_01622_amd.build [--debug]

Every source is compiled with hipcc for gfx950 only; packed fp32 instructions
are disabled in the device code (-packed-fp32-ops).  The host pass of hipcc
warns that it does not know that feature, which is harmless.
"""
from __future__ import annotations

import argparse
import os
import re
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libecmoe.so")
BUILD_DIR = os.path.join(ROOT, "_build")
SOURCES = ["router.hip", "topk.hip", "tc.hip", "movement.hip", "gemm.hip", "ec_api.cpp"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def flags(debug: bool):
    f = ["--offload-arch=gfx950", "-std=c++17", "-fPIC", "-O3",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-Wno-unused-result", "-Werror=uninitialized"]
    if debug:
        f += ["-g"]
    return f


def build(debug: bool = False, verbose: bool = False, jobs: int = 8) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    cc = hipcc()
    fl = flags(debug)

    def compile_one(src):
        obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
        cmd = [cc, *fl, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        err = "\n".join(ln for ln in r.stderr.splitlines()
                        if "packed-fp32-ops' is not a recognized feature" not in ln)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{err}")
        if verbose and err.strip():
            print(err, file=sys.stderr)
        return obj

    with ThreadPoolExecutor(max(1, jobs)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [cc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, OUT)
    return OUT


_RES_KEYS = {"VGPRs": "vgpr", "AGPRs": "agpr", "ScratchSize [bytes/lane]": "scratch",
             "Occupancy [waves/SIMD]": "occupancy", "LDS Size [bytes/block]": "lds"}


def resource_usage(src: str) -> dict:
    """Per-kernel register, scratch and LDS use of one source, as the compiler
    reports it for gfx950 (device-only compile to a temporary object)."""
    import tempfile
    with tempfile.TemporaryDirectory() as td:
        cmd = [hipcc(), *flags(False), "--cuda-device-only", "-x", "hip", "-c",
               os.path.join(CSRC, src), "-o", os.path.join(td, "res.o"),
               "-Rpass-analysis=kernel-resource-usage"]
        r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    out, cur = {}, None
    for ln in r.stderr.splitlines():
        m = re.search(r"remark: (?:\s*)(.+?): (\S+) \[-Rpass-analysis", ln)
        if not m:
            continue
        key, val = m.group(1).strip(), m.group(2)
        if key == "Function Name":
            cur = out.setdefault(val, {})
        elif cur is not None and key in _RES_KEYS:
            cur[_RES_KEYS[key]] = int(val)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--debug", action="store_true")
    ap.add_argument("-v", "--verbose", action="store_true")
    a = ap.parse_args()
    print(build(a.debug, a.verbose))


if __name__ == "__main__":
    main()
