"""Build libhcms.so (the HIP library behind include/hcms.h) for gfx950.

Usage: ``python -m paper_2607_01817_amd.build`` or ``build()`` from Python.
Every call recompiles.  Objects go to ``_build/`` beside this file; the
library is written in-tree as ``libhcms.so``.
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libhcms.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["api.cpp", "model.cpp", "pack.hip", "attention.hip", "attention_bwd.hip", "linear.hip"]

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    "-Wall", "-Wno-unused-result",
    # Packed fp32 VALU instructions are kept out of every kernel.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


# Resource limits checked on every kernel after compilation.  The kernels
# that load into LDS by inline asm count their own outstanding vector memory
# instructions (s_waitcnt vmcnt(N)); a register spill would add scratch
# accesses those counts do not include, and an SGPR reloaded from a VGPR lane
# (a VALU write) right before such a load is a dependency the compiler does
# not see inside the asm.  So no kernel may spill or use scratch.  The VGPR
# budgets keep room for a copy wave (at most 16 VGPRs) beside an attention
# workgroup's two waves per SIMD.
_RESOURCE_REMARK = "-Rpass-analysis=kernel-resource-usage"
VGPR_BUDGET = {"attention_dma_kernel": 248, "pack_kernel": 16, "unpack_kernel": 16}


def parse_resource_remarks(text: str) -> dict:
    """Per kernel (mangled name) the integer fields of the compiler's
    kernel-resource-usage remarks: VGPRs, SGPRs Spill, VGPRs Spill, ScratchSize."""
    out: dict = {}
    cur = None
    for ln in text.splitlines():
        if "remark:" not in ln or _RESOURCE_REMARK not in ln:
            continue
        body = ln.split("remark:", 1)[1].replace(f"[{_RESOURCE_REMARK}]", "").strip()
        key, _, val = body.partition(":")
        key, val = key.strip(), val.strip()
        if key == "Function Name":
            cur = val
            out[cur] = {}
        elif cur is not None and val.lstrip("-").isdigit():
            out[cur][key.split(" [")[0]] = int(val)
    return out


def resource_problems(res: dict) -> list:
    """Spills, scratch and VGPR budgets exceeded, as messages."""
    bad = []
    for name, r in res.items():
        for key in ("SGPRs Spill", "VGPRs Spill", "ScratchSize"):
            if r.get(key, 0) > 0:
                bad.append(f"{name}: {key} {r[key]}")
        for kern, cap in VGPR_BUDGET.items():
            # Mangled names carry each identifier as <length><name>.
            if f"{len(kern)}{kern}" in name and r.get("VGPRs", 0) > cap:
                bad.append(f"{name}: {r['VGPRs']} VGPRs > {cap}")
    return bad


def _compile(src: str, verbose: bool) -> tuple:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON, _RESOURCE_REMARK, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    text = r.stdout + r.stderr
    msgs = [ln for ln in text.splitlines()
            if "packed-fp32-ops" not in ln and _RESOURCE_REMARK not in ln and ln.strip()
            and not ln.lstrip()[:1].isdigit() and ln.strip() not in ("|", "^")
            and not ln.strip().startswith("| ")]
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n" + "\n".join(msgs))
    if msgs and verbose:
        print("\n".join(msgs), flush=True)
    return obj, parse_resource_remarks(text)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        done = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    objs = [o for o, _ in done]
    res = {k: v for _, r in done for k, v in r.items()}
    if not res:
        raise RuntimeError("no kernel-resource-usage remarks found: the resource guard cannot check "
                           "the kernels (compiler remark format changed?)")
    bad = resource_problems(res)
    if bad:
        raise RuntimeError("kernel resource limits exceeded:\n" + "\n".join(bad))
    if verbose:
        print(f"{len(res)} kernels: no spills, no scratch, VGPR budgets kept", flush=True)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
