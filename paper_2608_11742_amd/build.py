"""Build libdllm_rps.so for gfx950 with hipcc (in-tree, next to this file)."""
from __future__ import annotations

import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJ = os.path.join(ROOT, "_build", "obj")
LIB = os.path.join(HERE, "libdllm_rps.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = ["-Rpass-analysis=kernel-resource-usage", "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
         # packed fp32 instructions stay off: hipcc must not emit v_pk_{add,mul,fma}_f32
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-result"]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


# Kernels allowed a small spill area (mangled-name fragment -> bytes per lane).
# The LM head with 256-row tiles keeps a few loop-invariant scalars (row-scale
# indexing, descriptor words) in scratch: they are stored once and reloaded
# once per 256 x 256 x d tile, outside the MFMA loop, which spills nothing.
SCRATCH_ALLOWED = {"lmhead_kernelINS_6bf16_tELi256E": 64, "lmhead_kernelIfLi256E": 64}


def _scratch_users(remarks: str):
    """Kernels whose resource-usage remarks report more private scratch memory
    than they are allowed."""
    users, fn = [], None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            fn = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and int(m.group(1)) > 0:
            allowed = max((v for k, v in SCRATCH_ALLOWED.items() if k in (fn or "")), default=0)
            if int(m.group(1)) > allowed:
                users.append((fn, int(m.group(1))))
    return users


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.basename(src)[:-4] + ".o")
    cmd = [HIPCC, *FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    lines = (r.stderr or "").splitlines()
    err = "\n".join(l for l in lines if "packed-fp32-ops" not in l and "remark:" not in l
                    and "kernel-resource-usage" not in l and not re.match(r"^\s*(\d+\s*)?\|", l))
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if err.strip():
        print(err, file=sys.stderr)
    # register arrays indexed at run time end up in scratch memory and make a
    # kernel an order of magnitude slower: refuse such a build
    users = _scratch_users(r.stderr or "")
    if users:
        raise RuntimeError(f"{src}: kernels use scratch memory: {users}")
    return obj


def build(jobs: int = 8) -> str:
    os.makedirs(OBJ, exist_ok=True)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, sources()))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
