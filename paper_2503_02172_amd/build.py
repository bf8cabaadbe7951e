"""Build libkgq.so (HIP, gfx950) in-tree with hipcc.

Every HIP source is compiled with packed-FP32 instructions disabled
(``-Xclang -target-feature -Xclang -packed-fp32-ops``); the scorer is also
compiled with ``-fno-honor-nans`` so that min() on scalar operands needs no
NaN-canonicalising instruction in the inner loop. After linking, the
disassembly of the device code is checked for packed FP32 instructions.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build", "kgq")
OUT = os.path.join(HERE, "libkgq.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I" + os.path.join(ROOT, "include"),
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wall", "-Wno-unused-result"]
EXTRA = {"k_score.hip": ["-fno-honor-nans"]}
SOURCES = ["kgq_api.cpp", "plan.cpp", "k_embed.hip", "k_gemm.hip", "k_score.hip", "k_score_kl.hip", "k_topk.hip",
           "k_rank.hip", "k_cone_logice.hip"]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, src + ".o")
    cmd = [HIPCC] + COMMON + EXTRA.get(src, [])
    if src.endswith(".cpp"):
        cmd += ["-x", "hip"]
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in ln]
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n" + "\n".join(msgs))
    if msgs and verbose:
        print("\n".join(msgs))
    return obj


def check_no_packed_fp32(lib: str) -> None:
    """Fail if the device code contains packed FP32 arithmetic."""
    bundler = "/opt/rocm/llvm/bin/clang-offload-bundler"
    objdump = "/opt/rocm/llvm/bin/llvm-objdump"
    if not (os.path.exists(bundler) and os.path.exists(objdump)):
        return
    co = os.path.join(BUILD, "device.co")
    fb = os.path.join(BUILD, "device.fatbin")
    objs = [os.path.join(BUILD, s + ".o") for s in SOURCES if s.endswith(".hip")]
    bad = []
    for o in objs:
        # the device code object sits, bundled, in the .hip_fatbin section
        subprocess.run(["objcopy", "--dump-section", f".hip_fatbin={fb}", o], check=True,
                       capture_output=True)
        subprocess.run([bundler, "--type=o", f"--targets=hipv4-amdgcn-amd-amdhsa--{ARCH}",
                        f"--input={fb}", f"--output={co}", "--unbundle"], check=True,
                       capture_output=True, text=True)
        d = subprocess.run([objdump, "-d", co], capture_output=True, text=True, check=True).stdout
        if "v_" not in d:
            raise RuntimeError(f"no device code found in {o}")
        hits = re.findall(r"v_pk_(?:add|mul|fma)_f32", d)
        if hits:
            bad.append(f"{os.path.basename(o)}: {len(hits)}")
    if bad:
        raise RuntimeError("packed FP32 instructions in device code: " + ", ".join(bad))


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    check_no_packed_fp32(tmp)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
