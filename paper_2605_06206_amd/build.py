"""Build ``libfoe.so`` (gfx950) in-tree with hipcc.

Usage: ``python -m paper_2605_06206_amd.build`` (or ``build()`` from Python).
Every call recompiles.  The result is written next to this file.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(PKG_DIR, "libfoe.so")

SOURCES = ["foe_api.hip", "route.hip", "permute.hip", "ffn.hip", "combine.hip", "attention.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-result",
    # keep the compiler from forming packed fp32 math (v_pk_*_f32) by itself
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libfoe.so)")


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # the host pass warns that it does not know the packed-fp32 feature: harmless
    lines = [ln for ln in p.stdout.splitlines()
             if "packed-fp32-ops" not in ln or "error" in ln.lower()]
    return p.returncode, "\n".join(lines)


def build(verbose: bool = False, extra_flags=(), out_path: str = LIB_PATH) -> str:
    """Compile every source and link ``out_path`` (default: the in-tree library).
    ``extra_flags`` are appended to each compile line (e.g. ``-D`` tile macros)."""
    hipcc = _hipcc()
    with tempfile.TemporaryDirectory(prefix="foe_build_") as tmp:
        objs = []
        cmds = []
        for src in SOURCES:
            obj = os.path.join(tmp, src.replace(".hip", ".o"))
            objs.append(obj)
            cmds.append([hipcc, *HIPCC_FLAGS, *extra_flags, "-I", INCLUDE, "-I", CSRC, "-c",
                         os.path.join(CSRC, src), "-o", obj])
        jobs = min(len(cmds), int(os.environ.get("MAX_JOBS", "8")))
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            results = list(ex.map(_run, cmds))
        for cmd, (rc, out) in zip(cmds, results):
            if verbose and out.strip():
                print(out)
            if rc != 0:
                raise RuntimeError(f"hipcc failed ({rc}): {' '.join(cmd)}\n{out}")
        tmp_lib = os.path.join(tmp, "libfoe.so")
        rc, out = _run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp_lib, *objs])
        if rc != 0:
            raise RuntimeError(f"link failed ({rc}):\n{out}")
        staged = out_path + ".tmp"
        shutil.copyfile(tmp_lib, staged)
        os.replace(staged, out_path)
    return out_path


if __name__ == "__main__":
    path = build(verbose="-v" in sys.argv)
    print(path)
