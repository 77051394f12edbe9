"""Build libattuner.so for gfx950 with hipcc, in-tree.

    python -m paper_2609_36722_amd.build

Every ``csrc/*.hip`` file is compiled to an object under ``_build/`` at the
repository root (in parallel) and linked into ``paper_2609_36722_amd/libattuner.so``.
"""

from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(PKG_DIR, "libattuner.so")
# the same sources with device-side bounds tests (-DATTUNER_CHECKED)
CHECKED_LIB_PATH = os.path.join(PKG_DIR, "libattuner_checked.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# -packed-fp32-ops: no v_pk_{add,mul,fma}_f32 in generated code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON_FLAGS = [f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-result",
                "-I", INCLUDE, "-I", CSRC]
# Per-source extras (none at present).
EXTRA_FLAGS = {}


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # the host pass does not know the gfx950 feature name: drop that one warning line
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every HIP source and link libattuner.so and, from the same
    sources with -DATTUNER_CHECKED, libattuner_checked.so; return the first's path."""
    _build_one(LIB_PATH, BUILD_DIR, [], verbose, jobs)
    _build_one(CHECKED_LIB_PATH, os.path.join(BUILD_DIR, "checked"), ["-DATTUNER_CHECKED"], verbose, jobs)
    return LIB_PATH


def _build_one(lib_path: str, obj_dir: str, defines, verbose: bool, jobs: int) -> None:
    os.makedirs(obj_dir, exist_ok=True)
    srcs = sources()
    objs = [os.path.join(obj_dir, os.path.basename(s)[:-4] + ".o") for s in srcs]

    def compile_one(pair):
        src, obj = pair
        extra = EXTRA_FLAGS.get(os.path.basename(src), [])
        out = _run([HIPCC, *COMMON_FLAGS, *DEVICE_FLAGS, *defines, *extra, "-c", src, "-o", obj])
        return src, out

    with cf.ThreadPoolExecutor(max_workers=max(1, min(jobs, len(srcs)))) as ex:
        for src, out in ex.map(compile_one, zip(srcs, objs)):
            if verbose:
                print(f"[build] {os.path.relpath(src, ROOT)}", flush=True)
            if verbose and out.strip():
                print(out, flush=True)
    tmp = lib_path + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, lib_path)
    if verbose:
        print(f"[build] linked {os.path.relpath(lib_path, ROOT)}", flush=True)


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
