"""Builds libec2moe.so in-tree with hipcc for gfx950.

    python -m paper_2508_06024_amd.build

Every source under csrc/ is compiled to an object (in parallel) and linked into
paper_2508_06024_amd/libec2moe.so next to this file. With --incremental, sources whose
object is newer than the source and every project header it includes are not
recompiled (a development shortcut; the default rebuilds everything).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libec2moe.so")
BUILD_DIR = os.path.join(ROOT, "_build")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
          "-Wall", "-Wno-unused-function",
          # packed fp32 arithmetic stays off in all device code
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def sources():
    return sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


def _deps(path: str, seen=None) -> set:
    """The file and every project header it includes, transitively (#include "...")."""
    seen = set() if seen is None else seen
    if path in seen:
        return seen
    seen.add(path)
    for line in open(path):
        line = line.strip()
        if line.startswith('#include "'):
            name = line.split('"')[1]
            for d in (CSRC, INCLUDE):
                cand = os.path.join(d, name)
                if os.path.exists(cand):
                    _deps(cand, seen)
                    break
    return seen


def _up_to_date(src: str) -> bool:
    obj = os.path.join(BUILD_DIR, src + ".o")
    if not os.path.exists(obj):
        return False
    t = os.path.getmtime(obj)
    return all(t > os.path.getmtime(f) for f in _deps(os.path.join(CSRC, src)))


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, src + ".o")
    cmd = [HIPCC, *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    # the host pass does not know the device-only feature flag; drop that known warning
    noise = [ln for ln in r.stderr.splitlines() if "packed-fp32-ops" not in ln and ln.strip()]
    if noise:
        sys.stderr.write(f"[{src}]\n" + "\n".join(noise) + "\n")
    return obj


def build(verbose: bool = True, incremental: bool = False) -> str:
    if not shutil.which(HIPCC) and not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sources()
    todo = [s for s in srcs if not (incremental and _up_to_date(s))]
    if todo:
        with ThreadPoolExecutor(min(8, len(todo))) as ex:
            list(ex.map(_compile, todo))
    objs = [os.path.join(BUILD_DIR, s + ".o") for s in srcs]
    tmp = LIB + ".tmp"
    r = subprocess.run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,--no-undefined",
                        "-o", tmp, *objs],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB} from {len(srcs)} sources ({len(todo)} compiled)")
    return LIB


if __name__ == "__main__":
    build(incremental="--incremental" in sys.argv[1:])
