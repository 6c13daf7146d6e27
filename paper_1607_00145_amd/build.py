"""Build the gfx950 shared library libgett.so from csrc/ (hipcc, in-tree).

    python -m paper_1607_00145_amd.build [-j N] [--incremental] [--sanitize]

Objects go to _build/ at the repository root; the library to
paper_1607_00145_amd/lib/libgett.so.  --sanitize builds
paper_1607_00145_amd/lib/libgett_asan.so instead (objects in _build/asan/):
the host code (planner, C interface, launchers) instrumented with
AddressSanitizer and UndefinedBehaviorSanitizer, the device code as usual; a
process loads it with the sanitizer runtime preloaded (tests/run_sanitized.sh).
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libgett.so")
LIB_ASAN = os.path.join(LIBDIR, "libgett_asan.so")
# host-only sanitizer flags (each -fsanitize= right after -Xarch_host: the
# device code is not instrumented)
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer", "-g"]
ARCH = "gfx950"
ROCM_LIB = "/opt/rocm/lib"


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
          "-I" + os.path.join(ROOT, "include")]
# Packed fp32 instructions are turned off for every device compile.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


# Translation units built once per tile shape (GETT_TILE = 0 .. n-1) and once
# without it, so the kernel instantiations compile in parallel.
PER_TILE = {"launch_f32.hip": "kTilesF32", "launch_f64.hip": "kTilesF64"}


def tile_count(array: str) -> int:
    """Entries of a tile table in tiles.hpp."""
    text = open(os.path.join(CSRC, "tiles.hpp")).read()
    body = text[text.index(array + "[] = {"):]
    body = body[:body.index("};")]
    return sum(1 for line in body.splitlines() if line.strip().startswith("{"))


def jobs_of(src: str):
    """(source, tile or None) compile jobs of one source file."""
    if src in PER_TILE:
        return [(src, None)] + [(src, t) for t in range(tile_count(PER_TILE[src]))]
    return [(src, None)]


def sources():
    return sorted(f for f in os.listdir(CSRC) if f.endswith((".cpp", ".hip")))


def newest_input() -> float:
    """Modification time of the newest source or header the objects depend on."""
    files = [os.path.join(CSRC, f) for f in os.listdir(CSRC)]
    files += [os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))]
    return max(os.path.getmtime(f) for f in files)


def compile_one(job, incremental: bool = False, sanitize: bool = False) -> str:
    src, tile = job
    bdir = os.path.join(BUILD, "asan") if sanitize else BUILD
    os.makedirs(bdir, exist_ok=True)
    obj = os.path.join(bdir, src + ("" if tile is None else f".t{tile}") + ".o")
    if incremental and os.path.exists(obj) and os.path.getmtime(obj) >= newest_input():
        return obj
    cmd = [hipcc()] + COMMON + (SANITIZE if sanitize else [])
    if src.endswith(".hip"):
        cmd += DEVICE + ["-x", "hip"]
    if tile is not None:
        cmd += [f"-DGETT_TILE={tile}"]
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if r.stderr.strip():
        # hipcc's host pass does not know the device-only feature flag; drop that note
        lines = [l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip()]
        if lines:
            sys.stderr.write("\n".join(lines) + "\n")
    return obj


def build(jobs: int = 0, incremental: bool = False, sanitize: bool = False) -> str:
    """Compile every source (or, incremental, only those whose object is older
    than the newest source or header) and link libgett.so (libgett_asan.so
    with the host sanitizers)."""
    work = [j for src in sources() for j in jobs_of(src)]
    # the largest units first, so they do not end up last on one worker
    work.sort(key=lambda j: (j[0] not in PER_TILE, j[1] is None))
    jobs = jobs or min(len(work), os.cpu_count() or 4)
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda j: compile_one(j, incremental, sanitize), work))
    os.makedirs(LIBDIR, exist_ok=True)
    out = LIB_ASAN if sanitize else LIB
    tmp = out + f".tmp{os.getpid()}"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs + \
        ["-L" + ROCM_LIB, "-lrocblas", "-Wl,-rpath," + ROCM_LIB]
    if sanitize:
        cmd += ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("-j", type=int, default=0)
    ap.add_argument("--incremental", action="store_true",
                    help="recompile only objects older than the newest source or header")
    ap.add_argument("--sanitize", action="store_true",
                    help="host AddressSanitizer + UndefinedBehaviorSanitizer build (libgett_asan.so)")
    a = ap.parse_args()
    print(build(a.j, a.incremental, a.sanitize))
