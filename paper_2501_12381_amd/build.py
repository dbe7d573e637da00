"""Build libgspn.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

    python -m paper_2501_12381_amd.build        # or __graft_entry__.build()

Each source compiles to an object in parallel under _build/, then one link
produces paper_2501_12381_amd/libgspn.so next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libgspn.so")
ARCH = "gfx950"

# packed fp32 ops are disabled: hipcc still vectorises plain float code, but
# the packed forms are kept out of the code objects.
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-command-line-argument"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libgspn.so)")


# units that take minutes to compile (one large kernel each, or many
# instantiations); they start first so the parallel build is not left waiting
# on one of them at the end
SLOW_UNITS = ("gspn_widebwdlg_", "gspn_large_", "gspn_widebwd_", "gspn_resfwd_", "gspn_hadja_", "gspn_hadjb_",
              "gspn_widefwd_", "gspn_staged_")


def sources() -> list[str]:
    names = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    rank = lambda f: next((i for i, p in enumerate(SLOW_UNITS) if f.startswith(p)), len(SLOW_UNITS))
    return [os.path.join(CSRC, f) for f in sorted(names, key=rank)]


def _run(cmd: list[str]) -> None:
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}")
    for line in (r.stdout + r.stderr).splitlines():
        if "error" in line.lower():
            sys.stderr.write(line + "\n")


def _deps(dep_file: str) -> list[str]:
    """Files listed in a make-style dependency file written by the compiler."""
    try:
        text = open(dep_file).read().replace("\\\n", " ")
    except OSError:
        return []
    _, _, rest = text.partition(":")
    return rest.split()


def _up_to_date(obj: str) -> bool:
    deps = _deps(obj[:-2] + ".d")
    if not deps or not os.path.exists(obj):
        return False
    t = os.path.getmtime(obj)
    return all(os.path.exists(d) and os.path.getmtime(d) <= t for d in deps)


def build(verbose: bool = False, jobs: int | None = None, incremental: bool = False) -> str:
    """Compile every unit (incremental: only those whose sources or included
    headers changed since their object was built) and link libgspn.so."""
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    srcs = sources()
    objs = [os.path.join(BUILD, os.path.basename(s)[:-4] + ".o") for s in srcs]
    cmds = [[cc, *FLAGS, "-MMD", "-MF", o[:-2] + ".d", "-c", s, "-o", o] for s, o in zip(srcs, objs)
            if not (incremental and _up_to_date(o))]
    if verbose:
        for c in cmds:
            print(" ".join(c), flush=True)
    if cmds:
        with ThreadPoolExecutor(max_workers=jobs or min(8, len(cmds))) as ex:
            list(ex.map(_run, cmds))
    tmp = LIB + ".tmp"
    link = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(link), flush=True)
    _run(link)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, incremental="--incremental" in sys.argv))
