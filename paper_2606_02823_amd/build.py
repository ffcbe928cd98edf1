"""Build libqift.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2606_02823_amd.build          # or __graft_entry__.build()
    python -m paper_2606_02823_amd.build --stamps # the diagnostic libqift_stamps.so

Each .hip source under csrc/ is compiled to an object in _build/ (in
parallel), then linked into paper_2606_02823_amd/libqift.so.  The diagnostic
build recompiles the decode-chain sources with -DQIFT_CHAIN_STAMPS (wall-clock
phase stamps, read by chain_stamps.py) and links them with the other objects
into libqift_stamps.so; the product library is not touched.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libqift.so")
LIB_STAMPS = os.path.join(PKG, "libqift_stamps.so")
ARCH = os.environ.get("QIFT_OFFLOAD_ARCH", "gfx950")

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17", "-Wall", "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(os.path.dirname(PKG), "include"),
]


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str, outdir: str = BUILD, extra=()) -> str:
    obj = os.path.join(outdir, os.path.basename(src) + ".o")
    cmd = [hipcc(), *FLAGS, *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def _link(objs, lib: str) -> None:
    tmp = lib + ".tmp"
    # --no-undefined: a kernel whose host stub was not emitted fails here, not when the library loads
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,--no-undefined", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, lib)


def _sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = _sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    _link(objs, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def build_stamps(verbose: bool = True, reuse: bool = False) -> str:
    """libqift_stamps.so: the decode-chain sources with phase stamps, the rest as built for libqift.so
    (with reuse, the objects build() has just made)."""
    out = os.path.join(BUILD, "stamps")
    os.makedirs(out, exist_ok=True)
    srcs = _sources()
    stamped = [s for s in srcs if os.path.basename(s).startswith("qift_chain_")]
    plain = [s for s in srcs if s not in stamped]
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        if reuse:
            objs = [os.path.join(BUILD, os.path.basename(s) + ".o") for s in plain]
        else:
            objs = list(ex.map(_compile, plain))
        objs += list(ex.map(lambda s: _compile(s, out, ("-DQIFT_CHAIN_STAMPS",)), stamped))
    _link(objs, LIB_STAMPS)
    if verbose:
        print(f"built {LIB_STAMPS}")
    return LIB_STAMPS


if __name__ == "__main__":
    if "--stamps" in sys.argv[1:]:
        build_stamps()
    else:
        build()
