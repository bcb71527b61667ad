"""Build libgdninv.so (gfx950) in-tree.

    python paper_2606_06034_amd/csrc/build.py [--jobs N] [--verbose]

Compiles every csrc/*.hip and csrc/*.cpp with hipcc for gfx950 only and links
them into paper_2606_06034_amd/libgdninv.so.  Objects go to _build/ at the
repository root.  Always rebuilds objects whose source or headers changed.
"""

from __future__ import annotations

import argparse
import concurrent.futures as cf
import glob
import hashlib
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libgdninv.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
CFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-I", INCLUDE, "-I", HERE,
    # packed fp32 VALU ops are kept out of every code object
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results in architectural VGPRs (no accumulator-register copies)
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-Wno-unused-command-line-argument",
]


def _sources():
    return sorted(glob.glob(os.path.join(HERE, "*.hip")) + glob.glob(os.path.join(HERE, "*.cpp")))


def _includes(path: str, seen=None):
    """path plus every local header it includes, recursively."""
    seen = set() if seen is None else seen
    if path in seen:
        return seen
    seen.add(path)
    with open(path) as f:
        for line in f:
            line = line.strip()
            if line.startswith("#include \""):
                name = line.split('"')[1]
                for d in (os.path.dirname(path), HERE, INCLUDE):
                    cand = os.path.join(d, name)
                    if os.path.exists(cand):
                        _includes(cand, seen)
                        break
    return seen


def _digest(src: str) -> str:
    """Hash of a source, the local headers it includes and the compile flags,
    independent of where the repository is checked out."""
    root = os.path.dirname(os.path.dirname(HERE))
    h = hashlib.sha256()
    for p in sorted(_includes(src), key=lambda q: os.path.relpath(q, root)):
        h.update(os.path.relpath(p, root).encode())
        with open(p, "rb") as f:
            h.update(f.read())
    h.update(" ".join(CFLAGS).replace(root, "<repo>").encode())
    return h.hexdigest()[:16]


def _compile(src: str, verbose: bool, extra, force: bool = False) -> str:
    base = os.path.splitext(os.path.basename(src))[0]
    obj = os.path.join(BUILD, f"{base}.{_digest(src)}.o")
    if os.path.exists(obj) and not extra and not force:
        return obj
    lang = ["-x", "hip"]
    cmd = [HIPCC] + CFLAGS + list(extra) + lang + ["-c", src, "-o", obj + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{out}")
    if out.strip() and verbose:
        print(out)
    os.replace(obj + ".tmp", obj)
    return obj


def build(jobs: int = 8, verbose: bool = False, extra=(), force: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = _sources()
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, extra, force), srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=min(8, os.cpu_count() or 1))
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("--force", action="store_true", help="recompile every source")
    ap.add_argument("--resource-usage", action="store_true",
                    help="print per-kernel register / LDS / spill usage")
    a = ap.parse_args(argv)
    extra = ["-Rpass-analysis=kernel-resource-usage"] if a.resource_usage else []
    print(build(a.jobs, a.verbose or a.resource_usage, extra, a.force))


if __name__ == "__main__":
    sys.exit(main())
