"""Build libbo.so (HIP, gfx950) in-tree with hipcc.

Usage: python -m paper_2602_10729_amd.build [--jobs N] [--verbose]

Every source under csrc/ is compiled to an object in _build/, then linked
into paper_2602_10729_amd/libbo.so. Device code is built for gfx950 only,
with packed-FP32 instruction selection switched off.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libbo.so")

ARCH = "gfx950"
COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Wall", "-Wno-unused-result",
    "-I", os.path.join(ROOT, "include"),
]
DEVICE_ONLY = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found")
    return p


def sources():
    """Every source, the widest posterior instantiations first: they take
    longest to compile, so starting them first shortens a parallel build."""
    out = []
    for f in sorted(os.listdir(CSRC)):
        if f.endswith(".hip") or f.endswith(".cpp"):
            out.append(os.path.join(CSRC, f))

    def cost(path):
        m = re.match(r"posterior_dx(\d)", os.path.basename(path))
        return -int(m.group(1)) if m else 0
    return sorted(out, key=cost)


def _compile(src: str, verbose: bool, extra=(), bdir=BUILD) -> str:
    obj = os.path.join(bdir, os.path.basename(src) + ".o")
    cmd = [hipcc()] + COMMON + list(extra)
    if src.endswith(".hip"):
        cmd += DEVICE_ONLY + ["-x", "hip"]
    cmd += ["-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n{r.stdout}\n{r.stderr}")
    # the host pass does not know the packed-fp32 feature; drop that warning
    noise = [ln for ln in r.stderr.splitlines()
             if ln.strip() and "packed-fp32-ops" not in ln and "not a recognized feature" not in ln]
    if noise and verbose:
        print("\n".join(noise), file=sys.stderr)
    return obj


def build(jobs: int = 8, verbose: bool = False, extra_flags=(), out: str = LIB,
          build_dir: str = BUILD) -> str:
    """Compile every source and link ``out``. ``extra_flags`` (e.g. -D tuning
    macros) are added to every compile line."""
    os.makedirs(build_dir, exist_ok=True)
    srcs = sources()
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, extra_flags, build_dir), srcs))
    tmp = out + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=min(8, os.cpu_count() or 1))
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("-D", dest="defines", action="append", default=[],
                    help="extra preprocessor definition, e.g. -D BO_POST_WAVES=4")
    ap.add_argument("--out", default=LIB)
    ap.add_argument("--build-dir", default=BUILD)
    a = ap.parse_args(argv)
    print(build(a.jobs, a.verbose, ["-D" + d for d in a.defines], a.out, a.build_dir))


if __name__ == "__main__":
    main()
