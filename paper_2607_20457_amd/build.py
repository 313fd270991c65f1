"""Build the gfx950 shared library ``libpulsar.so`` from ``csrc/*.hip``.

Run ``python -m paper_2607_20457_amd.build`` (or ``__graft_entry__.build()``).
Each source is compiled to an object in parallel, then the objects are linked;
the library is written next to this file so that it travels with the tree.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libpulsar.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed: {' '.join(cmd[-3:])}")
    if verbose and res.stderr:
        sys.stderr.write(res.stderr)


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile every HIP source into ``libpulsar.so``; returns its path."""
    tmpdir = tempfile.mkdtemp(prefix="pulsar_build_")
    try:
        srcs = sources()
        objs = [os.path.join(tmpdir, os.path.basename(s) + ".o") for s in srcs]
        workers = max(1, min(len(srcs), os.cpu_count() or 1, 8))
        with cf.ThreadPoolExecutor(workers) as ex:
            futs = [ex.submit(_run, [HIPCC, *FLAGS, *extra_flags, "-c", "-o", o, s], verbose)
                    for s, o in zip(srcs, objs)]
            for f in futs:
                f.result()
        tmp = LIB + ".tmp"
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
        os.replace(tmp, LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv,
          extra_flags=["-Rpass-analysis=kernel-resource-usage"] if "--usage" in sys.argv else [])
