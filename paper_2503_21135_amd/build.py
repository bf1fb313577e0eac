"""Build the gfx950 kernel library libmoe_quant.so in-tree with hipcc."""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libmoe_quant.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math",
    # packed fp32 instructions are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
]


# compiled once per group size (64, 128), in parallel
SPLIT_BY_GROUP = ("ffn_stream.hip", "ffn_tile.hip")


def sources() -> list:
    """HIP kernel sources plus the host-only C++ of the library."""
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")) +
                  glob.glob(os.path.join(HERE, "csrc", "*.cpp")))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed: %s" % " ".join(cmd))


def build(verbose: bool = False) -> str:
    """Compile every HIP source into paper_2503_21135_amd/libmoe_quant.so:
    one object per source, compiled in parallel, then one link."""
    from concurrent.futures import ThreadPoolExecutor
    obj_dir = os.path.join(ROOT, "_build", "obj%d" % os.getpid())
    os.makedirs(obj_dir, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]
    units = []   # (source, extra flags): the kernel files once per group size
    for src in sources():
        name = os.path.basename(src)
        if name in SPLIT_BY_GROUP:
            units += [(src, ["-DMOE_FFN_NM=%d" % nm]) for nm in (2, 4)]
        else:
            units.append((src, []))
    objs = [os.path.join(obj_dir, "%d_%s.o" % (i, os.path.basename(u[0]))) for i, u in enumerate(units)]
    jobs = max(1, min(len(units), int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))
    with ThreadPoolExecutor(jobs) as ex:
        list(ex.map(lambda uo: _run([HIPCC] + FLAGS + uo[0][1] + ["-c"] + inc + [uo[0][0], "-o", uo[1]],
                                    verbose), zip(units, objs)))
    tmp = LIB + ".tmp%d" % os.getpid()
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + ["-o", tmp], verbose)
    os.replace(tmp, LIB)
    for o in objs:
        os.remove(o)
    os.rmdir(obj_dir)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
