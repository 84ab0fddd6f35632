"""Build the HIP library libxpress.so in-tree for gfx950.

    python -m paper_2608_02438_amd.build      (or call build())

Every .hip file under csrc/ is compiled by hipcc into one shared library next
to this file.  The library exports the C ABI declared in include/xpress.h.
"""
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libxpress.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # packed fp32 VALU forms stay off on this target
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result", "-Wno-unused-variable",
]


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = (r.stdout + r.stderr).strip()
    return r.returncode, [l for l in out.splitlines() if "packed-fp32-ops" not in l]


def build(verbose: bool = False) -> str:
    """Compile every HIP source (one hipcc process per file, in parallel) and
    link them into libxpress.so; returns its path."""
    from concurrent.futures import ThreadPoolExecutor
    objdir = os.path.join(ROOT, "_build", "obj")
    os.makedirs(objdir, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include")]
    compile_flags = [f for f in FLAGS if f != "-shared"]
    jobs = []
    for src in sources():
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        jobs.append((src, obj, [HIPCC, *compile_flags, *inc, "-c", src, "-o", obj]))
    if verbose:
        for _, _, cmd in jobs:
            print(" ".join(cmd), flush=True)
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        results = list(ex.map(lambda j: _run(j[2]), jobs))
    errs = [(j[0], lines) for j, (rc, lines) in zip(jobs, results) if rc != 0]
    if errs:
        raise RuntimeError("hipcc failed:\n" + "\n".join(
            f"{src}:\n" + "\n".join(lines) for src, lines in errs))
    if verbose:
        for (src, _, _), (_, lines) in zip(jobs, results):
            if lines:
                print("\n".join(lines))
    tmp = LIB + ".tmp"
    rc, lines = _run([HIPCC, *FLAGS, *[j[1] for j in jobs], "-o", tmp])
    if rc != 0:
        raise RuntimeError("link failed:\n" + "\n".join(lines))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
