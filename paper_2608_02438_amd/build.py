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


# Host AddressSanitizer: the host code only (argument validation, the
# handles, the launch sequences); device code is built as usual.
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
ASAN_LIB = os.path.join(ROOT, "_build", "libxpress_asan.so")


def asan_runtime() -> str:
    """Path of the host ASan runtime that a process loading ASAN_LIB must preload."""
    clang = os.path.join(os.path.dirname(os.path.dirname(HIPCC)), "lib", "llvm", "lib", "clang")
    for ver in sorted(os.listdir(clang), reverse=True):
        p = os.path.join(clang, ver, "lib", "linux", "libclang_rt.asan-x86_64.so")
        if os.path.exists(p):
            return p
    raise RuntimeError("host ASan runtime not found under " + clang)


def build(verbose: bool = False, asan: bool = False) -> str:
    """Compile every HIP source (one hipcc process per file, in parallel) and
    link them into libxpress.so (with asan: the host-ASan build ASAN_LIB);
    returns its path."""
    from concurrent.futures import ThreadPoolExecutor
    objdir = os.path.join(ROOT, "_build", "obj_asan" if asan else "obj")
    os.makedirs(objdir, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include")]
    compile_flags = [f for f in FLAGS if f != "-shared"] + (ASAN_FLAGS if asan else [])
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
    out = ASAN_LIB if asan else LIB
    tmp = out + ".tmp"
    rc, lines = _run([HIPCC, *FLAGS, *(ASAN_FLAGS if asan else []), *[j[1] for j in jobs],
                      "-o", tmp])
    if rc != 0:
        raise RuntimeError("link failed:\n" + "\n".join(lines))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, asan="--asan" in sys.argv))
