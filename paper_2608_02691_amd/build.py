"""Build libint2kv.so (HIP, gfx950) in-tree with hipcc.

Each ``csrc/*.hip`` file is compiled to an object under ``_build/`` in parallel, then linked
into ``paper_2608_02691_amd/libint2kv.so``. Always rebuilds (the build check compiles every
time it is called).

``build_host_asan()`` builds a second copy, ``_build/asan/libint2kv_asan.so``, whose host code
(argument validation, planning, workspace carving) is instrumented with AddressSanitizer; the
device code is the same as the release build's. It is loaded only by the CPU test that runs the
host-side checks under the sanitizer's runtime (preloaded with ``LD_PRELOAD``).
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libint2kv.so")
BUILD_DIR = os.path.join(ROOT, "_build")

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    "-I", os.path.join(ROOT, "include"),
]


def sources():
    return sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))


# host-only sanitizer flags: each -fsanitize= applies to the host pass alone
ASAN_HOST_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
ASAN_DIR = os.path.join(BUILD_DIR, "asan")
ASAN_LIB = os.path.join(ASAN_DIR, "libint2kv_asan.so")


def asan_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime (to preload), or '' if absent."""
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], stdout=subprocess.PIPE,
                       stderr=subprocess.DEVNULL)
    path = r.stdout.decode().strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        hits = sorted(glob.glob(os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(HIPCC))),
                                             "llvm", "lib", "clang", "*", "lib", "linux",
                                             "libclang_rt.asan-x86_64.so")))
        path = hits[-1] if hits else ""
    return path


def build_host_asan(verbose: bool = False) -> str:
    return build(verbose, extra_flags=ASAN_HOST_FLAGS, out=ASAN_LIB, obj_dir=ASAN_DIR,
                 link_flags=["-Xarch_host", "-fsanitize=address", "-shared-libasan"])


def build(verbose: bool = False, extra_flags=None, out: str = LIB, obj_dir: str = BUILD_DIR,
          link_flags=()) -> str:
    os.makedirs(obj_dir, exist_ok=True)
    flags = FLAGS + list(extra_flags or [])
    procs = []
    objs = []
    for src in sources():
        obj = os.path.join(obj_dir, os.path.basename(src) + ".o")
        objs.append(obj)
        cmd = [HIPCC, *flags, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    failed = []
    for src, p in procs:
        log, _ = p.communicate()
        text = log.decode(errors="replace")
        text = "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)
        if p.returncode != 0:
            failed.append((src, text))
        elif verbose and text.strip():
            print(text)
    if failed:
        msg = "\n".join(f"--- {s}\n{t}" for s, t in failed)
        raise RuntimeError(f"hipcc failed:\n{msg}")
    tmp = out + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *link_flags, "-o", tmp, *objs]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout.decode(errors="replace"))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
