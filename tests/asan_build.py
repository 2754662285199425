"""AddressSanitizer build of the library's host code, for the CPU tests of the
C ABI's error paths (test infrastructure; never loaded by a GPU run)."""

import concurrent.futures
import glob
import os

from paper_2506_20194_amd import build as B


def asan_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime (for LD_PRELOAD
    into an uninstrumented Python)."""
    for pat in ("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so",
                "/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"):
        hits = sorted(glob.glob(pat))
        if hits:
            return hits[-1]
    raise FileNotFoundError("no libclang_rt.asan-x86_64.so under /opt/rocm")


def build_asan(out_dir: str) -> str:
    """libduo with AddressSanitizer on its host code (argument validation,
    workspace carving, dispatch); device code is built as usual."""
    os.makedirs(out_dir, exist_ok=True)
    host_asan = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
    objs = [os.path.join(out_dir, os.path.splitext(s)[0] + ".o") for s in B.SOURCES]
    jobs = [[B.HIPCC, *B.FLAGS, *host_asan, "-c", os.path.join(B.CSRC, s), "-o", o] for s, o in zip(B.SOURCES, objs)]
    workers = min(len(jobs), max(1, min(16, os.cpu_count() or 1)))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        list(ex.map(B._run, jobs))
    out = os.path.join(out_dir, "libduo_asan.so")
    B._run([B.HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *objs, "-o", out,
            "-Xarch_host", "-fsanitize=address", "-shared-libsan"])
    return out
