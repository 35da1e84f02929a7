"""Sanitizer builds of the library's host code and of the CPU oracle, for
tests that run on the CPU only.

    python -m paper_2509_24626_amd.build_sanitized asan   # AddressSanitizer + UndefinedBehaviorSanitizer
    python -m paper_2509_24626_amd.build_sanitized tsan   # ThreadSanitizer

Every translation unit is compiled as in build.py; the sanitizer flags
apply to the host side only (each -fsanitize= follows -Xarch_host), so the
gfx950 kernels are built as usual and no GPU code is instrumented.  The
library goes to _lib/libsparseserve_<kind>.so and, for asan, the oracle
(built with the same clang, so both use one sanitizer runtime) to
oracle/liboracle_asan.so.  A process loads them through the environment
(SS_LIBRARY, ORACLE_LIBRARY) with the clang runtime preloaded; env() gives
that environment.
"""
import glob
import os
import subprocess
import sys

from . import build as B

LLVM = "/opt/rocm/llvm"
CLANG = os.path.join(LLVM, "bin", "clang")

FLAGS = {
    "asan": ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined"],
    "tsan": ["-fsanitize=thread"],
}
RUNTIME = {"asan": "libclang_rt.asan-x86_64.so", "tsan": "libclang_rt.tsan-x86_64.so"}


def runtime(kind):
    hits = sorted(glob.glob(os.path.join(LLVM, "lib", "clang", "*", "lib", "linux", RUNTIME[kind])))
    if not hits:
        raise FileNotFoundError(f"no {RUNTIME[kind]} under {LLVM}")
    return hits[-1]


def lib_path(kind):
    return os.path.join(B.LIBDIR, f"libsparseserve_{kind}.so")


def oracle_path(kind):
    return os.path.join(B.ROOT, "oracle", f"liboracle_{kind}.so")


def build(kind):
    host = []
    for f in FLAGS[kind] + ["-fno-omit-frame-pointer", "-g"]:
        host += ["-Xarch_host", f]
    objdir = os.path.join(B.ROOT, "_build", f"sparseserve_{kind}")
    os.makedirs(objdir, exist_ok=True)
    os.makedirs(B.LIBDIR, exist_ok=True)
    procs, objs = [], []
    for src in B.SOURCES:
        obj = os.path.join(objdir, src + ".o")
        objs.append(obj)
        cmd = [B.HIPCC, "-x", "hip", *B.COMMON, *host, "-c", os.path.join(B.CSRC, src), "-o", obj]
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        if p.returncode:
            print("\n".join(ln for ln in out.splitlines() if "packed-fp32-ops" not in ln), file=sys.stderr)
            failed.append(src)
    if failed:
        raise RuntimeError(f"hipcc failed for {failed}")
    out = lib_path(kind)
    link_san = ["-Xarch_host", FLAGS[kind][0], "-shared-libsan"]
    subprocess.run([B.HIPCC, "-shared", f"--offload-arch={B.ARCH}", "-fPIC", *objs, *link_san, "-o", out + ".tmp",
                    "-lpthread"], check=True)
    os.replace(out + ".tmp", out)
    outs = [out]
    if kind == "asan":
        o = oracle_path(kind)
        subprocess.run([CLANG, "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
                        *FLAGS[kind], "-fno-omit-frame-pointer", "-shared-libsan",
                        os.path.join(B.ROOT, "oracle", "oracle.c"), "-o", o + ".tmp", "-lm"], check=True)
        os.replace(o + ".tmp", o)
        outs.append(o)
    return outs


def env(kind, base=None):
    """Environment for a child process that runs on the sanitized builds."""
    e = dict(os.environ if base is None else base)
    e["LD_PRELOAD"] = runtime(kind)
    e["SS_LIBRARY"] = lib_path(kind)
    if kind == "asan":
        e["ORACLE_LIBRARY"] = oracle_path(kind)
        # Python and torch are not instrumented: their leaks and allocator
        # pairings are not this library's; every error stops the process
        e["ASAN_OPTIONS"] = "detect_leaks=0:alloc_dealloc_mismatch=0:halt_on_error=1:abort_on_error=0:exitcode=86"
        e["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1:exitcode=87"
    else:
        e["TSAN_OPTIONS"] = "halt_on_error=1:exitcode=88:report_signal_unsafe=0"
    return e


if __name__ == "__main__":
    for k in sys.argv[1:] or ["asan", "tsan"]:
        print("\n".join(build(k)))
