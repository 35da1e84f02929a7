"""Builds tests/c_gpu_step.c (a decode step through the C ABI alone, checked
against the oracle) with the host C compiler against the in-tree library,
the oracle's library and the HIP runtime.  Used by the tests only."""
import os
import shutil
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(out_path):
    """Compiles and links the program; returns its path, or None without gcc."""
    cc = shutil.which("gcc")
    if cc is None:
        return None
    import oracle
    from paper_2509_24626_amd import binding as ss
    oracle.lib()  # builds liboracle.so if it is missing or stale
    libdir = os.path.dirname(os.path.abspath(ss.LIB_PATH))
    oradir = os.path.join(ROOT, "oracle")
    rocm_lib = os.path.join(ROCM, "lib")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-isystem", os.path.join(ROCM, "include"),
                    os.path.join(ROOT, "tests", "c_gpu_step.c"), "-o", out_path,
                    "-L", libdir, "-lsparseserve", "-L", oradir, "-loracle", "-L", rocm_lib, "-lamdhip64", "-lm",
                    "-Wl,-rpath," + ":".join([libdir, oradir, rocm_lib])], check=True)
    return out_path
