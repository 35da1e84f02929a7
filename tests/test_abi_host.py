"""The C ABI on the CPU: the library loads, exports every function that
include/*.h declares, and rejects bad arguments before touching a GPU."""
import glob
import os
import re

import numpy as np
import pytest

from paper_2509_24626_amd import binding as ss

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"typedef[^;]*;", "", text)  # function-pointer types are not functions
        for m in re.finditer(r"\b(ss_\w+)\s*\(", text):
            names.add(m.group(1))
    return sorted(names)


def test_library_builds_and_loads():
    assert os.path.exists(ss.LIB_PATH)
    header = open(os.path.join(ROOT, "include", "sparseserve.h")).read()
    assert ss.ss_abi_version() == int(re.search(r"#define SS_ABI_VERSION (\d+)", header).group(1)) == 5


def test_every_declared_symbol_is_exported():
    L = ss.lib()
    names = declared_functions()
    assert len(names) >= 15, names
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing
    # and the binding covers exactly the declared set
    assert sorted(ss.exported_names()) == names


def test_status_strings():
    for code in range(6):
        assert ss.ss_status_string(code)
    assert ss.ss_status_string(99) == "unknown status"


def expect(status, fn, *args):
    with pytest.raises(ss.SparseServeError) as e:
        fn(*args)
    assert e.value.status == status, str(e.value)
    assert ss.ss_last_error()


FAKE = 0x1000  # never dereferenced: validation fails first


def test_unsupported_shapes_rejected():
    expect(ss.SS_ERR_UNSUPPORTED, ss.ss_build_metadata, FAKE, FAKE, FAKE, 1, 1, 4, 16, 64, FAKE, 0)
    expect(ss.SS_ERR_UNSUPPORTED, ss.ss_build_metadata, FAKE, FAKE, FAKE, 1, 1, 4, 12, 128, FAKE, 0)
    expect(ss.SS_ERR_UNSUPPORTED, ss.ss_score_blocks, FAKE, FAKE, FAKE, 1, 34, 2, 4, 128, FAKE, 0)  # G = 17
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_score_blocks, FAKE, FAKE, FAKE, 1, 9, 2, 4, 128, FAKE, 0)  # Hq % Hkv
    expect(ss.SS_ERR_UNSUPPORTED, ss.ss_select_topk, FAKE, FAKE, 1, 1, 70000, 4, FAKE, 0)
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_select_topk, FAKE, FAKE, 1, 1, 16, 0, FAKE, 0)  # k = 0
    expect(ss.SS_ERR_UNSUPPORTED, ss.ss_gather_blocks, FAKE, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 1000, 0)
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_gather_blocks, FAKE + 4, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 8192, 0)
    expect(ss.SS_ERR_UNSUPPORTED, ss.ss_sparse_attention, FAKE, FAKE, FAKE, FAKE, None, 8, 1, 8, 2, 64, 16, 4, 0.1, FAKE,
           0, 0, 0)
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_sparse_attention, FAKE, FAKE, FAKE, FAKE, None, 8, 1, 8, 2, 128, 16, 4,
           float("nan"), FAKE, 0, 0, 0)


def test_null_pointers_rejected():
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_build_metadata, None, FAKE, FAKE, 1, 1, 4, 16, 128, FAKE, 0)
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_score_topk, FAKE, FAKE, FAKE, 1, 8, 2, 4, 128, 2, FAKE, None, 0)
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_gather_blocks, None, 3, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 8192, 0)
    # a layer of the multi-layer step with no device buffers
    L = ss.ss_layer_buffers(B=2, Hq=8, Hkv=2, d=128, blk=16, nblk_max=16, k=4, parts=1)
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_decode_step_dev, [L], [FAKE], 0, [FAKE], [FAKE], 0)
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_decode_step, [L], 0, [FAKE], [FAKE], 0)


def test_empty_work_is_a_no_op():
    # zero sequences / zero misses enqueue nothing and succeed without a GPU
    ss.ss_build_metadata(None, None, None, 0, 2, 16, 16, 128, None, 0)
    ss.ss_score_blocks(None, None, None, 0, 8, 2, 16, 128, None, 0)
    ss.ss_select_topk(None, None, 0, 2, 16, 4, None, 0)
    ss.ss_gather_blocks(None, 0, None, None, None, None, None, None, 1, 1, 8192, 0)
    ss.ss_sparse_attention(None, None, None, None, None, 8, 0, 8, 2, 128, 16, 4, 0.1, None, None, 0, 0)
    ss.ss_decode_step_dev([], [], 0, [], [], 0)
    assert len(ss.ss_decode_step([], 0, [], [], 0)) == 0
    ss.ss_decode_step_dev([ss.ss_layer_buffers(B=0, Hq=8, Hkv=2, d=128, k=4)], [FAKE], 0, [FAKE], [FAKE], 0)


def test_score_topk_workspace_sizes():
    assert ss.ss_score_topk_workspace(64, 32, 8, 8192, 128, 128) == 64 * 8 * 8192 * 4
    assert ss.ss_score_topk_workspace(0, 32, 8, 8192, 128, 128) == 0
    assert ss.ss_score_topk_workspace(2, 30, 8, 100, 128, 8) == 0  # Hq not a multiple of Hkv
    assert ss.ss_score_topk_workspace(2, 32, 8, 100, 64, 8) == 0   # d other than 128


def test_attention_workspace_sizes():
    # split plan: several splits for few units, none for a single small unit
    assert ss.ss_sparse_attention_workspace(2, 8, 2, 128, 16, 16) == 0
    w = ss.ss_sparse_attention_workspace(32, 32, 8, 128, 16, 128)
    assert w > 0 and w % (4 * 130) == 0
    assert ss.ss_sparse_attention_workspace(1, 8, 2, 64, 16, 16) == 0  # unsupported -> 0
    expect(ss.SS_ERR_OOM, ss.ss_sparse_attention, FAKE, FAKE, FAKE, FAKE, FAKE, 2048, 32, 32, 8, 128, 16, 128, 0.1, FAKE,
           FAKE, w - 1, 0)


def test_host_alloc_rejects_bad_flags():
    expect(ss.SS_ERR_INVALID_ARG, ss.ss_host_alloc_mapped, 4096, 7)
    assert ss.ss_host_alloc_mapped(0) == (0, 0)


def test_header_and_host_calls_from_plain_c(tmp_path):
    """tests/c_abi_check.c, built as strict C99 against the in-tree library,
    calls the host-only entry points; the header also parses as C++."""
    import shutil
    import subprocess
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("no C compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    inc = os.path.join(root, "include")
    libdir = os.path.dirname(ss.LIB_PATH)
    exe = str(tmp_path / "c_abi_check")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", inc,
                    os.path.join(root, "tests", "c_abi_check.c"), "-o", exe, "-L", libdir, "-lsparseserve",
                    "-Wl,-rpath," + libdir], check=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout
    assert "c abi ok" in out
    cxx = shutil.which("g++")
    if cxx:
        src = tmp_path / "h.cpp"
        src.write_text('#include "sparseserve.h"\nint main() { return ss_abi_version() == SS_ABI_VERSION ? 0 : 1; }\n')
        subprocess.run([cxx, "-std=c++11", "-Wall", "-Werror", "-fsyntax-only", "-I", inc, str(src)], check=True)


def test_c_decode_step_program_builds(tmp_path):
    """tests/c_gpu_step.c, a whole decode step through the C ABI alone (run
    on the GPU by tests/test_gpu_c_abi.py), compiles as strict C99."""
    import c_step_build
    if c_step_build.build(str(tmp_path / "c_gpu_step")) is None:
        pytest.skip("no C compiler")
