"""A decode step driven from plain C through the library's C ABI, without
Python or torch in the process: metadata, scoring and top-k, the host
slot-table resolve, the gather from mapped DRAM and sparse attention over
three steps, each stage checked against the oracle inside the program
(tests/c_gpu_step.c)."""
import subprocess

import pytest

import c_step_build

pytestmark = pytest.mark.gpu


def test_decode_step_from_c(tmp_path):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    exe = c_step_build.build(str(tmp_path / "c_gpu_step"))
    if exe is None:
        pytest.skip("no C compiler")
    print("[gpu] running tests/c_gpu_step.c", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c gpu step ok" in r.stdout
    assert r.stdout.count("attention max abs error") == 3
