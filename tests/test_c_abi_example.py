"""The library used from plain C (tests/c_abi_example.c): the header compiles
as C11, the program links against the built library and the HIP runtime, and
on a GPU every element of C = A.B for a tridiagonal A with small-integer B
is bitwise the closed-form result at widths 1, 3, 8, 32, 64 and 100."""
import os
import subprocess

import pytest

import __graft_entry__ as entry


def _has_gpu():
    try:
        import torch

        return torch.cuda.is_available()
    except Exception:  # pragma: no cover
        return False


@pytest.mark.skipif(_has_gpu(), reason="a GPU is visible (the gpu test runs the example)")
def test_c_example_compiles_and_runs_host_only(tmp_path):
    exe = entry.build_c_example(str(tmp_path / "c_abi_example"))
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2, r.stdout + r.stderr  # no GPU: host-only plan, sd_spmm refused
    assert "analyse: m=4099 nnz=12295 row_max=3" in r.stdout
    assert "SD_ERR_NO_DEVICE" in r.stdout


@pytest.mark.gpu
@pytest.mark.skipif(not _has_gpu(), reason="needs a GPU")
def test_c_example_on_gpu():
    exe = entry.C_EXAMPLE
    assert os.path.exists(exe), "tests/c_abi_example is built by __graft_entry__.build()"
    print("case c_abi_example", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("ok")
    assert r.stdout.count("mismatches=0") == 6
