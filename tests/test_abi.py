"""The C ABI loads and exports every entry point include/ff8.h declares; host-side
argument validation returns the documented error codes before touching a GPU (CPU only)."""

import ctypes
import os
import re

import pytest

from paper_2511_02302_amd import ff8

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "ff8.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ff8_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ff8.library_path()):
        pytest.fail("libff8.so is not built (python -m paper_2511_02302_amd.build)")
    return ff8.load()


def test_every_declared_symbol_is_exported_and_bound(lib):
    names = _declared()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(ff8.EXPORTS) == names


def test_version_and_status_strings(lib):
    assert lib.ff8_version() >= 100
    assert lib.ff8_status_string(0) == b"ok"
    assert lib.ff8_status_string(2) == b"bad shape"


def test_rows_bound(lib):
    assert lib.ff8_rows_bound(1024, 2, 8) == 3072
    assert lib.ff8_rows_bound(16384, 8, 32) == 135168
    assert lib.ff8_rows_bound(8192, 8, 32) == 69632
    assert lib.ff8_rows_bound(10, 3, 2) == -1
    assert lib.ff8_permute_workspace_bytes(1024, 2, 8) == 4 * 8 * 4


def test_validation_errors_without_gpu(lib):
    vp = ctypes.c_void_p
    fake = vp(0x1000)
    assert lib.ff8_quant_rowwise(None, 4, 128, fake, fake, None) == 1
    assert lib.ff8_quant_rowwise(fake, 4, 100, fake, fake, None) == 2
    assert b"cols" in lib.ff8_last_error()
    assert lib.ff8_quant_block128(fake, 100, 128, fake, fake, None) == 2
    assert lib.ff8_scaling_aware_transpose(fake, fake, 130, 128, None, 0, fake, fake, None) == 2
    assert lib.ff8_grouped_gemm_fprop(fake, fake, fake, fake, fake, 0, 128, 128, 128, fake, None) == 3
    assert lib.ff8_grouped_gemm_wgrad(fake, fake, fake, fake, fake, 2, 128, 128, 128, fake, 2, None) == 3
    assert lib.ff8_grouped_gemm_dgrad(fake, fake, fake, fake, None, 2, 128, 128, 128, fake, None) == 1
    assert lib.ff8_grouped_gemm_fprop(fake, fake, fake, fake, fake, 1025, 128, 128, 128, fake, None) == 3
    assert b"1024" in lib.ff8_last_error()
    # permute: k > E, M_cap below the bound, workspace too small
    assert lib.ff8_permute_quant(fake, None, 16, 128, 3, 2, fake, 0, fake, fake, fake, 1024, fake, fake,
                                 fake, 1 << 20, None) == 3
    assert lib.ff8_permute_quant(fake, None, 16, 128, 2, 4, fake, 0, fake, fake, fake, 128, fake, fake,
                                 fake, 1 << 20, None) == 2
    assert lib.ff8_permute_quant(fake, None, 16, 128, 2, 4, fake, 0, fake, fake, fake, 640, fake, fake,
                                 fake, 0, None) == 3
    assert lib.ff8_unpermute(fake, fake, None, 4, 0, 128, 128, fake, None) == 3
    # an empty batch passes validation with NULL token-indexed arrays (no GPU here: the launch fails)
    assert lib.ff8_permute_quant(None, None, 0, 128, 2, 4, None, 0, None, fake, fake, 512, fake, fake,
                                 None, 0, None) != 1
    assert lib.ff8_swiglu_quant(fake, None, 0, 128, 100, fake, fake, None) == 2
    assert lib.ff8_baseline_copy(fake, fake, 17, None) == 2
