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
    assert lib.ff8_permute_workspace_bytes(1024, 2, 8) == 4 * 8 * 4  # 256-token chunks x experts x int32


def _no_gpu():
    torch = pytest.importorskip("torch")
    return torch.cuda.device_count() == 0  # counts devices without initialising one


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
    # T * k and M_cap must stay below 2^31 (int32 row maps and row indices)
    big_T = 1 << 28
    m_cap = lib.ff8_rows_bound(big_T, 8, 8)
    assert lib.ff8_permute_quant(fake, None, big_T, 128, 8, 8, fake, 1, fake, fake, fake, m_cap, fake, fake,
                                 None, 0, None) == 2
    # the router gradient keeps a row of dY in registers: H above 8192 is rejected
    assert lib.ff8_permute_quant_dprobs(fake, fake, 16, 8320, 2, 4, fake, fake, fake, 4096, fake, fake, fake, fake,
                                        None) == 2
    # an empty batch passes validation with NULL token-indexed arrays (no GPU here: the launch fails;
    # with a GPU present the launch would read the fake pointers, so it is not made there)
    if _no_gpu():
        assert lib.ff8_permute_quant(None, None, 0, 128, 2, 4, None, 0, None, fake, fake, 512, fake, fake,
                                     None, 0, None) != 1
    # the no-allocation permute holds a 1 MiB routing workspace: ceil(T / 256) * E above 2^18 is
    # rejected on the host, before any device call
    t_big = 8192 * 256 + 1
    m_big = lib.ff8_rows_bound(t_big, 8, 32)
    assert lib.ff8_permute_quant_noalloc(fake, None, t_big, 128, 8, 32, fake, 0, fake, fake, fake, m_big, fake, fake,
                                         128, None) == 3
    assert b"1048576 bytes" in lib.ff8_last_error()
    assert lib.ff8_permute_quant_noalloc(fake, None, 16, 128, 2, 4, fake, 0, fake, fake, fake, 640, fake, fake,
                                         24, None) == 3  # align
    # the batched transpose: n in [1, 4], every array and entry present, every extent a multiple of 128
    arr = lambda *v: (ctypes.c_void_p * len(v))(*v)
    cols = lambda *c: (ctypes.c_int64 * len(c))(*c)
    f5 = [0x1000] * 5
    sat_b = lib.ff8_scaling_aware_transpose_batch
    assert sat_b(0, arr(0x1000), arr(0x1000), cols(128), 128, None, 0, arr(0x1000), arr(0x1000), None) == 3
    assert sat_b(5, arr(*f5), arr(*f5), cols(*[128] * 5), 128, None, 0, arr(*f5), arr(*f5), None) == 3
    assert sat_b(1, None, arr(0x1000), cols(128), 128, None, 0, arr(0x1000), arr(0x1000), None) == 1
    assert sat_b(2, arr(0x1000, None), arr(0x1000, 0x1000), cols(128, 128), 128, None, 0, arr(0x1000, 0x1000),
                 arr(0x1000, 0x1000), None) == 1
    assert b"tensor 1" in lib.ff8_last_error()
    assert sat_b(2, arr(0x1000, 0x1000), arr(0x1000, 0x1000), cols(128, 200), 128, None, 0, arr(0x1000, 0x1000),
                 arr(0x1000, 0x1000), None) == 2
    assert lib.ff8_scaling_aware_transpose_batch_e8m0(1, arr(0x1000), arr(0x1000), cols(128), 100, None, 0,
                                                      arr(0x1000), arr(0x1000), None) == 2
    assert sat_b(1, arr(0x1000), arr(0x1000), cols(128), 128, fake, 0, arr(0x1000), arr(0x1000), None) == 3
    assert lib.ff8_swiglu_quant(fake, None, 0, 128, 100, fake, fake, None) == 2
    assert lib.ff8_baseline_copy(fake, fake, 17, None) == 2
    # operands of 4 GiB and more: the kernels address each operand with 32-bit byte offsets
    assert lib.ff8_grouped_gemm_fprop(fake, fake, fake, fake, fake, 1, 1 << 22, 128, 1024, fake, None) == 2
    assert b"4 GiB" in lib.ff8_last_error()
    assert lib.ff8_grouped_gemm_fprop(fake, fake, fake, fake, fake, 1, (1 << 22) - 128, 128, 1024, fake, None) != 2
    assert lib.ff8_grouped_gemm_dgrad(fake, fake, fake, fake, fake, 8, 128, 1 << 14, 1 << 15, fake, None) == 2
    assert lib.ff8_grouped_gemm_wgrad(fake, fake, fake, fake, fake, 2, 1 << 25, 128, 128, fake, 0, None) == 2


def test_binding_checks_every_shape():
    """The C ABI receives plain pointers and cannot see an undersized buffer, so the binding
    compares every tensor's shape with the extents it passes and raises before any call."""
    torch = pytest.importorskip("torch")
    u8, f32, bf16, i32 = torch.uint8, torch.float32, torch.bfloat16, torch.int32
    e = lambda *shape, dtype=u8: torch.empty(shape, dtype=dtype)
    M, K, N, E = 512, 256, 384, 4
    bad_calls = [
        lambda: ff8.ff8_quant_rowwise(e(M, K, dtype=bf16), e(M, K), e(M, 1, dtype=f32)),
        lambda: ff8.ff8_quant_block128(e(N, K, dtype=bf16), e(N, K), e(2, 2, dtype=f32)),
        lambda: ff8.ff8_scaling_aware_transpose(e(M, K), e(M, 2, dtype=f32), e(M // 128 - 1, K, 128), e(4, K, dtype=f32)),
        lambda: ff8.ff8_scaling_aware_transpose(e(M, K), e(M, 2, dtype=f32), e(K, M), e(4, K, dtype=f32)),  # not K-blocked
        lambda: ff8.ff8_scaling_aware_transpose_batch([e(M, K), e(M, N)], [e(M, 2, dtype=f32), e(M, 3, dtype=f32)],
                                                      [e(M // 128, K, 128), e(M // 128, N, 128)],
                                                      [e(M // 128, K, dtype=f32), e(M // 128, K, dtype=f32)]),
        lambda: ff8.ff8_scaling_aware_transpose_batch([e(M, K), e(M - 128, N)], [e(M, 2, dtype=f32), e(M, 3, dtype=f32)],
                                                      [e(M // 128, K, 128), e(M // 128, N, 128)],
                                                      [e(M // 128, K, dtype=f32), e(M // 128, N, dtype=f32)]),
        lambda: ff8.ff8_grouped_gemm_fprop(e(M, K), e(M, 2, dtype=f32), e(E, N, K), e(E, 3, 2, dtype=f32),
                                           e(E + 1, dtype=i32), e(M - 128, N, dtype=bf16)),
        lambda: ff8.ff8_grouped_gemm_dgrad(e(M, N), e(M, 3, dtype=f32), e(E, N, K), e(E, 3, 2, dtype=f32),
                                           e(E, dtype=i32), e(M, K, dtype=bf16)),
        lambda: ff8.ff8_grouped_gemm_wgrad(e(M // 128, N, 128), e(M // 128, N, dtype=f32), e(M // 128, K, 128),
                                           e(M // 128, K, dtype=f32), e(E + 1, dtype=i32), e(E, K, N, dtype=f32)),
        lambda: ff8.ff8_grouped_gemm_wgrad(e(M // 128, N, 128), e(M // 128, N, dtype=f32), e(M // 128 - 1, K, 128),
                                           e(M // 128, K, dtype=f32), e(E + 1, dtype=i32), e(E, N, K, dtype=f32)),
        lambda: ff8.ff8_swiglu_quant(e(M, 2 * K, dtype=bf16), e(M, K), e(M, 1, dtype=f32)),
        lambda: ff8.ff8_swiglu_bwd_quant(e(M, 2 * K, dtype=bf16), e(M, K, dtype=bf16), e(M, K), e(M, 4, dtype=f32)),
        lambda: ff8.ff8_unpermute(e(M, K, dtype=bf16), e(128, 2, dtype=i32), e(128, 1, dtype=f32),
                                  e(128, K, dtype=bf16)),
        lambda: ff8.ff8_permute_quant(e(128, K, dtype=bf16), None, 2, E, e(128, 2, dtype=i32), False,
                                      e(128, 2, dtype=i32), e(E + 1, dtype=i32), e(M - 1, dtype=i32), e(M, K),
                                      e(M, 2, dtype=f32)),
    ]
    for i, call in enumerate(bad_calls):
        with pytest.raises(ValueError, match="must (have shape|hold)"):
            call()
    # consistent shapes get past the shape checks (and stop at the device check here)
    with pytest.raises(ValueError, match="device tensor"):
        ff8.ff8_grouped_gemm_wgrad(e(M // 128, N, 128), e(M // 128, N, dtype=f32), e(M // 128, K, 128),
                                   e(M // 128, K, dtype=f32), e(E + 1, dtype=i32), e(E, N, K, dtype=f32))


def test_header_compiles_as_c_and_links(tmp_path):
    """include/ff8.h is plain C: a C99 program includes it, links libff8.so and calls the
    host-only entry points (no GPU needed for these)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "abi.c"
    src.write_text(r"""
#include <stdio.h>
#include <string.h>
#include "ff8.h"
int main(void) {
  if (ff8_version() <= 0) return 1;
  if (ff8_rows_bound(1024, 2, 8) != ff8_rows_bound_aligned(1024, 2, 8, 128)) return 2;
  if (ff8_rows_bound_aligned(1024, 2, 8, 48) != -1) return 3;
  int rc = ff8_quant_rowwise(NULL, 4, 128, (ff8_e4m3*)16, (float*)16, NULL);
  if (rc != FF8_ERR_NULL || strlen(ff8_last_error()) == 0) return 4;
  printf("%s\n", ff8_status_string(rc));
  return 0;
}
""")
    exe = tmp_path / "abi"
    lib_dir = os.path.dirname(ff8.library_path())
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                        "-L", lib_dir, "-lff8", "-Wl,-rpath," + lib_dir], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip() == "null pointer", (r.returncode, r.stdout, r.stderr)
