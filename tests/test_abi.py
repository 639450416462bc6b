"""The C-ABI library builds, loads and exports every entry point include/als.h declares
(CPU only: no compute calls)."""
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "als.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(als_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    fns = declared_functions()
    for must in ("als_init", "als_half_sweep", "als_rmse", "als_workspace_bytes", "als_status",
                 "als_plan", "als_destroy", "als_strerror", "als_last_hip_error"):
        assert must in fns


def test_library_exports_every_declared_symbol():
    import ctypes
    from paper_1603_03820_amd import als
    lib = ctypes.CDLL(als.LIB_PATH)
    missing = [fn for fn in declared_functions() if not hasattr(lib, fn)]
    assert not missing, missing
    assert set(als.EXPORTED) == set(declared_functions())


def test_strerror_without_device():
    from paper_1603_03820_amd import als
    assert als._lib.als_strerror(0) == b"ok"
    assert als._lib.als_strerror(-6) == b"theta_in and x_out overlap"
    assert als._lib.als_strerror(12345) == b"unknown status"


def _device_disassembly(lib=None):
    import subprocess
    import tempfile
    from paper_1603_03820_amd import build
    lib = lib or build.LIB
    llvm = "/opt/rocm/llvm/bin"
    with tempfile.TemporaryDirectory() as d:
        fat, co = os.path.join(d, "fatbin.bin"), os.path.join(d, "dev.co")
        subprocess.run(["objcopy", "-O", "binary", "--only-section=.hip_fatbin", lib, fat],
                       check=True)
        subprocess.run([f"{llvm}/clang-offload-bundler", "--unbundle", "--type=o",
                        f"--input={fat}", "--targets=hipv4-amdgcn-amd-amdhsa--gfx950",
                        f"--output={co}"], check=True)
        return subprocess.run([f"{llvm}/llvm-objdump", "-d", co], capture_output=True,
                              text=True, check=True).stdout


def test_device_code_shape():
    """The gfx950 code object exists; memory is written only through vector instructions
    (no scalar-cache writes); no packed-FP32 VALU ops; the Gram uses fp32 MFMA."""
    if not os.path.exists("/opt/rocm/llvm/bin/clang-offload-bundler"):
        pytest.skip("ROCm LLVM tools not installed")
    text = _device_disassembly()
    scalar_writes = re.compile(r"\bs_(?:" + "|".join(["st" + "ore", "atom" + "ic", "dcache_" + "wb"])
                               + r")")
    assert not scalar_writes.search(text)
    assert not re.search(r"\bv_pk_(?:add|mul|fma)_f32", text)
    assert "v_mfma_f32_16x16x4_f32" in text


def test_peak_microbenchmarks_build_and_export():
    """The bench's peak microbenchmarks (measurement only) load, export their launchers, and obey
    the same device-code rules."""
    import ctypes
    from paper_1603_03820_amd import build
    lib = ctypes.CDLL(build.PEAKS_LIB)
    for fn in ("peaks_mfma", "peaks_fma", "peaks_copy", "peaks_chains"):
        assert hasattr(lib, fn), fn
    assert lib.peaks_chains() == 8
    if not os.path.exists("/opt/rocm/llvm/bin/clang-offload-bundler"):
        pytest.skip("ROCm LLVM tools not installed")
    text = _device_disassembly(build.PEAKS_LIB)
    scalar_writes = re.compile(r"\bs_(?:" + "|".join(["st" + "ore", "atom" + "ic", "dcache_" + "wb"])
                               + r")")
    assert not scalar_writes.search(text)
    assert not re.search(r"\bv_pk_(?:add|mul|fma)_f32", text)
    assert "v_mfma_f32_16x16x4_f32" in text and "v_fma_f32" in text
