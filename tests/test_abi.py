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
    for fn in ("peaks_mfma", "peaks_fma", "peaks_pair", "peaks_copy", "peaks_chains",
               "peaks_fma_per_iter"):
        assert hasattr(lib, fn), fn
    assert lib.peaks_chains() == 8 and lib.peaks_fma_per_iter() == 64
    # argument checks run before any launch, so they are safe without a GPU
    V, I = ctypes.c_void_p, ctypes.c_int
    lib.peaks_pair.argtypes = [V, V, I, I, I, I, V]
    assert lib.peaks_pair(None, None, 1, 1, 1, 3, None) == -1
    buf = ctypes.create_string_buffer(4)
    assert lib.peaks_pair(buf, buf, 1, 1, 1, 0, None) == -1
    assert lib.peaks_pair(buf, buf, 1, 1, 1, 4, None) == -1
    if not os.path.exists("/opt/rocm/llvm/bin/clang-offload-bundler"):
        pytest.skip("ROCm LLVM tools not installed")
    text = _device_disassembly(build.PEAKS_LIB)
    scalar_writes = re.compile(r"\bs_(?:" + "|".join(["st" + "ore", "atom" + "ic", "dcache_" + "wb"])
                               + r")")
    assert not scalar_writes.search(text)
    assert not re.search(r"\bv_pk_(?:add|mul|fma)_f32", text)
    assert "v_mfma_f32_16x16x4_f32" in text and "v_fma_f32" in text


def _vgprs(tok):
    m = re.match(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def dpp_violations(text):
    """DPP instructions whose source VGPR (src0) a VALU instruction wrote less than two wait
    states earlier (s_nop N counts N + 1).  The DPP FMAs of the factorisation are inline
    assembly, so the compiler does not insert these wait states itself.  A linear scan per
    function: every textual predecessor counts, whichever way control reaches the DPP op."""
    bad, hist = [], []
    for line in text.splitlines():
        t = line.split("//")[0].strip()
        if t.endswith(">:"):
            hist = []
            continue
        if not t or t.endswith(":"):
            continue
        op = t.split()[0]
        if op == "s_nop":
            hist.append((set(), int(t.split()[1], 0) + 1))
            continue
        args = [a.strip() for a in t[len(op):].split(",")]
        if "_dpp" in op and len(args) > 1:
            src, ws = _vgprs(args[1].split()[0]), 0
            for written, n in reversed(hist):
                if ws >= 2:
                    break
                if written & src:
                    bad.append(t)
                    break
                ws += n
        written = set()
        if (op.startswith("v_") and not op.startswith(("v_readlane", "v_readfirstlane", "v_cmp"))
                and args and args[0]):
            written = _vgprs(args[0].split()[0])
        hist = (hist + [(written, 1)])[-8:]
    return bad


def test_dpp_sources_settled():
    """Every DPP instruction in the library reads its source at least two wait states after the
    source's last VALU write (the rule the factorisation's inline DPP FMAs keep by hand), and the
    check itself catches a planted violation."""
    if not os.path.exists("/opt/rocm/llvm/bin/clang-offload-bundler"):
        pytest.skip("ROCm LLVM tools not installed")
    text = _device_disassembly()
    assert text.count("_dpp") > 1000
    assert dpp_violations(text) == []
    planted = ("<k>:\n\tv_mul_f32_e32 v5, v1, v2\n"
               "\tv_fmac_f32_dpp v4, v5, v30 row_newbcast:1 row_mask:0xf bank_mask:0xf\n"
               "\tv_mul_f32_e32 v6, v1, v2\n\ts_nop 1\n"
               "\tv_fmac_f32_dpp v4, v6, v30 row_newbcast:1 row_mask:0xf bank_mask:0xf\n")
    assert len(dpp_violations(planted)) == 1


def test_bench_refuses_more_than_one_gpu():
    """bench.py --gpus N > 1 exits with a message before touching a GPU."""
    import json
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]


def test_bench_traffic_is_tied_to_workload_and_source():
    """bench.py reports the committed HBM-traffic figure only for the workload the counters were
    taken on, and only while the kernel source is the one they were taken on."""
    import hashlib
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    kv = {}
    for line in open(bench.traffic_file("movie_f100")):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    workload = kv["workload"]
    assert workload.startswith("movie:") and "f=100" in workload
    same_src = kv["source_sha256"] == hashlib.sha256(open(bench.KERNEL_SRC, "rb").read()).hexdigest()
    expect = float(kv["bytes_per_launch"]) if same_src else None
    assert bench.measured_traffic(workload) == expect
    assert bench.measured_traffic(workload.replace("f=100", "f=32")) is None
    assert bench.measured_traffic(workload.replace("movie", "music")) is None
    assert bench.measured_traffic(workload, tag="music_f100") is None


def test_bench_roofline_bound_rule():
    """The bench's bound: min(FP32 peak, HBM peak x AI): HBM below the ridge (19.7 flop/B),
    the FP32 datapath above it; and the committed counter bytes are found per workload and side
    while the kernel source is the one they were taken on."""
    import hashlib
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_mod2", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    ridge = bench.FP32_PEAK_TFLOPS * 1e3 / bench.HBM_PEAK_GBS
    assert abs(ridge - 19.66) < 0.01
    b, peak, ai = bench.roofline_bound(9.0e12, 1e12)          # AI 9: HBM
    assert b == "hbm" and abs(peak - 72.0) < 1e-9 and ai == 9.0
    b, peak, _ = bench.roofline_bound(30.0e12, 1e12)          # AI 30: FP32
    assert b == "mfma" and peak == bench.FP32_PEAK_TFLOPS
    # compulsory bytes of a half-sweep: indices + ratings, row pointers, both factors once
    assert bench.algorithmic_bytes(10, 3, 5, 2) == 8 * 10 + 8 * 4 + 4 * 5 * 2 + 4 * 3 * 2
    src = hashlib.sha256(open(bench.KERNEL_SRC, "rb").read()).hexdigest()
    for tag in ("movie_f32", "movie_f64", "movie_f128", "music_f100", "wiki_f100"):
        path = bench.traffic_file(tag)
        if not os.path.exists(path):
            continue
        kv = dict(l.split("=", 1) for l in open(path) if "=" in l and not l.startswith("#"))
        kv = {k.strip(): v.strip() for k, v in kv.items()}
        same = kv["source_sha256"] == src
        for side in ("user", "item"):
            got = bench.measured_traffic(kv["workload"], tag, f"bytes_{side}_launch")
            assert got == (float(kv[f"bytes_{side}_launch"]) if same else None)
        assert bench.measured_traffic(kv["workload"] + " ", tag) is None
