"""The paper's own numbers (tests/golden/paper_numbers.json, each with its citation) against the
workload shapes and the flop accounting used by the benchmark (CPU only)."""
import json
import os

import bench
import synth

HERE = os.path.dirname(os.path.abspath(__file__))
G = json.load(open(os.path.join(HERE, "golden", "paper_numbers.json")))


def test_workload_shapes_follow_table5():
    t = G["table5_datasets"]
    for name, ds in (("movie", "Netflix"), ("music", "YahooMusic"), ("wiki", "Hugewiki")):
        c, d = synth.CONFIGS[name], t[ds]
        for k in ("m", "n", "nnz"):
            assert abs(c[k] - d[k]) / d[k] < 0.02, (name, k)
        assert c["f"] == d["f"]
    # the one deliberate difference: lambda of the music shape (design reading R8)
    assert synth.CONFIGS["music"]["lam"] == 1.0 and t["YahooMusic"]["lambda"] == 1.4


def test_hermitian_footprint_example():
    e = G["section2_2_memory_example"]
    assert e["m"] * e["f"] ** 2 == e["hermitian_floats"] > e["device_floats"]


def test_flop_accounting_matches_table3():
    e = G["table3_cost_all_rows"]["example"]
    f, nnz, m = e["f"], e["nnz"], e["m"]
    assert nnz * f * (f + 1) // 2 == e["A_mults"]
    assert nnz + nnz * f + 2 * m * f == e["B_cost"]
    assert m * f ** 3 == e["solve"]
    # the benchmark counts multiply+add: twice Table 3's Gram multiplies, plus 2f per entry for b
    assert nnz * bench.F_h(f) == 2 * e["A_mults"] + 2 * f * nnz
    # Cholesky (f^3/3 + f^2/2 + f/6) and two triangular solves (2 f^2)
    assert abs(bench.F_s(f) - (f ** 3 / 3 + f ** 2 / 2 + f / 6 + 2 * f ** 2)) < 1e-9
