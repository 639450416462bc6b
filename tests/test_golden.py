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


def test_movie_row_mean_follows_section2_2():
    """The movie shape's rows: about 200 ratings per row over 17,770 columns, as the paper
    prints for Netflix."""
    e = G["section2_2_netflix_row_mean"]
    c = synth.CONFIGS["movie"]
    assert c["n"] == e["n"]
    assert abs(c["nnz"] / c["m"] - e["items_per_user"]) / e["items_per_user"] < 0.05


def test_flop_accounting_follows_table3_terms():
    """bench.py's per-entry and per-row counts are Table 3's terms (section 2.2), counted as
    multiply + add: the Gram's f(f+1)/2 multiplies per rating twice, plus 2f per rating for b
    (Table 3's N_z f multiplies for B_u, with its additions); and the Cholesky (f^3/3 + f^2/2 +
    f/6) with two triangular solves (2 f^2) in place of Table 3's f^3 for an unnamed solver."""
    for f in (1, 2, 10, 16, 100, 128):
        assert bench.F_h(f) == 2 * (f * (f + 1) // 2) + 2 * f
        assert abs(bench.F_s(f) - (f ** 3 / 3 + f ** 2 / 2 + f / 6 + 2 * f ** 2)) < 1e-9
        assert bench.F_s(f) <= f ** 3 + 3 * f ** 2
