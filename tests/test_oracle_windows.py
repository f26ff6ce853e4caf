"""Pins of the oracle's window variants (Tables 1 and 2; the sweep-range study of the
Experiment section) to the paper's printed tables, to the standard methods they generalize,
to the exhaustive sweep, and to an exact-rational brute force.  No GPU."""
from fractions import Fraction as Fr

import numpy as np
import pytest

import oracle
import workloads
from conftest import read_golden
from test_oracle_bruteforce import rn32
from test_oracle_pins import E4M3, bf_loss


def test_tight_offsets_are_tables_1_and_2():
    upper = {int(b, 2): int(d) for b, _, d in read_golden("table1_upper_bound.txt")}
    lower = {int(b, 2): int(d) for b, _, d in read_golden("table2_lower_bound.txt")}
    for b in range(8):
        assert oracle.window_tight("scalesweep_mse", 16, b) == (lower[b], upper[b])


@pytest.mark.parametrize("n", [16, 32, 64, 128])
def test_tight_offsets_of_the_other_windows(n):
    """Table 1 bounds every objective and block size (Lemmas 1 and 2 use neither); the lower
    end keeps the standard offset where Table 2 (MSE, n = 16) does not apply."""
    upper = {int(b, 2): int(d) for b, _, d in read_golden("table1_upper_bound.txt")}
    for b in range(8):
        lo_w, hi_w = oracle.window_tight("scalesweep_wmse", n, b)
        assert (lo_w, hi_w) == (oracle.window_lower("scalesweep_wmse", n), upper[b])
        if n > 16:
            assert oracle.window_tight("scalesweep_mse", n, b) == (
                oracle.window_lower("scalesweep_mse", n), upper[b])


def test_tight_window_never_wider_than_the_standard_one():
    for b in range(8):
        lo, hi = oracle.window_tight("scalesweep_mse", 16, b)
        assert lo <= 3 and hi <= 7
    # 11, 10, 10, 10, 10, 10, 9, 10 candidates: 80 / 8 = 10 on average instead of 11
    sizes = [sum(oracle.window_tight("scalesweep_mse", 16, b)) + 1 for b in range(8)]
    assert sizes == [11, 10, 10, 10, 10, 10, 9, 10]


@pytest.mark.parametrize("c0,mode,lo,hi,expect", [
    (40, "offsets", -3, 7, (37, 47)),
    (0, "offsets", -3, 7, (1, 7)),          # the standard window's clamp at the bottom
    (124, "offsets", -3, 7, (121, 126)),    # ... and at the top
    (5, "offsets", -16, -10, (1, 1)),       # wholly below code 1: code 1 alone
    (120, "offsets", 10, 20, (126, 126)),   # wholly above code 126: code 126 alone
    (60, "offsets", 0, 0, (60, 60)),
    (60, "offsets", -126, 126, (1, 126)),   # the exhaustive sweep
    (56, "tight", 99, -99, (53, 63)),       # b = 0: [-3, 7]; offsets ignored in tight mode
    (62, "tight", 0, 0, (60, 68)),          # b = 6: [-2, 6]
    (63, "tight", 0, 0, (60, 69)),          # b = 7: [-3, 6]
])
def test_window_codes(c0, mode, lo, hi, expect):
    assert oracle.window_codes("scalesweep_mse", 16, mode, lo, hi, c0) == expect


@pytest.mark.parametrize("mode,lo,hi", [("offsets", 2, 1), ("offsets", -127, 0),
                                        ("offsets", 0, 127), (2, 0, 0), (-1, -3, 7)])
def test_window_argument_errors(mode, lo, hi):
    x = np.ones((1, 16), np.float32)
    with pytest.raises(oracle.OracleError) as e:
        oracle.quantize_window(x, 16, None, mode, lo, hi)
    assert e.value.code == -5


@pytest.mark.parametrize("block", [16, 32, 64, 128])
def test_standard_offsets_reduce_to_the_methods(block):
    g = workloads.generator("cpu", 31, block)
    x = workloads.bf16_bits(workloads.llm_weight(8, 512, g, "cpu"))
    w = workloads.column_importance(512, g, "cpu").numpy()
    for method, weight in (("scalesweep_mse", None), ("scalesweep_wmse", w)):
        L = oracle.window_lower(method, block)
        ref = oracle.quantize(method, x, block, 256.0, 0.0, weight)
        got = oracle.quantize_window(x, block, weight, "offsets", -L, 7)
        assert got[0] == ref[0]
        assert np.array_equal(got[1], ref[1]) and np.array_equal(got[2], ref[2])


def test_exhaustive_window_is_the_full_sweep():
    rng = np.random.default_rng(7)
    x = (rng.standard_normal((16, 64)) * np.exp(rng.standard_normal((16, 1)))).astype(np.float32)
    w = workloads.column_importance(64, workloads.generator("cpu", 32), "cpu").numpy()
    for weight in (None, w):
        S, q, sc = oracle.quantize_window(x, 16, weight, "offsets", -126, 126)
        y = oracle.normalize(x, S)
        for r in range(16):
            for kb in range(4):
                wb = None if weight is None else weight[kb * 16:(kb + 1) * 16]
                full = oracle.block_sweep(y[r, kb * 16:(kb + 1) * 16], wb)["c_full"]
                assert sc[r, kb] == full


def test_zero_width_window_is_the_round_down_scale():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((32, 64)).astype(np.float32)
    S, q, sc = oracle.quantize_window(x, 16, None, "offsets", 0, 0)
    y = oracle.normalize(x, S)
    for r in range(32):
        for kb in range(4):
            ymax = max(abs(Fr(float(v))) for v in y[r, kb * 16:(kb + 1) * 16])
            c0 = max(c for c in range(127) if 6 * E4M3[c] <= ymax)
            assert sc[r, kb] == max(c0, 1)


def _bf_window_scales(x, block, w, lo_off, hi_off, S):
    rows, cols = x.shape
    out = np.zeros((rows, cols // block), np.uint8)
    for r in range(rows):
        for kb in range(cols // block):
            y = [rn32(Fr(float(v)) / Fr(S)) for v in x[r, kb * block:(kb + 1) * block]]
            ymax = max(abs(Fr(v)) for v in y)
            c0 = max(c for c in range(127) if 6 * E4M3[c] <= ymax)
            lo = min(max(c0 + lo_off, 1), 126)
            hi = min(max(c0 + hi_off, 1), 126)
            wb = None if w is None else w[kb * block:(kb + 1) * block]
            Js = {c: bf_loss(y, wb, E4M3[c]) for c in range(lo, hi + 1)}
            best = min(Js.values())
            out[r, kb] = min(c for c in Js if Js[c] == best)
    return out


@pytest.mark.parametrize("lo,hi", [(-5, 2), (-1, 9), (2, 4), (-12, -9), (-2, 12)])
def test_window_argmin_matches_exact_brute_force(lo, hi):
    rng = np.random.default_rng(100 + lo * 7 + hi)
    x = (rng.standard_normal((3, 32)) * rng.uniform(0.1, 10, (3, 1))).astype(np.float32)
    w = rng.uniform(0, 2, 32).astype(np.float32)
    for weight in (None, w):
        S, q, sc = oracle.quantize_window(x, 16, weight, "offsets", lo, hi, 256.0)
        assert np.array_equal(sc, _bf_window_scales(x, 16, weight, lo, hi, S))


@pytest.mark.parametrize("D", [256.0, 448.0])
def test_tight_window_matches_the_standard_one_where_the_lemmas_apply(D):
    """MSE, n = 16 on the C0 matrix: the per-mantissa window picks the standard window's code
    in every block whose base scale is normal with 11/7 s_base^FP8 <= 448 (Lemmas 1 and 3)."""
    x = workloads.c0_matrix()
    S_t, q_t, sc_t = oracle.quantize_window(x, 16, None, "tight", 0, 0, D)
    S_s, q_s, sc_s = oracle.quantize("scalesweep_mse", x, 16, D)
    assert S_t == S_s
    y = oracle.normalize(x, S_s).reshape(-1, 16)
    c0 = np.array([oracle.floor_fp8(float(np.abs(b).max()), 6.0) for b in y])
    s0 = np.array([oracle.e4m3(int(c)) for c in c0])
    applies = (c0 >= 8) & (11 * s0 <= 7 * 448)
    assert applies.mean() > 0.9
    same = sc_t.ravel() == sc_s.ravel()
    assert same[applies].all()
