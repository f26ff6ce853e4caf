"""Pins of the CPU oracle to things other than itself (no GPU).

Each test checks the oracle against what the paper or mathematics fixes: values the paper
prints (tests/golden/, each fixture citing its table or section), an independent library
decode (torch's float8 types), exact rational brute force on small inputs, closed forms and
the paper's lemmas as invariants.  A plausible mistake anywhere in the oracle -- a flipped
tie rule, a dropped weight, a wrong window bound, an off-by-one code, a lost sign -- fails
at least one of them (tests/test_oracle_mutants.py plants such mistakes and checks that).
"""
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch

import oracle
import workloads
from conftest import read_golden

FP4_POS = sorted({Fr(r[0]) for r in read_golden("e2m1_grid.txt") if Fr(r[0]) >= 0})


def torch_e4m3_values():
    """E4M3 values of codes 0..126 decoded by torch (an independent implementation)."""
    b = torch.arange(127, dtype=torch.uint8)
    return [Fr(float(v)) for v in b.view(torch.float8_e4m3fn).float().tolist()]


E4M3 = torch_e4m3_values()


def bf_round_fp4(a: Fr, s: Fr) -> int:
    """Brute-force nearest point of {v s : v in G_FP4} to a >= 0; exact ties -> even code."""
    if s == 0:
        return 0
    d = [abs(a - v * s) for v in FP4_POS]
    best = min(d)
    idx = [k for k in range(8) if d[k] == best]
    return idx[0] if len(idx) == 1 else [k for k in idx if k % 2 == 0][0]


def bf_loss(y, w, s: Fr) -> Fr:
    tot = Fr(0)
    for i, v in enumerate(y):
        a = abs(Fr(float(v)))
        e = a - FP4_POS[bf_round_fp4(a, s)] * s
        tot += (Fr(float(w[i])) if w is not None else 1) * e * e
    return tot


def bf_nearest_code(v: Fr) -> int:
    """Nearest E4M3 code (0..126) to v >= 0, ties to even code, saturating at 448."""
    d = [abs(v - e) for e in E4M3]
    best = min(d)
    idx = [c for c in range(127) if d[c] == best]
    return idx[0] if len(idx) == 1 else [c for c in idx if c % 2 == 0][0]


# --------------------------------------------------------------------------------------
# Number formats
# --------------------------------------------------------------------------------------

def test_e2m1_grid_is_the_papers():
    got = sorted({oracle.e2m1(k) for k in range(8)} | {-oracle.e2m1(k) for k in range(8)})
    want = sorted(float(r[0]) for r in read_golden("e2m1_grid.txt"))
    assert got == sorted(set(want))


def test_e4m3_decode_matches_torch_and_paper_facts():
    facts = {r[0]: float(r[1]) for r in read_golden("fp8_e4m3_facts.txt")}
    tab = oracle.e4m3_table()
    assert [Fr(float(v)) for v in tab] == E4M3
    pos = [v for v in tab if v > 0 and np.isfinite(v)]
    assert len(pos) == facts["positive_finite_count"]
    assert max(pos) == facts["max_value"]
    assert max(oracle.e2m1_table()) == facts["fp4_max_value"]
    # strictly increasing: the bit-pattern integer orders the values (Appendix A)
    assert all(tab[i] < tab[i + 1] for i in range(126))


def test_generic_eemm_formula_matches_torch_e5m2():
    """Appendix A's v(c, a, b) for E5M2 (bias 15) against torch's float8_e5m2 decode."""
    b = torch.arange(124, dtype=torch.uint8)            # finite positive-or-zero E5M2 codes
    ref = b.view(torch.float8_e5m2).float().tolist()
    got = [oracle.eemm_value(5, 2, c) for c in range(124)]
    assert got == ref


# --------------------------------------------------------------------------------------
# Rounding
# --------------------------------------------------------------------------------------

def _fp4_test_points(rng):
    pts = []
    for c in range(1, 127):
        s = float(E4M3[c])
        for k in range(7):
            mid = np.float32((float(FP4_POS[k]) + float(FP4_POS[k + 1])) / 2 * s)
            pts += [(mid, s), (np.nextafter(mid, np.float32(0)), s),
                    (np.nextafter(mid, np.float32(1e9)), s)]
        for v in FP4_POS:
            pts.append((np.float32(float(v) * s), s))
        for a in rng.uniform(0, 8 * s, 4).astype(np.float32):
            pts.append((a, s))
    return pts


def test_round_fp4_matches_exact_brute_force():
    rng = np.random.default_rng(1)
    for a, s in _fp4_test_points(rng):
        assert oracle.round_fp4(float(a), s) == bf_round_fp4(Fr(float(a)), Fr(s)), (a, s)


def test_round_fp4_zero_scale_and_saturation():
    assert oracle.round_fp4(5.0, 0.0) == 0
    assert oracle.round_fp4(1e30, 1.0) == 7
    assert oracle.round_fp4(0.0, 1.0) == 0


def test_nearest_fp8_matches_torch_rne():
    """Round-to-nearest-even onto E4M3 (AbsMax's rounding) against torch's conversion, for
    binary32 inputs below 464 (torch turns larger values into NaN; the oracle saturates)."""
    rng = np.random.default_rng(2)
    vals = list(rng.uniform(0, 464, 3000).astype(np.float32))
    vals += list(np.exp(rng.uniform(np.log(1e-4), np.log(400), 3000)).astype(np.float32))
    for c in range(126):                      # exact midpoints and neighbours
        m = np.float32((float(E4M3[c]) + float(E4M3[c + 1])) / 2)
        vals += [m, np.nextafter(m, np.float32(0)), np.nextafter(m, np.float32(1e9))]
    vals = [v for v in vals if v < 464]
    ref = torch.tensor(np.array(vals, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8)
    got = [oracle.nearest_fp8(float(v), 1.0) for v in vals]
    assert got == ref.tolist()
    assert oracle.nearest_fp8(1e6, 1.0) == 126          # reading: saturate at 448


def test_floor_and_nearest_fp8_of_ratio_brute_force():
    rng = np.random.default_rng(3)
    for _ in range(400):
        ymax = np.float32(rng.uniform(0, 3000))
        for den in (4, 6):
            v = Fr(float(ymax)) / den
            fl = max(c for c in range(127) if E4M3[c] <= v)
            assert oracle.floor_fp8(float(ymax), den) == fl
            assert oracle.nearest_fp8(float(ymax), den) == bf_nearest_code(v)


# --------------------------------------------------------------------------------------
# Tables 1-3 recomputed from the oracle's formats and rounding
# --------------------------------------------------------------------------------------

@pytest.mark.parametrize("a", [2, 5, 7, 9, 11])
def test_table1_upper_bound_per_mantissa(a):
    """Table 1: the largest round-down of (12/7) s_base over s_base in the FP8 interval
    starting at s_base^FP8 (closed at the top, as the printed sup values are)."""
    for b, sup, delta in read_golden("table1_upper_bound.txt"):
        b = int(b, 2)
        c0 = 8 * a + b
        s1 = oracle.e4m3(c0 + 1)
        c_sup = oracle.floor_fp8(12 * s1, 7)               # largest c with 7 E4M3(c) <= 12 s1
        carry, mant = int(sup[0]), int(sup[1:], 2)
        assert c_sup == 8 * a + mant + 8 * carry
        assert c_sup - c0 == int(delta)
        # Lemma 2 with alpha = 12/7, m = 3: ceil((1 - 7/12) 2^4) = 7 bounds every row
        assert c_sup - c0 <= 7


@pytest.mark.parametrize("a", [2, 5, 7, 9, 11])
def test_table2_lower_bound_per_mantissa(a):
    """Table 2: the smallest round-up of (4/5) s_base^FP8."""
    for b, inf, delta in read_golden("table2_lower_bound.txt"):
        b = int(b, 2)
        c0 = 8 * a + b
        s0 = oracle.e4m3(c0)
        c_inf = min(c for c in range(1, 127) if 5 * oracle.e4m3(c) >= 4 * s0)
        borrow, mant = int(inf[0]), int(inf[1:], 2)
        assert c_inf == 8 * a + mant - 8 * borrow
        assert c0 - c_inf == int(delta)


def _d(y, r):
    g = oracle.e2m1(oracle.round_fp4(y, r))
    return (y - r * g) ** 2


def _sup_delta(us, lams, r, lo, hi):
    pts = {lo, hi}
    for u in list(us) + [r]:
        for k in range(7):
            m = (oracle.e2m1(k) + oracle.e2m1(k + 1)) / 2 * u
            if lo <= m <= hi:
                pts.add(m)
    f = lambda y: sum(l * _d(y, u) for u, l in zip(us, lams)) - _d(y, r)
    return max(f(y) for y in pts)


def test_table3_convex_certificates():
    """Table 3: A = sup over [6, 6 rho_m] and B = sup over [0, 6 rho_m] of
    sum_j lambda_j d_{u_j}(y) - d_r(y), with rho_m = (m+1)/m for the mantissa m of s0 that
    makes r = j/m 2^k an FP8 ratio.  d_r uses the oracle's FP4 rounding."""
    m_of = {Fr(7, 9): 9, Fr(10, 13): 13, Fr(11, 14): 14}
    for row in read_golden("table3_certificates.txt"):
        r = Fr(row[0])
        us = [Fr(v) for v in row[1:4]]
        lams = [Fr(v) for v in row[4:7]]
        B_p, A_p, AB_p = (Fr(v) for v in row[7:10])
        assert sum(lams) == 1
        rho = Fr(m_of[r] + 1, m_of[r])
        B = _sup_delta([float(u) for u in us], [float(l) for l in lams], float(r), 0.0,
                       float(6 * rho))
        A = _sup_delta([float(u) for u in us], [float(l) for l in lams], float(r), 6.0,
                       float(6 * rho))
        assert B == pytest.approx(float(B_p), abs=1e-12)
        assert A == pytest.approx(float(A_p), abs=1e-12)
        assert A + 15 * B == pytest.approx(float(AB_p), abs=1e-12)
        assert A + 15 * B < 0


def test_table3_ratios_are_the_only_fp8_ratios_in_open_interval():
    """Proof of Lemma 3: the only FP8 ratios j/m 2^k (j, m in 8..15) in (3/4, 4/5)."""
    found = set()
    for j in range(8, 16):
        for m in range(8, 16):
            for k in range(-2, 3):
                r = Fr(j, m) * Fr(2) ** k
                if Fr(3, 4) < r < Fr(4, 5):
                    found.add(r)
    assert found == {Fr(7, 9), Fr(10, 13), Fr(11, 14)}


def test_window_bounds_n16_are_the_papers():
    for method, n, lo, hi in read_golden("windows.txt"):
        assert -oracle.window_lower(method, int(n)) == int(lo)
        assert oracle.window_upper() == int(hi)


@pytest.mark.parametrize("n,expect", [(16, 3), (32, 5), (64, 7), (128, 11)])
def test_mse_window_lower_offsets_follow_the_lemma3_argument(n, expect):
    """reading for n > 16: the r <= 3/4 step of the proof of Lemma 3 with n - 1 non-maximal
    coordinates excludes every ratio r < 24 / (28 + (n-1)/4); the lower offset is the largest
    code distance to the smallest FP8 ratio at or above that bound, over all mantissas."""
    rstar = Fr(24) / (28 + Fr(n - 1, 4))
    worst = 0
    for a in range(3, 12):
        for b in range(8):
            c0 = 8 * a + b
            cmin = min(c for c in range(1, 127) if E4M3[c] >= rstar * E4M3[c0])
            worst = max(worst, c0 - cmin)
    assert worst == expect
    assert oracle.window_lower("scalesweep_mse", n) == expect
    assert oracle.window_lower("scalesweep_wmse", n) == max(8, expect)


# --------------------------------------------------------------------------------------
# Objective and selection: brute force on tiny blocks
# --------------------------------------------------------------------------------------

def _lattice_blocks(rng, n, count):
    base = [float(v) for v in FP4_POS] + [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]
    out = []
    for _ in range(count):
        s = float(E4M3[rng.integers(20, 110)])
        v = np.array([rng.choice(base) * s for _ in range(n)], np.float32)
        v *= rng.choice([-1, 1], n).astype(np.float32)
        jig = rng.integers(0, 3, n)
        v = np.where(jig == 1, np.nextafter(v, np.float32(1e9)), v)
        v = np.where(jig == 2, np.float32(rng.uniform(0, 7 * s)), v)
        out.append(v.astype(np.float32))
    return out


@pytest.mark.parametrize("n", [1, 2, 4])
def test_block_loss_matches_exact_brute_force(n):
    rng = np.random.default_rng(10 + n)
    for y in _lattice_blocks(rng, n, 25):
        w = rng.uniform(0, 3, n).astype(np.float32)
        for c in list(range(1, 127, 5)) + [126]:
            s = E4M3[c]
            for ww in (None, w):
                exact = bf_loss(y, ww, s)
                got = oracle.block_loss(y, ww, float(s))
                assert got == pytest.approx(float(exact), rel=1e-14, abs=1e-300)


def test_block_loss_zero_scale_is_energy_and_exact_grid_is_zero():
    y = np.array([3.0, -1.5, 0.25, 6.0], np.float32)
    w = np.array([1.0, 2.0, 0.5, 4.0], np.float32)
    assert oracle.block_loss(y, w, 0.0) == float(np.sum(w.astype(np.float64) * y.astype(np.float64) ** 2))
    s = float(E4M3[60])
    g = np.array([6.0, -4.0, 0.5, 0.0, 1.5, -3.0], np.float32) * np.float32(s)
    assert oracle.block_loss(g, None, s) == 0.0


@pytest.mark.parametrize("n", [2, 4])
def test_windowed_argmin_matches_brute_force(n):
    rng = np.random.default_rng(20 + n)
    for y in _lattice_blocks(rng, n, 20):
        w = rng.uniform(0.1, 3, n).astype(np.float32)
        for method, ww in (("scalesweep_mse", None), ("scalesweep_wmse", w)):
            ymax = max(abs(Fr(float(v))) for v in y)
            c0 = max(c for c in range(127) if 6 * E4M3[c] <= ymax)
            L = 3 if method == "scalesweep_mse" else 8
            lo, hi = max(1, c0 - L), min(126, c0 + 7)
            Js = {c: bf_loss(y, ww, E4M3[c]) for c in range(lo, hi + 1)}
            best = min(Js.values())
            want = min(c for c in Js if Js[c] == best)
            info = oracle.block_sweep(y, ww, L, 7)
            assert (info["c0"], info["lo"], info["hi"]) == (c0, lo, hi)
            got = info["c_win"]
            if got != want:        # only an FP64 rounding tie-break may differ from exact
                assert float(Js[got] - best) <= 1e-14 * float(best)


def test_block_choose_sweeps_the_methods_window():
    rng = np.random.default_rng(30)
    for n in (16, 32, 64, 128):
        for y in workloads.random_blocks(12, n, rng, "t4"):
            w = rng.uniform(0.1, 3, n).astype(np.float32)
            for method, ww in (("scalesweep_mse", None), ("scalesweep_wmse", w)):
                L = oracle.window_lower(method, n)
                assert oracle.block_choose(method, y, w) == \
                    oracle.block_sweep(y, ww, L, 7)["c_win"]


def test_absmax_code_is_nearest_fp8_of_block_max_over_six():
    rng = np.random.default_rng(5)
    for kind in ("normal", "t4", "uniform"):
        for y in workloads.random_blocks(200, 16, rng, kind):
            ymax = max(abs(Fr(float(v))) for v in y)
            assert oracle.block_choose("absmax", y) == bf_nearest_code(ymax / 6)


def test_four_over_six_picks_lower_loss_of_its_two_codes():
    rng = np.random.default_rng(6)
    for y in workloads.random_blocks(150, 16, rng, "t4"):
        ymax = max(abs(Fr(float(v))) for v in y)
        c6, c4 = bf_nearest_code(ymax / 6), bf_nearest_code(ymax / 4)
        j6, j4 = bf_loss(y, None, E4M3[c6]), bf_loss(y, None, E4M3[c4])
        got = oracle.block_choose("four_over_six", y)
        assert got in (c6, c4)
        if abs(j4 - j6) > Fr(1, 10 ** 12) * j6:
            assert got == (c4 if j4 < j6 else c6)


def test_weighted_objective_reduces_to_unweighted_and_is_scale_invariant():
    rng = np.random.default_rng(7)
    for y in workloads.random_blocks(100, 16, rng, "t4"):
        ones = np.ones(16, np.float32)
        w = rng.uniform(0.01, 5, 16).astype(np.float32)
        assert oracle.block_choose("scalesweep_wmse", y, ones) == \
            oracle.block_sweep(y, None, 8, 7)["c_win"]
        assert oracle.block_choose("scalesweep_wmse", y, w) == \
            oracle.block_choose("scalesweep_wmse", y, w * np.float32(4))


# --------------------------------------------------------------------------------------
# Lemmas as invariants
# --------------------------------------------------------------------------------------

def test_lemma1_half_scale_is_never_worse():
    """Lemma 1: for s > max|y| / 3.5 (and s/2 an FP8 value), L(s) >= L(s/2)."""
    rng = np.random.default_rng(8)
    for kind in ("normal", "t4", "uniform"):
        for y in workloads.random_blocks(60, 16, rng, kind):
            w = rng.uniform(0, 4, 16).astype(np.float32)
            for ww in (None, w):
                J = oracle.block_sweep(y, ww, 3, 7)["J"]
                ymax = float(np.max(np.abs(y.astype(np.float64))))
                for c in range(16, 127):
                    if oracle.e4m3(c) * 3.5 > ymax:
                        assert oracle.e4m3(c - 8) * 2 == oracle.e4m3(c)
                        assert J[c] >= J[c - 8]


def _c0_blocks():
    x = workloads.c0_matrix()
    S = oracle.tensor_scale(x, 448.0)
    return oracle.normalize(x, S).reshape(-1, 16)


@pytest.mark.slow
def test_c0_window_contains_full_sweep_optimum_everywhere():
    """The 1024 x 1024 N(0,1) binary32 matrix, n = 16, MSE, S = amax / (6 * 448): the full
    sweep over all 126 codes and the [-3, +7] window agree on all 65,536 blocks, and the
    Lemma 3 bound (argmin >= 4/5 s_base^FP8) holds wherever its precondition does."""
    y = _c0_blocks()
    assert y.shape[0] == 65536
    misses = 0
    for blk in y:
        info = oracle.block_sweep(blk, None, 3, 7)
        if info["c_win"] != info["c_full"]:
            misses += 1
        c0 = info["c0"]
        s0 = oracle.e4m3(c0)
        if c0 >= 8 and 11 * s0 <= 7 * 448:
            assert 5 * oracle.e4m3(info["c_full"]) >= 4 * s0
    assert misses == 0


def test_lemma3_on_random_blocks():
    rng = np.random.default_rng(9)
    for kind in ("normal", "t4", "uniform"):
        for y in workloads.random_blocks(150, 16, rng, kind):
            info = oracle.block_sweep(y, None, 3, 7)
            c0, s0 = info["c0"], oracle.e4m3(info["c0"])
            if c0 >= 8 and 11 * s0 <= 7 * 448:
                assert 5 * oracle.e4m3(info["c_full"]) >= 4 * s0
                assert info["c_win"] == info["c_full"]


# --------------------------------------------------------------------------------------
# Scale quality: continuous optimum (appendix) as a lower bound
# --------------------------------------------------------------------------------------

def test_continuous_optimum_is_a_lower_bound_and_attained():
    rng = np.random.default_rng(11)
    for kind in ("normal", "t4"):
        for y in workloads.random_blocks(40, 16, rng, kind):
            w = rng.uniform(0.1, 3, 16).astype(np.float32)
            for ww in (None, w):
                lo, s_opt = oracle.continuous_opt(y, ww)
                J = oracle.block_sweep(y, ww, 3, 7)["J"]
                assert np.all(J[1:] >= lo * (1 - 1e-12))
                ymax = float(np.max(np.abs(y)))
                for s in np.geomspace(ymax / 40, ymax / 0.2, 4000):     # dense brute force
                    assert oracle.block_loss(y, ww, s) >= lo * (1 - 1e-12)
                assert oracle.block_loss(y, ww, s_opt) == pytest.approx(lo, rel=1e-9, abs=1e-12)
                c8, l8 = oracle.fp8_quantized_opt(y, ww)
                assert l8 >= lo * (1 - 1e-12)
                assert l8 >= J[1:].min()


def test_continuous_optimum_closed_forms():
    y = np.full(16, 3.7, np.float32)                     # equal values: exact fit, zero loss
    assert oracle.continuous_opt(y)[0] == pytest.approx(0.0, abs=1e-12)
    y = np.zeros(16, np.float32)
    assert oracle.continuous_opt(y)[0] == 0.0
    # one non-zero value a among zeros: a = 6 s is exact, loss 0
    y = np.zeros(16, np.float32)
    y[3] = 5.0
    assert oracle.continuous_opt(y)[0] == pytest.approx(0.0, abs=1e-12)
    # values a and 2a: both on the grid at s = a / 3 (3 s and 6 s)
    y = np.array([1.0, 2.0] * 8, np.float32)
    assert oracle.continuous_opt(y)[0] == pytest.approx(0.0, abs=1e-12)


def test_scalesweep_no_worse_than_absmax_and_four_over_six_at_equal_scale():
    """At D = 256 the AbsMax and 4/6 codes lie inside the window, so the window argmin can
    only be better (Introduction / Figure 1's ordering)."""
    x = workloads.c0_matrix()[:64]
    S = oracle.tensor_scale(x, 256.0)
    y = oracle.normalize(x, S).reshape(-1, 16)
    for blk in y:
        js = {m: oracle.block_loss(blk, None, oracle.e4m3(oracle.block_choose(m, blk)))
              for m in ("absmax", "four_over_six", "scalesweep_mse")}
        assert js["scalesweep_mse"] <= js["absmax"]
        assert js["scalesweep_mse"] <= js["four_over_six"]


# --------------------------------------------------------------------------------------
# Tensor level: global scale, packing, round trip, errors
# --------------------------------------------------------------------------------------

def test_global_scale_is_correctly_rounded_quotient():
    rng = np.random.default_rng(12)
    for D in (448.0, 256.0, 100.0):
        x = (rng.standard_normal((8, 64)) * rng.uniform(1e-3, 1e3)).astype(np.float32)
        S = oracle.tensor_scale(x, D)
        exact = Fr(float(np.max(np.abs(x)))) / (6 * Fr(D))
        S32 = np.float32(S)
        for nb in (np.nextafter(S32, np.float32(0)), np.nextafter(S32, np.float32(np.inf))):
            assert abs(Fr(float(S32)) - exact) <= abs(Fr(float(nb)) - exact)
    assert oracle.tensor_scale(np.zeros((2, 16), np.float32), 256.0) == 1.0
    tiny = np.zeros((1, 16), np.float32)
    tiny[0, 0] = np.float32(1e-45)
    assert oracle.tensor_scale(tiny, 448.0) > 0.0


@pytest.mark.parametrize("method", list(oracle.METHODS))
def test_power_of_two_equivariance(method):
    """x -> 4x scales S by exactly 4 and leaves y, codes and nibbles unchanged."""
    rng = np.random.default_rng(13)
    x = (rng.standard_normal((16, 64)) * 0.3).astype(np.float32)
    w = rng.uniform(0.1, 2, 64).astype(np.float32)
    S1, q1, s1 = oracle.quantize(method, x, 16, 256.0, weight=w)
    S2, q2, s2 = oracle.quantize(method, x * np.float32(4), 16, 256.0, weight=w)
    assert S2 == 4 * S1
    assert np.array_equal(q1, q2) and np.array_equal(s1, s2)


@pytest.mark.parametrize("method", list(oracle.METHODS))
def test_negation_flips_only_sign_bits(method):
    rng = np.random.default_rng(14)
    x = (rng.standard_normal((8, 64))).astype(np.float32)
    w = rng.uniform(0.1, 2, 64).astype(np.float32)
    S1, q1, s1 = oracle.quantize(method, x, 16, 256.0, weight=w)
    S2, q2, s2 = oracle.quantize(method, -x, 16, 256.0, weight=w)
    assert S1 == S2 and np.array_equal(s1, s2)
    assert np.array_equal(q1 ^ np.uint8(0x88), q2)


def _grid_tensor(rng, rows, cols, block, dtype):
    """A tensor on the NVFP4 grid whose dynamic S (D = 256) is the power of two 2^-3 and whose
    every block contains an element of magnitude 6 s."""
    S = 2.0 ** -3
    x = np.zeros((rows, cols), np.float64)
    for r in range(rows):
        for kb in range(cols // block):
            c = int(rng.integers(30, 121))
            ks = rng.integers(0, 8, block)
            ks[rng.integers(0, block)] = 7
            sg = rng.choice([-1.0, 1.0], block)
            if r == 0 and kb == 0:              # this block holds amax = 6 * 256 * S
                c, ks[0], sg[0] = 120, 7, 1.0
            x[r, kb * block:(kb + 1) * block] = sg * np.array([float(FP4_POS[k]) for k in ks]) \
                * float(E4M3[c]) * S
    x = x.astype(np.float32)
    if dtype == "bf16":
        return workloads.bf16_bits(torch.from_numpy(x).to(torch.bfloat16))
    return x


@pytest.mark.parametrize("method", list(oracle.METHODS))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("block", [16, 64])
def test_round_trip_on_the_grid_is_exact(method, dtype, block):
    rng = np.random.default_rng(15)
    x = _grid_tensor(rng, 6, 256, block, dtype)
    w = rng.uniform(0.1, 2, 256).astype(np.float32)
    S, q, sc = oracle.quantize(method, x, block, 256.0, weight=w)
    assert S == 2.0 ** -3
    xh = oracle.dequant(q, sc, S, block)
    xf = oracle.bf16_to_f32(x) if dtype == "bf16" else x
    assert np.array_equal(xh.view(np.uint32), xf.view(np.uint32))


def test_nibble_packing_order_and_sign_of_zero():
    x = np.zeros((1, 16), np.float32)
    x[0, 0] = 6.0      # -> code 7, low nibble of byte 0
    x[0, 1] = -3.0     # -> sign | code 5, high nibble of byte 0
    x[0, 2] = -0.0     # -> sign bit kept on zero
    S, q, sc = oracle.quantize("absmax", x, 16, 448.0, static_scale=1.0)
    assert sc[0, 0] == oracle.nearest_fp8(6.0, 6.0)
    assert q[0, 0] == (0x7 | (0xD << 4))
    assert q[0, 1] & 0x0F == 0x8


def test_scalesweep_zero_block_gets_code_one_and_absmax_code_zero():
    x = np.zeros((1, 32), np.float32)
    x[0, 16] = 1.0
    _, _, sc = oracle.quantize("scalesweep_mse", x, 16, 256.0)
    assert sc[0, 0] == 1
    _, q, sc = oracle.quantize("absmax", x, 16, 448.0)
    assert sc[0, 0] == 0 and np.all(q[0, :8] == 0)


def test_status_codes():
    x = np.zeros((4, 32), np.float32)
    assert oracle.quantize_status("scalesweep_mse", x) == 0
    assert oracle.quantize_status("scalesweep_mse", x, block=24) == -3
    assert oracle.quantize_status("scalesweep_mse", x, cols=30) == -2
    assert oracle.quantize_status("scalesweep_mse", x, fp8_range=0.0) == -5
    assert oracle.quantize_status("scalesweep_mse", x, fp8_range=500.0) == -5
    assert oracle.quantize_status("scalesweep_mse", x, static_scale=-1.0) == -5
    assert oracle.quantize_status("scalesweep_mse", x, static_scale=float("nan")) == -5
    assert oracle.quantize_status("scalesweep_wmse", x) == -1
    bad = np.ones(32, np.float32)
    bad[3] = -1
    assert oracle.quantize_status("scalesweep_wmse", x, weight=bad) == -5
    x[1, 3] = np.inf
    assert oracle.quantize_status("absmax", x) == -9
    x[1, 3] = 1e30
    assert oracle.quantize_status("absmax", x, static_scale=1e-20) == -9


def test_metrics_definitions_on_a_hand_example():
    x = np.array([[1.0, -2.0, 3.0, 0.0]], np.float32)
    xh = np.array([[1.5, -2.0, 2.0, 0.5]], np.float32)
    w = np.array([2.0, 1.0, 1.0, 4.0], np.float32)
    m = oracle.metrics(x, xh, w)
    assert m["mse"] == pytest.approx((0.25 + 0 + 1 + 0.25) / 4)
    assert m["nmse"] == pytest.approx(1.5 / 14)
    assert m["wmse"] == pytest.approx((0.5 + 0 + 1 + 1) / 8)
    assert m["nwmse"] == pytest.approx(2.5 / (2 + 4 + 9))


def test_c0_quality_ordering():
    """Figure 1's ordering on the N(0,1) matrix: AbsMax > 4/6 > ScaleSweep in NMSE, and the
    ScaleSweep objective sits above the sum of per-block continuous optima."""
    x = workloads.c0_matrix()[:128]
    res = {}
    for m, D in (("absmax", 448.0), ("four_over_six", 256.0), ("scalesweep_mse", 256.0)):
        S, q, sc = oracle.quantize(m, x, 16, D)
        res[m] = oracle.metrics(x, oracle.dequant(q, sc, S, 16))["nmse"]
    assert res["absmax"] > res["four_over_six"] > res["scalesweep_mse"]


def test_four_over_six_exact_tie_keeps_the_six_code():
    """A block exact on both grids ({0, 1.5, 3, 6} s lies in G s and in G 1.5 s): both losses
    are zero, and the tie keeps the scale that maps the block maximum to 6."""
    y = np.zeros(16, np.float32)
    y[:3] = [6.0, -3.0, 1.5]
    c6, c4 = oracle.nearest_fp8(6.0, 6.0), oracle.nearest_fp8(6.0, 4.0)
    assert (oracle.e4m3(c6), oracle.e4m3(c4)) == (1.0, 1.5)
    assert oracle.block_loss(y, None, 1.0) == oracle.block_loss(y, None, 1.5) == 0.0
    assert oracle.block_choose("four_over_six", y) == c6


def test_window_lower_edge_is_reached():
    """A block (found by a hill-climb on the oracle's full sweep) whose optimum sits exactly at
    the window's lower edge I(s_base^FP8) - 3 (Table 2, mantissa 000), and its power-of-two
    rescalings, which shift every code by a multiple of 8."""
    base = np.array([6.0, 1.221445893817698, 4.652834527496325, 3.3511210740080655,
                     4.989745833983692, 4.748865158786074, 0.406404801387671, 1.3845467685649486,
                     3.064249960616528, 1.2247963293421917, 1.21898021729173, 5.212238587925807,
                     1.2202789634017701, 0.413340576750549, 1.2165832546342012,
                     4.815861171136384], np.float32)
    for k in (-3, 0, 2, 5):
        y = base * np.float32(2.0 ** k)
        info = oracle.block_sweep(y, None, 3, 7)
        c0 = max(c for c in range(127) if 6 * E4M3[c] <= max(abs(Fr(float(v))) for v in y))
        assert info["c0"] == c0 == 56 + 8 * k
        assert info["c_full"] == c0 - 3
        assert oracle.block_choose("scalesweep_mse", y) == c0 - 3
