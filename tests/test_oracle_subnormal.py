"""Pins of the oracle's block-scale selection where the base code is an FP8 subnormal.

The Block Scale Optimization paragraph defines s_base^FP8 as the round-DOWN of max|y| / 6 onto
the FP8 grid, and the window is built around its bit pattern I(s_base^FP8).  For a normal base
code, rounding to nearest instead would shift the window up by one code exactly when
max|y| / 6 lies above an FP8 midpoint, and Lemma 1 (the half scale is never worse above
max|y| / 3.5) makes the extra top code lose to a code inside the window, so outputs hardly
differ.  Lemma 1's use needs s / 2 on the FP8 grid, which fails for the odd subnormal codes
(codes 1..7 are multiples of 2^-9; half of an odd one is not a grid point).  There the
window's edges decide the result: blocks with max|y| / 6 in [2^-10, 1.3 2^-6] reach their
window argmin at the upper edge c0 + 7 and would pick c0 + 8 if the window moved up.

Every expected value here comes from an integer-exact brute force written in this file
(binary32 inputs and FP8 values are dyadic, so everything is exact in scaled integers), never
from the oracle.
"""
from fractions import Fraction as Fr

import numpy as np
import pytest

import oracle
from test_oracle_pins import E4M3

SHIFT = 160                                   # 2^-149 (smallest binary32) and 2^-10 are integers here
G2 = [0, 1, 2, 3, 4, 6, 8, 12]                # twice the non-negative E2M1 values
E4M3_INT = [int(v * 2 ** SHIFT) for v in E4M3]


def _int(v) -> int:
    f = Fr(float(v)) * 2 ** SHIFT
    assert f.denominator == 1
    return int(f)


def exact_loss4(a_int, w_int, s_int):
    """4 * 2^(2 SHIFT) (times 2^SHIFT per weight) * the block loss at scale s, exactly: each
    |y| goes to the nearest point of {g s} (ties to the even E2M1 code), error 2|y| - 2g s."""
    tot = 0
    for i, a in enumerate(a_int):
        best_k, best_d = 0, None
        for k in range(8):
            d = abs(2 * a - G2[k] * s_int)
            if best_d is None or d < best_d or (d == best_d and k % 2 == 0):
                best_k, best_d = k, d
        e2 = 2 * a - G2[best_k] * s_int
        tot += (w_int[i] if w_int is not None else 1) * e2 * e2
    return tot


def exact_choose(y, w, L, U=7, round_base=True):
    """(code, c0, all window losses) of the windowed argmin, smallest code on a tie.  With
    round_base False the base code is the round-to-nearest (ties to even) of max|y| / 6,
    i.e. the planted misreading, used only to show which blocks tell the two apart."""
    a = [abs(_int(v)) for v in y]
    wi = None if w is None else [_int(v) for v in w]
    ymax = max(a)
    c0 = max(c for c in range(127) if 6 * E4M3_INT[c] <= ymax)
    if not round_base and c0 < 126:
        lo_v, hi_v = 6 * E4M3_INT[c0], 6 * E4M3_INT[c0 + 1]
        if 2 * ymax > lo_v + hi_v or (2 * ymax == lo_v + hi_v and (c0 + 1) % 2 == 0):
            c0 += 1
    lo, hi = max(1, c0 - L), min(126, c0 + U)
    J = {c: exact_loss4(a, wi, E4M3_INT[c]) for c in range(lo, hi + 1)}
    best = min(J.values())
    return min(c for c in J if J[c] == best), c0, J


def subnormal_blocks(seed, count, n):
    """Blocks whose max|y| / 6 lies in [2^-10, 1.3 2^-6] (base codes 1..8), in three shapes:
    uniform, normal and Student-t(4) around a planted maximum."""
    rng = np.random.default_rng(seed)
    out = []
    for t in range(count):
        kind = t % 3
        v = (rng.uniform(-1, 1, n) if kind == 0 else
             rng.standard_normal(n) if kind == 1 else rng.standard_t(4, n))
        smax = 2.0 ** rng.uniform(-10, -6 + np.log2(1.3))
        y = (v / np.abs(v).max() * 6 * smax).astype(np.float32)
        out.append((y, rng.uniform(0.1, 3, n).astype(np.float32)))
    return out


def _check_blocks(method, n, blocks):
    """Oracle block_choose against the brute force; returns how many blocks the planted
    round-to-nearest base code would get wrong."""
    L = 3 if method == "scalesweep_mse" else 8
    if n > 16:
        L = oracle.window_lower(method, n)
    telling = 0
    for y, w in blocks:
        ww = w if method == "scalesweep_wmse" else None
        want, c0, J = exact_choose(y, ww, L)
        got = oracle.block_choose(method, y, w)
        if got != want:      # only a binary64 rounding of an exact near-tie may differ
            assert got in J and (J[got] - J[want]) * 10 ** 14 <= J[want], (method, y, got, want)
        alt, c0n, _ = exact_choose(y, ww, L, round_base=False)
        if c0n != c0 and alt != want:
            telling += 1
    return telling


@pytest.mark.parametrize("method", ["scalesweep_mse", "scalesweep_wmse"])
def test_selection_with_subnormal_base_code_matches_exact_brute_force(method):
    blocks = subnormal_blocks(11 if method == "scalesweep_mse" else 12, 2400, 16)
    telling = _check_blocks(method, 16, blocks)
    # the sample holds blocks whose window edge decides the code (rounding the base code to
    # nearest would change them), so a base code that is not a round-down fails here
    assert telling >= 5, telling


def test_selection_with_subnormal_base_code_n32():
    blocks = subnormal_blocks(13, 200, 32)
    for method in ("scalesweep_mse", "scalesweep_wmse"):
        _check_blocks(method, 32, blocks)


def test_hand_made_block_round_down_base_code():
    """max|y| = 0.0881 gives max|y| / 6 = 0.014683, above the midpoint 0.014648 of codes 7
    (7 * 2^-9) and 8 (2^-6): the round-down base code is 7 and the MSE window [4, 14].  The
    other elements sit on the grid of code 15 (2^-6 * 15/8, with 3 * s = 0.08789 just below the
    maximum), which only a window moved up to [5, 15] could reach."""
    s15 = float(E4M3[15])
    y = np.array([0.0881] + [s15 * g for g in (3, 2, 1.5, 1, 0.5, -3, -2, -1.5, -1, -0.5, 3, 2, 1.5, 1, 0.5)],
                 np.float32)
    want, c0, J = exact_choose(y, None, 3)
    assert c0 == 7 and (min(J), max(J)) == (4, 14)
    assert oracle.block_choose("scalesweep_mse", y) == want
    alt, c0n, Jn = exact_choose(y, None, 3, round_base=False)
    assert c0n == 8 and alt == 15 != want


@pytest.mark.parametrize("method", ["scalesweep_mse", "scalesweep_wmse"])
def test_tensor_and_window_paths_with_subnormal_base_codes(method):
    """The tensor quantizer and the window-variant quantizer with S = 1 (so y = x exactly)
    on rows of such blocks: every scale byte is the brute force's."""
    n = 16
    blocks = subnormal_blocks(21 if method == "scalesweep_mse" else 22, 96, n)
    x = np.concatenate([b[0] for b in blocks]).reshape(6, 16 * n)
    w = np.concatenate([b[1] for b in blocks[:16]])
    ww = w if method == "scalesweep_wmse" else None
    L = 3 if method == "scalesweep_mse" else 8
    want = np.zeros((6, 16), np.uint8)
    for r in range(6):
        for kb in range(16):
            yb = x[r, kb * n:(kb + 1) * n]
            wb = None if ww is None else ww[kb * n:(kb + 1) * n]
            want[r, kb] = exact_choose(yb, wb, L)[0]
    S, q, sc = oracle.quantize(method, x, n, 256.0, 1.0, w)
    assert S == 1.0
    assert np.array_equal(sc, want)
    S, q, sc = oracle.quantize_window(x, n, ww, "offsets", -L, 7, 256.0, 1.0)
    assert np.array_equal(sc, want)
