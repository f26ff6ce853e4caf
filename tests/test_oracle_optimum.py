"""Pins of the oracle's reference scales (appendix "Optimal FP32 Scale for FP4 Quantization")
to an exact-rational brute force written here from the definitions: the optimal real block
scale minimizes a piecewise quadratic exactly, and the FP8-quantized optimum is the better of
the two FP8 values around it (values decoded by torch).  No GPU."""
from fractions import Fraction as Fr

import numpy as np
import pytest

import oracle
import workloads
from test_oracle_pins import E4M3, FP4_POS, bf_loss

MIDS = [(FP4_POS[k] + FP4_POS[k + 1]) / 2 for k in range(7)]


def exact_optimum(y, w=None):
    """min over real s > 0 of sum w (|y| - RNE_FP4(|y|/s) s)^2, with exact rationals: on each
    open piece between breakpoints |y_i| / m_k the rounding is fixed and the loss is
    A - 2 B s + C s^2; its infimum over the closed piece is at B / C clamped (the loss is
    continuous across breakpoints)."""
    a = [abs(Fr(float(v))) for v in y]
    wt = [Fr(1) if w is None else Fr(float(v)) for v in w] if w is not None else [Fr(1)] * len(a)
    bps = sorted({ai / m for ai in a if ai != 0 for m in MIDS})
    if not bps:
        return Fr(0)
    best = sum(wi * ai * ai for wi, ai in zip(wt, a))          # s -> infinity
    edges = [Fr(0)] + bps + [None]
    for lo, hi in zip(edges[:-1], edges[1:]):
        s_ref = (lo + hi) / 2 if hi is not None else 2 * lo
        A = B = C = Fr(0)
        for wi, ai in zip(wt, a):
            q = ai / s_ref
            g = FP4_POS[sum(1 for m in MIDS if q > m)]       # no ties inside an open piece
            A += wi * ai * ai
            B += wi * ai * g
            C += wi * g * g
        if C == 0:
            continue
        s = B / C
        s = max(s, lo)
        if hi is not None:
            s = min(s, hi)
        if s > 0:
            best = min(best, A - 2 * B * s + C * s * s)
    return best


@pytest.mark.parametrize("kind", ["normal", "t4"])
def test_continuous_optimum_matches_exact_rational_minimum(kind):
    rng = np.random.default_rng(21)
    for y in workloads.random_blocks(12, 16, rng, kind):
        w = rng.uniform(0.05, 4, 16).astype(np.float32)
        for ww in (None, w):
            J, s_opt = oracle.continuous_opt(y, ww)
            ref = exact_optimum(y, ww)
            assert J == pytest.approx(float(ref), rel=1e-12, abs=1e-300)
            # the minimizer attains it (loss evaluated exactly at the returned scale)
            assert float(bf_loss(y, ww, Fr(s_opt))) == pytest.approx(float(ref), rel=1e-9)


def test_continuous_optimum_on_other_block_sizes():
    rng = np.random.default_rng(22)
    for n in (32, 64):
        for y in workloads.random_blocks(3, n, rng, "t4"):
            J, _ = oracle.continuous_opt(y)
            assert J == pytest.approx(float(exact_optimum(y)), rel=1e-12)


def _bf_fp8_quantized(y, w, s_opt):
    """The FP8 values just below and just above s_opt (positive codes), the better by exact
    loss, the lower one on a tie."""
    v = Fr(s_opt)
    cf = max(c for c in range(127) if E4M3[c] <= v)
    cc = cf + 1 if E4M3[cf] < v and cf < 126 else cf
    cf, cc = max(cf, 1), max(cc, 1)
    jf, jc = bf_loss(y, w, E4M3[cf]), bf_loss(y, w, E4M3[cc])
    return (cc, jc) if jc < jf else (cf, jf)


def test_fp8_quantized_optimum_matches_brute_force():
    rng = np.random.default_rng(23)
    blocks = list(workloads.random_blocks(20, 16, rng, "normal"))
    blocks.append(np.zeros(16, np.float32))                  # all-zero block: s_opt = 1
    blocks.append(np.full(16, 1000.0, np.float32))           # s_opt above 448: code 126
    for y in blocks:
        w = rng.uniform(0.05, 4, 16).astype(np.float32)
        for ww in (None, w):
            _, s_opt = oracle.continuous_opt(y, ww)
            code, loss = oracle.fp8_quantized_opt(y, ww)
            c_ref, l_ref = _bf_fp8_quantized(y, ww, s_opt)
            assert code == c_ref
            assert loss == pytest.approx(float(l_ref), rel=1e-13, abs=1e-300)


def test_continuous_optimum_special_cases():
    assert oracle.continuous_opt(np.zeros(16, np.float32)) == (0.0, 1.0)
    # a single non-zero value a: exact at s = a / 6 (and other grid points), loss 0
    y = np.zeros(16, np.float32)
    y[5] = -7.0
    J, s = oracle.continuous_opt(y)
    assert J == 0.0
    assert float(bf_loss(y, None, Fr(s))) < 1e-28          # s is 7/6 rounded to binary64
