"""End-to-end pin of the oracle's tensor quantizer against an exact-rational brute force.

Every step is recomputed here from its definition with Python fractions: the global scale
S = RN32(amax / RN32(6 D)), the normalization y = RN32(x / S) (an exactly rounded binary32
quotient), the round-down / round-to-nearest onto the E4M3 grid (values decoded by torch), the
nearest-point FP4 rounding, the exact objective and the windowed argmin.  Small tensors only.
"""
import zlib
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch

import oracle
import workloads
from test_oracle_pins import E4M3, FP4_POS, bf_loss, bf_nearest_code, bf_round_fp4


def rn32(fr: Fr) -> float:
    """Round a rational to the nearest binary32 (ties to even), subnormals included."""
    if fr == 0:
        return 0.0
    sign = -1.0 if fr < 0 else 1.0
    a = abs(fr)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fr(2) ** e > a:
        e -= 1
    if Fr(2) ** (e + 1) <= a:
        e += 1
    ulp = Fr(2) ** (max(e, -126) - 23)
    n, rem = divmod(a, ulp)
    n = int(n)
    rem = rem / ulp
    if rem > Fr(1, 2) or (rem == Fr(1, 2) and n % 2 == 1):
        n += 1
    return sign * float(n * ulp)


def bf_quantize(method, x, block, D, static=0.0, w=None):
    rows, cols = x.shape
    if static:
        S = float(np.float32(static))
    else:
        amax = max(abs(Fr(float(v))) for v in x.ravel())
        S = 1.0 if amax == 0 else rn32(amax / Fr(rn32(6 * Fr(D))))
        if S == 0.0:
            S = float(np.float32(1e-45))
    q = np.zeros((rows, cols), np.uint8)
    sc = np.zeros((rows, cols // block), np.uint8)
    gaps = np.zeros((rows, cols // block))
    for r in range(rows):
        for kb in range(cols // block):
            xb = x[r, kb * block:(kb + 1) * block]
            y = [rn32(Fr(float(v)) / Fr(S)) for v in xb]
            yabs = [abs(Fr(v)) for v in y]
            ymax = max(yabs)
            wb = None if w is None else w[kb * block:(kb + 1) * block]
            if method == "absmax":
                c = bf_nearest_code(ymax / 6)
                gap = None
            elif method == "four_over_six":
                c6, c4 = bf_nearest_code(ymax / 6), bf_nearest_code(ymax / 4)
                j6, j4 = bf_loss(y, wb, E4M3[c6]), bf_loss(y, wb, E4M3[c4])
                c = c4 if j4 < j6 else c6
                gap = abs(j4 - j6) / max(j6, Fr(1, 10 ** 300))
            else:
                c0 = max(cc for cc in range(127) if 6 * E4M3[cc] <= ymax)
                L = oracle.window_lower(method, block)
                lo, hi = max(1, c0 - L), min(126, c0 + 7)
                ww = wb if method == "scalesweep_wmse" else None
                Js = {cc: bf_loss(y, ww, E4M3[cc]) for cc in range(lo, hi + 1)}
                best = min(Js.values())
                c = min(cc for cc in Js if Js[cc] == best)
                rest = [Js[cc] for cc in Js if Js[cc] != best]
                gap = (min(rest) - best) / max(best, Fr(1, 10 ** 300)) if rest else None
            sc[r, kb] = c
            gaps[r, kb] = float(gap) if gap is not None else np.inf
            for i, v in enumerate(y):
                k = bf_round_fp4(abs(Fr(v)), E4M3[c])
                q[r, kb * block + i] = (8 if np.signbit(v) else 0) | k
    packed = (q[:, 0::2] | (q[:, 1::2] << 4)).astype(np.uint8)
    return S, packed, sc, gaps


def _compare(method, x, block, D, static=0.0, w=None):
    S_o, q_o, sc_o = oracle.quantize(method, x, block, D, static, w)
    xf = oracle.bf16_to_f32(x) if x.dtype == np.uint16 else x
    S_b, q_b, sc_b, gaps = bf_quantize(method, xf, block, D, static, w)
    assert S_o == S_b
    near = gaps <= 1e-13          # FP64 objective vs exact rationals may only disagree here
    assert np.array_equal(sc_o[~near], sc_b[~near])
    rows_ok = ~near.any(axis=1)
    assert np.array_equal(q_o[rows_ok], q_b[rows_ok])


@pytest.mark.parametrize("method", list(oracle.METHODS))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("block", [16, 32])
def test_tensor_quantizer_matches_exact_brute_force(method, dtype, block):
    rng = np.random.default_rng(zlib.crc32(f"{method}/{dtype}/{block}".encode()))
    x = (rng.standard_t(4, (4, 64)) * rng.uniform(0.01, 3)).astype(np.float32)
    x[:, rng.integers(0, 64)] *= 10
    if dtype == "bf16":
        x = workloads.bf16_bits(torch.from_numpy(x).to(torch.bfloat16))
    w = rng.uniform(0.05, 4, 64).astype(np.float32)
    D = 448.0 if method == "absmax" else 256.0
    _compare(method, x, block, D, 0.0, w)
    _compare(method, x, block, D, 0.37, w)          # static global scale


def _division_sensitive_tensor():
    """A block whose normalized element x / S sits within half an ulp below the FP4 midpoint
    0.75 s with s = 1 (a tie that rounds up), found so that the correctly rounded quotient is
    exactly 0.75 while x * RN32(1/S) rounds below it: the element's FP4 code then depends on
    the normalization being a true division."""
    rng = np.random.default_rng(99)
    for _ in range(20000):
        S = np.float32(rng.uniform(0.05, 0.2))
        r = np.float32(1) / S
        base = np.float32(0.75) * S
        for d in range(-6, 7):
            x = np.float32(base)
            for _ in range(abs(d)):
                x = np.nextafter(x, np.float32(np.sign(d) * np.inf))
            if x / S == np.float32(0.75) and x * r < np.float32(0.75):
                blk = np.zeros((1, 16), np.float32)
                blk[0, 0] = np.float32(6.0) * S          # block max -> AbsMax scale 1.0
                blk[0, 1] = x
                if blk[0, 0] / S == np.float32(6.0):
                    return blk, float(S)
    raise AssertionError("no division-sensitive element found")


def test_normalization_is_a_correctly_rounded_division():
    x, S = _division_sensitive_tensor()
    _compare("absmax", x, 16, 448.0, static=S)
    _, q, sc = oracle.quantize("absmax", x, 16, 448.0, static_scale=S)
    assert oracle.e4m3(int(sc[0, 0])) == 1.0
    assert (q[0, 0] >> 4) == 2                      # 0.75 is a tie: even code 2 (value 1)
