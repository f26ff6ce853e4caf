"""Pins of the oracle's SwiGLU producer (the producer of the fused online quantizer) to
mathematics outside itself: Python's binary64 exp and an exact round-to-nearest-even onto
bfloat16 of the binary64 product.  No GPU."""
import math
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch

import oracle
import workloads


def test_exp_accuracy_and_range():
    rng = np.random.default_rng(1)
    xs = np.concatenate([rng.uniform(-80.0, 88.7, 40000), rng.uniform(-3, 3, 20000),   # and n ln2
                         np.arange(-115, 128) * math.log(2)]).astype(np.float32)
    worst = 0.0
    for x in xs:
        got = oracle.swiglu_exp(float(x))
        want = math.exp(float(x))
        if want > 3.4e38:
            assert got == math.inf or got > 2.0 ** 127
            continue
        worst = max(worst, abs(got / want - 1.0))
    assert worst < 2.0 ** -21, worst                      # a few binary32 ulps
    assert oracle.swiglu_exp(0.0) == 1.0
    assert oracle.swiglu_exp(-80.0) > 0.0 and oracle.swiglu_exp(-80.001) == 0.0
    assert oracle.swiglu_exp(89.0) == math.inf and oracle.swiglu_exp(88.7) < math.inf
    # monotone on a fine grid across a reduction boundary
    grid = np.float32(10.0) + np.arange(-2000, 2000, dtype=np.float32) * np.float32(2.0 ** -10)
    vals = [oracle.swiglu_exp(float(v)) for v in grid]
    assert all(a <= b for a, b in zip(vals, vals[1:]))


def bf16_of(v: float) -> int:
    """Nearest bfloat16 (ties to even) of a binary64 value, as a bit pattern; saturates to
    infinity past the largest finite bfloat16 + half an ulp."""
    if v == 0.0:
        return 0x8000 if math.copysign(1.0, v) < 0 else 0
    sign = 0x8000 if v < 0 else 0
    a = Fr(abs(v))
    best = None
    e = math.frexp(abs(v))[1] - 1                          # 2^e <= |v| < 2^(e+1)
    e = max(e, -126)
    ulp = Fr(2) ** (e - 7)
    k, rem = divmod(a, ulp)
    k = int(k)
    if rem > ulp / 2 or (rem == ulp / 2 and k % 2 == 1):
        k += 1
    val = k * ulp
    if val >= Fr(2) ** 128:
        return sign | 0x7F80
    f = np.float32(float(val))
    best = int(np.frombuffer(f.tobytes(), np.uint32)[0] >> 16)
    return sign | best


def near_boundary(v: float) -> bool:
    """Whether v lies within 2^-19 (relative) of a bfloat16 rounding boundary, where the
    binary32 rounding errors of the producer may decide the bfloat16 value."""
    if v == 0.0 or not math.isfinite(v):
        return False
    e = math.frexp(abs(v))[1] - 1
    ulp = 2.0 ** (max(e, -126) - 7)
    frac = (abs(v) / ulp) % 1.0
    return abs(frac - 0.5) * ulp < 2.0 ** -19 * abs(v)


def silu64(g: float) -> float:
    return g / (1.0 + math.exp(-g)) if g > -700 else -0.0


def test_swiglu_matches_binary64_reference():
    rng = np.random.default_rng(2)
    gate = workloads.bf16_bits(torch.from_numpy(rng.standard_normal(60000).astype(np.float32) * 3).to(torch.bfloat16))
    up = workloads.bf16_bits(torch.from_numpy(rng.standard_normal(60000).astype(np.float32)).to(torch.bfloat16))
    h = oracle.swiglu(gate, up)
    gf, uf = oracle.bf16_to_f32(gate), oracle.bf16_to_f32(up)
    hf = oracle.bf16_to_f32(h)
    differ = 0
    for i in range(len(h)):
        want = silu64(float(gf[i])) * float(uf[i])
        if int(h[i]) != bf16_of(want):
            assert near_boundary(want), (float(gf[i]), float(uf[i]), float(hf[i]), want)
            differ += 1
    assert differ < 60, differ


def test_swiglu_every_bfloat16_gate():
    """Every finite bfloat16 gate value with up = 1: the bfloat16 silu, within the same
    boundary allowance; the sign of zero and the saturated ends exactly."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    g = oracle.bf16_to_f32(bits)
    keep = np.isfinite(g)
    bits = bits[keep]
    one = np.full(bits.shape, 0x3F80, np.uint16)
    h = oracle.swiglu(bits, one)
    hf = oracle.bf16_to_f32(h)
    gf = oracle.bf16_to_f32(bits)
    for i in range(len(h)):
        gv = float(gf[i])
        want = silu64(gv)
        if gv > 80.0:                                         # e^-g vanishes: silu(g) = g
            assert hf[i] == gv
        elif gv <= -89.0:                                     # e^-g overflows: -0
            assert int(h[i]) == 0x8000
        elif int(h[i]) != bf16_of(want):
            assert near_boundary(want), (gv, float(hf[i]), want)
    assert int(oracle.swiglu(np.array([0x0000], np.uint16), np.array([0x3F80], np.uint16))[0]) == 0
    assert int(oracle.swiglu(np.array([0x8000], np.uint16), np.array([0x3F80], np.uint16))[0]) == 0x8000
    assert int(oracle.swiglu(np.array([0x0000], np.uint16), np.array([0xBF80], np.uint16))[0]) == 0x8000


def test_swiglu_rejects_non_finite():
    with pytest.raises(oracle.OracleError):
        oracle.swiglu(np.array([0x7F80], np.uint16), np.array([0x3F80], np.uint16))
    with pytest.raises(oracle.OracleError):
        oracle.swiglu(np.array([0x3F80], np.uint16), np.array([0x7FC0], np.uint16))
