"""The quotients the quantization kernels round with are the correctly rounded ones.

The kernels form y = RN32(x / S) and the emit step's u = RN32(y / M) (M the significand of the
chosen E4M3 scale) as a reciprocal product with one fused multiply-add correction
(Markstein), not with a division instruction.  The oracle divides in IEEE binary32.  These
CPU tests run that recipe, written out in tests/exact_quotient_check.c, against C's
division: every bfloat16 pattern against thousands of global scales, random binary32 inputs,
and random y against all eight E4M3 significands.  Any mismatch where it could change an
FP4 code fails.  (The recipe is stated here again rather than taken from the kernel source:
the test pins the arithmetic, and the GPU parity suite pins that the kernels use it.)
"""
import subprocess
from pathlib import Path

import pytest

HERE = Path(__file__).resolve().parent


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = tmp_path_factory.mktemp("eqc") / "exact_quotient_check"
    # -ffp-contract=off: the operations as written; libm's fmaf is correctly rounded
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-o", str(exe),
                    str(HERE / "exact_quotient_check.c"), "-lm"], check=True)
    return exe


def run(exe, mode, count):
    out = subprocess.run([str(exe), mode, str(count)], capture_output=True, text=True,
                         check=True, timeout=300).stdout.split()
    i = out.index("checked")
    return {k: int(v) for k, v in zip(out[i::2], out[i + 1::2])}, " ".join(out)


def test_normalization_all_bfloat16_patterns(checker):
    r, text = run(checker, "norm", 4000)
    assert r["mismatch"] == 0, text
    assert r["checked"] > 4000 * 50000     # finite patterns with |x| >= 2^-74, per scale
    assert r["nonfinite_ok"] > 0          # overflowing quotients stay non-finite


def test_normalization_random_binary32(checker):
    r, text = run(checker, "norm32", 60_000_000)
    assert r["mismatch"] == 0, text
    assert r["checked"] == 60_000_000


def test_emit_quotient_by_e4m3_significands(checker):
    r, text = run(checker, "sig", 12_000_000)
    assert r["mismatch"] == 0, text
    assert r["checked"] == 8 * 12_000_000 + 16
    assert r["tiny_ok"] > 0               # the underflow corner is exercised and harmless
