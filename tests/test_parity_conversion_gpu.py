"""The FP4 rounding the GPU path performs is the oracle's, at every E4M3 scale.

The kernels round to E2M1 with gfx950's scaled conversion instructions (round to nearest,
ties to the even code, saturating at 6, sign of zero kept, the scale operand contributing only
its power of two, the significand divided out beforehand).  This test pins that behaviour
through the C interface, using the window entry point with the zero-width window [0, 0]: each
block then takes exactly its round-down base code c0 = I(floor_FP8(max|y| / 6)), and with a
static global scale S = 1 the normalized values equal the binary32 input.  Every code 1..126 is
forced by a block maximum of exactly 6 E4M3(c); the other elements sit on every E2M1 grid point
and every midpoint between grid points, times the scale, and at k = 1 .. 64 ulps on either side
of them, in both signs, plus +-0 and values a few ulps above the saturation point 6 s.  A block
per code with its maximum one ulp below 6 E4M3(c) checks the round-down of the base code.
Nibbles and scale bytes are compared with the oracle bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
from test_parity_gpu import DEV, describe_mismatch

pytestmark = pytest.mark.gpu

GRID = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
MIDS = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]
ULPS = [0, 1, 2, 3, 4, 5, 6, 7, 8, 12, 16, 24, 32, 48, 64]


def e4m3_values():
    b = torch.arange(127, dtype=torch.uint8)
    return b.view(torch.float8_e4m3fn).float().numpy().astype(np.float32)


def step(v, k):
    """v moved k ulps (k < 0: downwards) along the binary32 line."""
    v = np.float32(v)
    to = np.float32(np.inf if k > 0 else -np.inf)
    for _ in range(abs(k)):
        v = np.nextafter(v, to)
    return v


def conversion_tensor():
    """Rows of 16 blocks of 16 binary32 values; returns (x, the code each block must take)."""
    E = e4m3_values()
    blocks, codes = [], []
    for c in range(1, 127):
        s = E[c]
        vals = []
        for p in GRID[1:] + MIDS:
            for k in ULPS:
                for kk in ({k, -k} if k else {0}):
                    v = step(np.float32(p) * s, kk)
                    if v <= np.float32(6) * s:
                        vals += [v, -v]
        for k in range(1, 9):                   # just above 6 s: saturates, c0 stays c
            v = step(np.float32(6) * s, k)
            vals += [v, -v]
        for k in range(1, 4):                   # positive subnormals and signed zeros
            v = step(np.float32(0), k)
            vals += [v, -v]
        vals += [np.float32(0.0), np.float32(-0.0)]
        for i in range(0, len(vals), 15):
            chunk = vals[i:i + 15]
            chunk += [np.float32(0.0)] * (15 - len(chunk))
            blocks.append([np.float32(6) * s] + chunk)
            codes.append(c)
        if c >= 2:                              # maximum one ulp below 6 E4M3(c): code c - 1
            t = E[c - 1]
            below = step(np.float32(6) * s, -1)
            mids = [np.float32(m) * t for m in MIDS] + [np.float32(g) * t for g in GRID[1:]]
            blk = [below] + [-mids[j % len(mids)] if j % 2 else mids[j % len(mids)] for j in range(15)]
            blocks.append(blk)
            codes.append(c - 1)
    pad = (-len(blocks)) % 16
    blocks += [[np.float32(6) * E[1]] + [np.float32(0.0)] * 15] * pad
    codes += [1] * pad
    x = np.array(blocks, dtype=np.float32).reshape(-1, 256)
    return x, np.array(codes, dtype=np.uint8).reshape(-1, 16)


@pytest.fixture(scope="module")
def nv():
    assert torch.cuda.is_available(), "GPU parity tests need a GPU"
    import paper_2606_07618_amd as nv
    return nv


def test_fp4_rounding_at_every_scale_code(nv):
    xh, codes = conversion_tensor()
    assert xh.shape[0] > 400
    x = torch.from_numpy(xh).to(DEV)
    for weight in (None, torch.ones(256, dtype=torch.float32, device=DEV)):
        q, sc, S = nv.quantize_window(x, 16, weight, "offsets", 0, 0, 256.0, 1.0)
        torch.cuda.synchronize()
        wh = None if weight is None else weight.cpu().numpy()
        S_ref, q_ref, sc_ref = oracle.quantize_window(xh, 16, wh, "offsets", 0, 0, 256.0, 1.0)
        assert S_ref == 1.0 and float(S.item()) == 1.0
        scg, qg = sc.cpu().numpy(), q.cpu().numpy()
        assert np.array_equal(sc_ref, codes)                      # the construction
        assert np.array_equal(scg, sc_ref), describe_mismatch(scg, sc_ref, "scales")
        assert np.array_equal(qg, q_ref), describe_mismatch(qg, q_ref, "nibbles")
        # both rounding directions and every magnitude code occur at every scale
        nib = np.stack([qg & 15, qg >> 4], -1).reshape(xh.shape)
        for c in (1, 7, 8, 63, 126):
            sel = np.repeat(codes == c, 16, axis=1)
            assert set(np.unique(nib[sel] & 7)) == set(range(8)), c
            assert set(np.unique(nib[sel] >> 3)) == {0, 1}, c
