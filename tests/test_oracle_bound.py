"""The saturation bound that the GPU sweeps use to skip lower window candidates, checked on
the oracle's exact block losses.  No GPU.

For a code c below the base code c0 (the largest code with 6 E4M3(c0) <= max|y|), the scale
s = E4M3(c) satisfies 6 s < y1 = max|y|, so y1 rounds to the saturated grid value 6 s and its
term w1 (y1 - 6 s)^2 alone bounds the block loss of c from below (Eq. weighted_quantization_loss
is a sum of non-negative terms).  A candidate whose bound exceeds another candidate's loss
cannot be the argmin, so skipping it does not change the window's argmin.
"""
import numpy as np
import pytest

import oracle


def _blocks(n, count, seed):
    rng = np.random.default_rng(seed)
    out = []
    for b in range(count):
        kind = b % 4
        scale = 2.0 ** rng.uniform(-4, 4)
        if kind == 0:
            v = rng.standard_t(4, n)
        elif kind == 1:
            v = rng.uniform(0.5, 1.0, n)                    # flat-topped
        elif kind == 2:
            v = rng.uniform(0.0, 1.0, n)
            v[rng.integers(n)] = 1.3
        else:
            v = rng.standard_normal(n) * np.exp(rng.normal(0, 1, n))
        out.append(np.abs(v * scale).astype(np.float32))
    return out


@pytest.mark.parametrize("n", [16, 32, 64, 128])
@pytest.mark.parametrize("weighted", [False, True])
def test_bound_holds_below_the_base_code(n, weighted):
    rng = np.random.default_rng(100 + n)
    checked = tight = 0
    for y in _blocks(n, 160, seed=n + 7 * weighted):
        w = rng.uniform(0.0, 3.0, n).astype(np.float32) if weighted else np.ones(n, np.float32)
        res = oracle.block_sweep(y, w if weighted else None, 11, 7)
        c0, J = res["c0"], res["J"]
        i1 = int(np.argmax(y))
        y1, w1 = float(y[i1]), float(w[i1])
        for c in range(max(1, c0 - 11), c0):
            s = oracle.e4m3(c)
            assert 6.0 * s < y1
            assert oracle.round_fp4(y1, s) == 7              # the largest element saturates
            bound = w1 * (y1 - 6.0 * s) ** 2
            assert J[c] >= bound, (c, J[c], bound)
            checked += 1
            tight += J[c] <= 2.0 * bound
    assert checked > 500 and tight > 20, (checked, tight)


def test_bound_is_the_loss_of_a_lone_element():
    """One nonzero element: every lower code's loss is exactly the saturated term."""
    for c0 in (20, 47, 90, 125):
        s0 = oracle.e4m3(c0)
        y = np.zeros(16, np.float32)
        y[5] = np.float32(6.0 * s0 * 1.01)
        w = np.full(16, 0.5, np.float32)
        w[5] = 2.5
        for weighted in (False, True):
            res = oracle.block_sweep(y, w if weighted else None, 8, 7)
            assert res["c0"] == c0
            w1 = 2.5 if weighted else 1.0
            for c in range(c0 - 8, c0):
                e = float(y[5]) - 6.0 * oracle.e4m3(c)
                assert res["J"][c] == w1 * e * e


def test_skipping_bounded_candidates_keeps_the_argmin():
    """Replays the skip rule on the oracle's losses: candidates whose bound exceeds the best
    loss of offsets -1..7 are dropped, and the window argmin (smallest code on ties) is
    unchanged, for both objectives and every block size."""
    rng = np.random.default_rng(5)
    for n in (16, 32, 64, 128):
        for method in ("scalesweep_mse", "scalesweep_wmse"):
            L = oracle.window_lower(method, n)
            for y in _blocks(n, 120, seed=3 * n):
                w = rng.uniform(0.0, 3.0, n).astype(np.float32)
                wt = w if method.endswith("wmse") else None
                res = oracle.block_sweep(y, wt, L, 7)
                c0, lo, hi, J = res["c0"], res["lo"], res["hi"], res["J"]
                i1 = int(np.argmax(y))
                w1 = float(w[i1]) if wt is not None else 1.0
                upper = range(max(lo, c0 - 1), hi + 1)
                jb = min(J[c] for c in upper)
                kept = [c for c in range(lo, hi + 1)
                        if c >= c0 - 1 or not w1 * (float(y[i1]) - 6.0 * oracle.e4m3(c)) ** 2 > jb]
                best = min(kept, key=lambda c: (J[c], c))
                assert best == res["c_win"], (n, method, best, res["c_win"])


def _top_rule_blocks(count, seed):
    """Blocks whose maximum sits anywhere in its FP8 interval (so that 3.5 E4M3(c0 + 7) falls on
    either side of it), from the shapes above plus blocks near the grid of code c0 + 7."""
    rng = np.random.default_rng(seed)
    out = _blocks(16, count, seed)
    for _ in range(count // 2):
        c0 = int(rng.integers(16, 110))
        s0 = oracle.e4m3(c0)
        y = np.abs(rng.standard_normal(16)) * s0
        y[0] = 6.0 * s0 * rng.uniform(1.0, oracle.e4m3(c0 + 1) / s0)
        st = oracle.e4m3(c0 + 7)
        snap = rng.random(16) < 0.5                        # some elements on the +7 grid
        y[1:][snap[1:]] = st * np.array([0.5, 1, 1.5, 2, 3])[rng.integers(0, 5, snap[1:].sum())]
        out.append(y.astype(np.float32))
    return out


def test_upper_lemma_rules_out_offset_seven():
    """Block Scale Upper Bound lemma on the oracle's exact losses: where 3.5 E4M3(c0 + 7) > max|y|
    (and c0 + 7 >= 16, so that half of it is the E4M3 value of c0 - 1), the loss of c0 + 7 is
    never below that of c0 - 1, with either objective, so c0 + 7 is never the window argmin."""
    rng = np.random.default_rng(41)
    fired = equal = 0
    for y in _top_rule_blocks(400, seed=41):
        w = rng.uniform(0.0, 3.0, 16).astype(np.float32)
        for wt in (None, w):
            res = oracle.block_sweep(y, wt, 8, 7)
            c0, J = res["c0"], res["J"]
            ct = c0 + 7
            if ct > 126 or ct < 16:
                continue
            assert oracle.e4m3(ct - 8) * 2.0 == oracle.e4m3(ct)
            if 3.5 * oracle.e4m3(ct) > float(np.max(y)):
                fired += 1
                equal += J[ct] == J[ct - 8]
                assert J[ct] >= J[ct - 8], (c0, J[ct], J[ct - 8])
                assert res["c_win"] != ct
    assert fired > 200, fired


def test_wmse_schedule_keeps_the_argmin():
    """Replays the WMSE n = 16 schedule of the GPU sweep on the oracle's exact losses:
    offsets -1..6 scored; lower offsets kept as the contiguous top range whose saturation bound
    is not above the best scored loss; offset +7 ruled out by the lemma where 3.5 s > max|y|,
    else kept unless the largest element's term exceeds the best scored loss.  The argmin over
    the kept candidates (smallest code on ties) is the window argmin."""
    rng = np.random.default_rng(43)
    for y in _top_rule_blocks(300, seed=43):
        w = rng.uniform(0.0, 3.0, 16).astype(np.float32)
        res = oracle.block_sweep(y, w, 8, 7)
        c0, lo, hi, J = res["c0"], res["lo"], res["hi"], res["J"]
        if c0 - 8 < 8 or c0 + 7 > 126:
            continue                                      # the GPU sweeps such waves in full
        i1 = int(np.argmax(y))
        y1, w1 = float(y[i1]), float(w[i1])
        scored = list(range(c0 - 1, c0 + 7))
        jb = min(J[c] for c in scored)
        low = [c for c in range(c0 - 8, c0 - 1) if not w1 * (y1 - 6.0 * oracle.e4m3(c)) ** 2 > jb]
        assert low == list(range(c0 - 1 - len(low), c0 - 1))     # a contiguous top range
        ct = c0 + 7
        st = oracle.e4m3(ct)
        top = []
        if not 3.5 * st > y1:
            g = oracle.e2m1(oracle.round_fp4(y1, st))
            if not w1 * (y1 - g * st) ** 2 > jb:
                top = [ct]
        best = min(scored + low + top, key=lambda c: (J[c], c))
        assert best == res["c_win"], (c0, best, res["c_win"])
