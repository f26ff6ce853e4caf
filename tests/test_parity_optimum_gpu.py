"""GPU parity of the reference-scale calls (nvfp4_block_optimum, nvfp4_block_loss,
nvfp4_sum_f64) against the oracle.  The optimum, its minimizer, the FP8-quantized code and
loss, and the exact block losses are compared bit for bit (both sides run the same sequence
of correctly rounded binary64 operations); the deterministic sum is compared with an exact
sum within its rounding bound.  Full-size tensors are checked on sampled blocks and through
properties that hold at any size."""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads
from test_parity_gpu import DEV, _edge_tensors

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def nv():
    assert torch.cuda.is_available(), "GPU parity tests need a GPU"
    import paper_2606_07618_amd as nv
    return nv


def oracle_blocks(xh, S, block, wh, rows=None):
    """Per-block (J_opt, s_opt, fp8 code, fp8 loss) from the oracle on y = RN32(x / S)."""
    y = oracle.normalize(xh if rows is None else xh[rows], S)
    nb = y.shape[1] // block
    out = np.zeros((y.shape[0], nb, 4))
    for r in range(y.shape[0]):
        for kb in range(nb):
            yb = y[r, kb * block:(kb + 1) * block]
            wb = None if wh is None else wh[kb * block:(kb + 1) * block]
            J, s = oracle.continuous_opt(yb, wb)
            c, l8 = oracle.fp8_quantized_opt(yb, wb)
            out[r, kb] = (J, s, c, l8)
    return out


def compare_optimum(got, ref, where=""):
    opt_loss, opt_scale, code, fp8_loss = (t.cpu().numpy() for t in got)
    for k, (g, name) in enumerate(((opt_loss, "opt_loss"), (opt_scale, "opt_scale"),
                                   (code.astype(np.float64), "fp8_code"),
                                   (fp8_loss, "fp8_loss"))):
        r = ref[..., k]
        bad = np.argwhere(~((g == r) | (np.isinf(g) & np.isinf(r))))
        assert len(bad) == 0, f"{where} {name}: {len(bad)} mismatches, first {bad[:3].tolist()}: gpu {g[tuple(bad[0])]!r} oracle {r[tuple(bad[0])]!r}"


@pytest.mark.parametrize("block", [16, 32, 64, 128])
@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_block_optimum_parity(nv, block, weighted, dtype):
    g = workloads.generator(DEV, 21, block, int(weighted))
    x = workloads.llm_weight(9, 512, g, DEV, outlier_frac=0.01).to(dtype)
    w = workloads.column_importance(512, g, DEV, tokens=64) if weighted else None
    _, _, S = nv.quantize(x, "scalesweep_mse", block)
    got = nv.block_optimum(x, S, block, w)
    torch.cuda.synchronize()
    ref = oracle_blocks(workloads.host_array(x), float(S.item()), block,
                        None if w is None else w.cpu().numpy())
    compare_optimum(got, ref, f"block {block}")


@pytest.mark.parametrize("name", list(_edge_tensors()))
def test_block_optimum_edge_tensors(nv, name):
    x = torch.from_numpy(_edge_tensors()[name]).to(DEV)
    S = torch.ones(1, device=DEV) if name == "midpoints" else nv.quantize(x, "absmax", 16)[2]
    w = torch.linspace(0.0, 2.0, x.shape[1], device=DEV)
    for weight in (None, w):
        got = nv.block_optimum(x, S, 16, weight)
        torch.cuda.synchronize()
        ref = oracle_blocks(workloads.host_array(x), float(S.item()), 16,
                            None if weight is None else weight.cpu().numpy())
        compare_optimum(got, ref, name)


@pytest.mark.parametrize("block", [16, 64])
def test_block_loss_parity(nv, block):
    g = workloads.generator(DEV, 22, block)
    x = workloads.llm_weight(33, 1024, g, DEV)
    w = workloads.column_importance(1024, g, DEV, tokens=64)
    xh, wh = workloads.host_array(x), w.cpu().numpy()
    for method, weight in (("absmax", None), ("four_over_six", None), ("scalesweep_mse", None),
                           ("scalesweep_wmse", w)):
        _, sc, S = nv.quantize(x, method, block, weight=weight)
        loss = nv.block_loss(x, S, sc, block, weight).cpu().numpy()
        y = oracle.normalize(xh, float(S.item()))
        scc = sc.cpu().numpy()
        ww = None if weight is None else wh
        for r in range(x.shape[0]):
            for kb in range(x.shape[1] // block):
                ref = oracle.block_loss(y[r, kb * block:(kb + 1) * block],
                                        None if ww is None else ww[kb * block:(kb + 1) * block],
                                        oracle.e4m3(int(scc[r, kb])))
                assert loss[r, kb] == ref, (method, r, kb)


@pytest.mark.parametrize("n", [0, 1, 255, 256 * 8 + 3, 1_000_003])
def test_sum_f64(nv, n):
    rng = np.random.default_rng(n)
    v = rng.standard_normal(n) * np.exp(rng.standard_normal(n) * 3)
    got = float(nv.sum_f64(torch.from_numpy(v).to(DEV)).item())
    exact = math.fsum(v.tolist())
    bound = n * 2.0 ** -52 * float(np.abs(v).sum()) + 1e-300
    assert abs(got - exact) <= bound
    again = float(nv.sum_f64(torch.from_numpy(v).to(DEV)).item())
    assert got == again                                   # fixed order


def test_block_optimum_full_size(nv):
    """q_proj of the Llama-3-8B layer at full size [4096, 4096]: sampled rows bit for bit, and
    at every block the optimum bounds the FP8 choices from below while the FP8-quantized
    optimum is never below the exhaustive FP8 sweep."""
    layer = workloads.llama8b_layer(DEV)
    x, w = layer["q_proj"]
    for weight in (None, w):
        _, sc_full, S = nv.quantize_window(x, 16, weight, "offsets", -126, 126)
        got = nv.block_optimum(x, S, 16, weight)
        full = nv.block_loss(x, S, sc_full, 16, weight)
        torch.cuda.synchronize()
        rows = np.sort(np.random.default_rng(4).choice(x.shape[0], 3, replace=False))
        ref = oracle_blocks(workloads.host_array(x), float(S.item()), 16,
                            None if weight is None else weight.cpu().numpy(), rows)
        compare_optimum([t[rows] for t in got], ref, "q_proj sampled")
        opt_loss, _, _, fp8_loss = got
        slack = 1e-12 * full + 1e-300
        assert bool((opt_loss <= full + slack).all())
        assert bool((full <= fp8_loss).all())


def test_gap_report_ordering(nv):
    """Figure 1's ordering on the 8192^2 workload's first 1024 rows: the exhaustive FP8 sweep
    is at least as good as every rule on its global scale, and ScaleSweep beats AbsMax and
    4/6."""
    x, w = workloads.square8192(DEV)
    x = x[:1024].contiguous()
    for weight in (None, w):
        rep = nv.gap_report(x, 16, weight)
        assert rep["exhaustive_fp8_sweep"] >= 0.0
        # rules on the same global scale (D = 256) as the exhaustive sweep
        for m in ("fp8_quantized_optimum", "four_over_six", "scalesweep_mse"):
            assert rep[m] >= rep["exhaustive_fp8_sweep"] - 1e-12, (m, rep)
        ss = rep["scalesweep_wmse"] if weight is not None else rep["scalesweep_mse"]
        assert ss < rep["absmax"] and ss < rep["four_over_six"]
