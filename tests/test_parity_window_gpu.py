"""GPU parity of the window variants (nvfp4_quant_scalesweep_window) against the oracle, bit
for bit: per-mantissa windows (Tables 1 and 2), explicit [l, r] offsets including windows
that leave the code range and the exhaustive sweep, both objectives, every block size."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from test_parity_gpu import DEV, _edge_tensors, describe_mismatch

pytestmark = pytest.mark.gpu

WINDOWS = [("tight", 0, 0), ("offsets", -3, 7), ("offsets", -8, 7), ("offsets", 0, 0),
           ("offsets", 2, 5), ("offsets", -16, 16), ("offsets", -20, -12), ("offsets", 5, 30),
           ("offsets", -126, 126)]


@pytest.fixture(scope="module")
def nv():
    assert torch.cuda.is_available(), "GPU parity tests need a GPU"
    import paper_2606_07618_amd as nv
    return nv


def check_window(nv, x, block, w, mode, lo, hi, static=0.0, D=256.0, rows_sample=None):
    q, sc, S = nv.quantize_window(x, block, w, mode, lo, hi, D, static)
    torch.cuda.synchronize()
    xh = workloads.host_array(x)
    wh = None if w is None else w.cpu().numpy()
    if rows_sample is None:
        S_ref, q_ref, sc_ref = oracle.quantize_window(xh, block, wh, mode, lo, hi, D, static)
        qg, scg = q.cpu().numpy(), sc.cpu().numpy()
    else:
        S_ref = static if static else oracle.tensor_scale(xh, D)
        _, q_ref, sc_ref = oracle.quantize_window(xh[rows_sample], block, wh, mode, lo, hi, D,
                                                  S_ref)
        qg, scg = q[rows_sample].cpu().numpy(), sc[rows_sample].cpu().numpy()
    S_gpu = S.cpu().numpy()[0]
    assert np.float32(S_gpu).view(np.uint32) == np.float32(S_ref).view(np.uint32), (S_gpu, S_ref)
    assert np.array_equal(scg, sc_ref), describe_mismatch(scg, sc_ref, "scales")
    assert np.array_equal(qg, q_ref), describe_mismatch(qg, q_ref, "nibbles")
    return q, sc, S


@pytest.mark.parametrize("window", WINDOWS, ids=[f"{m}{lo}_{hi}" for m, lo, hi in WINDOWS])
@pytest.mark.parametrize("objective", ["mse", "wmse"])
@pytest.mark.parametrize("block", [16, 32, 64, 128])
def test_window_parity(nv, window, objective, block):
    mode, lo, hi = window
    g = workloads.generator(DEV, 11, block, hi - lo)
    x = workloads.llm_weight(67, 4 * 128, g, DEV, outlier_frac=0.01)
    w = workloads.column_importance(512, g, DEV, tokens=128) if objective == "wmse" else None
    check_window(nv, x, block, w, mode, lo, hi)


@pytest.mark.parametrize("window", [("tight", 0, 0), ("offsets", -5, 9)])
@pytest.mark.parametrize("static", [0.0, 2.5e-4])
def test_window_parity_f32_and_static(nv, window, static):
    g = workloads.generator(DEV, 12, int(static > 0))
    x = workloads.llm_weight(45, 256, g, DEV).float()
    w = workloads.column_importance(256, g, DEV, tokens=64)
    for weight in (None, w):
        check_window(nv, x, 16, weight, *window, static=static)


@pytest.mark.parametrize("name", list(_edge_tensors()))
@pytest.mark.parametrize("window", [("tight", 0, 0), ("offsets", -126, 126), ("offsets", -12, 3)])
def test_window_edge_tensors(nv, name, window):
    x = torch.from_numpy(_edge_tensors()[name]).to(DEV)
    static = 1.0 if name == "midpoints" else 0.0
    w = torch.linspace(0.0, 2.0, x.shape[1], device=DEV)
    for weight in (None, w):
        check_window(nv, x, 16, weight, *window, static=static)


def test_standard_offsets_equal_the_standard_calls(nv):
    """[-3, 7] and [-8, 7] reproduce the ScaleSweep entry points exactly (n = 16)."""
    g = workloads.generator(DEV, 13)
    x = workloads.llm_weight(300, 1024, g, DEV)
    w = workloads.column_importance(1024, g, DEV, tokens=128)
    for weight, lo, method in ((None, -3, "scalesweep_mse"), (w, -8, "scalesweep_wmse")):
        a = nv.quantize_window(x, 16, weight, "offsets", lo, 7)
        b = nv.quantize(x, method, 16, weight=weight)
        torch.cuda.synchronize()
        for u, v in zip(a, b):
            assert torch.equal(u, v)


def test_tight_window_equals_standard_on_c0(nv):
    """Tables 1 and 2 prune only codes the lemmas exclude: same codes as [-3, 7] on C0."""
    x = torch.from_numpy(workloads.c0_matrix()).to(DEV)
    a = nv.quantize_window(x, 16, None, "tight", 0, 0, 448.0)
    b = nv.quantize(x, "scalesweep_mse", 16, fp8_range=448.0)
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)
    check_window(nv, x, 16, None, "tight", 0, 0, D=448.0)


@pytest.mark.parametrize("window", [("tight", 0, 0), ("offsets", -126, 126)])
def test_window_full_size_sampled(nv, window):
    """The largest Llama-3-8B weight (gate_proj [14336, 4096]) at full size; the oracle checks
    sampled rows with the whole tensor's global scale."""
    layer = workloads.llama8b_layer(DEV)
    x, w = layer["gate_proj"]
    rows = np.sort(np.random.default_rng(9).choice(x.shape[0], 6, replace=False))
    for weight in (None, w):
        check_window(nv, x, 16, weight, *window, rows_sample=rows)
