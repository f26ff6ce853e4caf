"""GPU parity of GPTQ with fixed block scales (nvfp4_ldlq) against the oracle, nibble for
nibble: both sides factor the damped, reordered Hessian and run LDLQ with the same binary64
operations in the same order.  Hessians are X^T X of seeded synthetic activations."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from test_parity_gpu import DEV, describe_mismatch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def nv():
    assert torch.cuda.is_available(), "GPU parity tests need a GPU"
    import paper_2606_07618_amd as nv
    return nv


def synthetic_hessian(n, tokens, seed, spread=0.7):
    """X^T X for X [tokens, n] with per-channel scales exp(N(0, spread^2)) and a shared
    low-rank component, in binary64 on the device."""
    g = workloads.generator(DEV, 61, seed)
    scale = torch.exp(torch.randn(n, generator=g, device=DEV, dtype=torch.float64) * spread)
    X = torch.randn((tokens, n), generator=g, device=DEV, dtype=torch.float64) * scale
    X += torch.randn((tokens, 4), generator=g, device=DEV, dtype=torch.float64) @ \
        torch.randn((4, n), generator=g, device=DEV, dtype=torch.float64)
    return (X.T @ X).contiguous()


def check(nv, w, H, method="scalesweep_wmse", block=16, damp=0.01, rows=None):
    q, sc, S = nv.gptq_quantize(w, H, method, block, damp)
    torch.cuda.synchronize()
    wh = workloads.host_array(w)
    sel = slice(None) if rows is None else rows
    q_ref = oracle.ldlq(wh[sel], H.cpu().numpy(), sc.cpu().numpy()[sel], float(S.item()), block,
                        damp)
    got = q.cpu().numpy()[sel]
    assert np.array_equal(got, q_ref), describe_mismatch(got, q_ref, "nibbles")
    return q, sc, S


@pytest.mark.parametrize("rows,cols", [(1, 64), (40, 128), (65, 192)])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_ldlq_parity_small(nv, rows, cols, dtype):
    g = workloads.generator(DEV, 62, rows, cols)
    w = workloads.llm_weight(rows, cols, g, DEV, outlier_frac=0.02).to(dtype)
    H = synthetic_hessian(cols, 3 * cols, rows)
    check(nv, w, H)


@pytest.mark.parametrize("rows,cols", [(130, 1024), (7, 1536)])
def test_ldlq_parity_many_tiles_every_row(nv, rows, cols):
    """Sixteen and twenty-four 64-column blocks: every look-ahead step of the factor and of the
    quantization (diagonal block beside the trailing update, tile beside the far columns) runs
    many times, with ragged row blocks; every row is compared."""
    g = workloads.generator(DEV, 65, rows, cols)
    w = workloads.llm_weight(rows, cols, g, DEV, outlier_frac=0.01)
    H = synthetic_hessian(cols, 2 * cols, rows, spread=0.9)
    check(nv, w, H)


def test_ldlq_workspace_contents_do_not_matter(nv):
    """The C call on a caller workspace filled with NaN, then reused for a second problem: only
    the upper triangle of the permuted Hessian is written and read as A, and whatever the
    kernels read elsewhere in the workspace feeds only discarded values, so both calls match
    the oracle."""
    import ctypes
    rows, cols, block = 40, 256, 16
    nbytes = nv.nvfp4_ldlq_workspace_bytes(rows, cols)
    ws = torch.full((nbytes // 8,), float("nan"), dtype=torch.float64, device=DEV)
    for seed in (66, 67):
        g = workloads.generator(DEV, seed)
        w = workloads.llm_weight(rows, cols, g, DEV).to(torch.bfloat16)
        H = synthetic_hessian(cols, 2 * cols, seed)
        _, sc, S = nv.quantize(w, "scalesweep_wmse", block, weight=torch.diagonal(H).float().contiguous())
        q = torch.empty((rows, cols // 2), dtype=torch.uint8, device=DEV)
        status = torch.zeros(1, dtype=torch.int32, device=DEV)
        stream = ctypes.c_void_p(torch.cuda.current_stream(DEV).cuda_stream)
        rc = nv.nvfp4_ldlq(ctypes.c_void_p(w.data_ptr()), 1, rows, cols, block,
                           ctypes.c_void_p(H.data_ptr()), ctypes.c_void_p(sc.data_ptr()),
                           ctypes.c_void_p(S.data_ptr()), ctypes.c_double(0.01),
                           ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(status.data_ptr()),
                           ctypes.c_void_p(ws.data_ptr()), nbytes, stream)
        assert rc == 0
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        q_ref = oracle.ldlq(workloads.host_array(w), H.cpu().numpy(), sc.cpu().numpy(),
                            float(S.item()), block, 0.01)
        got = q.cpu().numpy()
        assert np.array_equal(got, q_ref), describe_mismatch(got, q_ref, "nibbles")


@pytest.mark.parametrize("method,block", [("absmax", 16), ("four_over_six", 32),
                                          ("scalesweep_mse", 64), ("scalesweep_wmse", 128)])
def test_ldlq_parity_methods_and_blocks(nv, method, block):
    g = workloads.generator(DEV, 63, block)
    w = workloads.llm_weight(70, 256, g, DEV)
    H = synthetic_hessian(256, 300, block, spread=1.0)
    check(nv, w, H, method, block)


def test_ldlq_rank_deficient_hessian_is_damped(nv):
    """Fewer tokens than channels: X^T X is singular; the damping makes it definite."""
    g = workloads.generator(DEV, 64)
    w = workloads.llm_weight(16, 128, g, DEV)
    H = synthetic_hessian(128, 40, 7)
    check(nv, w, H)


def test_ldlq_diagonal_hessian_is_plain_rounding(nv):
    g = workloads.generator(DEV, 65)
    w = workloads.llm_weight(33, 128, g, DEV)
    H = torch.diag(torch.rand(128, generator=g, device=DEV, dtype=torch.float64) + 0.5)
    _, sc, S = nv.quantize(w, "scalesweep_mse", 16)
    q0, _, _ = nv.quantize(w, "scalesweep_mse", 16, static_scale=float(S.item()))
    q = nv.ldlq(w, H.contiguous(), sc, S)
    torch.cuda.synchronize()
    assert torch.equal(q, q0)


def test_ldlq_not_positive_definite_sets_status(nv):
    w = torch.ones((4, 64), dtype=torch.bfloat16, device=DEV)
    H = -torch.eye(64, dtype=torch.float64, device=DEV)
    _, sc, S = nv.quantize(w, "absmax", 16)
    with pytest.raises(nv.NVFP4Error):
        nv.ldlq(w, H, sc, S, 16, damp=0.0)


def test_ldlq_full_size_sampled(nv):
    """q_proj of the Llama-3-8B-shaped layer at full size [4096, 4096] with a Hessian from
    1024 synthetic tokens: every row on the GPU, three sampled rows through the oracle (same
    factorization), and GPTQ's purpose -- the proxy loss tr(E H E^T) below plain rounding
    with the same scales."""
    layer = workloads.llama8b_layer(DEV, with_weights=False)
    w = layer["q_proj"][0]
    H = synthetic_hessian(4096, 1024, 99)
    rows = np.array([0, 1234, 4095])
    q, sc, S = check(nv, w, H, rows=rows)
    q0, _, _ = nv.quantize(w, "scalesweep_wmse", 16,
                           weight=torch.diagonal(H).float().contiguous(),
                           static_scale=float(S.item()))
    wf = w.double()

    def proxy(qq):
        e = wf - nv.dequant(qq, sc, S, 16).double()
        return float(((e @ H) * e).sum().item())

    assert proxy(q) < proxy(q0)
