"""nvfp4_quant_batched_noalloc (the entry point for callers that cannot allocate: its scratch is
the library's fixed device array) against nvfp4_quant_batched with a caller workspace, bit for
bit, through the C interface: two calls in a row, the second on smaller inputs, every method."""
import ctypes

import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def nv():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_07618_amd as nv
    return nv


def descriptors(nv, xs, ws_col, outs):
    arr = (nv.nvfp4.NVFP4Tensor * len(xs))()
    for k, (x, w, (q, sc, S)) in enumerate(zip(xs, ws_col, outs)):
        arr[k] = nv.nvfp4.NVFP4Tensor(x.data_ptr(), x.shape[0], x.shape[1],
                                      None if w is None else w.data_ptr(), S.data_ptr(),
                                      q.data_ptr(), sc.data_ptr())
    return arr


def empty_outs(xs, block):
    return [(torch.full((x.shape[0], x.shape[1] // 2), 0xAB, dtype=torch.uint8, device=DEV),
             torch.full((x.shape[0], x.shape[1] // block), 0xCD, dtype=torch.uint8, device=DEV),
             torch.full((1,), -1.0, dtype=torch.float32, device=DEV)) for x in xs]


def run_both(nv, xs, ws_col, method, block, D):
    stream = ctypes.c_void_p(torch.cuda.current_stream(DEV).cuda_stream)
    mid = nv.METHOD_IDS[method]
    dt = 1 if xs[0].dtype == torch.bfloat16 else 0
    ref = empty_outs(xs, block)
    arr = descriptors(nv, xs, ws_col, ref)
    nbytes = nv.nvfp4_batched_workspace_bytes(len(xs))
    ws = torch.empty(nbytes // 4, dtype=torch.int32, device=DEV)
    assert nv.nvfp4_quant_batched(mid, ctypes.cast(arr, ctypes.c_void_p), len(xs), dt, block,
                                  ctypes.c_float(D), ctypes.c_void_p(ws.data_ptr()), nbytes,
                                  stream) == 0
    got = empty_outs(xs, block)
    arr2 = descriptors(nv, xs, ws_col, got)
    assert nv.nvfp4_quant_batched_noalloc(mid, ctypes.cast(arr2, ctypes.c_void_p), len(xs), dt,
                                          block, ctypes.c_float(D), stream) == 0
    torch.cuda.synchronize()
    for (q0, s0, S0), (q1, s1, S1) in zip(ref, got):
        assert torch.equal(S0.view(torch.int32), S1.view(torch.int32))
        assert torch.equal(s0, s1)
        assert torch.equal(q0, q1)


@pytest.mark.parametrize("method", ["absmax", "four_over_six", "scalesweep_mse", "scalesweep_wmse"])
def test_noalloc_matches_batched_two_calls(nv, method):
    D = 448.0 if method == "absmax" else 256.0
    g = workloads.generator(DEV, 71, nv.METHOD_IDS[method])
    shapes1 = [(512, 1024), (128, 1024), (128, 1024), (512, 1024), (1792, 1024), (1792, 1024),
               (1024, 1792)]
    xs = [workloads.llm_weight(r, c, g, DEV) for r, c in shapes1]
    wt = method in ("scalesweep_wmse", "four_over_six")
    ws_col = [workloads.column_importance(c, g, DEV, tokens=128) if wt else None for _, c in shapes1]
    run_both(nv, xs, ws_col, method, 16, D)
    # second call: fewer, smaller tensors (the scratch keeps the first call's contents)
    shapes2 = [(40, 256), (8, 256), (96, 512)]
    xs2 = [workloads.llm_weight(r, c, g, DEV) for r, c in shapes2]
    ws2 = [workloads.column_importance(c, g, DEV, tokens=64) if wt else None for _, c in shapes2]
    run_both(nv, xs2, ws2, method, 16, D)


def test_noalloc_other_block_size_and_binary32(nv):
    g = workloads.generator(DEV, 72)
    xs = [torch.randn((r, 512), generator=g, device=DEV) for r in (33, 7, 64)]
    run_both(nv, xs, [None] * 3, "scalesweep_mse", 64, 256.0)
    run_both(nv, xs[:2], [None] * 2, "scalesweep_mse", 32, 256.0)


def test_noalloc_rejects_more_tensors_than_its_scratch(nv):
    T = nv.nvfp4.NVFP4Tensor
    n = nv.NOALLOC_MAX_TENSORS + 1
    arr = (T * n)()
    stream = ctypes.c_void_p(torch.cuda.current_stream(DEV).cuda_stream)
    # rejected before any descriptor is read or anything launched
    assert nv.nvfp4_quant_batched_noalloc(2, ctypes.cast(arr, ctypes.c_void_p), n, 1, 16,
                                          ctypes.c_float(256.0), stream) == -10
    assert nv.nvfp4_quant_batched_noalloc(2, None, 0, 1, 16, ctypes.c_float(256.0), stream) == 0
    assert nv.nvfp4_quant_batched_noalloc(2, None, 3, 1, 16, ctypes.c_float(256.0), stream) == -1
