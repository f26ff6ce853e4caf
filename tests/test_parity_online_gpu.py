"""GPU parity of the online path (nvfp4_quant_online, nvfp4_channel_sq_norms) against the
oracle: codes and scale bytes bit for bit in both scale layouts (padding included), the
per-head importance vectors of K, V and Q, and the importance vectors themselves within one
binary32 ulp (both sides sum squares in binary64, in different orders, and round once)."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from test_parity_gpu import DEV, describe_mismatch

pytestmark = pytest.mark.gpu

METHODS = ["absmax", "four_over_six", "scalesweep_mse", "scalesweep_wmse"]


@pytest.fixture(scope="module")
def nv():
    assert torch.cuda.is_available(), "GPU parity tests need a GPU"
    import paper_2606_07618_amd as nv
    return nv


def run_online(nv, x, method, S, imp=None, groups=1, grows=1, layout="row_major", rows=None):
    rows_all, cols = x.shape
    nbytes = nv.nvfp4_scales_bytes(rows_all, cols, 16, nv.nvfp4.SCALE_LAYOUTS[layout])
    q = torch.empty((rows_all, cols // 2), dtype=torch.uint8, device=DEV)
    sc = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device=DEV)   # padding must be written
    nv.quantize_online(x, method, S, 16, imp, groups, grows, layout, out=(q, sc))
    torch.cuda.synchronize()
    xh = workloads.host_array(x)
    ih = None if imp is None else imp.cpu().numpy()
    if rows is None:
        q_ref, sc_ref = oracle.quantize_online(method, xh, S, 16, ih, groups, grows, layout)
        assert np.array_equal(q.cpu().numpy(), q_ref), describe_mismatch(q.cpu().numpy(), q_ref, "nibbles")
        got = sc.cpu().numpy()
        ref = sc_ref.reshape(-1)
        assert np.array_equal(got, ref), describe_mismatch(got[None], ref[None], "scales")
    else:
        # sampled rows: row r of the oracle's call keeps its own importance group
        for r in rows:
            g = (r // grows) % groups
            q_ref, sc_ref = oracle.quantize_online(method, xh[r:r + 1], S, 16,
                                                   None if ih is None else ih[g:g + 1])
            assert np.array_equal(q[r].cpu().numpy(), q_ref[0]), (method, r)
            k16 = cols // 16
            if layout == "row_major":
                got = sc.view(rows_all, k16)[r].cpu().numpy()
            else:
                offs = [oracle.swizzled_offset(int(r), k, k16) for k in range(k16)]
                got = sc.cpu().numpy()[offs]
            assert np.array_equal(got, sc_ref.reshape(-1)), (method, r)
    return q, sc


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("layout", ["row_major", "swizzled"])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_online_parity(nv, method, layout, dtype):
    g = workloads.generator(DEV, 31, METHODS.index(method))
    x = workloads.llm_weight(200, 80, g, DEV, scale=1.0, outlier_frac=0.05).to(dtype)   # k16 = 5
    imp = workloads.column_importance(80, g, DEV, tokens=64)[None].contiguous()
    run_online(nv, x, method, 0.004, imp, layout=layout)


@pytest.mark.parametrize("method", ["four_over_six", "scalesweep_wmse"])
def test_online_per_head_importance(nv, method):
    B, H, T, D = 2, 4, 37, 128
    g = workloads.generator(DEV, 32)
    x = (torch.randn((B, H, T, D), generator=g, device=DEV) *
         torch.exp(torch.randn((H, 1, D), generator=g, device=DEV))).to(torch.bfloat16)
    imp = torch.rand((H, D), generator=g, device=DEV) * 3
    run_online(nv, x.reshape(-1, D), method, 0.003, imp, H, T, "swizzled")


def test_online_row_major_matches_static_quantizer(nv):
    """One group, row-major scales: the static-scale single-tensor call's outputs."""
    g = workloads.generator(DEV, 33)
    x = workloads.llm_weight(300, 1024, g, DEV)
    w = workloads.column_importance(1024, g, DEV, tokens=64)
    for method in METHODS:
        wm = w if method in ("four_over_six", "scalesweep_wmse") else None
        q, sc, _ = nv.quantize(x, method, 16, weight=wm, static_scale=2e-4)
        q2, sc2 = nv.quantize_online(x, method, 2e-4, 16, w[None].contiguous())
        torch.cuda.synchronize()
        assert torch.equal(q, q2) and torch.equal(sc, sc2), method


def _ulp_diff(a, b):
    a = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    b = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return int(np.abs(a - b).max()) if a.size else 0


def test_channel_norms_parity(nv):
    B, Hq, Hkv, T, D, dm = 2, 8, 2, 300, 128, 256
    rep = Hq // Hkv
    g = workloads.generator(DEV, 34)
    K = torch.randn((B, Hkv, T, D), generator=g, device=DEV).to(torch.bfloat16)
    Q = torch.randn((B, Hq, T, D), generator=g, device=DEV)
    WO = workloads.llm_weight(dm, Hq * D, g, DEV)
    cases = [(K.reshape(-1, D), (T, Hkv, 1, rep)), (Q.reshape(-1, D), (T, Hq, rep, 1)),
             (WO.reshape(-1, D), (1, Hq, rep, 1)), (WO, (1, 1, 1, 1)), (Q.reshape(-1, D)[:0], (T, Hq, rep, 1))]
    for x, args in cases:
        got = nv.channel_sq_norms(x, *args)
        torch.cuda.synchronize()
        ref = oracle.channel_sq_norms(workloads.host_array(x), *args)
        assert got.shape == ref.shape
        assert _ulp_diff(got.cpu().numpy(), ref) <= 1, args


def test_online_full_size_attention_and_activations(nv):
    """The online workloads at full size (activations [8192, 4096]; K, V [16, 8, 4096, 128];
    Q [16, 32, 4096, 128]) with their importance vectors computed on the GPU (Q from K, K from
    Q, V from a synthetic W^O, activations from a synthetic weight), WMSE, swizzled scales;
    sampled rows against the oracle."""
    t = workloads.online_tensors(DEV)
    B, Hkv, T, D = t["k"].shape
    Hq = t["q"].shape[1]
    rep = Hq // Hkv
    g = workloads.generator(DEV, 35)
    WO = workloads.llm_weight(4096, Hq * D, g, DEV)
    W = workloads.llm_weight(4096, 4096, g, DEV)
    k2, q2, v2 = (t[n].reshape(-1, D) for n in ("k", "q", "v"))
    imp = {"q": nv.channel_sq_norms(k2, T, Hkv, 1, rep),
           "k": nv.channel_sq_norms(q2, T, Hq, rep, 1),
           "v": nv.channel_sq_norms(WO.reshape(-1, D), 1, Hq, rep, 1),
           "act": nv.channel_sq_norms(W)}
    rng = np.random.default_rng(5)
    for name, x, groups in (("act", t["act"], 1), ("k", k2, Hkv), ("v", v2, Hkv), ("q", q2, Hq)):
        S = float(x.float().abs().max().item()) / (6 * 256)
        rows = rng.choice(x.shape[0], 4, replace=False)
        run_online(nv, x, "scalesweep_wmse", S, imp[name], groups, T if name != "act" else 1,
                   "swizzled", rows=rows)
        run_online(nv, x, "scalesweep_mse", S, None, 1, 1, "swizzled", rows=rows)


def test_online_importance_offsets_past_2_32(nv):
    """Per-row importance vectors (imp_groups = rows) over more than 2^32 weights: the kernels
    address a block's weights in units of the block size, so rows whose weights start past
    2^32 elements read their own vectors.  [133120, 32768] bf16 (4.36 G elements, 8.7 GB) with a
    [133120, 32768] binary32 importance array (17.4 GB), WMSE with static S, row-major scales;
    sampled rows on both sides of the 2^32 mark against the oracle."""
    rows, cols = (1 << 17) + 2048, 1 << 15
    g = workloads.generator(DEV, 91, 1)
    x = torch.randn((rows, cols), generator=g, device=DEV, dtype=torch.bfloat16)
    imp = torch.rand((rows, cols), generator=g, device=DEV, dtype=torch.float32) + 0.1
    q, sc = nv.quantize_online(x, "scalesweep_wmse", 0.004, 16, imp, rows, 1)
    torch.cuda.synchronize()
    edge = (1 << 32) // cols                                       # first row past 2^32
    for r in (0, 12345, edge - 1, edge, edge + 1, rows - 1):
        xr = workloads.host_array(x[r:r + 1])
        ir = imp[r:r + 1].cpu().numpy()
        q_ref, sc_ref = oracle.quantize_online("scalesweep_wmse", xr, 0.004, 16, ir)
        assert np.array_equal(q[r].cpu().numpy(), q_ref[0]), r
        assert np.array_equal(sc[r].cpu().numpy(), sc_ref.reshape(-1)), r
    del x, imp, q, sc
    torch.cuda.empty_cache()
