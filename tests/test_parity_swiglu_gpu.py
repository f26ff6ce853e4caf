"""GPU parity of the fused producer + online quantizer (nvfp4_quant_online_swiglu) and of the
producer alone (nvfp4_swiglu) against the oracle, bit for bit: the oracle forms the SwiGLU
product from the same bfloat16 gate and up with its own implementation of the fixed binary32
arithmetic, then quantizes it as nvfp4_quant_online does."""
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


def mlp_inputs(rows, cols, seed, extremes=False):
    """gate ~ 3 N(0, 1) (pre-activations spread over silu's curved part), up ~ N(0, 1), with a
    few outlier channels; with extremes, values at and past the exp cut-offs, signed zeros and
    large magnitudes."""
    g = workloads.generator(DEV, 81, seed)
    gate = torch.randn((rows, cols), generator=g, device=DEV) * 3.0
    up = torch.randn((rows, cols), generator=g, device=DEV)
    ch = torch.randperm(cols, generator=g, device=DEV)[:4]
    up[:, ch] *= 20.0
    if extremes:
        special = torch.tensor([0.0, -0.0, 79.9, 80.0, 80.1, -88.9, -89.0, -89.5, -200.0, 200.0,
                                1e4, -1e4, 3e-30, -3e-30, 0.5, -0.5], device=DEV)
        gate[0, :special.numel()] = special
        gate[1, :special.numel()] = -special
        up[2, :special.numel()] = special
    return gate.to(torch.bfloat16).contiguous(), up.to(torch.bfloat16).contiguous()


def test_swiglu_every_bfloat16_gate(nv):
    """Every finite bfloat16 gate pattern (65,280 of them, padded to [4096, 16]), once with up = 1
    and once with up drawn from N(0, 1) with outliers: the producer's tabulated silu and its
    closed forms outside the table (|g| < 2^-40 and |g| >= 128) against the oracle, bit for bit."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    finite = np.isfinite(oracle.bf16_to_f32(bits))
    gb = bits[finite]
    gb = np.concatenate([gb, np.zeros(4096 * 16 - gb.size, np.uint16)]).reshape(4096, 16)
    gate = torch.from_numpy(gb.view(np.int16)).to(DEV).view(torch.bfloat16)
    g = workloads.generator(DEV, 81, 7)
    for up in (torch.ones((4096, 16), device=DEV),
               torch.randn((4096, 16), generator=g, device=DEV) * 3.0):
        up = up.to(torch.bfloat16).contiguous()
        h = nv.swiglu(gate, up)
        torch.cuda.synchronize()
        want = oracle.swiglu(workloads.bf16_bits(gate), workloads.bf16_bits(up))
        got = workloads.bf16_bits(h)
        assert np.array_equal(got, want), describe_mismatch(got, want, "h")


@pytest.mark.parametrize("shape", [(67, 512), (3, 1024), (130, 64)])
def test_swiglu_producer_matches_oracle(nv, shape):
    gate, up = mlp_inputs(*shape, seed=shape[0], extremes=True)
    h = nv.swiglu(gate, up)
    torch.cuda.synchronize()
    want = oracle.swiglu(workloads.bf16_bits(gate), workloads.bf16_bits(up))
    got = workloads.bf16_bits(h)
    assert np.array_equal(got, want), describe_mismatch(got, want, "h")


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("layout", ["row_major", "swizzled"])
def test_fused_quantizer_matches_oracle(nv, method, layout):
    gate, up = mlp_inputs(67, 512, seed=7, extremes=True)
    g = workloads.generator(DEV, 82)
    imp = workloads.column_importance(512, g, DEV, tokens=128)[None].contiguous()
    wt = imp if method in ("scalesweep_wmse", "four_over_six") else None
    S = 0.0123
    q, sc = nv.quantize_online_swiglu(gate, up, method, S, wt, layout=layout)
    torch.cuda.synchronize()
    h = oracle.swiglu(workloads.bf16_bits(gate), workloads.bf16_bits(up))
    q_ref, sc_ref = oracle.quantize_online(method, h, S, 16, None if wt is None else wt.cpu().numpy(),
                                           layout=layout)
    qg, scg = q.cpu().numpy(), sc.cpu().numpy()
    assert np.array_equal(scg, sc_ref), describe_mismatch(scg, sc_ref, "scales")
    assert np.array_equal(qg, q_ref), describe_mismatch(qg, q_ref, "nibbles")


@pytest.mark.parametrize("method", METHODS)
def test_fused_equals_producer_then_quantizer(nv, method):
    """The fusion changes nothing: the fused call equals nvfp4_swiglu then nvfp4_quant_online,
    with per-head importance groups as for attention tensors."""
    gate, up = mlp_inputs(256, 384, seed=9)
    g = workloads.generator(DEV, 83)
    imp = torch.stack([workloads.column_importance(384, g, DEV, tokens=64) for _ in range(4)]).contiguous()
    wt = imp if method in ("scalesweep_wmse", "four_over_six") else None
    for layout in ("row_major", "swizzled"):
        q1, s1 = nv.quantize_online_swiglu(gate, up, method, 0.02, wt, 4, 16, layout=layout)
        h = nv.swiglu(gate, up)
        q2, s2 = nv.quantize_online(h, method, 0.02, 16, wt, 4, 16, layout=layout)
        torch.cuda.synchronize()
        assert torch.equal(q1, q2) and torch.equal(s1, s2), (method, layout)


def test_fused_full_size_sampled(nv):
    """The MLP activation of 8192 tokens of a Llama-3-8B-shaped layer, [8192, 14336], in the
    launch configuration the benchmark times (swizzled scales, static S); sampled rows against
    the oracle, all rows against the unfused GPU path."""
    gate, up = mlp_inputs(8192, 14336, seed=11)
    rows = np.sort(np.random.default_rng(5).choice(8192, 24, replace=False))
    for method in ("absmax", "scalesweep_mse"):
        q, sc = nv.quantize_online_swiglu(gate, up, method, 0.004, layout="row_major")
        torch.cuda.synchronize()
        gh, uh = workloads.bf16_bits(gate[rows]), workloads.bf16_bits(up[rows])
        q_ref, sc_ref = oracle.quantize_online(method, oracle.swiglu(gh, uh), 0.004, 16)
        assert np.array_equal(sc[rows].cpu().numpy(), sc_ref)
        assert np.array_equal(q[rows].cpu().numpy(), q_ref)
        q1, s1 = nv.quantize_online_swiglu(gate, up, method, 0.004, layout="swizzled")
        q2, s2 = nv.quantize_online(nv.swiglu(gate, up), method, 0.004, 16, layout="swizzled")
        torch.cuda.synchronize()
        assert torch.equal(q1, q2) and torch.equal(s1, s2), method
