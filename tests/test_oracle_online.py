"""Pins of the oracle's online-quantization pieces (static global scale per the
implementation details; importance vectors of the WMSE section; the swizzled scale layout
of the operator benchmark) to independent definitions: a torch reshape/permute of the
padded scale matrix, per-row and per-group calls of the plain quantizer, exact sums of
squares and numpy's binary64 sums.  No GPU."""
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch

import oracle
import workloads


def swizzle_by_permute(scales: np.ndarray) -> np.ndarray:
    """The 128 x 4 tiled layout as a tensor view: pad [M, K] to multiples of (128, 4), view it
    as [M/128, 4, 32, K/4, 4] (row = tile*128 + i*32 + j, column = tile*4 + l) and order the
    axes (tile_m, tile_k, j, i, l)."""
    M, K = scales.shape
    Mp, Kp = -(-M // 128) * 128, -(-K // 4) * 4
    pad = np.zeros((Mp, Kp), scales.dtype)
    pad[:M, :K] = scales
    t = torch.from_numpy(pad).reshape(Mp // 128, 4, 32, Kp // 4, 4).permute(0, 3, 2, 1, 4)
    return t.contiguous().reshape(-1).numpy()


@pytest.mark.parametrize("M,K", [(1, 1), (128, 4), (130, 5), (300, 256), (7, 512)])
def test_swizzled_offsets_match_the_permuted_view(M, K):
    ids = (np.arange(M * K, dtype=np.int64) + 1).reshape(M, K)
    flat = swizzle_by_permute(ids)
    for m in range(0, M, max(1, M // 17)):
        for k in range(0, K, max(1, K // 13)):
            assert flat[oracle.swizzled_offset(m, k, K)] == ids[m, k]
    assert oracle.scales_bytes(M, 16 * K, 16, "swizzled") == flat.size


def test_swizzled_offsets_are_a_bijection():
    M, K = 256, 8
    offs = sorted(oracle.swizzled_offset(m, k, K) for m in range(M) for k in range(K))
    assert offs == list(range(M * K))


METHODS = ["absmax", "four_over_six", "scalesweep_mse", "scalesweep_wmse"]


@pytest.mark.parametrize("method", METHODS)
def test_online_row_major_single_group_is_the_static_quantizer(method):
    g = workloads.generator("cpu", 41)
    x = workloads.bf16_bits(workloads.llm_weight(20, 256, g, "cpu"))
    w = workloads.column_importance(256, g, "cpu").numpy()
    S = 2.0e-4
    wm = w if method in ("four_over_six", "scalesweep_wmse") else None
    _, q_ref, sc_ref = oracle.quantize(method, x, 16, 256.0, S, wm)
    q, sc = oracle.quantize_online(method, x, S, 16, w)
    assert np.array_equal(q, q_ref) and np.array_equal(sc, sc_ref)


@pytest.mark.parametrize("method", ["four_over_six", "scalesweep_wmse"])
def test_online_groups_follow_the_heads(method):
    """K-like rows [batch * heads * tokens, head_dim]: row r uses the vector of head
    (r / tokens) mod heads; equal to quantizing each head's rows with its own vector."""
    B, H, T, D = 2, 3, 5, 64
    rng = np.random.default_rng(42)
    x = (rng.standard_normal((B * H * T, D)) * np.exp(rng.standard_normal(D))).astype(np.float32)
    imp = rng.uniform(0.1, 3.0, (H, D)).astype(np.float32)
    S = 0.01
    q, sc = oracle.quantize_online(method, x, S, 16, imp, H, T)
    xr = x.reshape(B, H, T, D)
    for h in range(H):
        rows = xr[:, h].reshape(-1, D)
        _, q_h, sc_h = oracle.quantize(method, rows, 16, 256.0, S, imp[h])
        idx = np.array([(b * H + h) * T + t for b in range(B) for t in range(T)])
        assert np.array_equal(q[idx], q_h) and np.array_equal(sc[idx], sc_h)


@pytest.mark.parametrize("rows,cols", [(100, 64), (128, 512), (129, 48)])
def test_swizzled_scales_are_the_row_major_scales_permuted(rows, cols):
    rng = np.random.default_rng(rows + cols)
    x = rng.standard_normal((rows, cols)).astype(np.float32)
    _, sc_rm = oracle.quantize_online("scalesweep_mse", x, 0.005, 16)
    q, sc_sw = oracle.quantize_online("scalesweep_mse", x, 0.005, 16, layout="swizzled")
    assert np.array_equal(sc_sw, swizzle_by_permute(sc_rm))


def test_online_argument_errors():
    x = np.ones((4, 32), np.float32)
    for kw, code in (({"static_scale": 0.0}, -5), ({"static_scale": -1.0}, -5),
                     ({"block": 32, "layout": "swizzled"}, -5)):
        args = dict(static_scale=1.0, block=16, layout="row_major")
        args.update(kw)
        with pytest.raises(oracle.OracleError) as e:
            oracle.quantize_online("absmax", x, args["static_scale"], args["block"],
                                   layout=args["layout"])
        assert e.value.code == code
    with pytest.raises(oracle.OracleError) as e:
        oracle.quantize_online("scalesweep_wmse", x, 1.0, 16, None)
    assert e.value.code == -1


def test_channel_norms_exact_on_integers():
    rng = np.random.default_rng(43)
    x = rng.integers(-50, 50, (37, 24)).astype(np.float32)
    out = oracle.channel_sq_norms(x)
    ref = [sum(Fr(int(v)) ** 2 for v in x[:, c]) for c in range(24)]
    assert out.shape == (1, 24)
    assert [float(v) for v in out[0]] == [float(np.float32(float(r))) for r in ref]


def _ulp_close(a, b):
    a, b = np.asarray(a, np.float32), np.asarray(b, np.float32)
    return np.all(np.abs(a.view(np.int32).astype(np.int64) - b.view(np.int32).astype(np.int64)) <= 1)


def test_channel_norms_attention_groupings():
    """The importance vectors of the WMSE section for grouped-query attention (8 query heads
    sharing 2 KV heads): Q from K, K from Q, V from W^O, against numpy binary64 sums."""
    B, Hq, Hkv, T, D, dm = 2, 8, 2, 6, 16, 40
    rep = Hq // Hkv
    rng = np.random.default_rng(44)
    K = rng.standard_normal((B, Hkv, T, D)).astype(np.float32)
    Q = rng.standard_normal((B, Hq, T, D)).astype(np.float32)
    WO = rng.standard_normal((dm, Hq * D)).astype(np.float32)
    k64, q64, wo64 = (a.astype(np.float64) for a in (K, Q, WO))
    # importance of Q: squared norms of K's channels, per KV head, repeated over its Q heads
    imp_q = oracle.channel_sq_norms(K.reshape(-1, D), T, Hkv, 1, rep)
    ref_q = np.repeat((k64 ** 2).sum(axis=(0, 2)), rep, axis=0)
    assert imp_q.shape == (Hq, D) and _ulp_close(imp_q, ref_q.astype(np.float32))
    # importance of K: squared norms of Q's channels summed over the Q heads of a KV head
    imp_k = oracle.channel_sq_norms(Q.reshape(-1, D), T, Hq, rep, 1)
    ref_k = (q64 ** 2).sum(axis=(0, 2)).reshape(Hkv, rep, D).sum(axis=1)
    assert imp_k.shape == (Hkv, D) and _ulp_close(imp_k, ref_k.astype(np.float32))
    # importance of V: squared column norms of W^O, per head, summed over a KV head's Q heads
    imp_v = oracle.channel_sq_norms(WO.reshape(-1, D), 1, Hq, rep, 1)
    ref_v = (wo64 ** 2).sum(axis=0).reshape(Hkv, rep, D).sum(axis=1)
    assert imp_v.shape == (Hkv, D) and _ulp_close(imp_v, ref_v.astype(np.float32))
    # activations: squared column norms of the consuming weight [d_out, d_in]
    imp_a = oracle.channel_sq_norms(WO)
    assert _ulp_close(imp_a[0], (wo64 ** 2).sum(axis=0).astype(np.float32))


def test_channel_norms_bf16_input_and_errors():
    g = workloads.generator("cpu", 45)
    x = workloads.llm_weight(33, 64, g, "cpu")
    out = oracle.channel_sq_norms(workloads.bf16_bits(x))
    ref = (x.float().double() ** 2).sum(0).numpy().astype(np.float32)
    assert _ulp_close(out[0], ref)
    with pytest.raises(oracle.OracleError):
        oracle.channel_sq_norms(np.ones((4, 4), np.float32), 1, 3, 2, 1)   # 3 % 2 != 0
