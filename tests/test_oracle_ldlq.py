"""Pins of the oracle's GPTQ pass (implementation details, GPTQ paragraph: LDLQ, damping 0.01 x
mean Hessian diagonal, static reordering by descending diagonal, block scales fixed before the
pass) to independent routes: numpy's stable sort, numpy's Cholesky factorization, and the
column-update form of GPTQ written here with numpy's inverse and Cholesky.  No GPU."""
import numpy as np
import pytest

import oracle
import workloads


def hessian(n, rng, tokens=None, spread=1.0):
    X = rng.standard_normal((tokens or 4 * n, n)) * np.exp(spread * rng.standard_normal(n))
    return X.T @ X


def test_order_is_a_stable_descending_sort():
    rng = np.random.default_rng(1)
    H = hessian(40, rng)
    d = np.diag(H).copy()
    d[[3, 9, 17]] = d[5]                                   # ties keep index order
    np.fill_diagonal(H, d)
    assert np.array_equal(oracle.ldlq_order(H), np.argsort(-d, kind="stable"))


@pytest.mark.parametrize("n", [1, 7, 64])
def test_factor_matches_reversed_cholesky(n):
    """(U + I) D (U + I)^T of the damped, reordered Hessian equals the Cholesky factorization of
    the index-reversed matrix, read backwards (numpy)."""
    rng = np.random.default_rng(n)
    H = hessian(n, rng)
    U, D = oracle.ldlq_factor(H, 0.01)
    perm = oracle.ldlq_order(H)
    Hp = H[np.ix_(perm, perm)] + 0.01 * np.trace(H) / n * np.eye(n)
    J = np.eye(n)[::-1]
    C = np.linalg.cholesky(J @ Hp @ J)
    L = C / np.diag(C)
    U_ref = J @ L @ J - np.eye(n)
    D_ref = (np.diag(C) ** 2)[::-1]
    assert np.allclose(U, U_ref, rtol=1e-10, atol=1e-12)
    assert np.allclose(D, D_ref, rtol=1e-10)
    assert np.all(np.tril(U) == 0)


def gptq_columns(w, H, scales, S, block, damp=0.01):
    """GPTQ in its column-update form: U = upper Cholesky factor of the inverse damped,
    reordered Hessian; quantize column j, then subtract its scaled error from the later
    columns.  Returns nibbles [rows, n/2] like the quantizers."""
    rows, n = w.shape
    perm = np.argsort(-np.diag(H), kind="stable")
    Hp = H[np.ix_(perm, perm)] + damp * np.trace(H) / n * np.eye(n)
    Uc = np.linalg.cholesky(np.linalg.inv(Hp)).T
    W = w.astype(np.float64)[:, perm].copy()
    nib = np.zeros((rows, n), np.uint8)
    for j in range(n):
        c = perm[j]
        for r in range(rows):
            y = np.float32(np.float32(W[r, j]) / np.float32(S))
            s = oracle.e4m3(int(scales[r, c // block]))
            k = oracle.round_fp4(abs(float(y)), s)
            wq = oracle.e2m1(k) * s * float(np.float32(S)) * (-1 if np.signbit(y) else 1)
            nib[r, c] = (8 if np.signbit(y) else 0) | k
            err = (W[r, j] - wq) / Uc[j, j]
            W[r, j + 1:] -= err * Uc[j, j + 1:]
    return (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)


@pytest.mark.parametrize("n,rows", [(32, 12), (64, 8)])
def test_ldlq_equals_gptq(n, rows):
    rng = np.random.default_rng(100 + n)
    H = hessian(n, rng, spread=0.7)
    w = (rng.standard_normal((rows, n)) * 0.05).astype(np.float32)
    S, _, sc = oracle.quantize("scalesweep_wmse", w, 16, 256.0, 0.0, np.diag(H).astype(np.float32))
    q = oracle.ldlq(w, H, sc, S)
    q_ref = gptq_columns(w, H, sc, S, 16)
    # the two orders of operations differ, so a value on a rounding boundary could in principle
    # go either way; on these seeded problems every nibble agrees
    assert np.array_equal(q, q_ref)
    # and the proxy loss tr(E H E^T) agrees
    deq = lambda qq: oracle.dequant(qq, sc, S, 16).astype(np.float64)
    loss = lambda qq: np.einsum("ri,ij,rj->", w - deq(qq), H, w - deq(qq))
    assert loss(q) == pytest.approx(loss(q_ref), rel=1e-3)


def test_diagonal_hessian_is_plain_rounding():
    """With a diagonal Hessian U = 0: each value is rounded on its own with the fixed scale,
    i.e. the quantizer's own nibbles for the same scales."""
    rng = np.random.default_rng(7)
    n = 48
    H = np.diag(rng.uniform(0.5, 4.0, n))
    w = (rng.standard_normal((10, n)) * 0.1).astype(np.float32)
    S, q0, sc = oracle.quantize("scalesweep_mse", w, 16, 256.0)
    assert np.array_equal(oracle.ldlq(w, H, sc, S), q0)


def test_ldlq_lowers_the_proxy_loss():
    """GPTQ's purpose: tr(E H E^T) below plain rounding with the same scales."""
    rng = np.random.default_rng(8)
    n = 64
    H = hessian(n, rng, tokens=80, spread=0.5)
    g = workloads.generator("cpu", 51)
    w = workloads.bf16_bits(workloads.llm_weight(16, n, g, "cpu"))
    S, q0, sc = oracle.quantize("scalesweep_wmse", w, 16, 256.0, 0.0, np.diag(H).astype(np.float32))
    q = oracle.ldlq(w, H, sc, S)
    wf = oracle.bf16_to_f32(w).astype(np.float64)
    loss = lambda qq: np.einsum("ri,ij,rj->", wf - oracle.dequant(qq, sc, S), H,
                                wf - oracle.dequant(qq, sc, S))
    assert loss(q) < 0.9 * loss(q0)


def test_not_positive_definite_is_an_error():
    H = -np.eye(16)
    w = np.ones((2, 16), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.ldlq(w, H, np.full((2, 1), 56, np.uint8), 1.0, 16, 0.0)
