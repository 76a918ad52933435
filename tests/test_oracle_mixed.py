"""Pins of the mixed-precision (FP8) layer oracle against facts that do not
depend on it: exact agreement with the full-precision layer when every
quantised tensor is exactly representable, elementwise bounds from the E4M3
rounding bound, and the mask-gradient homogeneity identity."""
import numpy as np
import pytest

from oracle import fp8, mixed
from oracle import ttm as OT
from paper_2405_14377_amd import workloads as wl


def _exact_layer(rng, n, m, r, masks_p=None):
    """Integer cores whose dense weight is exact and FP8-representable (see
    workloads.integer_bond_diagonal_cores), optional 0/1 masks."""
    d = len(n)
    cores = [G.astype(np.float64) for G in wl.integer_bond_diagonal_cores(rng, n, m, r)]
    masks = None
    if masks_p is not None:
        masks = [(rng.random(r[k + 1]) < masks_p).astype(np.float64) for k in range(d - 1)]
    return cores, masks


@pytest.mark.parametrize("case", [((4, 6, 5), (3, 7, 4), (1, 6, 6, 1), 40, None),
                                  ((3, 4, 2, 5), (2, 5, 3, 4), (1, 8, 8, 8, 1), 33, 0.7),
                                  ((16, 8), (8, 16), (1, 16, 1), 20, None)])
def test_exact_when_representable(case):
    n, m, r, b, mp = case
    rng = np.random.default_rng(7)
    cores, masks = _exact_layer(rng, n, m, r, mp)
    N_in, N_out = int(np.prod(n)), int(np.prod(m))
    X = rng.integers(-8, 9, (b, N_in)).astype(np.float64)
    dY = rng.integers(-8, 9, (b, N_out)).astype(np.float64)
    W = OT.dense_weight(cores, masks)
    assert np.max(np.abs(W)) <= 16 and np.all(W == np.round(W))
    # the quantised tensors decode to themselves
    for T in (X, dY, W):
        c, s = fp8.quantize(T)
        assert np.array_equal(fp8.decode(c) / s, T)
    assert np.array_equal(mixed.forward_fp8(X, cores, masks), X @ W)
    dX8, dG8 = mixed.backward_fp8(X, dY, cores, masks)
    dX, dG = OT.backward_dense(X, dY, cores, masks)
    assert np.array_equal(dX8, dX)
    for a, c in zip(dG8, dG):
        assert np.allclose(a, c, rtol=1e-12, atol=1e-9)
    for a, c in zip(mixed.mask_grads_fp8(X, dY, cores, masks), OT.mask_grads_dense(X, dY, cores, masks)):
        assert np.allclose(a, c, rtol=1e-12, atol=1e-9)


def _qerr(T):
    """Elementwise bound of |value(code) / s - T| for T quantised as a tensor:
    half an E4M3 step, 2^-4 |T| for normal values and 2^-10 / s below 2^-6 / s."""
    _, s = fp8.quantize(T)
    return np.maximum(2.0 ** -4 * np.abs(T), 2.0 ** -10 / s)


def _random_layer(seed, n, m, r, b):
    rng = np.random.default_rng(seed)
    d = len(n)
    N_in = int(np.prod(n))
    sig = (N_in * np.prod(r[1:-1])) ** (-1.0 / (2 * d))
    cores = [sig * rng.standard_normal((r[k], m[k], n[k], r[k + 1])) for k in range(d)]
    masks = [(rng.random(r[k + 1]) < 0.8).astype(np.float64) for k in range(d - 1)]
    X = rng.standard_normal((b, N_in)).astype(np.float32).astype(np.float64)
    dY = rng.standard_normal((b, int(np.prod(m)))).astype(np.float32).astype(np.float64)
    return cores, masks, X, dY


@pytest.mark.parametrize("seed", [1, 2])
def test_error_bounds(seed):
    n, m, r, b = (4, 6, 5), (3, 7, 4), (1, 6, 5, 1), 64
    cores, masks, X, dY = _random_layer(seed, n, m, r, b)
    W = OT.dense_weight(cores, masks)
    W32 = W.astype(np.float32).astype(np.float64)
    eX, edY = _qerr(X), _qerr(dY)
    eW = _qerr(W32) + np.abs(W32 - W)
    aX, adY, aW = np.abs(X), np.abs(dY), np.abs(W)
    slack = 1 + 1e-9
    Y8, Y = mixed.forward_fp8(X, cores, masks), X @ W
    bY = eX @ aW + aX @ eW + eX @ eW
    assert np.all(np.abs(Y8 - Y) <= bY * slack)
    dX8, dG8 = mixed.backward_fp8(X, dY, cores, masks)
    dX, dG = OT.backward_dense(X, dY, cores, masks)
    assert np.all(np.abs(dX8 - dX) <= (edY @ aW.T + adY @ eW.T + edY @ eW.T) * slack)
    dW8, dW = mixed.dW_fp8(X, dY), X.T @ dY
    bW = eX.T @ adY + aX.T @ edY + eX.T @ edY
    assert np.all(np.abs(dW8 - dW) <= bW * slack)
    # dG_k is linear in dW with coefficients that are products of core
    # entries: bounded by the same contraction of |cores| with the dW bound
    bG = OT.project_dW(bW, [np.abs(G) for G in cores], masks)
    for a, c, bb in zip(dG8, dG, bG):
        assert np.all(np.abs(a - c) <= bb * slack + 1e-300)
    # and the quantisation really happened: errors of the expected size
    rel = np.linalg.norm(Y8 - Y) / np.linalg.norm(Y)
    assert 1e-3 < rel < 5e-2


def test_mask_grad_homogeneity():
    # W is linear in each mask: sum_c D_k[c] dD_k[c] = <dW, W> for every bond
    n, m, r, b = (3, 4, 5), (5, 2, 6), (1, 5, 4, 1), 50
    cores, masks, X, dY = _random_layer(3, n, m, r, b)
    masks = [mk * np.random.default_rng(4).uniform(0.5, 1.5, mk.shape) for mk in masks]
    dW8 = mixed.dW_fp8(X, dY)
    W = OT.dense_weight(cores, masks)
    ref = float(np.sum(dW8 * W))
    for Dk, g in zip(masks, mixed.mask_grads_fp8(X, dY, cores, masks)):
        assert abs(float(np.dot(Dk, g)) - ref) <= 1e-10 * max(1.0, abs(ref))


def test_rows_fp8_matches_full_forward():
    n, m, r, b = (4, 6, 5), (3, 7, 4), (1, 6, 5, 1), 64
    cores, masks, X, dY = _random_layer(5, n, m, r, b)
    rows = np.array([0, 7, 33, 63])
    cW, sW = mixed.quantized_weight(cores, masks)
    assert np.array_equal(mixed.rows_fp8(X, rows, cW, sW), mixed.forward_fp8(X, cores, masks)[rows])
    cWt, sWt = fp8.quantize(OT.dense_weight(cores, masks).astype(np.float32).T)
    dX, _ = mixed.backward_fp8(X, dY, cores, masks)
    assert np.allclose(mixed.rows_fp8(dY, rows, cWt, sWt), dX[rows], rtol=1e-12, atol=1e-12)
