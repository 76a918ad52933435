"""Mixed-precision layer on the GPU (the batch products on FP8 E4M3 codes,
the batch-free steps in fp32) against the oracle of oracle/mixed.py, and the
FP8 quantisation entry point against oracle/fp8.py.

* codes and scales: bit-exact (the rounding decision is taken on the same
  fp32 value x * s on both sides), padding included;
* layers whose dense weight is exact in fp32 (integer cores diagonal in
  their inner bonds): the GPU quantises the same W as the oracle, so Y and dX
  differ from the oracle only by the fp32 accumulation (relative 1e-4, the
  fp32 bar; bit-exact when the activations are small integers too); dG and
  dD go through the fp32 projections (relative 1e-4);
* Gaussian cores at the 768 -> 3072 shape: W is then rounded differently in
  fp32 (GPU chain) and fp64 (oracle), and a W code may flip where W s sits
  next to a rounding midpoint, so the GPU result is checked against the
  E4M3 error bound around the exact full-precision product (any valid
  rounding satisfies it) and for closeness to the oracle in norm.
"""
import zlib

import numpy as np
import pytest

from oracle import fp8 as OF
from oracle import mixed as OM
from oracle import ttm as OT
from paper_2405_14377_amd import comera as C
from paper_2405_14377_amd import workloads as wl
from tests.chunked import dw_fp8_rows
from tests.gpu_util import TTMRun, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu


def _quantize_gpu(x_np, act, ldq, ldt, want_q=True, want_qt=True):
    import torch
    rows, cols = x_np.shape
    x = to_dev(x_np, act)
    q = torch.full((rows, ldq), 0xAA, dtype=torch.uint8, device="cuda") if want_q else None
    qt = torch.full((cols, ldt), 0xAA, dtype=torch.uint8, device="cuda") if want_qt else None
    s = torch.zeros(1, dtype=torch.float32, device="cuda")
    ws = torch.empty(C.FP8_QUANTIZE_WS_BYTES, dtype=torch.uint8, device="cuda")
    C.comera_fp8_quantize(x, C.BF16 if act == "bf16" else C.F32, rows, cols, q, ldq, qt, ldt, s, ws)
    torch.cuda.synchronize()
    return (None if q is None else q.cpu().numpy(), None if qt is None else qt.cpu().numpy(), float(s.item()))


def _midpoints():
    """Values exactly halfway between neighbouring positive E4M3 values, and
    the values themselves (ties must go to the even code)."""
    v = OF.e4m3_table()[:0x7F]
    return np.concatenate([v, (v[:-1] + v[1:]) / 2])


@pytest.mark.parametrize("case", [
    ("normal", "f32", 1000, 777, 896, 1024),
    ("normal", "bf16", 64, 64, 64, 64),
    ("ties", "f32", 1, 253, 256, 128),
    ("tiny", "f32", 37, 5, 16, 64),
    ("zeros", "f32", 130, 70, 128, 256),
    ("huge", "f32", 9, 200, 256, 128),
    ("signed", "bf16", 257, 129, 256, 384),
    # 16-byte-load path (C a multiple of the chunk) with ragged tile edges
    ("normal", "f32", 1000, 776, 896, 1024),
    ("normal", "bf16", 333, 136, 256, 336),
    ("signed", "bf16", 129, 264, 264, 144),
])
def test_quantize_bit_exact(case):
    kind, act, rows, cols, ldq, ldt = case
    ldq, ldt = max(ldq, cols), max(ldt, rows)
    rng = np.random.default_rng(zlib.crc32(repr(case).encode()))
    if kind == "ties":
        x = _midpoints()[None, :cols] / 2.0 ** 3       # amax 448 / 8 -> s = 8: x s hits the midpoints exactly
        x = np.where(rng.random(x.shape) < 0.5, -x, x)
    elif kind == "tiny":
        x = rng.standard_normal((rows, cols)) * 1e-3
        x[0, 0] = 0.2                                   # most values fall in the subnormal codes
    elif kind == "zeros":
        x = np.zeros((rows, cols))
    elif kind == "huge":
        x = rng.standard_normal((rows, cols)) * 1e25   # scale clamped at 2^-60: saturating codes
    elif kind == "signed":
        x = rng.standard_normal((rows, cols)) * 0.01
        x[rng.random(x.shape) < 0.1] = -0.0
    else:
        x = rng.standard_normal((rows, cols)) * 3
    x = x.astype(np.float32)
    if act == "bf16":
        x = wl.to_bf16_values(x)
    codes, s_ref = OF.quantize(x)
    q, qt, s = _quantize_gpu(x, act, ldq, ldt)
    assert s == s_ref
    q_ref = np.zeros((rows, ldq), np.uint8)
    q_ref[:, :cols] = codes
    qt_ref = np.zeros((cols, ldt), np.uint8)
    qt_ref[:, :rows] = codes.T
    assert np.array_equal(q, q_ref)
    assert np.array_equal(qt, qt_ref)
    # one output only
    q2, _, _ = _quantize_gpu(x, act, ldq, ldt, want_qt=False)
    _, qt2, _ = _quantize_gpu(x, act, ldq, ldt, want_q=False)
    assert np.array_equal(q2, q_ref) and np.array_equal(qt2, qt_ref)


EXACT_CASES = [((8, 8, 12), (12, 8, 8), (1, 8, 8, 1), 200),
               ((4, 8, 4, 8), (8, 8, 8, 8), (1, 16, 16, 16, 1), 130),
               ((16, 8, 8, 1, 1, 1), (1, 1, 1, 8, 8, 16), (1, 4, 4, 4, 4, 4, 1), 64),
               ((5, 7), (3, 11), (1, 6, 1), 3)]


@pytest.mark.parametrize("reuse", [False, True])
@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", EXACT_CASES, ids=["768x768", "1024x4096", "tt6", "ragged"])
def test_integer_layer_bit_exact(case, act, reuse):
    """Small-integer activations and integer cores: every product is exact,
    so Y and dX equal the full-precision layer bit for bit (bf16 outputs:
    the exact value rounded once)."""
    n, m, r, b = case
    rng = np.random.default_rng(11)
    cores = wl.integer_bond_diagonal_cores(rng, n, m, r)
    masks = [(rng.random(r[k + 1]) < 0.75).astype(np.float32) for k in range(len(n) - 1)]
    run = TTMRun(n, m, r, cores, masks, b, act, force_order=0, reuse=reuse, fp8=True)
    X = rng.integers(-8, 9, (b, run.n_in)).astype(np.float32)
    dY = rng.integers(-8, 9, (b, run.n_out)).astype(np.float32)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    Y = to_np(run.forward(Xt))
    dX, dG = run.backward(Xt, dYt)
    Yo = OM.forward_fp8(X, cores, masks)
    dXo, dGo = OM.backward_fp8(X, dY, cores, masks)
    assert np.array_equal(Yo, OT.forward_dense(X, cores, masks))     # representable: no quantisation error
    rnd = (lambda a: wl.to_bf16_values(a.astype(np.float32))) if act == "bf16" else (lambda a: a)
    assert np.array_equal(Y, rnd(Yo))
    assert np.array_equal(to_np(dX), rnd(dXo))
    for a, c in zip(dG, dGo):
        assert rel_err(to_np(a), c) <= 1e-4


@pytest.mark.parametrize("reuse", [False, True])
@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", EXACT_CASES[:2] + EXACT_CASES[3:], ids=["768x768", "1024x4096", "ragged"])
def test_exact_weight_gaussian_activations(case, act, reuse):
    """W exact in fp32 on both sides, Gaussian activations: identical codes,
    results within the fp32 accumulation error (bf16: one output rounding)."""
    n, m, r, b = case
    rng = np.random.default_rng(12)
    cores = wl.integer_bond_diagonal_cores(rng, n, m, r)
    masks = [(rng.random(r[k + 1]) < 0.8).astype(np.float32) for k in range(len(n) - 1)]
    run = TTMRun(n, m, r, cores, masks, b, act, force_order=0, reuse=reuse, fp8=True)
    X = rng.standard_normal((b, run.n_in)).astype(np.float32)
    dY = rng.standard_normal((b, run.n_out)).astype(np.float32)
    if act == "bf16":
        X, dY = wl.to_bf16_values(X), wl.to_bf16_values(dY)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    Y = to_np(run.forward(Xt))
    dX, dG, dD = run.backward_masks(Xt, dYt)
    # fp32 bar 1e-4: accumulating K = 1024 products whose sum cancels to
    # about 1/32 of the sum of their magnitudes leaves ~1e-5 (measured 1.4e-5)
    tol = 1e-4 if act == "f32" else 4e-3
    assert rel_err(Y, OM.forward_fp8(X, cores, masks)) <= tol
    dXo, dGo = OM.backward_fp8(X, dY, cores, masks)
    assert rel_err(to_np(dX), dXo) <= tol
    for a, c in zip(dG, dGo):
        assert rel_err(to_np(a), c) <= 1e-4
    for a, c in zip(dD, OM.mask_grads_fp8(X, dY, cores, masks)):
        assert rel_err(to_np(a), c) <= 1e-4


def _qerr(T):
    _, s = OF.quantize(T)
    return np.maximum(2.0 ** -4 * np.abs(T), 2.0 ** -10 / s)


@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_ffn_up_within_fp8_bound(act):
    """768 -> 3072, ranks 30, Bernoulli(0.8) masks, Gaussian cores for unit
    output variance, 512 tokens: elementwise within the E4M3 error bound of
    the exact product and close to the oracle in norm."""
    shape = wl.TTMLayerShape("ffn_up", (8, 8, 12), (16, 16, 12), (1, 30, 30, 1))
    b = 512
    rng = np.random.default_rng(13)
    masks = wl.draw_masks(shape, ("bernoulli", 0.8), rng)
    sig = wl.unit_variance_sigma(shape, masks)
    cores = wl.random_cores(rng, shape, sig)
    n, m, r = shape.n, shape.m, shape.r
    run = TTMRun(n, m, r, cores, masks, b, act, force_order=0, reuse=True, fp8=True)
    X = rng.standard_normal((b, shape.n_in)).astype(np.float32)
    dY = rng.standard_normal((b, shape.n_out)).astype(np.float32)
    if act == "bf16":
        X, dY = wl.to_bf16_values(X), wl.to_bf16_values(dY)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    Y = to_np(run.forward(Xt))
    dX, dG = run.backward(Xt, dYt)
    dX = to_np(dX)
    W = OT.dense_weight(cores, masks)
    eW = _qerr(W) + 1e-6 * np.abs(W)               # either neighbour of a midpoint
    out_r = 2.0 ** -8 if act == "bf16" else 1e-6   # output rounding and fp32 accumulation
    bY = _qerr(X) @ np.abs(W) + np.abs(X) @ eW + _qerr(X) @ eW
    Yx = X.astype(np.float64) @ W
    assert np.all(np.abs(Y - Yx) <= bY * (1 + 1e-3) + out_r * np.abs(Y) + 1e-6 * np.max(np.abs(Yx)))
    bX = _qerr(dY) @ np.abs(W).T + np.abs(dY) @ eW.T + _qerr(dY) @ eW.T
    dXx = dY.astype(np.float64) @ W.T
    assert np.all(np.abs(dX - dXx) <= bX * (1 + 1e-3) + out_r * np.abs(dX) + 1e-6 * np.max(np.abs(dXx)))
    fro = lambda a, c: float(np.linalg.norm(a - c) / np.linalg.norm(c))
    close = 1e-3 if act == "f32" else 5e-3
    assert fro(Y, OM.forward_fp8(X, cores, masks)) <= close
    dXo, dGo = OM.backward_fp8(X, dY, cores, masks)
    assert fro(dX, dXo) <= close
    for a, c in zip(dG, dGo):
        assert fro(to_np(a), c) <= 1e-3


def test_fp8_smaller_batch_and_empty():
    """Calls with fewer tokens than planned (K of dW padded per call) and b = 0."""
    n, m, r = (8, 8, 12), (12, 8, 8), (1, 8, 8, 1)
    rng = np.random.default_rng(14)
    cores = wl.integer_bond_diagonal_cores(rng, n, m, r)
    run = TTMRun(n, m, r, cores, None, 700, "f32", force_order=0, fp8=True)
    for b in (700, 129, 1):
        X = rng.integers(-8, 9, (b, 768)).astype(np.float32)
        dY = rng.integers(-8, 9, (b, 768)).astype(np.float32)
        Xt, dYt = to_dev(X), to_dev(dY)
        assert np.array_equal(to_np(run.forward(Xt, b)), OM.forward_fp8(X, cores))
        dX, dG = run.backward(Xt, dYt, b)
        dXo, dGo = OM.backward_fp8(X, dY, cores)
        assert np.array_equal(to_np(dX), dXo)
        for a, c in zip(dG, dGo):
            assert rel_err(to_np(a), c) <= 1e-4
    assert run.forward(to_dev(np.zeros((1, 768))), 0).shape[0] == 0


@pytest.mark.parametrize("b", [8192, 8100])
@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_integer_layer_large_tiles(act, b):
    """8192 and 8100 tokens through 1024 -> 4096: the forward and dX products
    are large enough for the eight-wave 256 x 256 FP8 tiles (the bf16
    forward, 512 tiles, on the persistent kernel; 8100 tokens leave a ragged
    last row of tiles); still bit-exact."""
    n, m, r = (4, 8, 4, 8), (8, 8, 8, 8), (1, 16, 16, 16, 1)
    rng = np.random.default_rng(15)
    cores = wl.integer_bond_diagonal_cores(rng, n, m, r)
    run = TTMRun(n, m, r, cores, None, b, act, force_order=0, reuse=True, fp8=True)
    X = rng.integers(-8, 9, (b, run.n_in)).astype(np.float32)
    dY = rng.integers(-8, 9, (b, run.n_out)).astype(np.float32)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    Y = to_np(run.forward(Xt))
    dX, dG = run.backward(Xt, dYt)
    W = OT.dense_weight(cores)
    rnd = (lambda a: wl.to_bf16_values(a.astype(np.float32))) if act == "bf16" else (lambda a: a)
    assert np.array_equal(Y, rnd(X.astype(np.float64) @ W))
    assert np.array_equal(to_np(dX), rnd(dY.astype(np.float64) @ W.T))
    dGo = OT.project_dW(X.T.astype(np.float64) @ dY, cores)
    for a, c in zip(dG, dGo):
        assert rel_err(to_np(a), c) <= 1e-4


@pytest.mark.parametrize("li", [0, 1], ids=["up", "down"])
def test_fp8_large_pair_sampled(li):
    """The FP8 figures of the bench: 1024 <-> 4096, d = 4, ranks 64,
    Bernoulli(0.7) masks, 65536 tokens, bf16 activations, with the bench's
    plan settings (dense order, reuse).  Y and dX on 256 sampled rows: within
    the E4M3 bound of the exact product and close in norm to the oracle's FP8
    rows (scales from the whole tensors); every dG_k element by element
    against the oracle's FP8 dW over all 65536 tokens, projected in fp64."""
    from tests.test_gpu_ttm import _workload_layer
    sh, inp, X, dY, mask_active = _workload_layer(4, li, "bf16")
    b = X.shape[0]
    run = TTMRun(sh.n, sh.m, sh.r, inp.cores, inp.masks, b, "bf16", mask_active=mask_active, force_order=0,
                 reuse=True, fp8=True)
    Xt, dYt = to_dev(X, "bf16"), to_dev(dY, "bf16")
    Y = run.forward(Xt)
    dX, dG = run.backward(Xt, dYt)
    rows = np.random.default_rng(300 + li).choice(b, 256, replace=False)
    W = OT.dense_weight(inp.cores, inp.masks)
    cW, sW = OM.quantized_weight(inp.cores, inp.masks)
    cWt, sWt = OF.quantize(W.astype(np.float32).T)
    Yr, dXr = to_np(Y[rows]), to_np(dX[rows])
    fro = lambda a, c: float(np.linalg.norm(a - c) / np.linalg.norm(c))
    assert fro(Yr, OM.rows_fp8(X, rows, cW, sW)) <= 5e-3
    assert fro(dXr, OM.rows_fp8(dY, rows, cWt, sWt)) <= 5e-3
    eW = _qerr(W) + 1e-6 * np.abs(W)
    sX, sD = OF.pow2_scale(np.max(np.abs(X))), OF.pow2_scale(np.max(np.abs(dY)))   # whole-tensor scales
    qx = np.maximum(2.0 ** -4 * np.abs(X[rows]), 2.0 ** -10 / sX)
    qd = np.maximum(2.0 ** -4 * np.abs(dY[rows]), 2.0 ** -10 / sD)
    Yx = X[rows].astype(np.float64) @ W
    bY = qx @ np.abs(W) + np.abs(X[rows]) @ eW + qx @ eW
    assert np.all(np.abs(Yr - Yx) <= bY * (1 + 1e-3) + 2.0 ** -8 * np.abs(Yr) + 1e-6 * np.max(np.abs(Yx)))
    dXx = dY[rows].astype(np.float64) @ W.T
    bX = qd @ np.abs(W).T + np.abs(dY[rows]) @ eW.T + qd @ eW.T
    assert np.all(np.abs(dXr - dXx) <= bX * (1 + 1e-3) + 2.0 ** -8 * np.abs(dXr) + 1e-6 * np.max(np.abs(dXx)))
    # every dG_k element by element: the oracle's FP8 dW (codes of X and dY
    # with whole-tensor scales, exact products) over all 65536 tokens,
    # projected onto the cores in fp64; the GPU sums the same products in
    # fp32, then projects in fp32
    dGg = [to_np(g) for g in dG]
    dGr = OT.project_dW(dw_fp8_rows(X, dY), inp.cores, inp.masks)
    for k in range(4):
        err = rel_err(dGg[k], dGr[k])
        print(f"layer {li} dG{k}: {err:.3e}")
        assert err <= 1e-3, (k, err)

