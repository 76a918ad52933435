"""GPU parity of the TTM layer (forward Y = XW, backward dX and every dG_k)
against the fp64 oracle, through the C ABI.

Tolerances: max |gpu - ref| / max |ref| per output tensor <= 1e-4 for fp32
activations and <= 2e-2 for bf16 activations with fp32 accumulation.  The
oracle consumes exactly the bf16-rounded inputs the GPU sees.
"""
import numpy as np
import pytest

from oracle import ttm as OT
from paper_2405_14377_amd import workloads as wl
from tests.chunked import xt_dy_fp64
from tests.gpu_util import TTMRun, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


def _inputs(seed, n, m, r, b, act, masks="real"):
    rng = np.random.default_rng(seed)
    shape = wl.TTMLayerShape("t", tuple(n), tuple(m), tuple(r))
    d = len(n)
    D = None
    if masks == "real":
        D = [rng.standard_normal(r[k + 1]).astype(np.float32) for k in range(d - 1)]
        for Dk in D:
            if Dk.size > 1:
                Dk[rng.integers(Dk.size)] = 0.0
    cores = wl.random_cores(rng, shape)
    # unit output scale: sigma from the closed form with full ranks
    sig = (shape.n_in * np.prod(r[1:-1])) ** (-1.0 / (2 * d))
    cores = [(c * sig).astype(np.float32) for c in cores]
    X = rng.standard_normal((b, shape.n_in)).astype(np.float32)
    dY = rng.standard_normal((b, shape.n_out)).astype(np.float32)
    if act == "bf16":
        X, dY = wl.to_bf16_values(X), wl.to_bf16_values(dY)
    return cores, D, X, dY


def _check_layer(n, m, r, cores, D, X, dY, act, mask_active=None, tol=None):
    b = X.shape[0]
    tol = TOL[act] if tol is None else tol
    run = TTMRun(n, m, r, cores, D, b, act, mask_active=mask_active)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    Y = to_np(run.forward(Xt))
    dX, dG = run.backward(Xt, dYt)
    Yr = OT.forward_dense(X, cores, D)
    dXr, dGr = OT.backward_dense(X, dY, cores, D)
    errs = {"Y": rel_err(Y, Yr), "dX": rel_err(to_np(dX), dXr)}
    for k in range(len(n)):
        errs[f"dG{k}"] = rel_err(to_np(dG[k]), dGr[k])
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, (errs, tol)
    return errs


CASES = [
    # (seed, n, m, r, b)
    (1, (3,), (5,), (1, 1), 7),
    (2, (4, 3), (2, 5), (1, 3, 1), 1),
    (3, (3, 5, 11), (7, 2, 13), (1, 4, 3, 1), 300),          # several tiles, ragged in every dim
    (4, (1, 8, 1), (6, 1, 9), (1, 5, 2, 1), 130),            # unit modes
    (5, (2, 3, 2, 3), (3, 2, 4, 2), (1, 3, 4, 2, 1), 257),
    (6, (16, 8), (12, 20), (1, 17, 1), 129),
]


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_random_shapes(case, act):
    seed, n, m, r, b = case
    cores, D, X, dY = _inputs(seed, n, m, r, b, act)
    _check_layer(n, m, r, cores, D, X, dY, act)


REUSE_CASES = CASES + [(15, (2, 16), (3, 20), (1, 60, 1), 100)]   # last core too large for the W tile kernel


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", REUSE_CASES, ids=[f"s{c[0]}" for c in REUSE_CASES])
def test_reuse_forward_build(case, act):
    """With reuse on, backward takes the masked cores, chains and W that the
    forward left in the workspace: every output equals the rebuilding
    route's bit for bit and matches the oracle."""
    seed, n, m, r, b = case
    cores, D, X, dY = _inputs(seed, n, m, r, b, act)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    outs = []
    for reuse in (False, True):
        run = TTMRun(n, m, r, cores, D, b, act, reuse=reuse)
        Y = to_np(run.forward(Xt))
        dX, dG = run.backward(Xt, dYt)
        outs.append([Y, to_np(dX)] + [to_np(g) for g in dG])
    for a, c in zip(*outs):
        assert np.array_equal(a, c)
    Yr = OT.forward_dense(X, cores, D)
    dXr, dGr = OT.backward_dense(X, dY, cores, D)
    refs = [Yr, dXr] + list(dGr)
    errs = [rel_err(g, ref) for g, ref in zip(outs[1], refs)]
    assert max(errs) <= TOL[act], errs


@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_no_masks(act):
    n, m, r = (4, 6, 5), (3, 7, 4), (1, 6, 5, 1)
    cores, _, X, dY = _inputs(11, n, m, r, 200, act, masks=None)
    _check_layer(n, m, r, cores, None, X, dY, act)


def test_mask_compaction_matches_full_rank():
    """A plan told which mask entries are active (and so contracting only the
    surviving slices) gives the oracle's result, zero gradients on the
    inactive slices included."""
    n, m, r = (3, 4, 5), (5, 2, 6), (1, 6, 7, 1)
    rng = np.random.default_rng(12)
    cores, _, X, dY = _inputs(12, n, m, r, 150, "f32", masks=None)
    act1 = (rng.random(6) < 0.6).astype(np.uint8); act1[0] = 1
    act2 = (rng.random(7) < 0.6).astype(np.uint8); act2[-1] = 1
    D = [act1.astype(np.float32) * rng.uniform(0.5, 1.5, 6).astype(np.float32),
         act2.astype(np.float32) * rng.uniform(0.5, 1.5, 7).astype(np.float32)]
    mask_active = list(act1) + list(act2)
    _check_layer(n, m, r, cores, D, X, dY, "f32", mask_active=mask_active)


def test_zero_bond():
    import torch
    n, m, r = (3, 4), (2, 5), (1, 3, 1)
    cores, _, X, dY = _inputs(13, n, m, r, 20, "f32", masks=None)
    D = [np.zeros(3, np.float32)]
    run = TTMRun(n, m, r, cores, D, 20, "f32", mask_active=[0, 0, 0])
    Xt, dYt = to_dev(X), to_dev(dY)
    assert torch.count_nonzero(run.forward(Xt)).item() == 0
    dX, dG = run.backward(Xt, dYt)
    assert torch.count_nonzero(dX).item() == 0
    assert all(torch.count_nonzero(g).item() == 0 for g in dG)


def test_smaller_batch_than_planned():
    n, m, r = (4, 4, 6), (6, 4, 4), (1, 5, 5, 1)
    cores, D, X, dY = _inputs(14, n, m, r, 500, "f32")
    run = TTMRun(n, m, r, cores, D, 500, "f32")
    b = 77
    Xt, dYt = to_dev(X[:b]), to_dev(dY[:b])
    Y = to_np(run.forward(Xt, b=b))
    dX, dG = run.backward(Xt, dYt, b=b)
    assert rel_err(Y, OT.forward_dense(X[:b], cores, D)) <= 1e-4
    dXr, dGr = OT.backward_dense(X[:b], dY[:b], cores, D)
    assert rel_err(to_np(dX), dXr) <= 1e-4
    for k in range(3):
        assert rel_err(to_np(dG[k]), dGr[k]) <= 1e-4


def test_backward_is_bitwise_deterministic():
    import torch
    n, m, r = (8, 8, 12), (16, 16, 12), (1, 30, 30, 1)
    cores, D, X, dY = _inputs(15, n, m, r, 1024, "bf16")
    run = TTMRun(n, m, r, cores, D, 1024, "bf16")
    Xt, dYt = to_dev(X, "bf16"), to_dev(dY, "bf16")
    dX1, dG1 = run.backward(Xt, dYt)
    dX2, dG2 = run.backward(Xt, dYt)
    assert torch.equal(dX1, dX2)
    for a, b in zip(dG1, dG2):
        assert torch.equal(a, b)


# ------------------------------------------------------------------ workload configurations
def _workload_layer(wid, li, act, rows=None):
    w = wl.WORKLOADS[wid]
    sh = w.layers[li]
    inp = wl.ttm_layer_inputs(wid, li, sh, w.mask)
    b = w.batch
    X = wl.activations(wid, b, sh.n_in, 0, act, layer=li)
    dY = wl.activations(wid, b, sh.n_out, 1, act, layer=li)
    mask_active = [int(x != 0) for mk in inp.masks for x in mk]
    return sh, inp, X, dY, mask_active


@pytest.mark.parametrize("wid,act", [(0, "f32"), (1, "f32"), (1, "bf16"), (5, "f32"), (5, "bf16")])
def test_workload_full_parity(wid, act):
    sh, inp, X, dY, mask_active = _workload_layer(wid, 0, act)
    errs = _check_layer(sh.n, sh.m, sh.r, inp.cores, inp.masks, X, dY, act, mask_active=mask_active)
    print(f"workload {wid} {act}: {errs}")


@pytest.mark.parametrize("li", range(6))
def test_encoder_layers(li):
    """Six encoder linears, 16384 tokens, bf16: Y and dX on 1024 sampled rows,
    every dG_k in full (oracle dense route)."""
    sh, inp, X, dY, mask_active = _workload_layer(2, li, "bf16")
    run = TTMRun(sh.n, sh.m, sh.r, inp.cores, inp.masks, X.shape[0], "bf16", mask_active=mask_active)
    Xt, dYt = to_dev(X, "bf16"), to_dev(dY, "bf16")
    Y = run.forward(Xt)
    dX, dG = run.backward(Xt, dYt)
    rows = np.random.default_rng(100 + li).choice(X.shape[0], 1024, replace=False)
    W = OT.dense_weight(inp.cores, inp.masks)
    assert rel_err(to_np(Y[rows]), X[rows].astype(np.float64) @ W) <= TOL["bf16"]
    assert rel_err(to_np(dX[rows]), dY[rows].astype(np.float64) @ W.T) <= TOL["bf16"]
    dGr = OT.project_dW(X.astype(np.float64).T @ dY.astype(np.float64), inp.cores, inp.masks)
    for k in range(3):
        assert rel_err(to_np(dG[k]), dGr[k]) <= TOL["bf16"], k


@pytest.mark.parametrize("li", [0, 1])
def test_large_pair_full_size(li):
    """1024 <-> 4096, d = 4, 65536 tokens, bf16, one plan at the full batch
    (its token split of dW and the projections that sum the split partials):
    every dG_k element by element against the oracle's dense-W route over
    all 65536 tokens; Y and dX on 512 sampled rows; <dG_k, G_k> = <Y, dY> =
    <dX, X> (W is linear in each core)."""
    import torch
    sh, inp, X, dY, mask_active = _workload_layer(4, li, "bf16")
    b = X.shape[0]
    run = TTMRun(sh.n, sh.m, sh.r, inp.cores, inp.masks, b, "bf16", mask_active=mask_active)
    Xt, dYt = to_dev(X, "bf16"), to_dev(dY, "bf16")
    Y = run.forward(Xt)
    dX, dG = run.backward(Xt, dYt)
    rows = np.random.default_rng(200 + li).choice(b, 512, replace=False)
    W = OT.dense_weight(inp.cores, inp.masks)
    assert rel_err(to_np(Y[rows]), X[rows].astype(np.float64) @ W) <= TOL["bf16"]
    assert rel_err(to_np(dX[rows]), dY[rows].astype(np.float64) @ W.T) <= TOL["bf16"]
    ydy = float((Y.float() * dYt.float()).double().sum().item())
    xdx = float((dX.float() * Xt.float()).double().sum().item())
    assert abs(xdx - ydy) <= 1e-2 * abs(ydy)
    dGg = [to_np(g) for g in dG]
    del Y, dX, dG
    torch.cuda.empty_cache()
    dGr = OT.project_dW(xt_dy_fp64(X, dY), inp.cores, inp.masks)
    for k in range(4):
        err = rel_err(dGg[k], dGr[k])
        print(f"layer {li} dG{k}: {err:.3e}")
        assert err <= TOL["bf16"], (k, err)
        gk = float(np.sum(dGg[k] * inp.cores[k].astype(np.float64)))
        assert abs(gk - ydy) <= 1e-2 * abs(ydy), (k, gk, ydy)
