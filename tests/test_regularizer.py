"""comera_ttm_regularizer_grads (eq. pretrain-rank): argument errors on the
CPU (they return before any HIP call), and GPU parity with the oracle: the
loss gradients of a real backward call plus gamma dS^/dD and beta d||G||^2/dG,
for 2 to 4 cores, masks with zero entries, and partial outputs.

Tolerance: max |gpu - ref| / max |ref| <= 1e-5 per tensor for the added
terms (fp32 sums of at most a few hundred terms), on top of the dense-order
bar (1e-4) for the loss gradients they are added to.
"""
import ctypes

import numpy as np
import pytest

from oracle import regularizer as R
from oracle import ttm as OT
from paper_2405_14377_amd import comera as C


def _status(shape, gamma, beta, G, D, dG, dD):
    lib = C.load()
    return lib.comera_ttm_regularizer_grads(None if shape is None else ctypes.byref(shape), gamma, beta,
                                            G, D, dG, dD, None)


def _arr(n, val=0x1000):
    a = (ctypes.c_void_p * n)()
    for i in range(n):
        a[i] = val + 256 * i
    return a


def test_argument_errors():
    sh = C.ttm_shape((2, 3, 4), (3, 2, 2), (1, 3, 4, 1))
    assert _status(None, 0.1, 0.1, None, None, None, None) == C.ERR_INVALID_ARG
    assert _status(sh, -0.1, 0.1, None, None, None, None) == C.ERR_INVALID_ARG
    assert _status(sh, 0.1, float("nan"), None, None, None, None) == C.ERR_INVALID_ARG
    assert _status(sh, 0.1, 0.1, None, None, _arr(3), None) == C.ERR_INVALID_ARG       # dG without G
    assert _status(sh, 0.1, 0.1, None, None, None, _arr(2)) == C.ERR_INVALID_ARG       # dD without D
    bad = C.ttm_shape((2, 3), (3, 2), (1, 3, 2))
    assert _status(bad, 0.1, 0.1, None, None, None, None) == C.ERR_INVALID_ARG         # r[d] != 1
    # nothing requested: no launch, OK
    assert _status(sh, 0.1, 0.1, None, None, None, None) == C.OK


CASES = [
    (81, (4, 3), (2, 5), (1, 3, 1)),
    (82, (3, 5, 2), (2, 2, 7), (1, 4, 3, 1)),
    (83, (2, 3, 2, 3), (3, 2, 4, 2), (1, 3, 5, 2, 1)),
]


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_regularizer_grads_parity(case):
    import torch
    from tests.gpu_util import TTMRun, rel_err, to_dev, to_np
    seed, n, m, r = case
    print(f"regularizer seed={seed} n={n} m={m} r={r}", flush=True)
    rng = np.random.default_rng(seed)
    d = len(n)
    cores = [(0.5 * rng.standard_normal((r[k], m[k], n[k], r[k + 1]))).astype(np.float32) for k in range(d)]
    D = [(rng.uniform(0.2, 1.5, r[k]) * rng.choice([-1.0, 1.0], r[k])).astype(np.float32) for k in range(1, d)]
    for Dk in D:
        Dk[rng.integers(Dk.size)] = 0.0
    b = 40
    X = rng.standard_normal((b, int(np.prod(n)))).astype(np.float32)
    dY = rng.standard_normal((b, int(np.prod(m)))).astype(np.float32)
    gamma, beta = 1e-3, 5e-2
    run = TTMRun(n, m, r, cores, D, b, "f32")
    Xt, dYt = to_dev(X), to_dev(dY)
    dX, dG, dD = run.backward_masks(Xt, dYt)
    loss_dG = [to_np(g) for g in dG]
    loss_dD = [to_np(g) for g in dD]
    shape = C.ttm_shape(n, m, r)
    C.comera_ttm_regularizer_grads(shape, gamma, beta, run.G, run.D, dG, dD)
    torch.cuda.synchronize()
    # the added terms against the oracle's, on the loss gradients the GPU
    # returned: one fp32 rounding of the term and one of the sum (2^-24 each,
    # bounded by 2^-23 (|term| + |total|)); the size term also carries the
    # fp32 l1 norms of at most r entries (r 2^-24 relative)
    refG, refD = R.add_regularizer_grads(loss_dG, loss_dD, cores, D, m, n, gamma, beta)
    for k in range(d):
        term = refG[k] - loss_dG[k]
        assert np.all(np.abs(to_np(dG[k]) - refG[k]) <= 2.0 ** -23 * (np.abs(term) + np.abs(refG[k])) + 1e-30), k
    for k in range(d - 1):
        term = refD[k] - loss_dD[k]
        bound = 2.0 ** -23 * (np.abs(term) + np.abs(refD[k])) + 1e-5 * np.abs(term) + 1e-30
        assert np.all(np.abs(to_np(dD[k]) - refD[k]) <= bound), k
        assert np.all(to_np(dD[k])[D[k] == 0] == loss_dD[k][D[k] == 0])
    # and the totals against the oracle's loss gradients plus the terms
    dGr, dDr = OT.backward_dense(X, dY, cores, D)[1], OT.mask_grads_dense(X, dY, cores, D)
    totG, totD = R.add_regularizer_grads(dGr, dDr, cores, D, m, n, gamma, beta)
    for k in range(d):
        assert rel_err(to_np(dG[k]), totG[k]) <= 1e-4, ("total dG", k)
    for k in range(d - 1):
        assert rel_err(to_np(dD[k]), totD[k]) <= 1e-4, ("total dD", k)
    # partial outputs: only dD of the first bond, then only dG of the last core
    dD0 = [to_dev(np.ones(r[1], np.float32))] + [None] * (d - 2)
    C.comera_ttm_regularizer_grads(shape, gamma, 0.0, None, run.D, None, dD0)
    gD = R.size_relaxed_grad(D, m, n)[0]
    assert np.all(np.abs(to_np(dD0[0]) - (1.0 + gamma * gD)) <= 2.0 ** -23 * (1.0 + np.abs(gamma * gD)) + 1e-5 * np.abs(gamma * gD))
    dGl = [None] * (d - 1) + [to_dev(np.zeros_like(cores[-1]))]
    C.comera_ttm_regularizer_grads(shape, 0.0, beta, run.G, None, dGl, None)
    assert rel_err(to_np(dGl[-1]), 2 * beta * cores[-1].astype(np.float64)) <= 1e-6


@pytest.mark.gpu
def test_regularizer_grads_long_mask():
    """A bond of 300 entries (more than one pass of the 256 threads)."""
    import torch
    from tests.gpu_util import rel_err, to_dev, to_np
    n, m, r = (2, 3), (3, 2), (1, 300, 1)
    print(f"regularizer long mask r={r}", flush=True)
    rng = np.random.default_rng(84)
    cores = [rng.standard_normal((r[k], m[k], n[k], r[k + 1])).astype(np.float32) for k in range(2)]
    D = [(rng.uniform(0.2, 1.5, 300) * rng.choice([-1.0, 1.0], 300)).astype(np.float32)]
    D[0][::7] = 0.0
    G = [to_dev(c) for c in cores]
    Dt = [to_dev(D[0])]
    dG = [to_dev(np.zeros_like(c)) for c in cores]
    dD = [to_dev(np.zeros(300, np.float32))]
    C.comera_ttm_regularizer_grads(C.ttm_shape(n, m, r), 0.01, 0.2, G, Dt, dG, dD)
    torch.cuda.synchronize()
    refG, refD = R.add_regularizer_grads([np.zeros(c.shape) for c in cores], [np.zeros(300)], cores, D, m, n,
                                         0.01, 0.2)
    for k in range(2):
        assert rel_err(to_np(dG[k]), refG[k]) <= 1e-6
    assert rel_err(to_np(dD[0]), refD[0]) <= 300 * 2.0 ** -24 + 2.0 ** -23   # fp32 l1 norm of 300 entries
