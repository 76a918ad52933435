"""GPU parity of fp32 layers whose dW = X^T dY takes the straight-to-LDS
fp32 GEMM (operands M/N-contiguous, 128 x 128 tiles, K stages of 32, split
over the tokens): factor sizes that leave ragged last tiles in M and N, token
counts that are not a multiple of the split chunk, and the 768 -> 3072
layer at 4096 tokens.  Dense order; Y, dX and every dG_k against the oracle.

Tolerance as for fp32 layers: max |gpu - ref| / max |ref| <= 1e-4.
"""
import pytest

from oracle import ttm as OT
from tests.gpu_util import TTMRun, rel_err, to_dev, to_np
from tests.test_gpu_ttm import TOL, _inputs

pytestmark = pytest.mark.gpu

CASES = [
    # (seed, n, m, r, b)
    # N_in = 1088 (8.5 tiles), N_out = 1024, 4000 tokens (31.25 tiles)
    (111, (17, 8, 8), (8, 16, 8), (1, 8, 8, 1), 4000),
    # N_in = 1024, N_out = 1088, 2600 tokens
    (112, (8, 16, 8), (17, 8, 8), (1, 6, 10, 1), 2600),
    # the 768 -> 3072 layer's shape at 4096 tokens
    (113, (8, 8, 12), (16, 16, 12), (1, 12, 12, 1), 4096),
]


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_fp32_straight_to_lds_dw(case):
    seed, n, m, r, b = case
    print(f"gemm32 seed={seed} n={n} m={m} r={r} b={b}", flush=True)
    cores, D, X, dY = _inputs(seed, n, m, r, b, "f32")
    Yr = OT.forward_dense(X, cores, D)
    dXr, dGr = OT.backward_dense(X, dY, cores, D)
    run = TTMRun(n, m, r, cores, D, b, "f32", force_order=0)
    Xt, dYt = to_dev(X, "f32"), to_dev(dY, "f32")
    Y = to_np(run.forward(Xt))
    dX, dG = run.backward(Xt, dYt)
    errs = {"Y": rel_err(Y, Yr), "dX": rel_err(to_np(dX), dXr)}
    for k in range(len(n)):
        errs[f"dG{k}"] = rel_err(to_np(dG[k]), dGr[k])
    bad = {k: v for k, v in errs.items() if not v <= TOL["f32"]}
    assert not bad, bad
