"""GPU parity of bf16 layers whose forward product takes the persistent
straight-to-LDS GEMM (K-contiguous operands, plain bf16 output, one
workgroup per CU walking 256 x 256 tiles, part of each finished tile
stored during the next tile's first stages): ragged last tiles in M and N,
a tile count that leaves the last round partly empty, K stage counts of 12
and 17.  Dense order; Y, dX and every dG_k against the oracle on the
bf16-rounded inputs (the headline's 1024 <-> 4096 products at 65536 tokens
are covered on sampled rows by the full-size layer tests).

Tolerance as for bf16 layers: max |gpu - ref| / max |ref| <= 2e-2.
"""
import pytest

from oracle import ttm as OT
from tests.gpu_util import TTMRun, rel_err, to_dev, to_np
from tests.test_gpu_ttm import TOL, _inputs

pytestmark = pytest.mark.gpu

CASES = [
    # (seed, n, m, r, b)
    # forward 16300 x 4000 x 1088: ragged last tiles in M (16300 = 63.7
    # tiles) and N (4000 = 15.6 tiles), 17 K stages
    (121, (17, 8, 8), (10, 20, 20), (1, 8, 8, 1), 16300),
    # the encoder's 768 -> 3072 layer at 16400 tokens: forward 65 x 12 = 780
    # tiles, so 12 workgroups take a fourth tile; 12 K stages
    (123, (8, 8, 12), (16, 16, 12), (1, 12, 12, 1), 16400),
]


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_bf16_persistent_products(case):
    seed, n, m, r, b = case
    print(f"gemm_pers seed={seed} n={n} m={m} r={r} b={b}", flush=True)
    cores, D, X, dY = _inputs(seed, n, m, r, b, "bf16")
    Yr = OT.forward_dense(X, cores, D)
    dXr, dGr = OT.backward_dense(X, dY, cores, D)
    run = TTMRun(n, m, r, cores, D, b, "bf16", force_order=0)
    Xt, dYt = to_dev(X, "bf16"), to_dev(dY, "bf16")
    Y = to_np(run.forward(Xt))
    dX, dG = run.backward(Xt, dYt)
    errs = {"Y": rel_err(Y, Yr), "dX": rel_err(to_np(dX), dXr)}
    for k in range(len(n)):
        errs[f"dG{k}"] = rel_err(to_np(dG[k]), dGr[k])
    bad = {k: v for k, v in errs.items() if not v <= TOL["bf16"]}
    assert not bad, bad
