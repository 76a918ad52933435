"""GPU parity of the fused projection of dW onto the cores (eq. back Gi,
dense order) where its first step reads many split partials of dW: a
768 -> 768 layer at 16384 tokens splits the fp32 dW product over tokens
into more than eight slices, so the 1024-thread projection sums them in
several rounds of eight loads; every dG_k and dX against the oracle.

Tolerance as for the dense order: max |gpu - ref| / max |ref| <= 1e-4
(fp32), <= 2e-2 (bf16).
"""
import pytest

from oracle import ttm as OT
from tests.gpu_util import TTMRun, rel_err, to_dev, to_np
from tests.test_gpu_ttm import TOL, _inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("r", [(1, 8, 8, 1), (1, 30, 30, 1)], ids=["r8", "r30"])
def test_projection_many_dw_splits(act, r):
    n, m, b = (8, 8, 12), (12, 8, 8), 16384
    print(f"proj n={n} m={m} r={r} b={b} act={act}", flush=True)
    cores, D, X, dY = _inputs(71, n, m, r, b, act)
    dXr, dGr = OT.backward_dense(X, dY, cores, D)
    run = TTMRun(n, m, r, cores, D, b, act, force_order=0)
    dX, dG = run.backward(to_dev(X, act), to_dev(dY, act))
    errs = {"dX": rel_err(to_np(dX), dXr)}
    for k in range(3):
        errs[f"dG{k}"] = rel_err(to_np(dG[k]), dGr[k])
    bad = {k: v for k, v in errs.items() if not v <= TOL[act]}
    assert not bad, bad
