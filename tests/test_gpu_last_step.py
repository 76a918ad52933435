"""GPU parity of the W build for layers the one-launch three-core build
does not take (fold, chain steps and the W tile kernel, eq. TTM): two cores,
four and five cores, a last core with factors that rule out four-entry
stores in W, W^T or both, 256 entries per rank pair, ranks 1 and 64,
compacted bonds.  Dense order; Y, dX and
every dG_k against the oracle.

Tolerance as for the dense order: max |gpu - ref| / max |ref| <= 1e-4
(fp32), <= 2e-2 (bf16).
"""
import pytest

from oracle import ttm as OT
from tests.gpu_util import TTMRun, rel_err, to_dev, to_np
from tests.test_gpu_chain_steps import _masks
from tests.test_gpu_ttm import TOL, _inputs

pytestmark = pytest.mark.gpu

CASES = [
    # (seed, n, m, r, b, keep)
    # the 1024 -> 4096 layer's factors at a small batch, compacted ranks
    (101, (4, 8, 4, 8), (8, 8, 8, 8), (1, 64, 64, 64, 1), 24, 0.7),
    # two cores, last core 8 x 20 (W^T one-entry: n = 8 is fine, W: 20)
    (102, (16, 8), (12, 20), (1, 17, 1), 33, 1.0),
    # last core 11 x 13: one-entry stores in both layouts, rank 1
    (103, (7, 11), (13, 13), (1, 1, 1), 17, 1.0),
    # five cores, last core 4 x 3
    (104, (2, 3, 2, 2, 4), (3, 2, 2, 3, 3), (1, 5, 9, 16, 33, 1), 21, 1.0),
    # a 16 x 16 last core (256 entries per rank pair), rank 8, four cores
    (105, (2, 2, 3, 16), (2, 3, 2, 16), (1, 4, 6, 8, 1), 19, 1.0),
    # rank 64 into a 4 x 4 last core
    (106, (4, 4, 4, 4), (4, 4, 4, 4), (1, 8, 16, 64, 1), 15, 1.0),
]


@pytest.mark.parametrize("reuse", [False, True], ids=["rebuild", "reuse"])
@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_last_chain_step(case, act, reuse):
    seed, n, m, r, b, keep = case
    print(f"last-step seed={seed} n={n} m={m} r={r} b={b} keep={keep} act={act} reuse={reuse}", flush=True)
    cores, D, X, dY = _inputs(seed, n, m, r, b, act)
    D, active = _masks(seed, r, keep, D)
    Yr = OT.forward_dense(X, cores, D)
    dXr, dGr = OT.backward_dense(X, dY, cores, D)
    run = TTMRun(n, m, r, cores, D, b, act, mask_active=active, force_order=0, reuse=reuse)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    Y = to_np(run.forward(Xt))
    dX, dG = run.backward(Xt, dYt)
    errs = {"Y": rel_err(Y, Yr), "dX": rel_err(to_np(dX), dXr)}
    for k in range(len(n)):
        errs[f"dG{k}"] = rel_err(to_np(dG[k]), dGr[k])
    bad = {k: v for k, v in errs.items() if not v <= TOL[act]}
    assert not bad, bad
