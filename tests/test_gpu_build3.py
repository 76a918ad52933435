"""GPU parity of the one-launch build of a three-core layer (mask fold, the
chain step P_2 and W in one kernel, eq. TTM with eq. Wcompress) on shapes
that take its tile choices and store paths: the workload layers (tiles of
4 x 4 middle slices, 48-entry output runs, four-entry stores), slices of a
whole middle factor, a single pair per workgroup, fewer than 16 rows per
workgroup, odd last cores (one-entry stores in W, W^T or both), ranks 1, 2,
17, 60 and 64, compacted bonds, and a 256-entry last core.  The backward
reads the folded cores and P_2 the kernel writes, so dX and every dG_k check
them too.  Dense order; Y, dX and every dG_k against the oracle.

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
    # the 768 -> 3072 layer's factors, ranks compacted to about 24
    (91, (8, 8, 12), (16, 16, 12), (1, 30, 30, 1), 48, 0.8),
    # the encoder's 768 x 768 factors (tiles of 24 rows)
    (92, (8, 8, 12), (12, 8, 8), (1, 30, 30, 1), 40, 0.5),
    # the 3072 -> 768 factors, rank 64 on both bonds
    (93, (16, 16, 12), (8, 8, 12), (1, 64, 64, 1), 24, 1.0),
    # last core 11 x 13: one-entry stores in both layouts
    (94, (3, 5, 11), (7, 2, 13), (1, 4, 3, 1), 29, 1.0),
    # last core 2 x 14 (W^T one-entry), 3 x 4 middle slices
    (95, (2, 3, 2), (4, 4, 14), (1, 17, 2, 1), 37, 1.0),
    # unit factors, fewer than 16 rows per workgroup
    (96, (1, 8, 1), (6, 1, 9), (1, 5, 2, 1), 19, 1.0),
    # ranks 1 and 2; last core 7 x 2
    (97, (5, 3, 7), (3, 9, 2), (1, 1, 2, 1), 33, 1.0),
    # ranks 60 and 64 compacted from 65 and 70
    (98, (2, 3, 4), (3, 2, 4), (1, 65, 70, 1), 20, 0.9),
    # a 16 x 16 last core (256 entries per rank pair), rank 8
    (99, (16, 8, 16), (8, 16, 16), (1, 8, 8, 1), 16, 1.0),
]


@pytest.mark.parametrize("reuse", [False, True], ids=["rebuild", "reuse"])
@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_three_core_build(case, act, reuse):
    seed, n, m, r, b, keep = case
    print(f"build3 seed={seed} n={n} m={m} r={r} b={b} keep={keep} act={act} reuse={reuse}", flush=True)
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
