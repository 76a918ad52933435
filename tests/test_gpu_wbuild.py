"""GPU parity of the W build (last step of the batch-free chain, eq. TTM) on
shapes chosen to take each of its load and store paths: four-entry loads of
the chain slice and last core or one-entry loads, four-entry stores or
one-entry stores, with ragged last tiles in I and J.  The dense order builds
W^T for the forward and W for dX; with the forward's results reused, one
launch writes both layouts.  Y, dX and every dG_k against the oracle, fp32
and bf16 activations (bf16 builds bf16 copies of W).

Tolerance as for the dense order: max |gpu - ref| / max |ref| <= 1e-4
(fp32), <= 2e-2 (bf16).
"""
import numpy as np
import pytest

from oracle import ttm as OT
from tests.gpu_util import TTMRun, rel_err, to_dev, to_np
from tests.test_gpu_ttm import TOL, _inputs

pytestmark = pytest.mark.gpu

CASES = [
    # (seed, n, m, r, b): the last core is (n[-1], m[-1]) with rank A = r[-2]
    # 12 x 12 core, rank 8: both four-entry paths, ragged J tile
    (61, (4, 3, 12), (5, 4, 12), (1, 6, 8, 1), 70),
    # 4 x 3 core, rank 4, N_out = 15: four-entry loads, one-entry stores
    (62, (2, 3, 4), (5, 1, 3), (1, 3, 4, 1), 33),
    # 12 x 12 core, rank 5 over 9 values of J: one-entry loads, four-entry stores
    (63, (4, 2, 12), (3, 3, 12), (1, 4, 5, 1), 41),
    # 2 x 14 core, rank 2, 16 values of J in tiles of 7: only the ragged
    # last tile takes the four-entry paths, the others one-entry ones
    (66, (3, 2, 2), (4, 4, 14), (1, 3, 2, 1), 37),
    # 11 x 13 core: one-entry loads and stores
    (64, (3, 5, 11), (7, 2, 13), (1, 4, 3, 1), 29),
    # the 768 -> 3072 layer's last core (12 x 12, rank 30) at a small batch
    (65, (8, 8, 12), (16, 16, 12), (1, 30, 30, 1), 64),
]


@pytest.mark.parametrize("reuse", [False, True], ids=["rebuild", "reuse"])
@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_wbuild_paths(case, act, reuse):
    seed, n, m, r, b = case
    print(f"wbuild seed={seed} n={n} m={m} r={r} b={b} act={act} reuse={reuse}", flush=True)
    cores, D, X, dY = _inputs(seed, n, m, r, b, act)
    Yr = OT.forward_dense(X, cores, D)
    dXr, dGr = OT.backward_dense(X, dY, cores, D)
    run = TTMRun(n, m, r, cores, D, b, act, force_order=0, reuse=reuse)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    Y = to_np(run.forward(Xt))
    dX, dG = run.backward(Xt, dYt)
    errs = {"Y": rel_err(Y, Yr), "dX": rel_err(to_np(dX), dXr)}
    for k in range(len(n)):
        errs[f"dG{k}"] = rel_err(to_np(dG[k]), dGr[k])
    bad = {k: v for k, v in errs.items() if not v <= TOL[act]}
    assert not bad, bad
