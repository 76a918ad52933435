"""GPU parity of the inner chain steps of the W build (eq. TTM, the left
chains P_k for 0 < k < d - 1) and of the dG projection tiles (eq. back Gi) on
shapes that reach their edges: ranks 1, 2, 17, 33 and 63 (rank blocks of 16
zero-padded inside a tile), rank 64 (the largest the chain-step and
projection kernels take), ranks above 64 (the general GEMM and the unfused
projection instead), chain steps whose 64 x 64 output tiles are ragged in
both directions, projection steps wider than 256 columns (several column
chunks, the last one ragged), and compacted rank masks.  Dense order; Y, dX
and every dG_k against the oracle.

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
    # (seed, n, m, r, b, keep): keep = fraction of each bond's mask entries
    # left active (below 1: compacted bonds)
    # chain steps: 6 x 2205 (ragged columns) and 210 x 54 (ragged both ways);
    # projection steps 1260 x 20, 210 x 54 and 6 x 2205 (35 column chunks)
    (81, (3, 5, 2, 4), (2, 7, 3, 5), (1, 17, 63, 9, 1), 40, 0.6),
    # five cores, three inner chain steps, ranks 5 / 33 / 16 / 7
    (82, (2, 3, 2, 2, 3), (3, 2, 2, 3, 2), (1, 5, 33, 16, 7, 1), 24, 0.7),
    # rank 64 on both bonds, uncompacted
    (83, (4, 4, 4), (4, 4, 4), (1, 64, 64, 1), 16, 1.0),
    # ranks above 64: the general chain GEMM and the unfused projections
    (84, (2, 3, 4), (3, 2, 4), (1, 65, 70, 1), 20, 1.0),
    # ranks 1 and 2
    (85, (5, 3, 7), (3, 9, 2), (1, 1, 2, 1), 33, 1.0),
]


def _masks(seed, r, keep, D):
    """Masks with about (1 - keep) of each bond's entries zeroed (at least one
    kept), and the matching mask_active flags."""
    rng = np.random.default_rng(seed + 1000)
    out, active = [], []
    for k, Dk in enumerate(D):
        Dk = Dk.copy()
        if keep < 1.0:
            off = rng.random(Dk.size) >= keep
            if off.all():
                off[rng.integers(Dk.size)] = False
            Dk[off] = 0.0
        else:
            Dk[Dk == 0.0] = 1.0
        out.append(Dk)
        active += [int(x != 0.0) for x in Dk]
    return out, active


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_chain_steps_and_projection_tiles(case, act):
    seed, n, m, r, b, keep = case
    print(f"chain-steps seed={seed} n={n} m={m} r={r} b={b} keep={keep} act={act}", flush=True)
    cores, D, X, dY = _inputs(seed, n, m, r, b, act)
    D, active = _masks(seed, r, keep, D)
    Yr = OT.forward_dense(X, cores, D)
    dXr, dGr = OT.backward_dense(X, dY, cores, D)
    run = TTMRun(n, m, r, cores, D, b, act, mask_active=active, force_order=0)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    Y = to_np(run.forward(Xt))
    dX, dG = run.backward(Xt, dYt)
    errs = {"Y": rel_err(Y, Yr), "dX": rel_err(to_np(dX), dXr)}
    for k in range(len(n)):
        errs[f"dG{k}"] = rel_err(to_np(dG[k]), dGr[k])
    bad = {k: v for k, v in errs.items() if not v <= TOL[act]}
    assert not bad, bad
