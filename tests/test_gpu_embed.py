"""GPU parity of the TTM embedding lookup (Sec. 4.1) and its core gradients
against the fp64 oracle, through the C ABI.

Rows must match the oracle's rows for the same ids (fp32 tolerance 1e-4 on
max |gpu - ref| / max |ref|); repeated ids must give bitwise-identical rows;
the backward is bitwise reproducible run to run.
"""
import numpy as np
import pytest

from oracle import embed as OE
from paper_2405_14377_amd import workloads as wl
from tests.gpu_util import EmbedRun, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu


def _problem(seed, v, e, r, T, masks=True, std=0.5):
    rng = np.random.default_rng(seed)
    d = len(v)
    cores = [(rng.standard_normal((r[k], v[k], e[k], r[k + 1])) * std).astype(np.float32) for k in range(d)]
    D = None
    if masks and d > 1:
        D = [rng.standard_normal(r[k + 1]).astype(np.float32) for k in range(d - 1)]
        for Dk in D:
            if Dk.size > 1:
                Dk[0] = 0.0
    V = int(np.prod(v))
    ids = rng.integers(0, V, T).astype(np.int64)
    ids[T // 2:] = ids[: T - T // 2]          # repeated ids
    dY = rng.standard_normal((T, int(np.prod(e)))).astype(np.float32)
    return cores, D, ids, dY


def _check(v, e, r, cores, D, ids, dY, tol=1e-4):
    import torch
    T = ids.size
    run = EmbedRun(v, e, r, cores, D, T)
    ids_t = run.ids_dev(ids)
    Y = run.forward(ids_t)
    Yn = to_np(Y)
    Yr = OE.forward(ids, cores, D)
    assert rel_err(Yn, Yr) <= tol
    # rows of equal ids are bitwise equal
    first = {}
    for t, i in enumerate(ids.tolist()):
        if i in first:
            assert torch.equal(Y[t], Y[first[i]]), (t, i)
        else:
            first[i] = t
    dG = run.backward(ids_t, to_dev(dY))
    dGr = OE.backward(ids, dY, cores, D)
    for k in range(len(v)):
        assert rel_err(to_np(dG[k]), dGr[k]) <= tol, k
    assert int(run.err.item()) == 0
    return run, ids_t, dG


CASES = [
    (1, (7,), (5,), (1, 1), 9),
    (2, (3, 5), (2, 3), (1, 4, 1), 40),
    (3, (4, 3, 5), (2, 3, 2), (1, 3, 4, 1), 300),
    (4, (2, 3, 2, 3), (2, 1, 3, 2), (1, 2, 3, 2, 1), 1100),    # several sort tiles
    (5, (5, 1, 6), (3, 4, 1), (1, 3, 2, 1), 64),
    # shapes of the MFMA row / dA / dG_last kernels (E_p a multiple of 16)
    (6, (8, 4), (16, 12), (1, 17, 1), 500),                # d = 2: prefix table is core 0
    (7, (4, 4, 8), (4, 8, 7), (1, 5, 32, 1), 700),         # rank 32, E_last 7
    (8, (2, 3, 4), (4, 12, 16), (1, 3, 9, 1), 400),        # E_p 48, E_last 16
    (9, (3, 2, 5, 2), (2, 2, 4, 3), (1, 2, 3, 6, 1), 300),  # d = 4
]


@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_random_shapes(case):
    seed, v, e, r, T = case
    cores, D, ids, dY = _problem(seed, v, e, r, T)
    _check(v, e, r, cores, D, ids, dY)


def test_out_of_range_ids_flagged():
    v, e, r = (3, 4), (2, 3), (1, 3, 1)
    cores, D, ids, dY = _problem(7, v, e, r, 20)
    bad = ids.copy()
    bad[3] = 12          # == V
    bad[9] = -1
    run = EmbedRun(v, e, r, cores, D, 20)
    ids_t = run.ids_dev(bad)
    Y = to_np(run.forward(ids_t))
    assert int(run.err.item()) == 1
    good = np.array([i for i in range(20) if i not in (3, 9)])
    assert np.all(Y[3] == 0) and np.all(Y[9] == 0)
    assert rel_err(Y[good], OE.forward(bad[good], cores, D)) <= 1e-4
    run.err.zero_()
    dG = run.backward(ids_t, to_dev(dY))
    assert int(run.err.item()) == 1
    dGr = OE.backward(bad[good], dY[good], cores, D)
    for k in range(2):
        assert rel_err(to_np(dG[k]), dGr[k]) <= 1e-4


def test_all_tokens_one_id():
    """The hottest possible id: every token the same (work split into many
    items, summed in a fixed order)."""
    v, e, r = (4, 8), (4, 6), (1, 5, 1)
    cores, D, ids, dY = _problem(8, v, e, r, 3000)
    ids[:] = 17
    _check(v, e, r, cores, D, ids, dY)


@pytest.mark.parametrize("v,e,r", [((16, 32), (2, 4), (1, 3, 1)), ((8, 8, 8), (2, 3, 4), (1, 3, 5, 1))])
def test_two_pass_sort_many_blocks(v, e, r):
    """Vocabularies above 256 ids take two radix passes; with several
    thousand skewed tokens the second pass sees its own per-block digit
    counts, which differ from the first pass's."""
    cores, D, _, _ = _problem(11, v, e, r, 8)
    V = int(np.prod(v))
    T = 5000
    ids = wl.token_ids(T, V, "zipf1.1", 77)
    dY = np.random.default_rng(12).standard_normal((T, int(np.prod(e)))).astype(np.float32)
    _check(v, e, r, cores, D, ids, dY)


@pytest.mark.parametrize("dist", ["zipf1.1", "uniform"])
def test_workload_parity_and_determinism(dist):
    import torch
    w = wl.WORKLOADS[3]
    cores = wl.embed_cores(w)
    ids = wl.token_ids(w.n_tokens, int(np.prod(w.v)), dist, wl.seed_of(3, 20))
    dY = wl.activations(3, w.n_tokens, int(np.prod(w.e)), 1, "f32")
    run, ids_t, dG = _check(w.v, w.e, w.r, cores, None, ids, dY)
    dG2 = run.backward(ids_t, to_dev(dY))
    for a, b in zip(dG, dG2):
        assert torch.equal(a, b)
    # permuting the tokens permutes nothing in the result beyond rounding
    perm = np.random.default_rng(1).permutation(ids.size)
    dG3 = run.backward(run.ids_dev(ids[perm]), to_dev(dY[perm]))
    for a, b in zip(dG, dG3):
        assert rel_err(to_np(b), to_np(a)) <= 1e-5


@pytest.mark.parametrize("case", CASES[5:], ids=[f"s{c[0]}" for c in CASES[5:]])
def test_reuse_forward_and_hot_prefix(case):
    """Backward taking the forward's prefix table from the workspace equals
    the rebuilding backward bit for bit; ids crowded under a few prefixes
    (the dA sums split over waves) still match the oracle."""
    import torch
    from paper_2405_14377_amd import comera as C
    seed, v, e, r, T = case
    cores, D, ids, dY = _problem(seed, v, e, r, T)
    Vs = v[-1]
    rng = np.random.default_rng(seed + 100)
    ids = (rng.integers(0, 3, T) * Vs + rng.integers(0, Vs, T)).astype(np.int64)   # prefixes 0..2 only
    run = EmbedRun(v, e, r, cores, D, T)
    ids_t, dY_t = run.ids_dev(ids), to_dev(dY)
    run.forward(ids_t)
    a = run.backward_ex(ids_t, dY_t, C.EMBED_REUSE_FORWARD)
    b = run.backward_ex(ids_t, dY_t, 0)
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    dGr = OE.backward(ids, dY, cores, D)
    for k in range(len(v)):
        assert rel_err(to_np(a[k]), dGr[k]) <= 1e-4, k
