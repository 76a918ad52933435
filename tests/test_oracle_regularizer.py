"""Pins of the regulariser-gradient oracle (eq. pretrain-rank) against facts
that do not depend on it: central differences of S^(D) and ||G||^2, the
exact size S(D) equal to S^ on 0/1 masks and equal to a count of the core
entries that survive the masks, and the two-core special case."""
import itertools

import numpy as np
import pytest

from oracle import regularizer as R

SHAPES = [
    ((4, 3), (2, 5), (1, 3, 1)),
    ((3, 5, 2), (2, 2, 7), (1, 4, 3, 1)),
    ((2, 3, 2, 3), (3, 2, 4, 2), (1, 3, 4, 2, 1)),
    ((2, 2, 3, 2, 2), (3, 2, 2, 2, 2), (1, 2, 3, 3, 2, 1)),
]


def _masks(rng, r, away_from_zero=True):
    out = []
    for k in range(1, len(r) - 1):
        x = rng.uniform(0.2, 1.5, r[k]) * rng.choice([-1.0, 1.0], r[k])
        out.append(x if away_from_zero else np.where(rng.random(r[k]) < 0.3, 0.0, x))
    return out


@pytest.mark.parametrize("shape", SHAPES, ids=[f"d{len(s[0])}" for s in SHAPES])
def test_size_gradient_central_differences(shape):
    n, m, r = shape
    rng = np.random.default_rng(len(n))
    D = _masks(rng, r)
    g = R.size_relaxed_grad(D, m, n)
    h = 1e-6
    for k, Dk in enumerate(D):
        for c in range(Dk.size):
            Dp = [x.copy() for x in D]
            Dm = [x.copy() for x in D]
            Dp[k][c] += h
            Dm[k][c] -= h
            fd = (R.size_relaxed(Dp, m, n) - R.size_relaxed(Dm, m, n)) / (2 * h)
            assert abs(fd - g[k][c]) <= 1e-6 * max(1.0, abs(fd)), (k, c, fd, g[k][c])


def test_zero_entries_get_no_size_gradient():
    n, m, r = SHAPES[1]
    D = _masks(np.random.default_rng(3), r, away_from_zero=False)
    for Dk, gk in zip(D, R.size_relaxed_grad(D, m, n)):
        assert np.all(gk[Dk == 0] == 0)
        assert np.all(gk[Dk != 0] != 0)


def test_l2_gradient_central_differences():
    rng = np.random.default_rng(5)
    cores = [rng.standard_normal((2, 3, 2, 3)), rng.standard_normal((3, 2, 2, 1))]
    g = R.l2_grad(cores)
    h = 1e-6
    for k, G in enumerate(cores):
        for idx in itertools.product(*[range(x) for x in G.shape]):
            Gp = [x.copy() for x in cores]
            Gm = [x.copy() for x in cores]
            Gp[k][idx] += h
            Gm[k][idx] -= h
            fd = (R.l2(Gp) - R.l2(Gm)) / (2 * h)
            assert abs(fd - g[k][idx]) <= 1e-6 * max(1.0, abs(fd))


@pytest.mark.parametrize("shape", SHAPES, ids=[f"d{len(s[0])}" for s in SHAPES])
def test_exact_size_counts_surviving_core_entries(shape):
    """With 0/1 masks, S counts the entries (a, x, y, c) of every core whose
    left and right rank indices both survive (the outer bonds always do), and
    the relaxation equals it."""
    n, m, r = shape
    rng = np.random.default_rng(11)
    D = [(rng.random(r[k]) < 0.6).astype(np.float64) for k in range(1, len(r) - 1)]
    d = len(n)
    count = 0
    for j in range(d):
        left = np.ones(r[j]) if j == 0 else D[j - 1]
        right = np.ones(r[j + 1]) if j == d - 1 else D[j]
        for a, x, y, c in itertools.product(range(r[j]), range(m[j]), range(n[j]), range(r[j + 1])):
            if left[a] != 0 and right[c] != 0:
                count += 1
    assert R.size_exact(D, m, n) == count
    assert R.size_relaxed(D, m, n) == count


def test_two_cores():
    n, m, r = SHAPES[0]
    D = [np.array([0.5, -2.0, 0.0])]
    s = R.core_sizes(m, n)
    assert R.size_relaxed(D, m, n) == (s[0] + s[1]) * 2.5
    assert np.array_equal(R.size_relaxed_grad(D, m, n)[0], np.array([1.0, -1.0, 0.0]) * (s[0] + s[1]))


def test_add_regularizer_grads_is_the_sum():
    n, m, r = SHAPES[1]
    rng = np.random.default_rng(2)
    cores = [rng.standard_normal((r[k], m[k], n[k], r[k + 1])) for k in range(3)]
    D = _masks(rng, r)
    dG = [rng.standard_normal(G.shape) for G in cores]
    dD = [rng.standard_normal(x.shape) for x in D]
    gG, gD = R.add_regularizer_grads(dG, dD, cores, D, m, n, gamma=0.0, beta=0.0)
    assert all(np.array_equal(a, b) for a, b in zip(gG, dG))
    assert all(np.array_equal(a, b) for a, b in zip(gD, dD))
    gG, gD = R.add_regularizer_grads(dG, dD, cores, D, m, n, gamma=0.25, beta=0.5)
    assert all(np.allclose(a, b + G) for a, b, G in zip(gG, dG, cores))
