"""Pins for the fp64 TT/TTM embedding oracle.

* explicit index sums on tiny shapes (forward rows and core gradients, masks);
* the worked example of Sec. 4.1 (two index vectors sharing a prefix) and the
  prefix/suffix-table route of eq. emb_A1, emb_A2, emb_unique;
* the embedding gradient equals the TTM-layer gradient with one-hot inputs;
* central finite differences for every core gradient.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import embed, ttm

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _problem(seed, v, e, r, T=7, masks=True):
    rng = np.random.default_rng(seed)
    d = len(v)
    cores = [rng.standard_normal((r[k], v[k], e[k], r[k + 1])) for k in range(d)]
    D = [rng.standard_normal(r[k + 1]) for k in range(d - 1)] if masks else None
    if D:
        for Dk in D:
            if Dk.size > 1:
                Dk[0] = 0.0
    V = int(np.prod(v))
    ids = rng.integers(0, V, T)
    ids[-1] = ids[0]                       # a repeated id
    dY = rng.standard_normal((T, int(np.prod(e))))
    return cores, D, ids, dY


def _brute(v, e, r, cores, D, ids, dY):
    d = len(v)
    E = int(np.prod(e))
    Dm = [np.ones(r[k + 1]) if D is None else D[k] for k in range(d - 1)]
    Y = np.zeros((ids.size, E))
    dG = [np.zeros(c.shape) for c in cores]
    for t, idv in enumerate(ids):
        z = []
        x = int(idv)
        for k in reversed(range(d)):
            z.append(x % v[k]); x //= v[k]
        z = z[::-1]
        for et in itertools.product(*[range(x) for x in e]):
            col = 0
            for k in range(d):
                col = col * e[k] + et[k]
            for at in itertools.product(*[range(r[k]) for k in range(1, d)]):
                a = (0,) + at + (0,)
                fac = [cores[k][a[k], z[k], et[k], a[k + 1]] for k in range(d)]
                msk = np.prod([Dm[k][a[k + 1]] for k in range(d - 1)])
                Y[t, col] += np.prod(fac) * msk
                for k in range(d):
                    rest = np.prod([fac[l] for l in range(d) if l != k]) * msk
                    dG[k][a[k], z[k], et[k], a[k + 1]] += dY[t, col] * rest
    return Y, dG


@pytest.mark.parametrize("seed,v,e,r", [
    (1, (3, 2), (2, 3), (1, 3, 1)),
    (2, (2, 3, 2), (2, 2, 3), (1, 2, 3, 1)),
    (3, (3, 2, 2), (3, 1, 2), (1, 3, 2, 1)),
    (4, (2, 2, 2, 2), (2, 1, 2, 2), (1, 2, 2, 2, 1)),
])
def test_embed_brute_force(seed, v, e, r):
    cores, D, ids, dY = _problem(seed, v, e, r)
    Yb, dGb = _brute(v, e, r, cores, D, ids, dY)
    np.testing.assert_allclose(embed.forward(ids, cores, D), Yb, rtol=1e-12, atol=1e-13)
    T = embed.table(cores, D)
    np.testing.assert_allclose(T[ids], Yb, rtol=1e-12, atol=1e-13)
    dG = embed.backward(ids, dY, cores, D)
    for k in range(len(v)):
        np.testing.assert_allclose(dG[k], dGb[k], rtol=1e-12, atol=1e-13)


def test_digits_row_major():
    v = (5, 3, 4)
    ids = np.arange(60)
    z = embed.digits(ids, v)
    assert z.shape == (3, 60)
    assert np.array_equal(z[:, 0], [0, 0, 0])
    assert np.array_equal(z[:, 1], [0, 0, 1])          # last factor varies fastest
    assert np.array_equal(z[:, 4], [0, 1, 0])
    assert np.array_equal(z[:, 12], [1, 0, 0])
    assert np.array_equal(z[:, 59], [4, 2, 3])


def test_paper_prefix_example():
    g = json.load(open(os.path.join(GOLDEN, "emb_prefix_example.json")))
    v, e, r = g["v"], g["e"], g["r"]
    vecs = np.array(g["digit_vectors"])
    ids = np.array([((zv[0] * v[1] + zv[1]) * v[2] + zv[2]) * v[3] + zv[3] for zv in vecs])
    z = embed.digits(ids, v)
    assert np.array_equal(z.T, vecs)
    assert np.array_equal(z[:2, 0], g["shared_prefix"]) and np.array_equal(z[:2, 1], g["shared_prefix"])
    # eq. emb_A1 / emb_A2 / emb_unique: prefix table over (z1,z2), suffix table over (z3,z4)
    rng = np.random.default_rng(0)
    cores = [rng.standard_normal((r[k], v[k], e[k], r[k + 1])) for k in range(4)]
    A1 = np.einsum("avec,cwfd->avwefd", cores[0], cores[1])[0]          # [v1, v2, e1, e2, r2]
    A1 = A1.reshape(v[0] * v[1], e[0] * e[1], r[2])
    A2 = np.einsum("avec,cwfd->avwefd", cores[2], cores[3])[..., 0]      # [r2, v3, v4, e3, e4]
    A2 = A2.reshape(r[2], v[2] * v[3], e[2] * e[3])
    J1 = z[0] * v[1] + z[1]
    J2 = z[2] * v[3] + z[3]
    assert J1[0] == J1[1]                      # the shared prefix entry is one row of A1
    rows = np.einsum("kEa,akF->kEF", A1[J1], A2[:, J2, :]).reshape(2, -1)
    np.testing.assert_allclose(embed.forward(ids, cores), rows, rtol=1e-12)


@pytest.mark.parametrize("seed", [5, 6])
def test_embed_grad_equals_ttm_grad_of_onehot(seed):
    v, e, r = (3, 2, 2), (2, 3, 2), (1, 2, 3, 1)
    cores, D, ids, dY = _problem(seed, v, e, r, T=9)
    V = int(np.prod(v))
    onehot = np.zeros((ids.size, V)); onehot[np.arange(ids.size), ids] = 1.0
    lin = [np.swapaxes(c, 1, 2) for c in cores]          # linear layout: m = e (out), n = v (in)
    np.testing.assert_allclose(ttm.forward_direct(onehot, lin, D), embed.forward(ids, cores, D), rtol=1e-12)
    _, dGl = ttm.backward_dense(onehot, dY, lin, D)
    dG = embed.backward(ids, dY, cores, D)
    for k in range(3):
        np.testing.assert_allclose(np.swapaxes(dGl[k], 1, 2), dG[k], rtol=1e-11, atol=1e-13)


def test_embed_finite_differences():
    v, e, r = (2, 3, 2), (2, 2, 2), (1, 3, 2, 1)
    cores, D, ids, dY = _problem(8, v, e, r, T=5)
    h = 1e-6
    dG = embed.backward(ids, dY, cores, D)

    def loss(cs):
        return float(np.sum(embed.forward(ids, cs, D) * dY))

    for k in range(3):
        for idx in np.ndindex(*cores[k].shape):
            cp = [c.copy() for c in cores]; cp[k][idx] += h
            cm = [c.copy() for c in cores]; cm[k][idx] -= h
            fd = (loss(cp) - loss(cm)) / (2 * h)
            assert abs(fd - dG[k][idx]) < 1e-6 * max(1.0, abs(fd))
