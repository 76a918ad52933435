"""fp64 oracle for the TTM embedding table (Sec. 4.1; test infrastructure only).

Layout (Sec. 4.1, the table T in R^{m x n} reshaped to m_1 x n_1 x ... x m_d x n_d):
core t is G_t[r_t, v_t, e_t, r_{t+1}] with v_t the row (vocabulary) factor and
e_t the column (embedding) factor; V = prod v_t rows, E = prod e_t columns.
A row id is converted to its tensor index (z_1, ..., z_d) row-major, first
factor most significant.  Optional masks D_t sit on core t's right bond as in
eq. Wcompress.

T[id, e] = sum_a prod_t G~_t[a_t, z_t, e_t, a_{t+1}]
Y[k, :] = T[ids[k], :]                     (the lookup T[I, :] of Sec. 4.1)
dG_t = d<Y, dY>/dG_t, accumulated token by token in token order (the paper
does not state the backward; it follows from the lookup being linear in each
core).
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np

from .ttm import masked_cores


def digits(ids, v: Sequence[int]) -> np.ndarray:
    """Tensor index of each row id, row-major: returns int64 [d, T]."""
    ids = np.asarray(ids, dtype=np.int64)
    d = len(v)
    z = np.empty((d, ids.size), dtype=np.int64)
    rem = ids.copy()
    for t in reversed(range(d)):
        z[t] = rem % v[t]
        rem = rem // v[t]
    return z


def table(cores, masks=None) -> np.ndarray:
    """Dense table T [V, E] by a left-to-right chain of the cores."""
    Gt = masked_cores(cores, masks)
    P = np.ones((1, 1, 1))                       # [Vl, El, a]
    for G in Gt:                                 # [a, v, e, c]
        T = np.einsum("VEa,avec->VvEec", P, G, optimize=True)
        V, v, E, e, c = T.shape
        P = T.reshape(V * v, E * e, c)
    return P[:, :, 0]


def _slices(Gt, z):
    """G~_t[:, z_t(k), :, :] for every token k, as [T, a, e, c]."""
    return [np.transpose(G[:, zt, :, :], (1, 0, 2, 3)) for G, zt in zip(Gt, z)]


def forward(ids, cores, masks=None) -> np.ndarray:
    """Rows T[ids, :] (fp64) by contracting each token's core slices left to right."""
    Gt = masked_cores(cores, masks)
    v = [G.shape[1] for G in Gt]
    z = digits(ids, v)
    S = _slices(Gt, z)
    T = z.shape[1]
    R = S[0][:, 0, :, :]                          # [T, e_0, a_1]
    for t in range(1, len(Gt)):
        R = np.einsum("kEa,kaec->kEec", R, S[t], optimize=True)
        R = R.reshape(T, -1, S[t].shape[3])
    return R[:, :, 0]


def backward(ids, dY, cores, masks=None) -> List[np.ndarray]:
    """dG_t for every core; token contributions are added in token order."""
    Gt = masked_cores(cores, masks)
    d = len(Gt)
    v = [G.shape[1] for G in Gt]
    e = [G.shape[2] for G in Gt]
    z = digits(ids, v)
    S = _slices(Gt, z)
    T = z.shape[1]
    dY = np.asarray(dY, dtype=np.float64)
    # left environments L[t] = prod of slices < t: [T, E_<t, a_t]
    L = [np.ones((T, 1, 1))]
    for t in range(d - 1):
        Lt = np.einsum("kEa,kaec->kEec", L[t], S[t], optimize=True)
        L.append(Lt.reshape(T, -1, S[t].shape[3]))
    # right environments R[t] = prod of slices > t: [T, a_{t+1}, E_>t]
    R = [None] * d
    R[d - 1] = np.ones((T, 1, 1))
    for t in reversed(range(d - 1)):
        Rt = np.einsum("kaec,kcE->kaeE", S[t + 1], R[t + 1], optimize=True)
        R[t] = Rt.reshape(T, S[t + 1].shape[1], -1)
    out = []
    for t in range(d):
        El = int(np.prod(e[:t], dtype=np.int64))
        Er = int(np.prod(e[t + 1:], dtype=np.int64))
        dY3 = dY.reshape(T, El, e[t], Er)
        contrib = np.einsum("kAeB,kAa,kcB->kaec", dY3, L[t], R[t], optimize=True)  # [T, a, e_t, c]
        if masks is not None and t < d - 1:
            contrib = contrib * np.asarray(masks[t], np.float64)[None, None, None, :]
        g = np.zeros(Gt[t].shape)
        np.add.at(np.transpose(g, (1, 0, 2, 3)), z[t], contrib)
        out.append(g)
    return out
