"""fp64 oracle for one TTM linear layer Y = X W (test infrastructure only).

Conventions (the paper's, and the readings taken where it leaves a choice):

* Core k (0-based here, k = 0..d-1) is G_k[r_k, m_k, n_k, r_{k+1}] with
  r_0 = r_d = 1: ``m`` is the output factor, ``n`` the input factor (the TTM
  format of eq. TTM in Sec. 2, read with the paper's linear-layer statement
  Y = XW, W in R^{N_in x N_out}, of Sec. 4.2).
* Multi-indices are row-major with the first factor most significant:
  i = ((i_0 n_1 + i_1) n_2 + i_2) ..., likewise j over the m_k.
* Rank masks (eq. Wcompress, Sec. 3.1): a diagonal D_k of length r_{k+1}
  sits between cores k and k+1 (k = 0..d-2); it is folded into core k's right
  bond.  ``masks=None`` means all ones.
* W[i, j] = sum_a prod_k G~_k[a_k, j_k, i_k, a_{k+1}] with G~_k = G_k D_k.

Two independent routes are provided:

* dense-W: rebuild W by a left-to-right chain of pairwise contractions, then
  Y = XW, dX = dY W^T (eq. back X), dW = X^T dY and dG_k = <dW, dW/dG_k>
  (eq. back Gi) as a contraction of dW with the partial chains left and right
  of core k;
* direct: never forms W.  Y is a right-to-left sweep of X through the cores
  (one pairwise contraction per core); dX is a left-to-right sweep of dY; dG_k
  is the contraction, over the batch and the modes outside core k, of the
  forward state entering core k with the backward state entering core k.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def masked_cores(cores: Sequence[np.ndarray], masks: Optional[Sequence[np.ndarray]]) -> List[np.ndarray]:
    """G~_k = G_k with D_k applied on its right bond (eq. Wcompress)."""
    d = len(cores)
    out = []
    for k in range(d):
        G = _f64(cores[k])
        if masks is not None and k < d - 1:
            G = G * _f64(masks[k])[None, None, None, :]
        out.append(G)
    return out


def _check(cores):
    d = len(cores)
    assert d >= 1
    assert cores[0].shape[0] == 1 and cores[-1].shape[3] == 1, "r_0 = r_d = 1"
    for k in range(d - 1):
        assert cores[k].shape[3] == cores[k + 1].shape[0], "bond mismatch"


def left_chain(Gt: Sequence[np.ndarray], upto: int) -> np.ndarray:
    """P[I, J, a] = contraction of cores 0..upto-1: I over their n's, J over their m's, a = r_upto."""
    P = np.ones((1, 1, 1))
    for k in range(upto):
        G = Gt[k]                                   # [a, j, i, c]
        T = np.einsum("IJa,ajic->IiJjc", P, G, optimize=True)
        I, i, J, j, c = T.shape
        P = T.reshape(I * i, J * j, c)
    return P


def right_chain(Gt: Sequence[np.ndarray], start: int) -> np.ndarray:
    """Q[a, I, J] = contraction of cores start..d-1: a = r_start, I over their n's, J over their m's."""
    d = len(Gt)
    Q = np.ones((1, 1, 1))
    for k in reversed(range(start, d)):
        G = Gt[k]                                   # [a, j, i, c]
        T = np.einsum("ajic,cIJ->aiIjJ", G, Q, optimize=True)
        a, i, I, j, J = T.shape
        Q = T.reshape(a, i * I, j * J)
    return Q


def dense_weight(cores, masks=None) -> np.ndarray:
    """W [N_in, N_out] (fp64) by the left-to-right chain of eq. TTM / eq. Wcompress."""
    _check(cores)
    Gt = masked_cores(cores, masks)
    return left_chain(Gt, len(Gt))[:, :, 0]


# ----------------------------------------------------------------------------- dense-W route
def forward_dense(X, cores, masks=None) -> np.ndarray:
    """Y = X W (Sec. 4.2, eq. forward)."""
    return _f64(X) @ dense_weight(cores, masks)


def project_dW(dW: np.ndarray, cores, masks=None) -> List[np.ndarray]:
    """dG_k = <dW, dW/dG_k> for every k (eq. back Gi), from dW [N_in, N_out]."""
    _check(cores)
    Gt = masked_cores(cores, masks)
    d = len(Gt)
    dW = _f64(dW)
    out = []
    for k in range(d):
        r0, mk, nk, r1 = Gt[k].shape
        P = left_chain(Gt, k)                       # [Il, Jl, r0]
        Q = right_chain(Gt, k + 1)                  # [r1, Ir, Jr]
        Il, Jl, Ir, Jr = P.shape[0], P.shape[1], Q.shape[1], Q.shape[2]
        dW6 = dW.reshape(Il, nk, Ir, Jl, mk, Jr)
        T = np.tensordot(dW6, P, axes=([0, 3], [0, 1]))          # [i, Ir, j, Jr, a]
        T = np.tensordot(T, Q, axes=([1, 3], [1, 2]))            # [i, j, a, c]
        g = T.transpose(2, 1, 0, 3).copy()                        # [a, j, i, c]
        if masks is not None and k < d - 1:
            g *= _f64(masks[k])[None, None, None, :]
        out.append(g)
    return out


def backward_dense(X, dY, cores, masks=None) -> Tuple[np.ndarray, List[np.ndarray]]:
    """dX = dY W^T (eq. back X) and every dG_k (eq. back Gi) through dense W."""
    W = dense_weight(cores, masks)
    X = _f64(X)
    dY = _f64(dY)
    dX = dY @ W.T
    dW = X.T @ dY
    return dX, project_dW(dW, cores, masks)


# ----------------------------------------------------------------------------- direct route
def sweep_right_to_left(X, Gt) -> Tuple[np.ndarray, List[np.ndarray]]:
    """Contract X with cores d-1, ..., 0 one at a time.

    Returns (Y, F) where F[k] is the state entering core k, laid out
    [b, I_<k, i_k, a_{k+1}, J_>k].
    """
    d = len(Gt)
    X = _f64(X)
    b = X.shape[0]
    n = [G.shape[2] for G in Gt]
    m = [G.shape[1] for G in Gt]
    Z = X
    Mr = 1
    F = [None] * d
    for k in reversed(range(d)):
        Nl = int(np.prod(n[:k], dtype=np.int64))
        Z5 = Z.reshape(b, Nl, n[k], Gt[k].shape[3], Mr)
        F[k] = Z5
        Z = np.einsum("bNicM,ajic->bNajM", Z5, Gt[k], optimize=True)   # [b, Nl, a_k, m_k, Mr]
        Mr *= m[k]
    return Z.reshape(b, -1), F


def sweep_left_to_right(dY, Gt) -> Tuple[np.ndarray, List[np.ndarray]]:
    """Contract dY with cores 0, ..., d-1 one at a time over their output modes.

    Returns (dX, H) where H[k] is the state entering core k, laid out
    [b, I_<k, a_k, j_k, J_>k].
    """
    d = len(Gt)
    dY = _f64(dY)
    b = dY.shape[0]
    n = [G.shape[2] for G in Gt]
    m = [G.shape[1] for G in Gt]
    Z = dY
    Nl = 1
    H = []
    for k in range(d):
        Mr = int(np.prod(m[k + 1:], dtype=np.int64))
        Z5 = Z.reshape(b, Nl, Gt[k].shape[0], m[k], Mr)
        H.append(Z5)
        Z = np.einsum("bNajM,ajic->bNicM", Z5, Gt[k], optimize=True)   # [b, Nl, n_k, a_{k+1}, Mr]
        Nl *= n[k]
    return Z.reshape(b, -1), H


def forward_direct(X, cores, masks=None) -> np.ndarray:
    """Y = X W without forming W: right-to-left sweep of eq. forward."""
    _check(cores)
    Y, _ = sweep_right_to_left(X, masked_cores(cores, masks))
    return Y


def backward_direct(X, dY, cores, masks=None) -> Tuple[np.ndarray, List[np.ndarray]]:
    """dX (eq. back X) by a left-to-right sweep of dY; dG_k (eq. back Gi) as the
    meet of the forward state and the backward state at core k."""
    _check(cores)
    Gt = masked_cores(cores, masks)
    d = len(Gt)
    _, F = sweep_right_to_left(X, Gt)
    dX, H = sweep_left_to_right(dY, Gt)
    dG = []
    for k in range(d):
        g = np.einsum("bNajM,bNicM->ajic", H[k], F[k], optimize=True)
        if masks is not None and k < d - 1:
            g = g * _f64(masks[k])[None, None, None, :]
        dG.append(g)
    return dX, dG


# ----------------------------------------------------------------------------- mask gradients
def _mask_list(cores, masks) -> List[np.ndarray]:
    d = len(cores)
    return [np.ones(cores[k].shape[3]) if masks is None else _f64(masks[k]) for k in range(d - 1)]


def mask_grads_dense(X, dY, cores, masks=None) -> List[np.ndarray]:
    """dD_k[c] = <dW, dW/dD_k[c]> for every bond k = 0..d-2 (chain rule through
    eq. Wcompress), dW = X^T dY."""
    return mask_grads_from_dW(_f64(X).T @ _f64(dY), cores, masks)


def mask_grads_from_dW(dW, cores, masks=None) -> List[np.ndarray]:
    """dD_k[c] = <dW, dW/dD_k[c]> for a given dW [N_in, N_out].  W is linear in
    D_k, so dW/dD_k[c] is the layer rebuilt with D_k replaced by the unit
    vector e_c and the other masks kept."""
    _check(cores)
    dW = _f64(dW)
    base = _mask_list(cores, masks)
    out = []
    for k in range(len(cores) - 1):
        g = np.zeros(base[k].shape[0])
        for c in range(g.shape[0]):
            mk = [m.copy() for m in base]
            mk[k] = np.zeros_like(mk[k])
            mk[k][c] = 1.0
            g[c] = float(np.sum(dW * dense_weight(cores, mk)))
        out.append(g)
    return out


def mask_grads_direct(X, dY, cores, masks=None) -> List[np.ndarray]:
    """dD_k[c] = sum_{a, j, i} dG~_k[a, j, i, c] G_k[a, j, i, c], where dG~_k is
    the gradient with respect to the masked core G~_k = G_k D_k: the meet of
    the forward and the backward sweep at core k (as in backward_direct,
    before the mask factor)."""
    _check(cores)
    Gt = masked_cores(cores, masks)
    _, F = sweep_right_to_left(X, Gt)
    _, H = sweep_left_to_right(dY, Gt)
    out = []
    for k in range(len(cores) - 1):
        g = np.einsum("bNajM,bNicM->ajic", H[k], F[k], optimize=True)
        out.append(np.einsum("ajic,ajic->c", g, _f64(cores[k])))
    return out


def mask_grad_term_scale(X, dY, cores, masks=None) -> List[np.ndarray]:
    """sum_{a, j, i} |dG~_k[a, j, i, c] G_k[a, j, i, c]| per entry c: the
    scale of the terms whose sum is dD_k[c].  A perturbation of relative size
    e in every dG~_k changes dD_k[c] by at most e times this, however much
    the terms cancel (the error scale for gradients from rounded states)."""
    _check(cores)
    Gt = masked_cores(cores, masks)
    _, F = sweep_right_to_left(X, Gt)
    _, H = sweep_left_to_right(dY, Gt)
    out = []
    for k in range(len(cores) - 1):
        g = np.einsum("bNajM,bNicM->ajic", H[k], F[k], optimize=True)
        out.append(np.einsum("ajic->c", np.abs(g * _f64(cores[k]))))
    return out
