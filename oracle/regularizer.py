"""fp64 oracle of the early-stage regulariser gradients (test infrastructure
only: imported by tests/, never by the library).

The early stage of training (Sec. 3.2, eq. pretrain-rank) minimises
L(G, D) + gamma * S^(D) + beta * ||G||^2, where S^ is the size of the
compressed layer with each ||D_k||_0 replaced by ||D_k||_1:

    S^(D) = s_1 ||D_1||_1 + s_d ||D_{d-1}||_1
            + sum_{j=2}^{d-1} s_j ||D_{j-1}||_1 ||D_j||_1,

and ||G||^2 is the sum of the squared entries of all cores.  Readings (the
section states the formula for a tensor train; the garbled double sum over
layers is read as one sum of the per-layer expression):

* s_j, the variables of core j per pair of rank indices, is m_j n_j for a
  TTM core [r_{j-1}, m_j, n_j, r_j];
* the derivative of |x| at 0 is taken as 0 (the subgradient the sign
  function gives), so entries that are exactly zero get no size gradient;
* the regulariser acts on the mask values it is given; a layer with one core
  has no masks and S^ = 0.

Pinned in tests/test_oracle_regularizer.py: central differences of S^ and
||G||^2, S^ = S (the exact size) for 0/1 masks, S counted entry by entry on
the cores, and the two-core special case.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def core_sizes(m: Sequence[int], n: Sequence[int]) -> List[int]:
    """s_j = m_j n_j, the entries of core j per pair of rank indices."""
    return [int(a) * int(b) for a, b in zip(m, n)]


def _size(norms: List[float], s: List[int]) -> float:
    d = len(s)
    if d < 2:
        return 0.0
    tot = s[0] * norms[0] + s[d - 1] * norms[d - 2]
    for j in range(1, d - 1):
        tot += s[j] * norms[j - 1] * norms[j]
    return float(tot)


def size_exact(masks, m, n) -> float:
    """S(D) of Sec. 3.1: the formula with ||D_k||_0."""
    return _size([float(np.count_nonzero(Dk)) for Dk in masks], core_sizes(m, n))


def size_relaxed(masks, m, n) -> float:
    """S^(D) of eq. pretrain-rank's relaxation: the formula with ||D_k||_1."""
    return _size([float(np.sum(np.abs(np.asarray(Dk, np.float64)))) for Dk in masks], core_sizes(m, n))


def size_relaxed_grad(masks, m, n) -> List[np.ndarray]:
    """dS^/dD_k[c] = sign(D_k[c]) (left_k + right_k): bond k (0-based, between
    cores k and k+1) enters core k's term (s_k alone for the first core, else
    s_k ||D_{k-1}||_1) and core k+1's term (s_{k+1} alone for the last core,
    else s_{k+1} ||D_{k+1}||_1)."""
    s = core_sizes(m, n)
    d = len(s)
    norms = [float(np.sum(np.abs(np.asarray(Dk, np.float64)))) for Dk in masks]
    out = []
    for k in range(d - 1):
        left = s[k] if k == 0 else s[k] * norms[k - 1]
        right = s[k + 1] if k + 1 == d - 1 else s[k + 1] * norms[k + 1]
        out.append(np.sign(np.asarray(masks[k], np.float64)) * (left + right))
    return out


def l2(cores) -> float:
    """||G||^2: the squared entries of every core."""
    return float(sum(np.sum(np.asarray(G, np.float64) ** 2) for G in cores))


def l2_grad(cores) -> List[np.ndarray]:
    return [2.0 * np.asarray(G, np.float64) for G in cores]


def add_regularizer_grads(dG, dD, cores, masks, m, n, gamma: float, beta: float
                          ) -> Tuple[List[np.ndarray], List[np.ndarray]]:
    """The loss gradients (dG_k, dD_k) plus those of gamma S^(D) and
    beta ||G||^2."""
    gG = l2_grad(cores)
    gD = size_relaxed_grad(masks, m, n)
    return ([np.asarray(a, np.float64) + beta * g for a, g in zip(dG, gG)],
            [np.asarray(a, np.float64) + gamma * g for a, g in zip(dD, gD)])
