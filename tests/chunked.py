"""Token-chunked forms of two oracle quantities, for the full-size parity
tests (65536 tokens): the same sums over tokens, taken over row chunks so
that no fp64 copy of a whole activation tensor is held at once.  Only
oracle/ primitives and numpy matmuls are used; tests/test_oracle_chunked.py
pins both against the whole-tensor oracle functions."""
from __future__ import annotations

import numpy as np

from oracle import fp8 as OF


def xt_dy_fp64(X, dY, chunk: int = 8192) -> np.ndarray:
    """X^T dY in fp64 over every token (dW of eq. back Gi)."""
    acc = np.zeros((X.shape[1], dY.shape[1]))
    for c0 in range(0, X.shape[0], chunk):
        acc += X[c0:c0 + chunk].astype(np.float64).T @ dY[c0:c0 + chunk].astype(np.float64)
    return acc


def dw_fp8_rows(X, dY, chunk: int = 8192) -> np.ndarray:
    """The oracle's FP8 dW, decode(q(X))^T decode(q(dY)) / (sX sD), with each
    scale taken from its whole tensor (a row's codes depend only on that row
    and the scale)."""
    sX = OF.pow2_scale(float(np.max(np.abs(np.asarray(X, np.float32)))))
    sD = OF.pow2_scale(float(np.max(np.abs(np.asarray(dY, np.float32)))))
    acc = np.zeros((X.shape[1], dY.shape[1]))
    for c0 in range(0, X.shape[0], chunk):
        cx = OF.encode((np.asarray(X[c0:c0 + chunk], np.float32) * np.float32(sX)).astype(np.float64))
        cd = OF.encode((np.asarray(dY[c0:c0 + chunk], np.float32) * np.float32(sD)).astype(np.float64))
        acc += OF.decode(cx).T @ OF.decode(cd)
    return acc / (sX * sD)
