"""fp64 oracle of the mixed-precision TTM layer (test infrastructure only).

The appendix on mixed-precision CoMERA splits the contractions of a training
step by whether they carry the batch index: those that do run in a low
precision (FP8 in its runtime table), the batch-free ones in full precision.
On the dense order of Sec. 4.2 the batch contractions are the three products

    Y = X W,   dX = dY W^T,   dW = X^T dY,

and everything else (building W from the cores, projecting dW onto the
cores, the rank-mask gradients) is batch-free.  Readings used here (the
appendix fixes neither the format, the scaling nor which operand copy is
quantised):

* each product reads OCP E4M3 codes of both operands, one power-of-two scale
  per tensor (oracle.fp8.quantize); the three tensors quantised are X, dY and
  W, each once per step;
* W is the fp64 dense weight rounded to fp32 (the precision the layer holds
  it in) before it is quantised;
* a product is the exact sum of the decoded codes' products, divided by the
  two scales;
* dG_k and dD_k are the full-precision functions of that dW (project_dW, and
  the mask-gradient definition of oracle.ttm).

Pinned in tests/test_oracle_mixed.py: exact agreement with the full-precision
layer when every quantised tensor is representable, elementwise error bounds
from the E4M3 rounding bound, and the mask-gradient homogeneity identity.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

from . import fp8
from . import ttm


def quantized_weight(cores, masks=None) -> Tuple[np.ndarray, float]:
    """(E4M3 codes of W [N_in, N_out], scale) with W rounded to fp32 first."""
    W32 = ttm.dense_weight(cores, masks).astype(np.float32)
    return fp8.quantize(W32)


def forward_fp8(X, cores, masks=None) -> np.ndarray:
    """Y = X W with both operands as E4M3 codes (fp64 result)."""
    cW, sW = quantized_weight(cores, masks)
    cX, sX = fp8.quantize(X)
    return (fp8.decode(cX) @ fp8.decode(cW)) / (sX * sW)


def dW_fp8(X, dY) -> np.ndarray:
    """dW = X^T dY with both operands as E4M3 codes (fp64 result)."""
    cX, sX = fp8.quantize(X)
    cD, sD = fp8.quantize(dY)
    return (fp8.decode(cX).T @ fp8.decode(cD)) / (sX * sD)


def backward_fp8(X, dY, cores, masks=None) -> Tuple[np.ndarray, List[np.ndarray]]:
    """dX = dY W^T on codes of dY and W; dG_k projected from the FP8 dW in fp64."""
    cW, sW = quantized_weight(cores, masks)
    cD, sD = fp8.quantize(dY)
    dX = (fp8.decode(cD) @ fp8.decode(cW).T) / (sD * sW)
    return dX, ttm.project_dW(dW_fp8(X, dY), cores, masks)


def mask_grads_fp8(X, dY, cores, masks=None) -> List[np.ndarray]:
    """dD_k[c] = <dW, dW/dD_k[c]> with the FP8 dW."""
    return ttm.mask_grads_from_dW(dW_fp8(X, dY), cores, masks)


def rows_fp8(A, rows, B_codes, sB: float) -> np.ndarray:
    """Rows `rows` of (A quantised as a whole tensor) @ decode(B_codes) / sB:
    the scale of A comes from all of A, the codes only for the rows asked
    for (sampled checks of large products)."""
    A32 = np.asarray(A, dtype=np.float32)
    sA = fp8.pow2_scale(float(np.max(np.abs(A32))) if A32.size else 0.0)
    cA = fp8.encode((A32[rows] * np.float32(sA)).astype(np.float64))
    return (fp8.decode(cA) @ fp8.decode(B_codes)) / (sA * sB)
