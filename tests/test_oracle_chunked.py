"""The token-chunked helpers of the full-size parity tests equal the
whole-tensor oracle quantities (CPU)."""
import numpy as np

from oracle import mixed as OM
from tests.chunked import dw_fp8_rows, xt_dy_fp64


def _data(seed, b=300, nin=24, nout=40):
    rng = np.random.default_rng(seed)
    X = (rng.standard_normal((b, nin)) * 3.0).astype(np.float32)
    dY = rng.standard_normal((b, nout)).astype(np.float32)
    X[5, 7] = 100.0          # the amax sits in one chunk only
    return X, dY


def test_xt_dy_chunks_equal_whole():
    X, dY = _data(0)
    ref = X.astype(np.float64).T @ dY.astype(np.float64)
    for chunk in (1, 7, 64, 300, 1000):
        assert np.allclose(xt_dy_fp64(X, dY, chunk), ref, rtol=1e-13, atol=1e-12)


def test_fp8_dw_chunks_equal_whole():
    X, dY = _data(1)
    ref = OM.dW_fp8(X, dY)
    for chunk in (1, 7, 64, 300, 1000):
        got = dw_fp8_rows(X, dY, chunk)
        assert np.allclose(got, ref, rtol=1e-13, atol=1e-12 * np.max(np.abs(ref)))
