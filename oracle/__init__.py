"""CPU fp64 oracle for TTM linear layers and the TT/TTM embedding.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke entry point and the
benchmark's CPU-baseline leg may import this package.  The product path (the
HIP library and its Python binding) never calls it and shares no code with it.

Everything here is plain numpy in float64, written from the paper's
definitions (tensor-train-matrix format, eq. TTM; rank-masked cores,
eq. Wcompress; the linear layer and its gradients, eq. forward / eq. back Gi /
eq. back X of Sec. 4.2; the TTM embedding lookup of Sec. 4.1).  Each pairwise
contraction is one library call (numpy einsum / tensordot / matmul); there is
no blocking, fusion or reordering beyond what the definition states.

Pins (tests marked ``not gpu``): explicit index sums on tiny shapes, the
Kronecker special case (all ranks 1), d = 1 as a plain matmul, central finite
differences, the rank-mask deletion invariant, inner-product identities, and
the paper's own large-batch path (Alg. path, eq. path-T1 .. path-gGi<d) on the
unit-mode TT layout.  No function in this package is "parity unpinned".
"""
from . import ttm, embed, fp8, mixed, regularizer  # noqa: F401
