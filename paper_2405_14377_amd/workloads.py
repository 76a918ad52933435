"""Seeded synthetic workloads for TTM layers and the TT embedding.

This module only draws random inputs and describes shapes.  It holds none of
the layer arithmetic, so both the CPU oracle's tests and the GPU path may use
it.  Everything is drawn on the host with numpy ``default_rng``; bf16
activations are produced by a single round-to-nearest-even cast of the fp32
draw (torch on the CPU), and the oracle reads exactly those rounded values.

Seeds: ``1000 * workload_id + tensor_id + 100 * layer`` with tensor ids
X = 0, dY = 1, cores 2.., masks 10.., ids 20.

Core scale: with X, cores iid zero mean and 0/1 masks the output variance of a
TTM layer is ``N_in * prod(rho_k) * sigma^(2d)`` (rho_k = active entries on bond
k), so ``sigma = (N_in * prod rho_k) ** (-1 / (2 d))`` gives Var(Y) ~ 1.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np


@dataclass(frozen=True)
class TTMLayerShape:
    """TTM linear layer: cores G_k[r_{k-1}, m_k, n_k, r_k]; Y[b, N_out] = X[b, N_in] W."""
    name: str
    n: Tuple[int, ...]          # input factors, N_in = prod(n)
    m: Tuple[int, ...]          # output factors, N_out = prod(m)
    r: Tuple[int, ...]          # bond ranks, r[0] = r[d] = 1

    @property
    def d(self) -> int:
        return len(self.n)

    @property
    def n_in(self) -> int:
        return int(np.prod(self.n))

    @property
    def n_out(self) -> int:
        return int(np.prod(self.m))

    def core_shapes(self):
        return [(self.r[k], self.m[k], self.n[k], self.r[k + 1]) for k in range(self.d)]


@dataclass(frozen=True)
class TTMWorkload:
    wid: int
    name: str
    layers: Tuple[TTMLayerShape, ...]
    batch: int
    dtypes: Tuple[str, ...]     # activation dtypes to run ("f32", "bf16")
    mask: Tuple                 # ("ones",) | ("bernoulli", p) | ("half",)


@dataclass(frozen=True)
class EmbedWorkload:
    wid: int
    name: str
    v: Tuple[int, ...]          # vocabulary (row) factors
    e: Tuple[int, ...]          # embedding (column) factors
    r: Tuple[int, ...]
    n_tokens: int
    core_std: float
    id_dists: Tuple[str, ...]   # ("zipf1.1", "uniform")


_QKVO = dict(n=(8, 8, 12), m=(12, 8, 8))
_UP = dict(n=(8, 8, 12), m=(16, 16, 12))
_DOWN = dict(n=(16, 16, 12), m=(8, 8, 12))

WORKLOADS = {
    0: TTMWorkload(0, "ttm768x768_d3_r8_b32_f32",
                   (TTMLayerShape("ttm768x768", (8, 8, 12), (12, 8, 8), (1, 8, 8, 1)),),
                   32, ("f32",), ("ones",)),
    1: TTMWorkload(1, "ttm768x3072_d3_r30_b4096",
                   (TTMLayerShape("ffn_up", (8, 8, 12), (16, 16, 12), (1, 30, 30, 1)),),
                   4096, ("f32", "bf16"), ("bernoulli", 0.8)),
    2: TTMWorkload(2, "encoder6_d3_r30_b16384_bf16",
                   tuple(TTMLayerShape(nm, **sh, r=(1, 30, 30, 1)) for nm, sh in
                         (("q", _QKVO), ("k", _QKVO), ("v", _QKVO), ("o", _QKVO),
                          ("ffn_up", _UP), ("ffn_down", _DOWN))),
                   16384, ("bf16",), ("half",)),
    3: EmbedWorkload(3, "ttembed32768x768_d3_r30_b16384", (32, 32, 32), (8, 8, 12),
                     (1, 30, 30, 1), 16384, 0.1, ("zipf1.1", "uniform")),
    4: TTMWorkload(4, "ttm1024x4096_d4_r64_b65536_bf16",
                   (TTMLayerShape("up", (4, 8, 4, 8), (8, 8, 8, 8), (1, 64, 64, 64, 1)),
                    TTMLayerShape("down", (8, 8, 8, 8), (4, 8, 4, 8), (1, 64, 64, 64, 1))),
                   65536, ("bf16",), ("bernoulli", 0.7)),
    # the paper's TT layout (Sec. 4.2): input cores [r, 1, n_k, r] then output
    # cores [r, m_k, 1, r], i.e. a TTM layer with unit modes and a rank-30
    # bond between the input and the output half
    5: TTMWorkload(5, "tt_layout_768x3072_768x768_r30_b4096",
                   (TTMLayerShape("tt_ffn_up", (8, 8, 12, 1, 1, 1), (1, 1, 1, 16, 16, 12), (1,) + (30,) * 5 + (1,)),
                    TTMLayerShape("tt_qkvo", (8, 8, 12, 1, 1, 1), (1, 1, 1, 12, 8, 8), (1,) + (30,) * 5 + (1,))),
                   4096, ("f32", "bf16"), ("bernoulli", 0.8)),
    # the TT shapes of the paper's mixed-precision runtime table (appendix,
    # Tab. LP-time): 1024 -> 4096 as (16, 8, 8 | 16, 16, 16) and 1024 -> 1024
    # as (16, 8, 8 | 8, 8, 16), ranks 32, 40000 tokens
    6: TTMWorkload(6, "tt_layout_1024x4096_1024x1024_r32_b40000",
                   (TTMLayerShape("tt_1024x4096", (16, 8, 8, 1, 1, 1), (1, 1, 1, 16, 16, 16), (1,) + (32,) * 5 + (1,)),
                    TTMLayerShape("tt_1024x1024", (16, 8, 8, 1, 1, 1), (1, 1, 1, 8, 8, 16), (1,) + (32,) * 5 + (1,))),
                   40000, ("bf16",), ("ones",)),
}


def seed_of(wid: int, tensor_id: int, layer: int = 0) -> int:
    return 1000 * wid + tensor_id + 100 * layer


def to_bf16_values(x: np.ndarray) -> np.ndarray:
    """Round fp32 -> bf16 (RNE, via torch on the CPU) and return the values as fp32."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def draw_masks(shape: TTMLayerShape, kind: Tuple, rng: np.random.Generator) -> List[np.ndarray]:
    """Per-bond 0/1 mask vectors D_k (k = 1..d-1), fp32."""
    out = []
    for k in range(1, shape.d):
        rk = shape.r[k]
        if kind[0] == "ones":
            mk = np.ones(rk, np.float32)
        elif kind[0] == "bernoulli":
            mk = (rng.random(rk) < kind[1]).astype(np.float32)
            if mk.sum() == 0:
                mk[rng.integers(rk)] = 1.0
        elif kind[0] == "half":
            mk = np.ones(rk, np.float32)
            mk[rng.permutation(rk)[: rk // 2]] = 0.0
        else:
            raise ValueError(kind)
        out.append(mk)
    return out


def unit_variance_sigma(shape: TTMLayerShape, masks: Sequence[np.ndarray]) -> float:
    rho = [float(np.count_nonzero(mk)) for mk in masks]
    return float((shape.n_in * np.prod(rho)) ** (-1.0 / (2 * shape.d)))


@dataclass
class TTMLayerInputs:
    shape: TTMLayerShape
    cores: List[np.ndarray]
    masks: List[np.ndarray]
    sigma: float


def ttm_layer_inputs(wid: int, layer: int, shape: TTMLayerShape, mask_kind: Tuple) -> TTMLayerInputs:
    mrng = np.random.default_rng(seed_of(wid, 10, layer))
    masks = draw_masks(shape, mask_kind, mrng)
    sigma = unit_variance_sigma(shape, masks)
    cores = []
    for k, cs in enumerate(shape.core_shapes()):
        crng = np.random.default_rng(seed_of(wid, 2 + k, layer))
        cores.append((crng.standard_normal(cs) * sigma).astype(np.float32))
    return TTMLayerInputs(shape, cores, masks, sigma)


def activations(wid: int, batch: int, width: int, tensor_id: int, dtype: str, layer: int = 0,
                rows: Optional[int] = None) -> np.ndarray:
    """X (tensor_id 0) or dY (tensor_id 1) ~ N(0, 1), [batch, width], fp32 values (bf16-rounded if asked)."""
    rng = np.random.default_rng(seed_of(wid, tensor_id, layer))
    x = rng.standard_normal((batch, width), dtype=np.float32)
    if rows is not None:
        x = x[:rows]
    return to_bf16_values(x) if dtype == "bf16" else x


def embed_cores(w: EmbedWorkload, v=None, e=None, r=None, seed_wid=None) -> List[np.ndarray]:
    v = w.v if v is None else v
    e = w.e if e is None else e
    r = w.r if r is None else r
    wid = w.wid if seed_wid is None else seed_wid
    cores = []
    for k in range(len(v)):
        rng = np.random.default_rng(seed_of(wid, 2 + k))
        cores.append((rng.standard_normal((r[k], v[k], e[k], r[k + 1])) * w.core_std).astype(np.float32))
    return cores


def token_ids(n_tokens: int, vocab: int, dist: str, seed: int) -> np.ndarray:
    """int64 ids in [0, vocab).  'zipfS': bounded Zipf p(id) ~ (id+1)^-S, hot ids small; 'uniform'."""
    rng = np.random.default_rng(seed)
    if dist == "uniform":
        return rng.integers(0, vocab, n_tokens, dtype=np.int64)
    if dist.startswith("zipf"):
        s = float(dist[4:])
        p = (np.arange(1, vocab + 1, dtype=np.float64)) ** (-s)
        p /= p.sum()
        return rng.choice(vocab, size=n_tokens, p=p).astype(np.int64)
    raise ValueError(dist)


def random_ttm_shape(rng: np.random.Generator, d: int, max_factor: int = 4, max_rank: int = 4,
                     allow_unit: bool = True) -> TTMLayerShape:
    lo = 1 if allow_unit else 2
    n = tuple(int(rng.integers(lo, max_factor + 1)) for _ in range(d))
    m = tuple(int(rng.integers(lo, max_factor + 1)) for _ in range(d))
    r = (1,) + tuple(int(rng.integers(1, max_rank + 1)) for _ in range(d - 1)) + (1,)
    return TTMLayerShape(f"rand_d{d}", n, m, r)


def random_cores(rng: np.random.Generator, shape: TTMLayerShape, scale: float = 1.0) -> List[np.ndarray]:
    return [(rng.standard_normal(cs) * scale).astype(np.float32) for cs in shape.core_shapes()]


def integer_bond_diagonal_cores(rng: np.random.Generator, n, m, r) -> List[np.ndarray]:
    """Cores with entries in {-1, 0, 1}, the inner ones diagonal in their bond
    (G[a, :, :, c] = 0 for a != c).  Every entry of the dense weight is then a
    sum of at most r_1 products of +-1: an integer of magnitude <= r_1, exact
    in fp32 whatever the contraction order, and exactly representable in FP8
    E4M3 after a power-of-two scaling while r_1 <= 16."""
    d = len(n)
    cores = []
    for k in range(d):
        G = rng.integers(-1, 2, (r[k], m[k], n[k], r[k + 1])).astype(np.float32)
        if 0 < k < d - 1:
            G *= np.eye(r[k], dtype=np.float32)[:, None, None, :]
        cores.append(G)
    return cores
