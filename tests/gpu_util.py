"""Helpers for the GPU parity tests: run the HIP library through its C ABI
on seeded inputs and return numpy arrays.  No arithmetic of the method lives
here; the expected values come from ``oracle/``."""
from __future__ import annotations

import numpy as np

from paper_2405_14377_amd import comera as C


def torch_dev():
    import torch
    return torch, torch.device("cuda", 0)


def rel_err(got, ref) -> float:
    """max |got - ref| / max |ref| over one output tensor."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    if scale == 0.0:
        return float(np.max(np.abs(got))) if got.size else 0.0
    return float(np.max(np.abs(got - ref)) / scale)


def to_dev(x, dtype="f32"):
    torch, dev = torch_dev()
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32)))
    t = t.to(dev)
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t


def to_np(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


class TTMRun:
    """Plan + device buffers for one TTM layer."""

    def __init__(self, n, m, r, cores, masks, b, act="f32", mask_active=None, force_order=-1, reuse=False,
                 fp8=False):
        torch, dev = torch_dev()
        self.act = act
        self.b = b
        self.plan = C.TTMPlan(n, m, r, C.BF16 if act == "bf16" else C.F32, batch=b, mask_active=mask_active,
                              force_order=force_order)
        if reuse:
            self.plan.set_reuse_forward(True)
        if fp8:
            self.plan.set_fp8(True)
        self.G = [to_dev(c) for c in cores]
        self.D = None if masks is None else [to_dev(mk) for mk in masks]
        self.ws = torch.empty(max(self.plan.workspace_bytes, 1), dtype=torch.uint8, device=dev)
        self.n_in = int(np.prod(n))
        self.n_out = int(np.prod(m))
        self.tdt = torch.bfloat16 if act == "bf16" else torch.float32

    def forward(self, X, b=None):
        torch, dev = torch_dev()
        b = self.b if b is None else b
        Y = torch.empty((b, self.n_out), dtype=self.tdt, device=dev)
        C.comera_ttm_forward(self.plan.handle, b, X, self.G, self.D, Y, self.ws)
        return Y

    def backward(self, X, dY, b=None, want_dx=True, want_dg=True):
        torch, dev = torch_dev()
        b = self.b if b is None else b
        dX = torch.empty((b, self.n_in), dtype=self.tdt, device=dev) if want_dx else None
        dG = [torch.empty_like(g) for g in self.G] if want_dg else None
        C.comera_ttm_backward(self.plan.handle, b, X, dY, self.G, self.D, dX, dG, self.ws)
        return dX, dG


    def backward_masks(self, X, dY, b=None, want_dx=True, want_dg=True):
        torch, dev = torch_dev()
        b = self.b if b is None else b
        dX = torch.empty((b, self.n_in), dtype=self.tdt, device=dev) if want_dx else None
        dG = [torch.empty_like(g) for g in self.G] if want_dg else None
        dD = [torch.empty(self.G[k].shape[3], dtype=torch.float32, device=dev) for k in range(len(self.G) - 1)]
        C.comera_ttm_backward_masks(self.plan.handle, b, X, dY, self.G, self.D, dX, dG, dD, self.ws)
        return dX, dG, dD


class EmbedRun:
    def __init__(self, v, e, r, cores, masks, n_tokens):
        torch, dev = torch_dev()
        self.shape = C.tt_embed_shape(v, e, r)
        self.n = n_tokens
        self.E = int(np.prod(e))
        self.G = [to_dev(c) for c in cores]
        self.D = None if masks is None else [to_dev(mk) for mk in masks]
        self.ws = torch.empty(max(C.comera_tt_embed_workspace_bytes(self.shape, n_tokens), 1), dtype=torch.uint8,
                              device=dev)
        self.err = torch.zeros(1, dtype=torch.int32, device=dev)

    def ids_dev(self, ids):
        torch, dev = torch_dev()
        return torch.from_numpy(np.asarray(ids, np.int64)).to(dev)

    def forward(self, ids_t):
        torch, dev = torch_dev()
        Y = torch.empty((self.n, self.E), dtype=torch.float32, device=dev)
        C.comera_tt_embed_forward(self.shape, ids_t, self.n, self.G, self.D, Y, self.ws, self.err)
        return Y

    def backward_ex(self, ids_t, dY_t, flags):
        dG = [torch_dev()[0].empty_like(g) for g in self.G]
        C.comera_tt_embed_backward_ex(self.shape, ids_t, self.n, dY_t, self.G, self.D, dG, flags, self.ws, self.err)
        return dG

    def backward(self, ids_t, dY_t, deterministic=1):
        dG = [torch_dev()[0].empty_like(g) for g in self.G]
        C.comera_tt_embed_backward(self.shape, ids_t, self.n, dY_t, self.G, self.D, dG, deterministic, self.ws,
                                   self.err)
        return dG
