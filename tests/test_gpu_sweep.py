"""GPU parity of every contraction order of the Prop. 4.1 family (Sec. 4.2):
each order forced through the planner must give the oracle's Y, dX and every
dG_k.  Covers single-core and multi-core groups, both sweep directions,
unit modes, rank masks with compaction, batches below the planned one, the
768 -> 768 rank-8 layer at 32 tokens (where a sweep does fewer flops than
the dense order) and the paper's TT layout (Sec. 4.2: input cores then
output cores, a rank-r bottleneck) written as a TTM layer with unit modes.

Tolerances as for the dense order: max |gpu - ref| / max |ref| per output
tensor <= 1e-4 (fp32 activations), <= 2e-2 (bf16 activations).
"""
import numpy as np
import pytest

from oracle import ttm as OT
from paper_2405_14377_amd import comera as C
from paper_2405_14377_amd import workloads as wl
from tests.gpu_util import TTMRun, rel_err, to_dev, to_np
from tests.test_gpu_ttm import TOL, _inputs

pytestmark = pytest.mark.gpu


def _all_orders(n, m, r, cores, D, X, dY, act, mask_active=None, b_run=None, orders=None, reuse=False):
    b_plan = X.shape[0]
    b = b_plan if b_run is None else b_run
    Xb, dYb = X[:b], dY[:b]
    Yr = OT.forward_dense(Xb, cores, D)
    dXr, dGr = OT.backward_dense(Xb, dYb, cores, D)
    probe = C.TTMPlan(n, m, r, C.BF16 if act == "bf16" else C.F32, batch=b_plan, mask_active=mask_active)
    idx = range(probe.num_orders) if orders is None else orders
    bad, seen = {}, 0
    for i in idx:
        info = probe.order_info(i)
        if not info["executable"]:
            continue
        seen += 1
        print(f"order {i} {info['desc']} b={b} act={act}", flush=True)
        run = TTMRun(n, m, r, cores, D, b_plan, act, mask_active=mask_active, force_order=i, reuse=reuse)
        Xt, dYt = to_dev(Xb, act), to_dev(dYb, act)
        Y = to_np(run.forward(Xt, b=b))
        dX, dG = run.backward(Xt, dYt, b=b)
        errs = {"Y": rel_err(Y, Yr), "dX": rel_err(to_np(dX), dXr)}
        for k in range(len(n)):
            errs[f"dG{k}"] = rel_err(to_np(dG[k]), dGr[k])
        worst = {k: v for k, v in errs.items() if not v <= TOL[act]}
        if worst:
            bad[info["desc"]] = worst
    assert seen > 0
    assert not bad, bad


SHAPES = [
    # (seed, n, m, r, b)
    (21, (4, 3), (2, 5), (1, 3, 1), 9),
    (22, (3, 5, 11), (7, 2, 13), (1, 4, 3, 1), 150),         # ragged in every dim
    (23, (1, 8, 1), (6, 1, 9), (1, 5, 2, 1), 70),            # unit modes
    (24, (2, 3, 2, 3), (3, 2, 4, 2), (1, 3, 4, 2, 1), 65),   # d = 4: 15 orders
    (25, (8, 8, 12), (12, 8, 8), (1, 8, 8, 1), 33),
]


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", SHAPES, ids=[f"s{c[0]}" for c in SHAPES])
def test_every_order(case, act):
    seed, n, m, r, b = case
    cores, D, X, dY = _inputs(seed, n, m, r, b, act)
    _all_orders(n, m, r, cores, D, X, dY, act)


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("case", SHAPES, ids=[f"s{c[0]}" for c in SHAPES])
def test_every_order_reusing_forward(case, act):
    """Backward calls that take the group matrices and activation states the
    forward left in the workspace: the oracle's results for every order, and
    bit for bit the rebuilding route's."""
    seed, n, m, r, b = case
    cores, D, X, dY = _inputs(seed, n, m, r, b, act)
    _all_orders(n, m, r, cores, D, X, dY, act, reuse=True)
    probe = C.TTMPlan(n, m, r, C.BF16 if act == "bf16" else C.F32, batch=b)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    for i in range(probe.num_orders):
        if not probe.order_info(i)["executable"]:
            continue
        outs = []
        for reuse in (False, True):
            run = TTMRun(n, m, r, cores, D, b, act, force_order=i, reuse=reuse)
            Y = run.forward(Xt)
            dX, dG = run.backward(Xt, dYt)
            outs.append([Y, dX] + dG)
        for a, c in zip(*outs):
            assert np.array_equal(to_np(a), to_np(c)), i


def test_every_order_compacted_masks_smaller_batch():
    """Inactive mask entries removed by the plan, and a call with fewer
    tokens than planned."""
    n, m, r = (3, 4, 5), (5, 2, 6), (1, 6, 7, 1)
    rng = np.random.default_rng(26)
    cores, _, X, dY = _inputs(26, n, m, r, 120, "f32", masks=None)
    act1 = (rng.random(6) < 0.6).astype(np.uint8); act1[0] = 1
    act2 = (rng.random(7) < 0.6).astype(np.uint8); act2[-1] = 1
    D = [act1.astype(np.float32) * rng.uniform(0.5, 1.5, 6).astype(np.float32),
         act2.astype(np.float32) * rng.uniform(0.5, 1.5, 7).astype(np.float32)]
    _all_orders(n, m, r, cores, D, X, dY, "f32", mask_active=list(act1) + list(act2), b_run=47)


def test_low_rank_layer_all_orders():
    """768 -> 768, ranks (1, 8, 8, 1), 32 tokens, fp32: every order in full."""
    w = wl.WORKLOADS[0]
    sh = w.layers[0]
    inp = wl.ttm_layer_inputs(0, 0, sh, w.mask)
    X = wl.activations(0, w.batch, sh.n_in, 0, "f32", layer=0)
    dY = wl.activations(0, w.batch, sh.n_out, 1, "f32", layer=0)
    mask_active = [int(x != 0) for mk in inp.masks for x in mk]
    _all_orders(sh.n, sh.m, sh.r, inp.cores, inp.masks, X, dY, "f32", mask_active=mask_active)


@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_paper_tt_layout(act):
    """The paper's TT layout for a 768 x 3072 weight at rank 30: three input
    cores [r, 1, n_k, r] then three output cores [r, m_k, 1, r]; the planner
    picks the left-to-right sweep over the groups (inputs)(outputs), i.e.
    T = X A, Y = T B with the rank-30 bottleneck T."""
    n = (8, 8, 12, 1, 1, 1)
    m = (1, 1, 1, 16, 16, 12)
    r = (1, 30, 30, 30, 30, 30, 1)
    cores, D, X, dY = _inputs(27, n, m, r, 512, act)
    p = C.TTMPlan(n, m, r, C.BF16 if act == "bf16" else C.F32, batch=512)
    assert p.order_info(p.chosen)["desc"] == "sweep-lr [0,1,2][3,4,5]"
    _all_orders(n, m, r, cores, D, X, dY, act, orders=[p.chosen, 0])


@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_paper_mixed_precision_table_tt_shape(act):
    """The TT shape of the appendix's runtime table, 1024 x 4096 as
    (16, 8, 8 | 16, 16, 16) at rank 32, with 2048 tokens: the sweep's
    products have a side of 32 against K up to 4096 (split over K, skinny
    tiles), and its meets have 32 rows against 2048 tokens."""
    n = (16, 8, 8, 1, 1, 1)
    m = (1, 1, 1, 16, 16, 16)
    r = (1, 32, 32, 32, 32, 32, 1)
    cores, D, X, dY = _inputs(29, n, m, r, 2048, act)
    p = C.TTMPlan(n, m, r, C.BF16 if act == "bf16" else C.F32, batch=2048)
    assert p.order_info(p.chosen)["desc"] == "sweep-lr [0,1,2][3,4,5]"
    _all_orders(n, m, r, cores, D, X, dY, act, orders=[p.chosen])


def test_sweep_backward_partial_outputs():
    """dX only, dG only, and a subset of dG for a sweep order."""
    import torch
    n, m, r = (3, 4, 5), (4, 3, 6), (1, 5, 4, 1)
    cores, D, X, dY = _inputs(28, n, m, r, 90, "f32")
    probe = C.TTMPlan(n, m, r, batch=90)
    descs = [probe.order_info(i)["desc"] for i in range(probe.num_orders)]
    dXr, dGr = OT.backward_dense(X, dY, cores, D)
    for desc in ("sweep-rl [0][1][2]", "sweep-lr [0][1,2]"):
        run = TTMRun(n, m, r, cores, D, 90, "f32", force_order=descs.index(desc))
        Xt, dYt = to_dev(X), to_dev(dY)
        dX, _ = run.backward(Xt, dYt, want_dg=False)
        assert rel_err(to_np(dX), dXr) <= 1e-4, desc
        _, dG = run.backward(Xt, dYt, want_dx=False)
        for k in range(3):
            assert rel_err(to_np(dG[k]), dGr[k]) <= 1e-4, (desc, k)
        dG1 = [None, torch.empty_like(run.G[1]), None]
        C.comera_ttm_backward(run.plan.handle, 90, Xt, dYt, run.G, run.D, None, dG1, run.ws)
        assert rel_err(to_np(dG1[1]), dGr[1]) <= 1e-4, desc


def test_sweep_backward_bitwise_deterministic():
    import torch
    n, m, r = (8, 8, 12), (12, 8, 8), (1, 8, 8, 1)
    cores, D, X, dY = _inputs(29, n, m, r, 256, "bf16")
    probe = C.TTMPlan(n, m, r, C.BF16, batch=256)
    i = [probe.order_info(j)["desc"] for j in range(probe.num_orders)].index("sweep-rl [0][1][2]")
    run = TTMRun(n, m, r, cores, D, 256, "bf16", force_order=i)
    Xt, dYt = to_dev(X, "bf16"), to_dev(dY, "bf16")
    dX1, dG1 = run.backward(Xt, dYt)
    dX2, dG2 = run.backward(Xt, dYt)
    assert torch.equal(dX1, dX2)
    for a, b in zip(dG1, dG2):
        assert torch.equal(a, b)


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("b", [1, 513, 1537, 5000])
def test_fused_order_token_groups(b, act):
    """The fused single-core sweep with more tokens than workgroups (the
    backward keeps at most 512 workgroups, each summing its token groups'
    meets into its own partial in order; above 1024 tokens the forward takes
    several tokens per workgroup): the oracle's Y, dX and every dG_k, and a
    second backward bit for bit equal to the first."""
    import torch
    n, m, r = (3, 4, 2), (2, 5, 3), (1, 5, 4, 1)
    cores, D, X, dY = _inputs(40 + b, n, m, r, b, act)
    probe = C.TTMPlan(n, m, r, C.BF16 if act == "bf16" else C.F32, batch=b)
    last = probe.num_orders - 1
    assert probe.order_info(last)["kind"] == C.ORDER_FUSED_RL and probe.order_info(last)["executable"]
    _all_orders(n, m, r, cores, D, X, dY, act, orders=[last])
    run = TTMRun(n, m, r, cores, D, b, act, force_order=last)
    Xt, dYt = to_dev(X, act), to_dev(dY, act)
    dX1, dG1 = run.backward(Xt, dYt)
    dX2, dG2 = run.backward(Xt, dYt)
    assert torch.equal(dX1, dX2)
    for g1, g2 in zip(dG1, dG2):
        assert torch.equal(g1, g2)
