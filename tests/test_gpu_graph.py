"""HIP-graph capture of a whole training step (TTM forward + backward, and
the embedding lookup forward + backward), the analogue of the CUDA-graph
execution of Sec. 4.3: every replay must reproduce the eager results bit
for bit.  Between replays the program does its own eager work (new inputs
copied into the captured buffers, eager calls of the same plan on another
workspace) and synchronises, and every replay is checked."""
import numpy as np
import pytest

from oracle import ttm as OT
from paper_2405_14377_amd import comera as C
from paper_2405_14377_amd import workloads as wl
from tests.gpu_util import EmbedRun, TTMRun, rel_err, to_dev, to_np

pytestmark = pytest.mark.gpu


def _ttm_inputs(seed, n, m, r, b, act, sets):
    rng = np.random.default_rng(seed)
    shape = wl.TTMLayerShape("g", tuple(n), tuple(m), tuple(r))
    d = len(n)
    sig = (shape.n_in * np.prod(r[1:-1])) ** (-1.0 / (2 * d))
    cores = [(c * sig).astype(np.float32) for c in wl.random_cores(rng, shape)]
    D = [rng.uniform(0.5, 1.5, r[k + 1]).astype(np.float32) for k in range(d - 1)]
    xs = []
    for _ in range(sets):
        X = rng.standard_normal((b, shape.n_in)).astype(np.float32)
        dY = rng.standard_normal((b, shape.n_out)).astype(np.float32)
        if act == "bf16":
            X, dY = wl.to_bf16_values(X), wl.to_bf16_values(dY)
        xs.append((X, dY))
    return cores, D, xs


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("reuse", [False, True])
@pytest.mark.parametrize("case", [((4, 6, 5), (3, 7, 4), (1, 6, 5, 1), 200, -1),
                                  ((8, 8, 12), (12, 8, 8), (1, 8, 8, 1), 32, -1),
                                  ((3, 4, 5), (5, 2, 6), (1, 3, 4, 1), 64, 1)],
                         ids=["dense", "w0", "sweep"])
def test_ttm_step_graph_replays(case, reuse, act):
    import torch
    n, m, r, b, order = case
    cores, D, xs = _ttm_inputs(31, n, m, r, b, act, 3)
    run = TTMRun(n, m, r, cores, D, b, act, force_order=order, reuse=reuse)
    ref_run = TTMRun(n, m, r, cores, D, b, act, force_order=order, reuse=reuse)
    Xs, dYs = to_dev(xs[0][0], act), to_dev(xs[0][1], act)
    Ys = torch.empty((b, run.n_out), dtype=run.tdt, device="cuda")
    dXs = torch.empty((b, run.n_in), dtype=run.tdt, device="cuda")
    dGs = [torch.empty_like(g) for g in run.G]

    def step():
        C.comera_ttm_forward(run.plan.handle, b, Xs, run.G, run.D, Ys, run.ws)
        C.comera_ttm_backward(run.plan.handle, b, Xs, dYs, run.G, run.D, dXs, dGs, run.ws)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            step()
        torch.cuda.synchronize()
        for rep in range(2):
            for X, dY in xs:
                Xt, dYt = to_dev(X, act), to_dev(dY, act)
                # eager reference on its own workspace, then the replay
                Yr = ref_run.forward(Xt)
                dXr, dGr = ref_run.backward(Xt, dYt)
                torch.cuda.synchronize()
                Xs.copy_(Xt)
                dYs.copy_(dYt)
                g.replay()
                torch.cuda.synchronize()
                assert torch.equal(Ys, Yr), rep
                assert torch.equal(dXs, dXr), rep
                for a, c in zip(dGs, dGr):
                    assert torch.equal(a, c), rep
        # the last replay also matches the oracle
        X, dY = xs[-1]
        tol = 1e-4 if act == "f32" else 2e-2
        assert rel_err(to_np(Ys), OT.forward_dense(X, cores, D)) <= tol
        dXo, dGo = OT.backward_dense(X, dY, cores, D)
        assert rel_err(to_np(dXs), dXo) <= tol
        for a, c in zip(dGs, dGo):
            assert rel_err(to_np(a), c) <= tol
    del g


def test_embed_step_graph_replays():
    import torch
    v, e, r = (4, 5, 6), (2, 3, 4), (1, 3, 4, 1)
    rng = np.random.default_rng(32)
    cores = [(0.3 * rng.standard_normal((r[k], v[k], e[k], r[k + 1]))).astype(np.float32) for k in range(3)]
    n = 300
    V, E = int(np.prod(v)), int(np.prod(e))
    ids_sets = [rng.integers(0, V, n), rng.zipf(1.5, n) % V, np.full(n, 7)]
    dY_sets = [rng.standard_normal((n, E)).astype(np.float32) for _ in ids_sets]
    run = EmbedRun(v, e, r, cores, None, n)
    ref = EmbedRun(v, e, r, cores, None, n)
    ids_s = run.ids_dev(ids_sets[0])
    dY_s = to_dev(dY_sets[0])
    Y_s = torch.empty((n, E), device="cuda")
    dG_s = [torch.empty_like(g) for g in run.G]

    def step():
        C.comera_tt_embed_forward(run.shape, ids_s, n, run.G, None, Y_s, run.ws, run.err)
        C.comera_tt_embed_backward(run.shape, ids_s, n, dY_s, run.G, None, dG_s, 1, run.ws, run.err)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            step()
        torch.cuda.synchronize()
        for rep in range(2):
            for ids, dY in zip(ids_sets, dY_sets):
                it, dYt = ref.ids_dev(ids), to_dev(dY)
                Yr = ref.forward(it)
                dGr = ref.backward(it, dYt)
                torch.cuda.synchronize()
                ids_s.copy_(it)
                dY_s.copy_(dYt)
                g.replay()
                torch.cuda.synchronize()
                assert torch.equal(Y_s, Yr), rep
                for a, c in zip(dG_s, dGr):
                    assert torch.equal(a, c), rep
    assert int(run.err.item()) == 0
    del g


@pytest.mark.parametrize("reuse", [False, True])
@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_fp8_step_graph_replays(act, reuse):
    """The mixed-precision layer (FP8 products): the quantisers write their
    scales into the workspace on every call, so replays with new inputs must
    match eager calls bit for bit."""
    import torch
    n, m, r, b = (8, 8, 12), (12, 8, 8), (1, 8, 8, 1), 300
    cores, D, xs = _ttm_inputs(33, n, m, r, b, act, 3)
    run = TTMRun(n, m, r, cores, D, b, act, force_order=0, reuse=reuse, fp8=True)
    ref_run = TTMRun(n, m, r, cores, D, b, act, force_order=0, reuse=reuse, fp8=True)
    Xs, dYs = to_dev(xs[0][0], act), to_dev(xs[0][1], act)
    Ys = torch.empty((b, run.n_out), dtype=run.tdt, device="cuda")
    dXs = torch.empty((b, run.n_in), dtype=run.tdt, device="cuda")
    dGs = [torch.empty_like(g) for g in run.G]

    def step():
        C.comera_ttm_forward(run.plan.handle, b, Xs, run.G, run.D, Ys, run.ws)
        C.comera_ttm_backward(run.plan.handle, b, Xs, dYs, run.G, run.D, dXs, dGs, run.ws)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            step()
        torch.cuda.synchronize()
        for rep in range(2):
            for X, dY in xs:
                Xt, dYt = to_dev(X, act), to_dev(dY, act)
                Yr = ref_run.forward(Xt)
                dXr, dGr = ref_run.backward(Xt, dYt)
                torch.cuda.synchronize()
                Xs.copy_(Xt)
                dYs.copy_(dYt)
                g.replay()
                torch.cuda.synchronize()
                assert torch.equal(Ys, Yr), rep
                assert torch.equal(dXs, dXr), rep
                for a, c in zip(dGs, dGr):
                    assert torch.equal(a, c), rep
    del g


def test_model_step_graph_replays():
    """One graph for a whole model-shaped step (Sec. 4.3): the 32768 x 768
    TT embedding, then the six TTM layers of the encoder workload (q, k, v
    read the embedded rows in bf16, o reads v, the feed-forward pair reads
    o), their backward in reverse, the input gradients of q, k and v summed
    into the embedding's dY, and the embedding backward.  The layers keep
    the workload's cores and masks at 2048 tokens.  Every replay (three
    input sets, twice each, with eager work between) must equal the same
    sequence run eagerly on other workspaces, bit for bit; the last replay's
    embedding gradient is also checked against the oracle."""
    import torch
    from oracle import embed as OE
    b = 2048
    enc = wl.WORKLOADS[2]
    ew = wl.WORKLOADS[3]
    rng = np.random.default_rng(41)
    ecores = wl.embed_cores(ew)
    V = int(np.prod(ew.v))

    def layers():
        out = []
        for li, sh in enumerate(enc.layers):
            inp = wl.ttm_layer_inputs(2, li, sh, enc.mask)
            active = [int(x != 0) for mk in inp.masks for x in mk]
            out.append((sh, TTMRun(sh.n, sh.m, sh.r, inp.cores, inp.masks, b, "bf16", mask_active=active,
                                   reuse=True)))
        return out

    def model(L, emb, bufs):
        (ids, dYq, dYk, dYd), o = bufs["in"], bufs["out"]
        C.comera_tt_embed_forward(emb.shape, ids, b, emb.G, None, o["Ye"], emb.ws, emb.err)
        o["X0"].copy_(o["Ye"])
        names = [sh.name for sh, _ in L]
        run = dict(zip(names, [r for _, r in L]))
        fwd = [("q", "X0", "Yq"), ("k", "X0", "Yk"), ("v", "X0", "Yv"), ("o", "Yv", "Yo"),
               ("ffn_up", "Yo", "Yu"), ("ffn_down", "Yu", "Yd")]
        for nm, xi, yo in fwd:
            C.comera_ttm_forward(run[nm].plan.handle, b, o[xi], run[nm].G, run[nm].D, o[yo], run[nm].ws)
        bwd = [("ffn_down", "Yu", dYd, "dYu"), ("ffn_up", "Yo", "dYu", "dYo"), ("o", "Yv", "dYo", "dYv"),
               ("v", "X0", "dYv", "dXv"), ("k", "X0", dYk, "dXk"), ("q", "X0", dYq, "dXq")]
        for nm, xi, dy, dx in bwd:
            dyt = o[dy] if isinstance(dy, str) else dy
            C.comera_ttm_backward(run[nm].plan.handle, b, o[xi], dyt, run[nm].G, run[nm].D, o[dx],
                                  o["dG_" + nm], run[nm].ws)
        o["dYe"].copy_(o["dXq"])
        o["dYe"].add_(o["dXk"])
        o["dYe"].add_(o["dXv"])
        C.comera_tt_embed_backward(emb.shape, ids, b, o["dYe"], emb.G, None, o["dGe"], 1, emb.ws, emb.err)

    def buffers(L, emb):
        dev, bf = "cuda", torch.bfloat16
        o = {"Ye": torch.empty((b, emb.E), device=dev), "dYe": torch.empty((b, emb.E), device=dev),
             "X0": torch.empty((b, emb.E), dtype=bf, device=dev),
             "dGe": [torch.empty_like(g) for g in emb.G]}
        for nm, width in (("Yq", 768), ("Yk", 768), ("Yv", 768), ("Yo", 768), ("Yu", 3072), ("Yd", 768),
                          ("dYu", 3072), ("dYo", 768), ("dYv", 768), ("dXv", 768), ("dXk", 768), ("dXq", 768)):
            o[nm] = torch.empty((b, width), dtype=bf, device=dev)
        for sh, r in L:
            o["dG_" + sh.name] = [torch.empty_like(g) for g in r.G]
        return o

    def draw():
        ids = wl.token_ids(b, V, "zipf1.1", int(rng.integers(1 << 30)))
        return (ids, wl.to_bf16_values(rng.standard_normal((b, 768)).astype(np.float32)),
                wl.to_bf16_values(rng.standard_normal((b, 768)).astype(np.float32)),
                wl.to_bf16_values(rng.standard_normal((b, 768)).astype(np.float32)))

    def upload(emb, s):
        ids, dq, dk, dd = s
        return emb.ids_dev(ids), to_dev(dq, "bf16"), to_dev(dk, "bf16"), to_dev(dd, "bf16")

    L, Lr = layers(), layers()
    emb, embr = EmbedRun(ew.v, ew.e, ew.r, ecores, None, b), EmbedRun(ew.v, ew.e, ew.r, ecores, None, b)
    sets = [draw() for _ in range(3)]
    cap = {"in": upload(emb, sets[0]), "out": buffers(L, emb)}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        model(L, emb, cap)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            model(L, emb, cap)
        torch.cuda.synchronize()
        for rep in range(2):
            for s in sets:
                ref = {"in": upload(embr, s), "out": buffers(Lr, embr)}
                model(Lr, embr, ref)
                torch.cuda.synchronize()
                for dst, src in zip(cap["in"], ref["in"]):
                    dst.copy_(src)
                g.replay()
                torch.cuda.synchronize()
                for k, v in ref["out"].items():
                    got = cap["out"][k]
                    if isinstance(v, list):
                        for a, c in zip(got, v):
                            assert torch.equal(a, c), (rep, k)
                    else:
                        assert torch.equal(got, v), (rep, k)
    assert int(emb.err.item()) == 0
    ids = sets[-1][0]
    dGo = OE.backward(ids, to_np(cap["out"]["dYe"]).astype(np.float64), ecores)
    for a, c in zip(cap["out"]["dGe"], dGo):
        assert rel_err(to_np(a), c) <= 1e-4
    del g
