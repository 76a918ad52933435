#!/usr/bin/env python3
"""Throughput of the TTM-layer hot path on one MI355X.

A step is one pass of the whole path over one batch: forward Y = X W and
backward dX = dY W^T plus every dG_k, through the C ABI, for the largest
configuration: the TTM pair 1024 -> 4096 and 4096 -> 1024 (d = 4, factors
(4, 8, 4, 8) / (8, 8, 8, 8), ranks (1, 64, 64, 64, 1), Bernoulli(0.7) rank
masks, 65536 tokens, bf16 activations with fp32 accumulation), both layers
per step.  Plans are made once, outside the timed region.  Beside it: the
dense GEMM baseline, the roofline of the dominant kernel, the 768 -> 3072
layer (fp32 and bf16), the other workloads, the FP8 layers and the CPU
oracle.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "TT-layer fwd+bwd tokens/s; % of MFMA or HBM roofline; speedup vs dense GEMM"
PEAK = {"f32": 157.3e12, "bf16": 2.5e15}
HBM_PEAK = 8.0e12
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SRCS = [os.path.join(ROOT, "paper_2405_14377_amd", "csrc", f) for f in ("gemm.hip", "api_ttm.hip")]
EMBED_SRCS = [os.path.join(ROOT, "paper_2405_14377_amd", "csrc", f) for f in ("embed_kernels.hip", "api_embed.hip")]
HEADLINE_WID = 4              # the 1024 <-> 4096 d4 r64 pair, 65536 tokens, bf16
COPY_BYTES = 1 << 28          # plain device copy used to scale the HBM byte counters


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# ------------------------------------------------------------------ inputs
def layer_inputs(wid, li, act, gen_seed):
    """Cores/masks from the seeded workload recipe; activations drawn on the device."""
    import numpy as np
    import torch
    from paper_2405_14377_amd import workloads as wl
    w = wl.WORKLOADS[wid]
    sh = w.layers[li]
    inp = wl.ttm_layer_inputs(wid, li, sh, w.mask)
    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(gen_seed)
    tdt = torch.bfloat16 if act == "bf16" else torch.float32
    X = torch.randn((w.batch, sh.n_in), generator=g, device=dev, dtype=torch.float32).to(tdt)
    dY = torch.randn((w.batch, sh.n_out), generator=g, device=dev, dtype=torch.float32).to(tdt)
    G = [torch.from_numpy(c).to(dev) for c in inp.cores]
    D = [torch.from_numpy(mk).to(dev) for mk in inp.masks]
    mask_active = [int(x != 0) for mk in inp.masks for x in mk]
    return sh, inp, X, dY, G, D, mask_active, w.batch


class Layer:
    def __init__(self, sh, X, dY, G, D, mask_active, b, act, force_order=-1, fp8=False):
        import torch
        from paper_2405_14377_amd import comera as C
        self.C = C
        self.sh, self.X, self.dY, self.G, self.D, self.b, self.act = sh, X, dY, G, D, b, act
        self.plan = C.TTMPlan(sh.n, sh.m, sh.r, C.BF16 if act == "bf16" else C.F32, batch=b,
                              mask_active=mask_active, force_order=0 if fp8 else force_order)
        # a training step: the backward follows the forward on the same
        # workspace and cores, so it takes the forward's W and core copies
        self.plan.set_reuse_forward(True)
        if fp8:
            self.plan.set_fp8(True)
        dev = X.device
        self.ws = torch.empty(self.plan.workspace_bytes, dtype=torch.uint8, device=dev)
        self.Y = torch.empty((b, sh.n_out), dtype=X.dtype, device=dev)
        self.dX = torch.empty((b, sh.n_in), dtype=X.dtype, device=dev)
        self.dG = [torch.empty_like(g) for g in G]

    # every call goes to the caller's current stream
    def forward(self):
        self.C.comera_ttm_forward(self.plan.handle, self.b, self.X, self.G, self.D, self.Y, self.ws, None)

    def backward(self):
        self.C.comera_ttm_backward(self.plan.handle, self.b, self.X, self.dY, self.G, self.D, self.dX, self.dG,
                                   self.ws, None)

    def step(self):
        self.forward()
        self.backward()


def time_loop(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return e0.elapsed_time(e1) / steps, wall


def graph_loop(fn, steps, warmup):
    """Capture one call of fn as a HIP graph on the current stream and time
    `steps` replays of it (after `warmup` replays).  Returns (ms per replay,
    None) or (None, reason) when the capture fails."""
    import torch
    s = torch.cuda.current_stream()
    fn()                      # lazy initialisation happens outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    try:
        with torch.cuda.graph(g, stream=s):
            fn()
    except Exception as e:   # reported, never silently replaced by the eager time
        return None, f"capture failed: {type(e).__name__}: {e}"[:200]
    ms, _ = time_loop(g.replay, steps, warmup)
    del g
    return ms, None


def dense_step_fn(sh, X, dY):
    """Three plain GEMMs of the same shapes (W materialised): Y = X W,
    dX = dY W^T, dW = X^T dY; all operands contiguous."""
    import torch
    dev = X.device
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    W = (torch.randn((sh.n_in, sh.n_out), generator=g, device=dev) / sh.n_in ** 0.5).to(X.dtype)
    Wt = W.t().contiguous()
    Xt = X.t().contiguous()

    def fn():
        torch.matmul(X, W)
        torch.matmul(dY, Wt)
        torch.matmul(Xt, dY)
    return fn


# ------------------------------------------------------------------ roofline
def source_sha(files=None):
    h = hashlib.sha256()
    for f in (KERNEL_SRCS if files is None else files):
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def traffic_from_profile(kernel_tag, act):
    """HBM bytes per launch from a committed counter summary, if it was taken
    on the current kernel sources (the GEMM sources, or the files the summary
    lists); else None."""
    path = os.path.join(PROFILES, f"traffic_{kernel_tag}_{act}.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m_sha = re.search(r"source_sha256_16:\s*([0-9a-f]+)", txt)
    m_b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    m_src = re.search(r"^sources:\s*(.+)$", txt, re.M)
    files = [os.path.join(ROOT, f) for f in m_src.group(1).split()] if m_src else None
    if files and not all(os.path.exists(f) for f in files):
        return None
    if not m_sha or not m_b or m_sha.group(1) != source_sha(files):
        return None
    return float(m_b.group(1))


def kernel_roofline(layer, steps, act, tag=""):
    """Mean duration of each batch-product kernel from HIP events recorded by
    the library on its launch stream, over `steps` instrumented steps."""
    import torch
    C = layer.C
    C.comera_ttm_plan_set_timing(layer.plan.handle, True)
    for _ in range(steps):
        layer.step()
    torch.cuda.synchronize()
    sh, b = layer.sh, layer.b
    flops = 2.0 * b * sh.n_in * sh.n_out        # per launch of each of the three products
    out = {}
    for kt, kid in (("fwd", C.KERNEL_FWD), ("dx", C.KERNEL_DX), ("dw", C.KERNEL_DW)):
        ms, cnt = C.comera_ttm_plan_kernel_time(layer.plan.handle, kid)
        out[kt] = {"avg_ms": ms, "launches": cnt, "tflops": flops / (ms * 1e-3) / 1e12 if ms > 0 else 0.0}
    C.comera_ttm_plan_set_timing(layer.plan.handle, False)
    dom = max(out, key=lambda t: out[t]["avg_ms"])
    ach = out[dom]["tflops"]
    peak = PEAK[act] / 1e12
    # the counter summary is keyed by the product it measured: M x N x K and
    # whether the operands are K-contiguous (fwd, dX) or M/N-contiguous (dW)
    shape = {"fwd": (b, sh.n_out, sh.n_in, "kc"), "dx": (b, sh.n_in, sh.n_out, "kc"),
             "dw": (sh.n_in, sh.n_out, b, "mn")}[dom]
    ttag = "gemm_{}x{}x{}_{}".format(*shape)
    traffic = traffic_from_profile(ttag, act)
    roof = {"bound": "mfma", "achieved": round(ach, 3), "peak": peak, "unit": "TFLOP/s",
            "frac": round(ach / peak, 4), "traffic": traffic,
            "kernel": f"gemm {dom} ({act}{', ' + tag if tag else ''}; {shape[0]}x{shape[1]}x{shape[2]} {shape[3]})",
            "flops_per_launch": flops, "avg_ms": round(out[dom]["avg_ms"], 5),
            "traffic_profile": f"profiles/traffic_{ttag}_{act}.md"}
    return roof, out


# ------------------------------------------------------------------ profile summaries (CPU only)
def _read_csv(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def _find(dirpath, suffix):
    for root, _, files in os.walk(dirpath):
        for fn in files:
            if fn.endswith(suffix):
                return os.path.join(root, fn)
    raise FileNotFoundError(f"no *{suffix} under {dirpath}")


def kernel_stats_summary(prof_dir, out_path, command, top=25):
    """Short text table of a rocprofv3 --kernel-trace --stats run."""
    rows = _read_csv(_find(prof_dir, "kernel_stats.csv"))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = ["# rocprofv3 kernel statistics", "", "command:", "", "```", command, "```", "",
             "| calls | avg us | total ms | % | kernel |", "|---:|---:|---:|---:|---|"]
    for r in rows[:top]:
        name = r["Name"].replace("comera::(anonymous namespace)::", "").replace("|", "/")
        if len(name) > 120:
            name = name[:117] + "..."
        lines.append(f"| {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {float(r['TotalDurationNs']) / 1e6:.3f} | "
                     f"{float(r['Percentage']):.1f} | `{name}` |")
    open(out_path, "w").write("\n".join(lines) + "\n")


def headline_products(prof_dir, out_path):
    """Append to a kernel-statistics summary of the headline run the mean
    duration of each of its two K-contiguous products, which share one
    kernel and grid: in the kernel trace every layer's step starts with its
    fold launch (the up layer's fold grid is the first one seen) and its
    first two persistent-kernel launches after it are the forward and dX
    (up layer: 65536 x 4096 x 1024, then 65536 x 1024 x 4096; down layer
    the other way round)."""
    rows = sorted(_read_csv(_find(prof_dir, "kernel_trace.csv")), key=lambda r: int(r["Start_Timestamp"]))
    up_grid = None
    dur = {"65536x4096x1024": [], "65536x1024x4096": []}
    layer, seen = None, 0
    for r in rows:
        name = r["Kernel_Name"]
        if "fold_kernel" in name:
            g = (r["Grid_Size_X"], r["Grid_Size_Y"])
            up_grid = up_grid or g
            layer, seen = ("up" if g == up_grid else "down"), 0
        elif "gemm_dma_pers_kernel<false>" in name and layer and seen < 2:
            first = (layer == "up") == (seen == 0)
            dur["65536x4096x1024" if first else "65536x1024x4096"].append(
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
            seen += 1
    lines = ["", "Per product of `gemm_dma_pers_kernel<false>` (kernel trace of the same run; each layer's two",
             "launches after its fold are its forward and dX; "
             f"`python3 bench.py --headline-products {os.path.relpath(prof_dir, ROOT)} {os.path.relpath(out_path, ROOT)}`,",
             "no GPU needed for this step):", "",
             "| product | calls | avg us |", "|---|---:|---:|"]
    for k, v in dur.items():
        if v:
            lines.append(f"| {k.replace('x', ' x ')} K-contiguous | {len(v)} | {sum(v) / len(v):.2f} |")
    open(out_path, "a").write("\n".join(lines) + "\n")
    return {k: (len(v), sum(v) / len(v) if v else 0.0) for k, v in dur.items()}


def traffic_summary(fetch_dir, write_dir, kernel, grid, tag, act, out_path, commands, sources=None, out_bytes=None):
    """HBM bytes per launch of one kernel from two counter passes (FETCH_SIZE,
    WRITE_SIZE, KiB per dispatch), each scaled by what the same counter reads
    for a plain device copy of COPY_BYTES.  out_bytes: products that share
    one kernel and grid are told apart by their output size, the launches
    whose scaled write counter lies within 2 % of it; the fetch counter is
    read for the same dispatch ids (the two passes run one deterministic
    launch sequence)."""
    def rows_of(d, counter):
        rows = [r for r in _read_csv(_find(d, "counter_collection.csv")) if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        k = [(int(r["Dispatch_Id"]), float(r["Counter_Value"])) for r in rows
             if kernel in r["Kernel_Name"] and (grid is None or int(r["Grid_Size"]) == grid)]
        c = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        if not k or not c:
            raise RuntimeError(f"{counter}: {len(k)} kernel dispatches, {len(c)} copy dispatches")
        return k, max(c)
    kfr, cf = rows_of(fetch_dir, "FETCH_SIZE")
    kwr, cw = rows_of(write_dir, "WRITE_SIZE")
    if out_bytes:
        if [i for i, _ in kfr] != [i for i, _ in kwr]:
            raise RuntimeError("the two counter passes dispatched the kernel under different ids")
        keep = {i for i, v in kwr if abs(v * 1024 * (COPY_BYTES / 1024.0 / cw) - out_bytes) <= 0.02 * out_bytes}
        kfr = [(i, v) for i, v in kfr if i in keep]
        kwr = [(i, v) for i, v in kwr if i in keep]
        if not kwr:
            raise RuntimeError(f"no dispatch writes {out_bytes} bytes")
    kf, nf = sum(v for _, v in kfr) / len(kfr), len(kfr)
    kw, nw = sum(v for _, v in kwr) / len(kwr), len(kwr)
    sf = COPY_BYTES / 1024.0 / cf
    sw = COPY_BYTES / 1024.0 / cw
    hbm = kf * 1024 * sf + kw * 1024 * sw
    lines = ["# HBM traffic per launch", "",
             f"kernel: `{kernel}`" + (f" (grid size {grid} work-items)" if grid else "") +
             (f", the dispatches that write {int(out_bytes)} bytes" if out_bytes else ""),
             f"tag: {tag} ({act})"] + \
            ([f"sources: {' '.join(os.path.relpath(f, ROOT) for f in sources)}"] if sources else []) + [
             f"source_sha256_16: {source_sha(sources)}",
             f"fetch_kib_per_dispatch: {kf:.1f} (mean of {nf})",
             f"write_kib_per_dispatch: {kw:.1f} (mean of {nw})",
             f"copy_{COPY_BYTES}_bytes_fetch_kib: {cf:.1f} -> scale {sf:.4f}",
             f"copy_{COPY_BYTES}_bytes_write_kib: {cw:.1f} -> scale {sw:.4f}",
             f"hbm_bytes_per_launch: {hbm:.6e}", "", "commands:", "", "```"] + commands + ["```"]
    open(out_path, "w").write("\n".join(lines) + "\n")
    return hbm


def calib_copy():
    """A plain device-to-device copy of COPY_BYTES (the scale for the byte counters)."""
    import torch
    src = torch.ones(COPY_BYTES // 4, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()


# ------------------------------------------------------------------ CPU oracle
def cpu_info():
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        blas = max((i.get("num_threads", 0) for i in threadpool_info()), default=None)
    except Exception:
        pass
    return model, len(os.sched_getaffinity(0)), blas


def _time_reps(fn, min_s):
    reps, t0 = 0, time.perf_counter()
    while True:
        fn()
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_s:
            return reps, el


def _ttm_route_rate(wid, tokens, route, min_s):
    """tokens/s of one oracle route over every layer of a workload, on its
    first `tokens` tokens (the same rows the GPU gets; work per token is
    constant, so the rate is exact in work)."""
    from oracle import ttm as OT
    from paper_2405_14377_amd import workloads as wl
    w = wl.WORKLOADS[wid]
    act = w.dtypes[-1]
    data = []
    for li, sh in enumerate(w.layers):
        inp = wl.ttm_layer_inputs(wid, li, sh, w.mask)
        X = wl.activations(wid, tokens, sh.n_in, 0, act, layer=li)
        dY = wl.activations(wid, tokens, sh.n_out, 1, act, layer=li)
        data.append((X, dY, inp.cores, inp.masks))
    if route == "dense":
        fwd, bwd = OT.forward_dense, OT.backward_dense
    else:
        fwd, bwd = OT.forward_direct, OT.backward_direct

    def step():
        for X, dY, cores, masks in data:
            fwd(X, cores, masks)
            bwd(X, dY, cores, masks)
    reps, el = _time_reps(step, min_s)
    return {"tokens_per_s": round(reps * tokens / el, 1), "tokens": tokens, "reps": reps, "seconds": round(el, 2),
            "layers": len(w.layers), "dtype_in": act}


def _embed_rate(tokens, min_s):
    import numpy as np
    from oracle import embed as OE
    from paper_2405_14377_amd import workloads as wl
    w = wl.WORKLOADS[3]
    cores = wl.embed_cores(w)
    V, E = int(np.prod(w.v)), int(np.prod(w.e))
    ids = wl.token_ids(w.n_tokens, V, "zipf1.1", wl.seed_of(3, 20))[:tokens]
    dY = np.random.default_rng(wl.seed_of(3, 1)).standard_normal((tokens, E)).astype(np.float32)

    def step():
        OE.forward(ids, cores)
        OE.backward(ids, dY, cores)
    reps, el = _time_reps(step, min_s)
    return {"tokens_per_s": round(reps * tokens / el, 1), "tokens": tokens, "reps": reps, "seconds": round(el, 2),
            "ids": "zipf1.1"}


def cpu_baseline():
    """The fp64 oracle as it stands, on the host cores: the headline workload
    (the 1024 <-> 4096 pair, both layers) on a 1024-token slice by the dense-W
    route (the value) and on a 128-token slice by the direct route; the
    768 -> 768 and 768 -> 3072 layers at full size, the six encoder layers on
    a 1024-token slice, the embedding on a 2048-token slice."""
    model, aff, blas = cpu_info()
    head = _ttm_route_rate(HEADLINE_WID, 1024, "dense", 5.0)
    direct = _ttm_route_rate(HEADLINE_WID, 128, "direct", 2.0)
    others = {
        "w0_768x768_full_dense_w": _ttm_route_rate(0, 32, "dense", 1.0),
        "w0_768x768_full_direct": _ttm_route_rate(0, 32, "direct", 1.0),
        "w1_768x3072_full_dense_w": _ttm_route_rate(1, 4096, "dense", 1.0),
        "w1_768x3072_slice256_direct": _ttm_route_rate(1, 256, "direct", 1.0),
        "w2_encoder6_slice1024_dense_w": _ttm_route_rate(2, 1024, "dense", 1.0),
        "w3_embedding_slice2048": _embed_rate(2048, 1.0),
    }
    cores = min(aff, blas) if blas else aff
    return {"value": head["tokens_per_s"], "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{head['reps']} steps of the 1024<->4096 d4 r64 pair (both layers) on its first 1024 tokens "
                      f"(bf16-rounded inputs, fp64 math), dense-W route (forward_dense + backward_dense), "
                      f"{head['seconds']} s",
            "cpu_model": model, "affinity_cpus": aff, "blas_threads": blas,
            "direct_route": direct, "other_configs": others}


# ------------------------------------------------------------------ other workloads
def graph_entry(gms, gerr, dgms, dgerr):
    """Graph-replay figures of one step (ours and the dense baseline's)."""
    e = {"ms_per_step": None if gms is None else round(gms, 5),
         "dense_ms_per_step": None if dgms is None else round(dgms, 5)}
    if gms is not None and dgms is not None:
        e["speedup_vs_dense"] = round(dgms / gms, 3)
    if gerr or dgerr:
        e["error"] = gerr or dgerr
    return e


def other_workloads(steps, warmup):
    import numpy as np
    import torch
    from paper_2405_14377_amd import comera as C
    from paper_2405_14377_amd import workloads as wl
    res = {}
    # TTM layer workloads
    for wid, act in ((0, "f32"), (2, "bf16"), (5, "f32"), (5, "bf16")):
        w = wl.WORKLOADS[wid]
        layers, dense = [], []
        for li in range(len(w.layers)):
            sh, inp, X, dY, G, D, ma, b = layer_inputs(wid, li, act, 1000 * wid + li)
            layers.append(Layer(sh, X, dY, G, D, ma, b, act))
            dense.append(dense_step_fn(sh, X, dY))
        k = steps if wid != 4 else max(3, steps // 4)
        ms, _ = time_loop(lambda: [l.step() for l in layers], k, warmup)
        dms, _ = time_loop(lambda: [f() for f in dense], k, warmup)
        gms, gerr = graph_loop(lambda: [l.step() for l in layers], k, warmup)
        dgms, dgerr = graph_loop(lambda: [f() for f in dense], k, warmup)
        fl = sum(6.0 * l.b * l.sh.n_in * l.sh.n_out for l in layers)
        fl_alg = 0.0
        for l in layers:
            o = l.plan.order_info(l.plan.chosen)
            fl_alg += o["flops_fwd"] + o["flops_bwd"]
        entry = {"workload": w.name, "dtype": act, "tokens": w.batch, "layers": len(layers),
                 "ms_per_step": round(ms, 4), "tokens_per_s": round(w.batch / (ms * 1e-3), 1),
                 "tflops_gemm_equiv": round(fl / (ms * 1e-3) / 1e12, 2),
                 "tflops_algorithmic": round(fl_alg / (ms * 1e-3) / 1e12, 2),
                 "dense_ms_per_step": round(dms, 4), "speedup_vs_dense": round(dms / ms, 3),
                 "graph": graph_entry(gms, gerr, dgms, dgerr)}
        if wid == 2:
            rr = [kernel_roofline(l, max(2, k // 2), act, f"encoder layer {i}") for i, l in enumerate(layers)]
            entry["kernels_ms"] = [{t: round(v["avg_ms"], 4) for t, v in r.items()} for _, r in rr]
            # the step's dominant product (longest mean launch) and its roofline
            entry["roofline"] = max((r for r, _ in rr), key=lambda r: r["avg_ms"])
        entry["orders"] = [l.plan.order_info(l.plan.chosen)["desc"] for l in layers]
        res[f"w{wid}_{act}"] = entry
        del layers, dense
        torch.cuda.empty_cache()
    # embedding
    w = wl.WORKLOADS[3]
    dev = torch.device("cuda", 0)
    cores = [torch.from_numpy(c).to(dev) for c in wl.embed_cores(w)]
    shape = C.tt_embed_shape(w.v, w.e, w.r)
    V, E, n = int(np.prod(w.v)), int(np.prod(w.e)), w.n_tokens
    ws = torch.empty(C.comera_tt_embed_workspace_bytes(shape, n), dtype=torch.uint8, device=dev)
    Y = torch.empty((n, E), device=dev)
    dG = [torch.empty_like(c) for c in cores]
    g = torch.Generator(device=dev)
    g.manual_seed(3000)
    dYe = torch.randn((n, E), generator=g, device=dev)
    table = torch.randn((V, E), generator=g, device=dev) * 0.1
    table.requires_grad_(True)
    for dist in ("zipf1.1", "uniform"):
        ids = torch.from_numpy(wl.token_ids(n, V, dist, wl.seed_of(3, 20))).to(dev)
        stream = None             # the current stream

        def step():
            # a training step: the backward takes the forward's prefix table
            C.comera_tt_embed_forward(shape, ids, n, cores, None, Y, ws, None, stream)
            C.comera_tt_embed_backward_ex(shape, ids, n, dYe, cores, None, dG, C.EMBED_REUSE_FORWARD, ws, None, stream)

        def fstep():
            C.comera_tt_embed_forward(shape, ids, n, cores, None, Y, ws, None, stream)

        def dense():
            out = torch.nn.functional.embedding(ids, table)
            out.backward(dYe)
            table.grad = None

        ms, _ = time_loop(step, steps, warmup)
        fms, _ = time_loop(fstep, steps, warmup)
        dms, _ = time_loop(dense, steps, warmup)
        gms, gerr = graph_loop(step, steps, warmup)
        byt = 2.0 * n * E * 4            # output write + dY read (algorithmic floor)
        # the row kernel (the forward's dominant launch): HBM bytes per launch
        # from its counter summary (mean over the Zipf and uniform runs)
        Vp, Ep = int(np.prod(w.v[:-1])), int(np.prod(w.e[:-1]))
        rows_tag = f"embed_rows_{V}x{E}_b{n}"
        rows = {"hbm_bytes": traffic_from_profile(rows_tag, "f32"),
                "algorithmic_bytes": float(n * E * 4 + Vp * Ep * w.r[-2] * 4),
                "traffic_profile": f"profiles/traffic_{rows_tag}_f32.md"}
        res[f"w3_{dist}"] = {"workload": w.name, "dtype": "f32", "tokens": n, "ms_per_step": round(ms, 4),
                             "fwd_ms": round(fms, 4), "tokens_per_s": round(n / (ms * 1e-3), 1),
                             "gbps_floor_bytes": round(byt / (ms * 1e-3) / 1e9, 1),
                             "hbm_frac": round(byt / (ms * 1e-3) / HBM_PEAK, 4),
                             "dense_ms_per_step": round(dms, 4), "speedup_vs_dense": round(dms / ms, 3),
                             "rows_kernel": rows, "graph": graph_entry(gms, gerr, None, None)}
    return res


def dense_fp8_step_fn(sh, X, dY):
    """The three dense products on FP8 E4M3 operands with per-tensor scales
    (torch._scaled_mm, bf16 out), operands quantised inside the step as the
    mixed-precision layer does; None with the reason if torch cannot run it."""
    import torch
    dev = X.device
    f8 = torch.float8_e4m3fn
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    W = torch.randn((sh.n_in, sh.n_out), generator=g, device=dev) / sh.n_in ** 0.5

    def q(t):
        s = 448.0 / t.abs().amax().float().clamp(min=1e-30)
        return (t.float() * s).to(f8), (1.0 / s).reshape(())

    def fn():
        x8, sx = q(X)
        w8t, sw = q(W.t().contiguous())  # [N_out, N_in] row-major: its transpose is the column-major B
        d8, sd = q(dY)
        torch._scaled_mm(x8, w8t.t(), scale_a=sx, scale_b=sw, out_dtype=torch.bfloat16)
        w8, _ = q(W)
        torch._scaled_mm(d8, w8.t(), scale_a=sd, scale_b=sw, out_dtype=torch.bfloat16)
        xt8, _ = q(X.t().contiguous())
        dt8, _ = q(dY.t().contiguous())
        torch._scaled_mm(xt8, dt8.t(), scale_a=sx, scale_b=sd, out_dtype=torch.float32)
    try:
        fn()
        torch.cuda.synchronize()
    except Exception as e:
        return None, f"{type(e).__name__}: {e}"[:160]
    return fn, None


def fp8_workloads(steps, warmup):
    """Mixed-precision layers (batch products on FP8 codes) beside the same
    layers in bf16 (the planner's order) and the dense products in bf16 and
    FP8, for the layer shapes of the large-batch workloads."""
    import torch
    from paper_2405_14377_amd import workloads as wl
    res = {}
    for wid in (1, 4, 6):
        w = wl.WORKLOADS[wid]
        for li in range(len(w.layers)):
            sh, inp, X, dY, G, D, ma, b = layer_inputs(wid, li, "bf16", 1000 * wid + li)
            k = steps if wid == 1 else max(3, steps // 4)
            lay = Layer(sh, X, dY, G, D, ma, b, "bf16", fp8=True)
            log(f"[fp8] {w.name} {sh.name}: {k} steps")
            ms, _ = time_loop(lay.step, k, warmup)
            C = lay.C
            C.comera_ttm_plan_set_timing(lay.plan.handle, True)
            for _ in range(max(2, k // 2)):
                lay.step()
            torch.cuda.synchronize()
            flops = 2.0 * b * sh.n_in * sh.n_out
            kern = {}
            for tag, kid in (("fwd", C.KERNEL_FWD), ("dx", C.KERNEL_DX), ("dw", C.KERNEL_DW)):
                kms, _ = C.comera_ttm_plan_kernel_time(lay.plan.handle, kid)
                kern[tag] = {"ms": round(kms, 5), "tflops": round(flops / (kms * 1e-3) / 1e12, 1),
                             "frac_fp8_peak": round(flops / (kms * 1e-3) / 5.0e15, 4)}
            C.comera_ttm_plan_set_timing(lay.plan.handle, False)
            del lay
            torch.cuda.empty_cache()
            ref = Layer(sh, X, dY, G, D, ma, b, "bf16")
            bms, _ = time_loop(ref.step, k, warmup)
            order = ref.plan.order_info(ref.plan.chosen)["desc"]
            del ref
            torch.cuda.empty_cache()
            dms, _ = time_loop(dense_step_fn(sh, X, dY), k, warmup)
            f8fn, f8err = dense_fp8_step_fn(sh, X, dY)
            d8ms = time_loop(f8fn, k, warmup)[0] if f8fn else None
            res[f"w{wid}_{sh.name}"] = {
                "workload": w.name, "layer": sh.name, "tokens": b, "activations": "bf16",
                "fp8_ms_per_step": round(ms, 4), "fp8_tokens_per_s": round(b / (ms * 1e-3), 1),
                "fp8_gemm_kernels": kern,
                "bf16_ms_per_step": round(bms, 4), "bf16_order": order,
                "dense_bf16_ms_per_step": round(dms, 4),
                "dense_fp8_ms_per_step": None if d8ms is None else round(d8ms, 4),
                "dense_fp8_error": f8err,
                "fp8_speedup_vs_dense_bf16": round(dms / ms, 3),
                "fp8_speedup_vs_dense_fp8": None if d8ms is None else round(d8ms / ms, 3),
                "fp8_speedup_vs_bf16_layer": round(bms / ms, 3)}
            del X, dY, G, D
            torch.cuda.empty_cache()
    return res


def order_timings(wids, steps, warmup):
    """Every executable contraction order of each layer of the given
    workloads, timed forward and backward separately, beside the dense
    torch.matmul step of the same shapes."""
    import torch
    from paper_2405_14377_amd import workloads as wl
    out = []
    for wid in wids:
        w = wl.WORKLOADS[wid]
        for act in w.dtypes:
            for li in range(len(w.layers)):
                sh, inp, X, dY, G, D, ma, b = layer_inputs(wid, li, act, 1000 * wid + li)
                probe = Layer(sh, X, dY, G, D, ma, b, act)
                chosen = probe.plan.chosen
                infos = [probe.plan.order_info(i) for i in range(probe.plan.num_orders)]
                del probe
                dense = 6.0 * b * sh.n_in * sh.n_out
                dms, _ = time_loop(dense_step_fn(sh, X, dY), steps, warmup)
                rec = {"workload": w.name, "layer": sh.name, "dtype": act, "tokens": b, "chosen": chosen,
                       "dense_gemm_ms": round(dms, 5), "orders": []}
                for i, o in enumerate(infos):
                    if not o["executable"]:
                        rec["orders"].append({"i": i, "desc": o["desc"], "executable": False})
                        continue
                    fl = o["flops_fwd"] + o["flops_bwd"]
                    k = steps if fl < 5 * dense else max(2, steps // 5)
                    log(f"[orders] {w.name} {sh.name} {act} order {i} {o['desc']}: {k} steps")
                    lay = Layer(sh, X, dY, G, D, ma, b, act, force_order=i)
                    fms, _ = time_loop(lay.forward, k, min(warmup, 2))
                    bms, _ = time_loop(lay.backward, k, min(warmup, 2))
                    rec["orders"].append({"i": i, "desc": o["desc"], "fwd_ms": round(fms, 5), "bwd_ms": round(bms, 5),
                                          "step_ms": round(fms + bms, 5),
                                          "flops_vs_dense": round(fl / dense, 4),
                                          "tflops": round(fl / ((fms + bms) * 1e-3) / 1e12, 2),
                                          "speedup_vs_dense_gemm": round(dms / (fms + bms), 3)})
                    del lay
                    torch.cuda.empty_cache()
                out.append(rec)
                del X, dY, G, D
                torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-extra", action="store_true", help="skip the other workloads")
    ap.add_argument("--dtype", default="bf16", choices=["f32", "bf16"], help="dtype tag of a traffic summary")
    ap.add_argument("--headline-only", action="store_true", help="only the headline workload (profiling runs)")
    ap.add_argument("--workload", type=int, default=None, metavar="WID",
                    help="only this workload's steps (3 = the embedding), eager, one JSON line (profiling runs)")
    ap.add_argument("--act", default="bf16", choices=["f32", "bf16"], help="activation dtype for --workload")
    ap.add_argument("--calib-copy", action="store_true", help="also run a plain device copy of known size")
    ap.add_argument("--stats-summary", nargs=3, metavar=("PROF_DIR", "OUT_MD", "COMMAND"),
                    help="write a kernel-statistics table from a rocprofv3 run (no GPU)")
    ap.add_argument("--traffic-summary", nargs=5, metavar=("FETCH_DIR", "WRITE_DIR", "KERNEL", "GRID", "TAG"),
                    help="write profiles/traffic_<TAG>_<dtype>.md from two counter runs (no GPU); GRID 0 = any")
    ap.add_argument("--commands", nargs="*", default=[], help="commands recorded in a summary")
    ap.add_argument("--sources", nargs="*", default=None,
                    help="source files (repository paths) a traffic summary is keyed to (default: the GEMM sources)")
    ap.add_argument("--headline-products", nargs=2, metavar=("PROF_DIR", "OUT_MD"),
                    help="append the per-product means of the headline's persistent GEMM to a summary (no GPU)")
    ap.add_argument("--out-bytes", type=float, default=None,
                    help="traffic summary: only the dispatches whose output (write counter) is this many bytes")
    ap.add_argument("--fp8-only", action="store_true", help="only the mixed-precision (FP8) figures")
    ap.add_argument("--orders", type=int, nargs="*", default=None, metavar="WORKLOAD",
                    help="time every contraction order of these workloads (default 0 1 5) and exit")
    args = ap.parse_args()
    if args.stats_summary:
        kernel_stats_summary(*args.stats_summary)
        return
    if args.headline_products:
        print(headline_products(*args.headline_products))
        return
    if args.traffic_summary:
        fd, wd, kern, grid, tag = args.traffic_summary
        srcs = [os.path.join(ROOT, f) for f in args.sources] if args.sources else None
        hbm = traffic_summary(fd, wd, kern, int(grid) or None, tag, args.dtype,
                              os.path.join(PROFILES, f"traffic_{tag}_{args.dtype}.md"), args.commands, srcs,
                              args.out_bytes)
        print(f"hbm bytes per launch: {hbm:.4e}")
        return
    ws = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or ws != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path (a layer would shard by tokens, "
              "with one all-reduce of the core gradients per step). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    from paper_2405_14377_amd import comera as C
    C.load()
    # every GPU call, ours and the baselines', goes to one dedicated stream
    # of default priority (the legacy null stream adds per-launch cost)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        run_gpu(args)
        torch.cuda.synchronize()


def run_layers(wid, act, steps, warmup, seed_base, roof_tag=None):
    """Time whole steps (every layer of workload wid, forward then backward)
    beside the dense GEMMs of the same shapes, eager and under graph replay;
    with roof_tag, also the per-kernel roofline of each layer."""
    import torch
    from paper_2405_14377_amd import workloads as wl
    w = wl.WORKLOADS[wid]
    layers, dense = [], []
    for li in range(len(w.layers)):
        sh, inp, X, dY, G, D, ma, b = layer_inputs(wid, li, act, seed_base + li)
        layers.append(Layer(sh, X, dY, G, D, ma, b, act))
        dense.append(dense_step_fn(sh, X, dY))
    b = w.batch

    def step():
        for lay in layers:
            lay.step()

    def dstep():
        for f in dense:
            f()
    log(f"[bench] {w.name} {act}: warmup {warmup}, timing {steps} steps")
    torch.cuda.synchronize()
    ms, wall = time_loop(step, steps, warmup)
    dms, _ = time_loop(dstep, steps, warmup)
    gms, gerr = graph_loop(step, steps, warmup)
    dgms, dgerr = graph_loop(dstep, steps, warmup)
    res = {"workload": w.name, "dtype": act, "tokens": b, "layers": len(layers), "ms_per_step": ms, "wall_s": wall,
           "tokens_per_s": b / (ms * 1e-3), "dense_ms": dms, "speedup_vs_dense": dms / ms,
           "graph": graph_entry(gms, gerr, dgms, dgerr),
           "orders": [lay.plan.order_info(lay.plan.chosen)["desc"] for lay in layers]}
    if gms is not None:
        res["graph"]["tokens_per_s"] = round(b / (gms * 1e-3), 1)
    if roof_tag is not None:
        roofs, kerns = [], {}
        for lay in layers:
            tag = f"{roof_tag}_{lay.sh.name}" if len(layers) > 1 else roof_tag
            roof, kern = kernel_roofline(lay, steps, act, tag)
            roofs.append(roof)
            kerns[lay.sh.name] = {t: round(v["avg_ms"], 5) for t, v in kern.items()}
        res["roofline"] = max(roofs, key=lambda r: r["avg_ms"])
        res["kernels_ms"] = kerns
    log(f"[bench]   {ms:.4f} ms/step, dense {dms:.4f} ms")
    del layers, dense
    torch.cuda.empty_cache()
    return res


def embed_steps(dist, steps, warmup):
    """The embedding training step (forward, then backward on the forward's
    prefix table) for one id distribution; eager."""
    import numpy as np
    import torch
    from paper_2405_14377_amd import comera as C
    from paper_2405_14377_amd import workloads as wl
    w = wl.WORKLOADS[3]
    dev = torch.device("cuda", 0)
    cores = [torch.from_numpy(c).to(dev) for c in wl.embed_cores(w)]
    shape = C.tt_embed_shape(w.v, w.e, w.r)
    V, E, n = int(np.prod(w.v)), int(np.prod(w.e)), w.n_tokens
    ws = torch.empty(C.comera_tt_embed_workspace_bytes(shape, n), dtype=torch.uint8, device=dev)
    Y = torch.empty((n, E), device=dev)
    dG = [torch.empty_like(c) for c in cores]
    g = torch.Generator(device=dev)
    g.manual_seed(3000)
    dYe = torch.randn((n, E), generator=g, device=dev)
    ids = torch.from_numpy(wl.token_ids(n, V, dist, wl.seed_of(3, 20))).to(dev)

    def step():
        C.comera_tt_embed_forward(shape, ids, n, cores, None, Y, ws, None, None)
        C.comera_tt_embed_backward_ex(shape, ids, n, dYe, cores, None, dG, C.EMBED_REUSE_FORWARD, ws, None, None)
    ms, _ = time_loop(step, steps, warmup)
    return {"workload": w.name, "ids": dist, "ms_per_step": round(ms, 5), "tokens_per_s": round(n / (ms * 1e-3), 1)}


def run_gpu(args):
    if args.workload is not None:
        if args.workload == 3:
            print(json.dumps([embed_steps(dist, args.steps, args.warmup) for dist in ("zipf1.1", "uniform")]))
        else:
            r = run_layers(args.workload, args.act, args.steps, args.warmup, 1000 * args.workload)
            print(json.dumps(r))
        if args.calib_copy:
            calib_copy()
        return
    if args.orders is not None:
        wids = args.orders or [0, 1, 5]
        for rec in order_timings(wids, args.steps, args.warmup):
            print(json.dumps(rec), flush=True)
        return
    if args.fp8_only:
        print(json.dumps(fp8_workloads(args.steps, args.warmup)), flush=True)
        return
    main_run = run_layers(HEADLINE_WID, "bf16", args.steps, args.warmup, 4000, roof_tag="ttm1024x4096")
    out = {
        "metric": METRIC,
        "value": round(main_run["tokens_per_s"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_run["ms_per_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations, cores scaled for unit output variance)",
        "config": {"workload": "ttm_pair_1024x4096_4096x1024_d4_r64_mask0.7_b65536_bf16 (both layers per step)",
                   "global_batch": 65536, "parallelism": "none (1 GPU)"},
        "roofline": main_run["roofline"],
        "speedup_vs_dense_gemm": round(main_run["speedup_vs_dense"], 3),
        "dense_gemm_ms_per_step": round(main_run["dense_ms"], 5),
        "kernels_ms": main_run["kernels_ms"],
        "orders": main_run["orders"],
        "graph_replay": main_run["graph"],
        "stream": "one dedicated stream (default priority) for every GPU call, ours and the baseline's",
    }
    if not args.headline_only:
        for act in ("f32", "bf16"):
            r = run_layers(1, act, args.steps, args.warmup, 1000 + (act == "bf16"), roof_tag="ttm768x3072")
            out[f"ttm768x3072_{act}"] = {
                "value": round(r["tokens_per_s"], 1), "ms_per_step": round(r["ms_per_step"], 5),
                "speedup_vs_dense_gemm": round(r["speedup_vs_dense"], 3),
                "dense_gemm_ms_per_step": round(r["dense_ms"], 5), "roofline": r["roofline"],
                "kernels_ms": r["kernels_ms"], "graph_replay": r["graph"]}
    if args.calib_copy:
        calib_copy()
    if not args.no_extra and not args.headline_only:
        log("[bench] other workloads")
        out["other_workloads"] = other_workloads(max(5, args.steps // 2), 3)
        log("[bench] mixed-precision (FP8) layers")
        out["fp8_layers"] = fp8_workloads(max(5, args.steps // 2), 3)
    if not args.no_cpu and not args.headline_only:
        log("[bench] CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline()
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
