"""Drive every compute entry point of libcomera.so through its host path in
launch check mode (no GPU: each kernel launch is validated against the
gfx950 limits and recorded instead of issued; no device memory is touched,
so the device pointers below are placeholders that are never dereferenced).

Run as a program, it prints one JSON line: the number of calls made, the
calls whose status differs from the expected one, and the launches outside
the limits.  tests/test_launch_sizing.py runs it in a child process, so a
host arithmetic trap (SIGFPE from an integer division by zero) or a crash in
the launch sizing shows up as the child's signal instead of ending pytest."""
from __future__ import annotations

import itertools
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2405_14377_amd import comera as C  # noqa: E402

_next = [0x100000000]


def fake(nbytes=1):
    """A distinct 256-byte-aligned placeholder address (never dereferenced)."""
    p = _next[0]
    _next[0] += (int(nbytes) + 0x10000 + 255) // 256 * 256
    return p


def ttm_cases():
    shapes = [
        ((5,), (3,), (1, 1)),                                   # d = 1
        ((1, 1, 1), (1, 1, 1), (1, 2, 3, 1)),                   # unit modes
        ((2, 3, 4), (4, 3, 2), (1, 1, 1, 1)),                   # rank 1
        ((3, 5), (2, 7), (1, 4, 1)),                            # N below one tile
        ((2, 2), (2, 2), (1, 300, 1)),                          # rank above the compaction limit
        ((8, 8, 12), (12, 8, 8), (1, 8, 8, 1)),                 # 768 -> 768 r8
        ((8, 8, 12), (16, 16, 12), (1, 30, 30, 1)),             # 768 -> 3072 r30
        ((16, 16, 12), (8, 8, 12), (1, 30, 30, 1)),             # 3072 -> 768 r30
        ((4, 8, 4, 8), (8, 8, 8, 8), (1, 64, 64, 64, 1)),       # 1024 -> 4096 d4 r64
        ((8, 8, 12, 1, 1, 1), (1, 1, 1, 16, 16, 12), (1,) + (30,) * 5 + (1,)),   # TT layout
        ((16, 8, 8, 1, 1, 1), (1, 1, 1, 16, 16, 16), (1,) + (32,) * 5 + (1,)),
        ((3, 1, 7, 2), (1, 5, 2, 3), (1, 3, 1, 5, 1)),          # ragged with unit factors
    ]
    for n, m, r in shapes:
        d = len(n)
        nmask = sum(r[1:d])
        for batch in (0, 1, 33, 4096, 65536):
            for act in (C.F32, C.BF16):
                masks = [None]
                if nmask:
                    masks.append([1 if (i % 3) else 0 for i in range(nmask)])       # compaction
                    masks.append([0] * r[1] + [1] * (nmask - r[1]))                  # an empty bond
                for ma in masks:
                    yield n, m, r, batch, act, ma


def run_ttm(n, m, r, batch, act, ma, out):
    shape = C.ttm_shape(n, m, r, act)
    st, h = C.comera_ttm_plan(shape, batch, ma, -1, raise_on_error=False)
    out["calls"] += 1
    if st != C.OK:
        out["bad_status"].append({"call": "plan", "n": n, "m": m, "r": r, "b": batch, "st": st})
        return
    norders = C.comera_ttm_plan_num_orders(h)
    infos = [C.comera_ttm_plan_order_info(h, i) for i in range(norders)]
    C.comera_ttm_plan_destroy(h)
    d = len(n)
    nin, nout = 1, 1
    for k in range(d):
        nin *= n[k]
        nout *= m[k]
    esz = 2 if act == C.BF16 else 4
    orders = [i for i, o in enumerate(infos) if o["executable"]]
    if batch > 4096:
        orders = orders[:1]
    for order in orders:
        for reuse, fp8 in ((0, 0), (1, 0), (0, 1), (1, 1)):
            if fp8 and order != 0:
                continue
            st, h = C.comera_ttm_plan(shape, batch, ma, order, raise_on_error=False)
            out["calls"] += 1
            if st != C.OK:
                out["bad_status"].append({"call": "plan", "order": order, "n": n, "b": batch, "st": st})
                continue
            lib = C.load()
            lib.comera_ttm_plan_set_reuse_forward(h, reuse)
            if fp8:
                s8 = lib.comera_ttm_plan_set_fp8(h, 1)
                if s8 == C.ERR_UNSUPPORTED:
                    C.comera_ttm_plan_destroy(h)
                    continue
            wsb = C.comera_ttm_workspace_bytes(h)
            ws = fake(wsb)
            G = [fake(4 * r[k] * m[k] * n[k] * r[k + 1]) for k in range(d)]
            D = [fake(4 * r[k + 1]) for k in range(d - 1)]
            dG = [fake(4 * r[k] * m[k] * n[k] * r[k + 1]) for k in range(d)]
            dD = [fake(4 * r[k + 1]) for k in range(d - 1)]
            for b in sorted({batch, max(batch // 2, 0), min(batch, 1)}):
                X, Y, dY, dX = fake(esz * b * nin), fake(esz * b * nout), fake(esz * b * nout), fake(esz * b * nin)
                Gp, Dp, dGp, dDp = C._ptr_array(G), C._ptr_array(D) if d > 1 else None, C._ptr_array(dG), \
                    C._ptr_array(dD) if d > 1 else None
                calls = [
                    ("forward", lambda: lib.comera_ttm_forward(h, b, X, Gp, Dp, Y, ws, wsb, 0)),
                    ("backward", lambda: lib.comera_ttm_backward(h, b, X, dY, Gp, Dp, dX, dGp, ws, wsb, 0)),
                    ("backward dX only", lambda: lib.comera_ttm_backward(h, b, X, dY, Gp, Dp, dX, None, ws, wsb, 0)),
                    ("backward dG only", lambda: lib.comera_ttm_backward(h, b, X, dY, Gp, Dp, None, dGp, ws, wsb, 0)),
                    ("backward masks", lambda: lib.comera_ttm_backward_masks(h, b, X, dY, Gp, Dp, dX, dGp, dDp, ws,
                                                                              wsb, 0)),
                ]
                if not reuse and not fp8:
                    st = lib.comera_ttm_forward_noalloc(h, b, X, Gp, Dp, Y, 0)
                    out["calls"] += 1
                    if st not in (C.OK, C.ERR_UNSUPPORTED) or (st != C.OK and order == 0 and wsb < (48 << 20)):
                        out["bad_status"].append({"call": "forward noalloc", "order": order, "n": n, "m": m, "r": r,
                                                  "b": b, "act": act, "st": st})
                for name, fn in calls:
                    st = fn()
                    out["calls"] += 1
                    if st != C.OK:
                        out["bad_status"].append({"call": name, "order": order, "reuse": reuse, "fp8": fp8, "n": n,
                                                  "m": m, "r": r, "b": b, "act": act, "st": st})
            C.comera_ttm_plan_destroy(h)
    # regulariser
    G = C._ptr_array([fake(4 * r[k] * m[k] * n[k] * r[k + 1]) for k in range(d)])
    D = C._ptr_array([fake(4 * r[k + 1]) for k in range(d - 1)]) if d > 1 else None
    st = C.load().comera_ttm_regularizer_grads(shape, 0.5, 0.25, G, D, G, D, 0)
    out["calls"] += 1
    if st != C.OK:
        out["bad_status"].append({"call": "regularizer", "n": n, "st": st})


def embed_cases():
    shapes = [
        ((50,), (7,), (1, 1)),
        ((4, 8), (3, 5), (1, 6, 1)),
        ((7, 3), (16, 2), (1, 30, 1)),
        ((32, 32, 32), (8, 8, 12), (1, 30, 30, 1)),
        ((2, 3, 4, 5), (2, 2, 3, 4), (1, 3, 5, 7, 1)),
        ((16, 16), (48, 16), (1, 64, 1)),
        ((1, 1, 3), (4, 1, 2), (1, 2, 2, 1)),
    ]
    for v, e, r in shapes:
        for n in (0, 1, 15, 16, 17, 255, 1023, 1024, 1025, 16384, 65537):
            yield v, e, r, n


def run_embed(v, e, r, n, out):
    lib = C.load()
    shape = C.tt_embed_shape(v, e, r)
    d = len(v)
    E = 1
    for x in e:
        E *= x
    wsb = C.comera_tt_embed_workspace_bytes(shape, n)
    ws = fake(wsb)
    G = C._ptr_array([fake(4 * r[k] * v[k] * e[k] * r[k + 1]) for k in range(d)])
    dG = C._ptr_array([fake(4 * r[k] * v[k] * e[k] * r[k + 1]) for k in range(d)])
    D = C._ptr_array([fake(4 * r[k + 1]) for k in range(d - 1)]) if d > 1 else None
    ids, Y, dY, err = fake(8 * n), fake(4 * n * E), fake(4 * n * E), fake(4)
    calls = [
        ("embed forward", lambda: lib.comera_tt_embed_forward(shape, ids, n, G, D, Y, ws, wsb, err, 0)),
        ("embed backward", lambda: lib.comera_tt_embed_backward(shape, ids, n, dY, G, D, dG, 1, ws, wsb, err, 0)),
        ("embed backward reuse", lambda: lib.comera_tt_embed_backward_ex(shape, ids, n, dY, G, D, dG,
                                                                        C.EMBED_REUSE_FORWARD, ws, wsb, err, 0)),
    ]
    for name, fn in calls:
        st = fn()
        out["calls"] += 1
        if st not in (C.OK, C.ERR_UNSUPPORTED):
            out["bad_status"].append({"call": name, "v": v, "e": e, "r": r, "n": n, "st": st})


def run_fp8(out):
    lib = C.load()
    for rows, cols in itertools.product((0, 1, 127, 128, 129, 4096, 65536), (1, 16, 100, 1024, 4096)):
        for dtype in (C.F32, C.BF16):
            ldq = (cols + 127) // 128 * 128
            ldt = (rows + 127) // 128 * 128
            st = lib.comera_fp8_quantize(fake(4 * rows * cols), dtype, rows, cols, fake(rows * ldq), ldq,
                                         fake(cols * max(ldt, 1)), max(ldt, 1), fake(4), fake(4096),
                                         C.FP8_QUANTIZE_WS_BYTES, 0)
            out["calls"] += 1
            if st != C.OK:
                out["bad_status"].append({"call": "fp8 quantize", "rows": rows, "cols": cols, "st": st})


def main():
    C.comera_debug_launch_check(True)
    out = {"calls": 0, "bad_status": []}
    for case in ttm_cases():
        run_ttm(*case, out)
    for case in embed_cases():
        run_embed(*case, out)
    run_fp8(out)
    log = C.comera_debug_launch_log()
    C.comera_debug_launch_check(False)
    out["launches"] = len(log)
    out["bad_launches"] = [x for x in log if not x["ok"]][:20]
    out["kernels"] = sorted({x["kernel"] for x in log})
    out["bad_status"] = out["bad_status"][:20]
    print(json.dumps(out))


if __name__ == "__main__":
    main()
