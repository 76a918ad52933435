// extern "C" entry points for one TTM linear layer: comera_ttm_forward and
// comera_ttm_backward.  Every step runs as a kernel on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstring>

#include "internal.h"

using namespace comera;

namespace {

inline char *at(void *ws, size_t off) { return reinterpret_cast<char *>(ws) + off; }

struct DenseBuild {
    float *gc[kMaxCores];      // folded cores, layout [rho_k][n_k][m_k][rho_{k+1}]
    float *P[kMaxCores + 1];   // P[k] = product of cores 0..k-1 as [I_<k][J_<k][rho_k], k = 1..d-1
};

// Steps shared by forward and backward: fold the masks into compacted core
// copies (eq. Wcompress), then the left chains P_1..P_{d-1} and W (eq. TTM)
// as one GEMM per core; the last one writes W[N_in, N_out] (or, with
// transpose, W^T[N_out, N_in]) in the activation dtype.
int build_dense(const comera_ttm_plan_s *p, const float *const *G, const float *const *D, void *ws, void *stream,
                DenseBuild &bd, bool transpose) {
    const DenseLayout &L = p->dense;
    const int d = p->d;
    FoldArgs fa;
    std::memset(&fa, 0, sizeof(fa));
    fa.d = d;
    fa.nfold = d;
    fa.compacted = p->compacted ? 1 : 0;
    fa.swap = 1;
    for (int k = 0; k < d; ++k) {
        fa.G[k] = G[k];
        fa.D[k] = (D && k < d - 1) ? D[k] : nullptr;
        bd.gc[k] = reinterpret_cast<float *>(at(ws, L.gc[k]));
        fa.Gc[k] = bd.gc[k];
        fa.m[k] = int(p->s.m[k]);
        fa.n[k] = int(p->s.n[k]);
    }
    for (int k = 0; k <= d; ++k) {
        fa.r[k] = int(p->s.r[k]);
        fa.rc[k] = int(p->rho[k]);
        fa.act[k] = p->act[k];
    }
    int e = launch_fold(fa, stream);
    if (e) return e;
    const bool bf = p->s.act == COMERA_BF16;
    if (d == 1) {
        // W = G_0[0, :, :, 0]^T: a GEMM with a single 1 on the left
        float *ones = reinterpret_cast<float *>(at(ws, L.ones));
        e = launch_fill_one(ones, stream);
        if (e) return e;
        return chain_gemm(ones, bd.gc[0], at(ws, L.w), bf, 1, 1, 1, int(p->s.n[0]), int(p->s.m[0]), 1, stream,
                          transpose ? kChainT : kChainNormal);
    }
    bd.P[1] = bd.gc[0];  // rho_0 = 1: [n_0][m_0][rho_1] is the folded core itself
    int64_t Il = p->s.n[0], Jl = p->s.m[0];
    for (int k = 1; k < d; ++k) {
        const bool last = k == d - 1;
        void *out = last ? at(ws, L.w) : at(ws, L.p[k + 1]);
        int qb = 0;
        if (last && wbuild_tiles(Il, Jl, int(p->rho[k]), int(p->s.n[k]), int(p->s.m[k]), transpose, qb)) {
            WBuildArgs wa;
            wa.P = bd.P[k];
            wa.G = bd.gc[k];
            wa.out = out;
            wa.NI = Il;
            wa.NJ = Jl;
            wa.A = int(p->rho[k]);
            wa.nx = int(p->s.n[k]);
            wa.ny = int(p->s.m[k]);
            wa.transpose = transpose ? 1 : 0;
            wa.out_bf16 = bf ? 1 : 0;
            wa.QB = qb;
            return launch_wbuild(wa, stream);
        }
        e = chain_gemm(bd.P[k], bd.gc[k], out, last && bf, Il, Jl, int(p->rho[k]), int(p->s.n[k]), int(p->s.m[k]),
                       int(p->rho[k + 1]), stream, last && transpose ? kChainT : kChainNormal);
        if (e) return e;
        if (!last) bd.P[k + 1] = reinterpret_cast<float *>(out);
        Il *= p->s.n[k];
        Jl *= p->s.m[k];
    }
    return 0;
}

comera_status hip_status(int e) { return e ? COMERA_ERR_HIP : COMERA_OK; }

// Core gradients from the split partials of dW (eq. back Gi): one fused
// projection step per core k = d-1 .. 1 (right environment E_k and the meet
// with P_k), then the expand kernel sums the meet partials (and, for core 0,
// the slices of E_1) in a fixed order, unswaps, applies the masks and writes
// zeros on inactive slices.
comera_status project_dense(const comera_ttm_plan_s *p, const DenseBuild &bd, const float *dw_part, int splits,
                            const float *const *D, float *const *dG, void *ws, void *stream) {
    const DenseLayout &L = p->dense;
    const int d = p->d;
    const float *En = dw_part;
    int nin = splits;
    int64_t in_stride = p->N_in * p->N_out;
    int64_t Il = p->N_in, Jl = p->N_out;
    ExpandArgs xa;
    std::memset(&xa, 0, sizeof(xa));
    for (int k = d - 1; k >= 1; --k) {
        Il /= p->s.n[k];
        Jl /= p->s.m[k];
        const int A = int(p->rho[k]);
        const int64_t rows = Il * Jl, cols = p->s.n[k] * p->s.m[k] * p->rho[k + 1];
        ProjArgs pa;
        pa.En = En;
        pa.nin = nin;
        pa.in_stride = in_stride;
        pa.Gc = bd.gc[k];
        pa.P = dG[k] ? bd.P[k] : nullptr;
        pa.Eout = reinterpret_cast<float *>(at(ws, L.e[k]));
        pa.out_stride = rows * A;
        // E_k blocked for step k-1: [(I', J')][(x', y')][a], I = I' n_{k-1} + x',
        // J = J' m_{k-1} + y'
        const int64_t nxp = p->s.n[k - 1], nyp = p->s.m[k - 1], NJp = Jl / nyp;
        pa.rmap.nd = 4;
        pa.rmap.radix[1] = nxp;
        pa.rmap.radix[2] = NJp;
        pa.rmap.radix[3] = nyp;
        pa.rmap.stride[0] = NJp * nxp * nyp * A;
        pa.rmap.stride[1] = nyp * A;
        pa.rmap.stride[2] = nxp * nyp * A;
        pa.rmap.stride[3] = A;
        pa.part = reinterpret_cast<float *>(at(ws, L.gpart[k]));
        pa.rows = rows;
        pa.cols = cols;
        pa.A = A;
        pa.RT = L.proj_rt[k];
        pa.CT = L.proj_ct[k];
        if (int e = launch_proj(pa, stream)) return hip_status(e);
        xa.part[k] = pa.part;
        xa.splits[k] = L.meet_splits[k];
        En = pa.Eout;
        nin = L.e_slices[k];
        in_stride = pa.out_stride;
    }
    xa.part[0] = En;     // P_0 = 1: the gradient of core 0 is E_1 (or dW when d = 1)
    xa.splits[0] = nin;
    xa.d = d;
    xa.compacted = p->compacted ? 1 : 0;
    xa.swap = 1;
    for (int k = 0; k < d; ++k) {
        xa.D[k] = (D && k < d - 1) ? D[k] : nullptr;
        xa.dG[k] = dG[k];
        xa.m[k] = int(p->s.m[k]);
        xa.n[k] = int(p->s.n[k]);
    }
    for (int k = 0; k <= d; ++k) {
        xa.r[k] = int(p->s.r[k]);
        xa.rc[k] = int(p->rho[k]);
        xa.act[k] = p->act[k];
    }
    return hip_status(launch_expand(xa, stream));
}

}  // namespace

namespace comera {

void timing_begin(comera_ttm_plan_s *p, int kernel, void *stream, void **ev0) {
    *ev0 = nullptr;
    if (!p->timing.on) return;
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return;
    hipEventRecord(e, hipStream_t(stream));
    *ev0 = e;
    (void)kernel;
}

void timing_end(comera_ttm_plan_s *p, int kernel, void *stream, void *ev0) {
    if (!p->timing.on || !ev0) return;
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) {
        hipEventDestroy(hipEvent_t(ev0));
        return;
    }
    hipEventRecord(e, hipStream_t(stream));
    p->timing.ev[kernel].push_back({ev0, e});
}

void timing_clear(comera_ttm_plan_s *p) {
    for (auto &v : p->timing.ev) {
        for (auto &pr : v) {
            hipEventDestroy(hipEvent_t(pr.first));
            hipEventDestroy(hipEvent_t(pr.second));
        }
        v.clear();
    }
}

}  // namespace comera

extern "C" {

comera_status comera_ttm_forward(comera_ttm_plan_t p, int64_t b, const void *X, const float *const *G,
                                 const float *const *D, void *Y, void *ws, size_t ws_bytes, void *stream) {
    if (!p || b < 0 || b > p->batch) return COMERA_ERR_INVALID_ARG;
    if (b == 0) return COMERA_OK;
    if (!X || !Y) return COMERA_ERR_INVALID_ARG;
    const size_t esz = p->s.act == COMERA_BF16 ? 2 : 4;
    if (p->zero) return hip_status(launch_fill_zero(Y, size_t(b) * size_t(p->N_out) * esz, stream));
    if (!G) return COMERA_ERR_INVALID_ARG;
    for (int k = 0; k < p->d; ++k)
        if (!G[k]) return COMERA_ERR_INVALID_ARG;
    if (!ws || ws_bytes < p->ws_bytes) return COMERA_ERR_WORKSPACE;
    DenseBuild bd;
    int e = build_dense(p, G, D, ws, stream, bd, true);
    if (e) return COMERA_ERR_HIP;
    // Y[b, N_out] = X[b, N_in] W (eq. forward), W^T read row by row
    void *ev;
    timing_begin(p, COMERA_KERNEL_FWD, stream, &ev);
    GemmArgs g;
    g.dtype = p->s.act;
    g.a_kc = true;
    g.b_kc = true;
    g.out_bf16 = p->s.act == COMERA_BF16;
    g.A = X;
    g.B = at(ws, p->dense.w);
    g.C = Y;
    g.M = b;
    g.N = p->N_out;
    g.K = p->N_in;
    g.lda = p->N_in;
    g.ldb = p->N_in;
    g.rmap = remap_linear(p->N_out);
    g.cmap = remap_linear(1);
    e = launch_gemm(g, stream);
    timing_end(p, COMERA_KERNEL_FWD, stream, ev);
    return hip_status(e);
}

comera_status comera_ttm_backward(comera_ttm_plan_t p, int64_t b, const void *X, const void *dY,
                                  const float *const *G, const float *const *D, void *dX, float *const *dG,
                                  void *ws, size_t ws_bytes, void *stream) {
    if (!p || b < 0 || b > p->batch) return COMERA_ERR_INVALID_ARG;
    const int d = p->d;
    const size_t esz = p->s.act == COMERA_BF16 ? 2 : 4;
    bool want_dg = false;
    if (dG)
        for (int k = 0; k < d; ++k) want_dg = want_dg || dG[k];
    // nothing flows when the batch is empty or a bond is fully masked
    if (b == 0 || p->zero) {
        int e = 0;
        if (dX && b > 0) e = launch_fill_zero(dX, size_t(b) * size_t(p->N_in) * esz, stream);
        for (int k = 0; want_dg && k < d && !e; ++k)
            if (dG[k])
                e = launch_fill_zero(dG[k], sizeof(float) * size_t(p->s.r[k] * p->s.m[k] * p->s.n[k] * p->s.r[k + 1]),
                                     stream);
        return hip_status(e);
    }
    if (!dY || !G || (want_dg && !X)) return COMERA_ERR_INVALID_ARG;
    for (int k = 0; k < d; ++k)
        if (!G[k]) return COMERA_ERR_INVALID_ARG;
    if (!ws || ws_bytes < p->ws_bytes) return COMERA_ERR_WORKSPACE;
    const DenseLayout &L = p->dense;
    DenseBuild bd;
    int e = build_dense(p, G, D, ws, stream, bd, false);
    if (e) return COMERA_ERR_HIP;
    if (dX) {
        // dX[b, N_in] = dY[b, N_out] W^T  (eq. back X)
        void *ev;
        timing_begin(p, COMERA_KERNEL_DX, stream, &ev);
        GemmArgs g;
        g.dtype = p->s.act;
        g.a_kc = true;
        g.b_kc = true;
        g.out_bf16 = p->s.act == COMERA_BF16;
        g.A = dY;
        g.B = at(ws, L.w);
        g.C = dX;
        g.M = b;
        g.N = p->N_in;
        g.K = p->N_out;
        g.lda = p->N_out;
        g.ldb = p->N_out;
        g.rmap = remap_linear(p->N_in);
        g.cmap = remap_linear(1);
        if (L.dx_splits > 1) {
            g.C = at(ws, L.dx_part);
            g.splits = L.dx_splits;
            g.kchunk = L.dx_kchunk;
            g.split_stride = b * p->N_in;
        }
        e = launch_gemm(g, stream);
        if (!e && L.dx_splits > 1)
            e = launch_sum_splits(reinterpret_cast<const float *>(at(ws, L.dx_part)), reinterpret_cast<float *>(dX),
                                  b * p->N_in, L.dx_splits, stream);
        timing_end(p, COMERA_KERNEL_DX, stream, ev);
        if (e) return COMERA_ERR_HIP;
    }
    if (!want_dg) return COMERA_OK;
    // dW = X^T dY (split over tokens, fixed-order split sum), written blocked
    // as E_d[(I_<, J_<)][(x, y)] with x = i_{d-1}, y = j_{d-1}
    const int64_t nl = p->s.n[d - 1], ml = p->s.m[d - 1];
    const int64_t NJl = p->N_out / ml;
    const int splits = int((b + L.dw_kchunk - 1) / L.dw_kchunk);
    float *dw = reinterpret_cast<float *>(at(ws, L.dw));
    float *dwp = (splits > 1 || L.proj) ? reinterpret_cast<float *>(at(ws, L.dw_part)) : dw;
    {
        void *ev;
        timing_begin(p, COMERA_KERNEL_DW, stream, &ev);
        GemmArgs g;
        g.dtype = p->s.act;
        g.a_kc = false;
        g.b_kc = false;
        g.out_bf16 = false;
        g.A = X;
        g.B = dY;
        g.C = dwp;
        g.M = p->N_in;
        g.N = p->N_out;
        g.K = b;
        g.lda = p->N_in;
        g.ldb = p->N_out;
        g.rmap.nd = 2;
        g.rmap.radix[1] = nl;
        g.rmap.stride[0] = NJl * nl * ml;
        g.rmap.stride[1] = ml;
        g.cmap.nd = 2;
        g.cmap.radix[1] = ml;
        g.cmap.stride[0] = nl * ml;
        g.cmap.stride[1] = 1;
        g.splits = splits;
        g.kchunk = L.dw_kchunk;
        g.split_stride = p->N_in * p->N_out;
        e = launch_gemm(g, stream);
        timing_end(p, COMERA_KERNEL_DW, stream, ev);
        if (e) return COMERA_ERR_HIP;
    }
    if (L.proj) return project_dense(p, bd, dwp, splits, D, dG, ws, stream);
    if (splits > 1) {
        e = launch_sum_splits(dwp, dw, p->N_in * p->N_out, splits, stream);
        if (e) return COMERA_ERR_HIP;
    }
    // right environments E_k = dW contracted with cores k..d-1, each written
    // blocked for the next step (eq. back Gi, read right to left)
    float *E[kMaxCores + 1];
    E[d] = dw;
    int64_t Il = p->N_in, Jl = p->N_out;
    for (int k = d - 1; k >= 1; --k) {
        Il /= p->s.n[k];
        Jl /= p->s.m[k];
        E[k] = reinterpret_cast<float *>(at(ws, L.e[k]));
        e = adjoint_gemm(E[k + 1], bd.gc[k], E[k], Il, Jl, int(p->rho[k]), int(p->s.n[k]), int(p->s.m[k]),
                         int(p->rho[k + 1]), int(p->s.n[k - 1]), int(p->s.m[k - 1]), L.adj_splits[k],
                         reinterpret_cast<float *>(at(ws, L.adj_part)), stream);
        if (e) return COMERA_ERR_HIP;
    }
    // core gradients: meet of P_k and E_{k+1}, then expand to the full layout
    ExpandArgs xa;
    std::memset(&xa, 0, sizeof(xa));
    xa.d = d;
    xa.compacted = p->compacted ? 1 : 0;
    xa.swap = 1;
    Il = 1;
    Jl = 1;
    for (int k = 0; k < d; ++k) {
        if (k == 0) {
            xa.part[0] = E[1];    // P_0 = 1: the gradient of core 0 is E_1 itself
            xa.splits[0] = 1;
        } else {
            float *part = reinterpret_cast<float *>(at(ws, L.gpart[k]));
            if (dG[k]) {
                e = meet_gemm(bd.P[k], E[k + 1], part, Il, Jl, int(p->rho[k]), int(p->s.n[k]), int(p->s.m[k]),
                              int(p->rho[k + 1]), L.meet_splits[k], stream);
                if (e) return COMERA_ERR_HIP;
            }
            xa.part[k] = part;
            xa.splits[k] = L.meet_splits[k];
        }
        xa.D[k] = (D && k < d - 1) ? D[k] : nullptr;
        xa.dG[k] = dG[k];
        xa.m[k] = int(p->s.m[k]);
        xa.n[k] = int(p->s.n[k]);
        Il *= p->s.n[k];
        Jl *= p->s.m[k];
    }
    for (int k = 0; k <= d; ++k) {
        xa.r[k] = int(p->s.r[k]);
        xa.rc[k] = int(p->rho[k]);
        xa.act[k] = p->act[k];
    }
    return hip_status(launch_expand(xa, stream));
}

comera_status comera_ttm_plan_set_timing(comera_ttm_plan_t p, int32_t enable) {
    if (!p) return COMERA_ERR_INVALID_ARG;
    p->timing.on = enable != 0;
    if (!p->timing.on) timing_clear(p);
    return COMERA_OK;
}

comera_status comera_ttm_plan_kernel_time(comera_ttm_plan_t p, int32_t kernel, double *avg_ms, int32_t *count) {
    if (!p || kernel < 0 || kernel > 2) return COMERA_ERR_INVALID_ARG;
    auto &v = p->timing.ev[kernel];
    double tot = 0;
    int n = 0;
    comera_status st = COMERA_OK;
    for (auto &pr : v) {
        float ms = 0.f;
        if (hipEventSynchronize(hipEvent_t(pr.second)) != hipSuccess ||
            hipEventElapsedTime(&ms, hipEvent_t(pr.first), hipEvent_t(pr.second)) != hipSuccess) {
            st = COMERA_ERR_HIP;
        } else {
            tot += ms;
            ++n;
        }
        hipEventDestroy(hipEvent_t(pr.first));
        hipEventDestroy(hipEvent_t(pr.second));
    }
    v.clear();
    if (avg_ms) *avg_ms = n ? tot / n : 0.0;
    if (count) *count = n;
    return st;
}

}  // extern "C"
