// extern "C" entry points for one TTM linear layer: comera_ttm_forward and
// comera_ttm_backward.  Every step runs as a kernel on the caller's stream.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>
#include <mutex>

#include "internal.h"

using namespace comera;

namespace {

inline char *at(void *ws, size_t off) { return reinterpret_cast<char *>(ws) + off; }

thread_local char g_last_hip_error[160];

}  // namespace

namespace comera {

int note_hip(int e, const char *where) {
    if (e)
        snprintf(g_last_hip_error, sizeof(g_last_hip_error), "%s (%d) in %s", hipGetErrorName(hipError_t(e)), e,
                 where);
    return e;
}

void dense_ptrs(const comera_ttm_plan_s *sp, void *ws, DenseBuild &bd) {
    std::memset(&bd, 0, sizeof(bd));
    for (int k = 0; k < sp->d; ++k) bd.gc[k] = reinterpret_cast<float *>(at(ws, sp->dense.gc[k]));
}

int fold_cores(const comera_ttm_plan_s *p, const float *const *G, const float *const *D, float *const *dst,
               const CoreStrides *st, void *stream) {
    const int d = p->d;
    FoldArgs fa;
    std::memset(&fa, 0, sizeof(fa));
    fa.d = d;
    fa.nfold = d;
    fa.compacted = p->compacted ? 1 : 0;
    for (int k = 0; k < d; ++k) {
        fa.G[k] = G[k];
        fa.D[k] = (D && k < d - 1) ? D[k] : nullptr;
        fa.Gc[k] = dst[k];
        fa.m[k] = int(p->s.m[k]);
        fa.n[k] = int(p->s.n[k]);
        fa.st[k] = st[k];
    }
    for (int k = 0; k <= d; ++k) {
        fa.r[k] = int(p->s.r[k]);
        fa.rc[k] = int(p->rho[k]);
        fa.act[k] = p->act[k];
    }
    return note_hip(launch_fold(fa, stream), "fold");
}

// Left chains P_1..P_{d-1} and W (eq. TTM) as one GEMM per core from the
// folded cores; the last step writes W[N_in, N_out] (want & kWantW) and / or
// W^T[N_out, N_in] (want & kWantWT) in the activation dtype.
int build_chain(const comera_ttm_plan_s *sp, void *ws, DenseBuild &bd, int want, void *stream) {
    const DenseLayout &L = sp->dense;
    const int d = sp->d;
    const bool bf = sp->s.act == COMERA_BF16 && !sp->fp8;   // FP8 layers build W in fp32
    bd.w = at(ws, L.w);
    bd.wt = at(ws, L.wt);
    if (d == 1) {
        // W = G_0[0, :, :, 0]^T: the folded core [n][m] itself in fp32, else
        // a GEMM with a single 1 on the left
        if (!bf && want == kWantW) {
            bd.w = bd.gc[0];
            return 0;
        }
        float *ones = reinterpret_cast<float *>(at(ws, L.ones));
        int e = note_hip(launch_fill_one(ones, stream), "fill");
        for (int t = 0; t < 2 && !e; ++t) {
            const bool tr = t == 1;
            if (!(want & (tr ? kWantWT : kWantW))) continue;
            e = note_hip(chain_gemm(ones, bd.gc[0], tr ? bd.wt : bd.w, bf, 1, 1, 1, int(sp->s.n[0]),
                                    int(sp->s.m[0]), 1, stream, tr ? kChainT : kChainNormal),
                         "chain GEMM");
        }
        return e;
    }
    bd.P[1] = bd.gc[0];  // rho_0 = 1: [n_0][m_0][rho_1] is the folded core itself
    int64_t Il = sp->s.n[0], Jl = sp->s.m[0];
    for (int k = 1; k < d; ++k) {
        const bool last = k == d - 1;
        if (!last) {
            void *out = at(ws, L.p[k + 1]);
            int e = 0;
            if (lchain_supported(int(sp->rho[k]))) {
                LChainArgs la;
                la.P = bd.P[k];
                la.G = bd.gc[k];
                la.out = reinterpret_cast<float *>(out);
                la.NI = Il;
                la.NJ = Jl;
                la.A = int(sp->rho[k]);
                la.nx = int(sp->s.n[k]);
                la.ny = int(sp->s.m[k]);
                la.C = int(sp->rho[k + 1]);
                e = launch_lchain(la, stream);
            } else {
                e = chain_gemm(bd.P[k], bd.gc[k], out, false, Il, Jl, int(sp->rho[k]), int(sp->s.n[k]),
                               int(sp->s.m[k]), int(sp->rho[k + 1]), stream, kChainNormal);
            }
            if (e) return note_hip(e, "chain GEMM");
            bd.P[k + 1] = reinterpret_cast<float *>(out);
            Il *= sp->s.n[k];
            Jl *= sp->s.m[k];
            continue;
        }
        int qi = 0, qj = 0;
        if (wbuild_tiles(Il, Jl, int(sp->rho[k]), int(sp->s.n[k]), int(sp->s.m[k]), qi, qj)) {
            WBuildArgs wa;
            wa.P = bd.P[k];
            wa.G = bd.gc[k];
            wa.out = (want & kWantW) ? bd.w : nullptr;
            wa.out_t = (want & kWantWT) ? bd.wt : nullptr;
            wa.NI = Il;
            wa.NJ = Jl;
            wa.A = int(sp->rho[k]);
            wa.nx = int(sp->s.n[k]);
            wa.ny = int(sp->s.m[k]);
            wa.out_bf16 = bf ? 1 : 0;
            wa.QI = qi;
            wa.QJ = qj;
            return note_hip(launch_wbuild(wa, stream), "W build");
        }
        for (int t = 0; t < 2; ++t) {
            const bool tr = t == 1;
            if (!(want & (tr ? kWantWT : kWantW))) continue;
            int e = chain_gemm(bd.P[k], bd.gc[k], tr ? bd.wt : bd.w, bf, Il, Jl, int(sp->rho[k]), int(sp->s.n[k]),
                               int(sp->s.m[k]), int(sp->rho[k + 1]), stream, tr ? kChainT : kChainNormal);
            if (e) return note_hip(e, "chain GEMM");
        }
    }
    return 0;
}

void built_dense(const comera_ttm_plan_s *p, void *ws, DenseBuild &bd, int want) {
    dense_ptrs(p, ws, bd);
    bd.P[1] = bd.gc[0];
    for (int k = 1; k + 1 < p->d; ++k) bd.P[k + 1] = reinterpret_cast<float *>(at(ws, p->dense.p[k + 1]));
    bd.w = at(ws, p->dense.w);
    bd.wt = at(ws, p->dense.wt);
    // build_chain keeps a single fp32 core as W itself
    if (p->d == 1 && (p->s.act != COMERA_BF16 || p->fp8) && want == kWantW) bd.w = bd.gc[0];
}

int dw_gemm(const comera_ttm_plan_s *sp, const void *A, int64_t lda, const void *B, int64_t ldb, int64_t K,
            void *ws, float **dwp, int *splits_out, void *stream, const float *oscale) {
    const DenseLayout &L = sp->dense;
    const int d = sp->d;
    // written blocked as E_d[(I_<, J_<)][(x, y)] with x = i_{d-1}, y = j_{d-1}
    const int64_t nl = sp->s.n[d - 1], ml = sp->s.m[d - 1];
    const int64_t NJl = sp->N_out / ml;
    const int splits = int((K + L.dw_kchunk - 1) / L.dw_kchunk);
    float *dw = reinterpret_cast<float *>(at(ws, L.dw));
    float *part = (splits > 1 || L.proj) ? reinterpret_cast<float *>(at(ws, L.dw_part)) : dw;
    GemmArgs g;
    g.dtype = oscale ? kDtypeFp8 : sp->s.act;
    g.a_kc = oscale != nullptr;
    g.b_kc = oscale != nullptr;
    g.out_bf16 = false;
    g.oscale = oscale;
    g.A = A;
    g.B = B;
    g.C = part;
    g.M = sp->N_in;
    g.N = sp->N_out;
    g.K = K;
    g.lda = lda;
    g.ldb = ldb;
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
    g.split_stride = sp->N_in * sp->N_out;
    *dwp = part;
    *splits_out = splits;
    return note_hip(launch_gemm(g, stream), "dW GEMM");
}

// Core gradients from the split partials of dW (eq. back Gi).  Fused route:
// one projection step per core k = d-1 .. 1 (right environment E_k and the
// meet with P_k); the gradient of core 0 is E_1 (or dW itself when d = 1)
// as slices.  Otherwise: the fixed-order split sum, one adjoint GEMM per
// environment and one meet GEMM per core.
int project_cores(const comera_ttm_plan_s *sp, const DenseBuild &bd, const float *dwp, int splits,
                  const bool *want, void *ws, const float **part, int *nsplit, void *stream) {
    const DenseLayout &L = sp->dense;
    const int d = sp->d;
    if (L.proj) {
        const float *En = dwp;
        int nin = splits;
        int64_t in_stride = sp->N_in * sp->N_out;
        int64_t Il = sp->N_in, Jl = sp->N_out;
        for (int k = d - 1; k >= 1; --k) {
            Il /= sp->s.n[k];
            Jl /= sp->s.m[k];
            const int A = int(sp->rho[k]);
            const int64_t rows = Il * Jl, cols = sp->s.n[k] * sp->s.m[k] * sp->rho[k + 1];
            ProjArgs pa;
            pa.En = En;
            pa.nin = nin;
            pa.in_stride = in_stride;
            pa.Gc = bd.gc[k];
            pa.P = want[k] ? bd.P[k] : nullptr;
            pa.Eout = reinterpret_cast<float *>(at(ws, L.e[k]));
            pa.out_stride = rows * A;
            // E_k blocked for step k-1: [(I', J')][(x', y')][a], I = I' n_{k-1} + x',
            // J = J' m_{k-1} + y'
            const int64_t nxp = sp->s.n[k - 1], nyp = sp->s.m[k - 1], NJp = Jl / nyp;
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
            if (int e = launch_proj(pa, stream)) return note_hip(e, "projection");
            part[k] = pa.part;
            nsplit[k] = L.meet_splits[k];
            En = pa.Eout;
            nin = L.e_slices[k];
            in_stride = pa.out_stride;
        }
        part[0] = En;
        nsplit[0] = nin;
        return 0;
    }
    float *dw = reinterpret_cast<float *>(at(ws, L.dw));
    if (splits > 1) {
        if (int e = launch_sum_splits(dwp, dw, sp->N_in * sp->N_out, splits, stream)) return note_hip(e, "split sum");
    } else {
        dw = const_cast<float *>(dwp);
    }
    // right environments E_k = dW contracted with cores k..d-1, each written
    // blocked for the next step (eq. back Gi, read right to left)
    float *E[kMaxCores + 1];
    E[d] = dw;
    int64_t Il = sp->N_in, Jl = sp->N_out;
    for (int k = d - 1; k >= 1; --k) {
        Il /= sp->s.n[k];
        Jl /= sp->s.m[k];
        E[k] = reinterpret_cast<float *>(at(ws, L.e[k]));
        int e = adjoint_gemm(E[k + 1], bd.gc[k], E[k], Il, Jl, int(sp->rho[k]), int(sp->s.n[k]), int(sp->s.m[k]),
                             int(sp->rho[k + 1]), int(sp->s.n[k - 1]), int(sp->s.m[k - 1]), L.adj_splits[k],
                             reinterpret_cast<float *>(at(ws, L.adj_part)), stream);
        if (e) return note_hip(e, "adjoint GEMM");
    }
    // meets of P_k and E_{k+1}
    part[0] = E[1];    // P_0 = 1: the gradient of core 0 is E_1 itself
    nsplit[0] = 1;
    Il = sp->s.n[0];
    Jl = sp->s.m[0];
    for (int k = 1; k < d; ++k) {
        float *gp = reinterpret_cast<float *>(at(ws, L.gpart[k]));
        if (want[k]) {
            int e = meet_gemm(bd.P[k], E[k + 1], gp, Il, Jl, int(sp->rho[k]), int(sp->s.n[k]), int(sp->s.m[k]),
                              int(sp->rho[k + 1]), L.meet_splits[k], stream);
            if (e) return note_hip(e, "meet GEMM");
        }
        part[k] = gp;
        nsplit[k] = L.meet_splits[k];
        Il *= sp->s.n[k];
        Jl *= sp->s.m[k];
    }
    return 0;
}

// The expand kernel sums the partials of each core in a fixed order,
// unfolds the compacted layout, applies the masks and writes zeros on
// inactive slices.
int expand_cores(const comera_ttm_plan_s *p, const float *const *part, const int *nsplit, const CoreStrides *st,
                 const float *const *D, float *const *dG, void *stream) {
    const int d = p->d;
    ExpandArgs xa;
    std::memset(&xa, 0, sizeof(xa));
    xa.d = d;
    xa.compacted = p->compacted ? 1 : 0;
    for (int k = 0; k < d; ++k) {
        xa.part[k] = part[k];
        xa.splits[k] = nsplit[k];
        xa.st[k] = st[k];
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
    return note_hip(launch_expand(xa, stream), "expand");
}

int mask_grads(const comera_ttm_plan_s *p, const float *const *part, const int *nsplit, const CoreStrides *st,
               const float *const *G, float *const *dD, void *stream) {
    if (!dD) return 0;
    const int d = p->d;
    MaskGradArgs ma;
    std::memset(&ma, 0, sizeof(ma));
    ma.d = d;
    ma.compacted = p->compacted ? 1 : 0;
    for (int k = 0; k < d; ++k) {
        ma.part[k] = part[k];
        ma.splits[k] = nsplit[k];
        ma.st[k] = st[k];
        ma.G[k] = G[k];
        ma.dD[k] = k < d - 1 ? dD[k] : nullptr;
        ma.m[k] = int(p->s.m[k]);
        ma.n[k] = int(p->s.n[k]);
    }
    for (int k = 0; k <= d; ++k) {
        ma.r[k] = int(p->s.r[k]);
        ma.rc[k] = int(p->rho[k]);
        ma.act[k] = p->act[k];
    }
    return note_hip(launch_mask_grad(ma, stream), "mask gradients");
}

}  // namespace comera

namespace {

// placement of the folded cores of the dense order: [rho_k][n_k][m_k][rho_{k+1}]
void dense_strides(const comera_ttm_plan_s *p, CoreStrides *st) {
    for (int k = 0; k < p->d; ++k)
        st[k] = core_strides(int(p->rho[k]), int(p->s.m[k]), int(p->s.n[k]), int(p->rho[k + 1]), true);
}

// fold, chains and W of the dense order
int build_dense(const comera_ttm_plan_s *p, const float *const *G, const float *const *D, void *ws, void *stream,
                DenseBuild &bd, int want) {
    dense_ptrs(p, ws, bd);
    CoreStrides st[kMaxCores];
    dense_strides(p, st);
    if (p->d == 3 && (want & (kWantW | kWantWT))) {
        Build3Args ba;
        std::memset(&ba, 0, sizeof(ba));
        int n[3], m[3];
        for (int k = 0; k < 3; ++k) {
            n[k] = int(p->s.n[k]);
            m[k] = int(p->s.m[k]);
        }
        if (build3_tiles(n, m, int(p->rho[1]), int(p->rho[2]), ba.SX, ba.SY, ba.PX, ba.PY) &&
            (!p->compacted || (p->s.r[1] <= 256 && p->s.r[2] <= 256))) {
            const bool bf = p->s.act == COMERA_BF16 && !p->fp8;
            for (int k = 0; k < 3; ++k) {
                ba.G[k] = G[k];
                ba.Gc[k] = bd.gc[k];
                ba.st[k] = st[k];
                ba.n[k] = n[k];
                ba.m[k] = m[k];
            }
            ba.D[0] = D ? D[0] : nullptr;
            ba.D[1] = D ? D[1] : nullptr;
            ba.P2 = reinterpret_cast<float *>(at(ws, p->dense.p[2]));
            bd.P[1] = bd.gc[0];
            bd.P[2] = ba.P2;
            bd.w = at(ws, p->dense.w);
            bd.wt = at(ws, p->dense.wt);
            ba.w = (want & kWantW) ? bd.w : nullptr;
            ba.wt = (want & kWantWT) ? bd.wt : nullptr;
            ba.act1 = p->act[1];
            ba.act2 = p->act[2];
            ba.r1 = int(p->s.r[1]);
            ba.r2 = int(p->s.r[2]);
            ba.A = int(p->rho[1]);
            ba.C = int(p->rho[2]);
            ba.compacted = p->compacted ? 1 : 0;
            ba.out_bf16 = bf ? 1 : 0;
            return note_hip(launch_build3(ba, stream), "W build (three cores)");
        }
    }
    if (int e = fold_cores(p, G, D, bd.gc, st, stream)) return e;
    return build_chain(p, ws, bd, want, stream);
}

inline uint8_t *codes(void *ws, size_t off) { return reinterpret_cast<uint8_t *>(at(ws, off)); }

// Mixed-precision forward (the batch product on FP8 codes, the batch-free
// build of W in fp32): W -> W^T codes (and W codes for a backward call that
// reuses them), X -> X codes (and X^T codes likewise), Y = X8 W8 / (sX sW).
comera_status fp8_forward(comera_ttm_plan_t p, int64_t b, const void *X, const float *const *G,
                          const float *const *D, void *Y, void *ws, void *stream) {
    const Fp8Layout &F = p->f8;
    DenseBuild bd;
    if (build_dense(p, G, D, ws, stream, bd, kWantW)) return COMERA_ERR_HIP;
    float *sc = reinterpret_cast<float *>(at(ws, F.sc));
    float *pmax = reinterpret_cast<float *>(at(ws, F.pmax));
    int e = note_hip(launch_fp8_quant(bd.w, COMERA_F32, p->N_in, p->N_out, pmax, p->reuse ? codes(ws, F.w8) : nullptr,
                                      F.nout_p, codes(ws, F.w8t), F.nin_p, sc + kScW, nullptr, nullptr, nullptr,
                                      nullptr, stream),
                     "FP8 codes of W");
    if (!e)
        e = note_hip(launch_fp8_quant(X, p->s.act, b, p->N_in, pmax, codes(ws, F.x8), F.nin_p,
                                      p->reuse ? codes(ws, F.x8t) : nullptr, F.b_p, sc + kScX, sc + kScW,
                                      sc + kScFwd, nullptr, nullptr, stream),
                     "FP8 codes of X");
    if (e) return COMERA_ERR_HIP;
    void *ev;
    timing_begin(p, COMERA_KERNEL_FWD, stream, &ev);
    GemmArgs g;
    g.dtype = kDtypeFp8;
    g.a_kc = true;
    g.b_kc = true;
    g.out_bf16 = p->s.act == COMERA_BF16;
    g.A = codes(ws, F.x8);
    g.B = codes(ws, F.w8t);
    g.C = Y;
    g.M = b;
    g.N = p->N_out;
    g.K = F.nin_p;
    g.lda = F.nin_p;
    g.ldb = F.nin_p;
    g.rmap = remap_linear(p->N_out);
    g.cmap = remap_linear(1);
    g.oscale = sc + kScFwd;
    e = note_hip(launch_gemm(g, stream), "forward GEMM (FP8)");
    timing_end(p, COMERA_KERNEL_FWD, stream, ev);
    return e ? COMERA_ERR_HIP : COMERA_OK;
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

namespace {

// Dense order: build W^T (and W for a backward that reuses it), then
// Y[b, N_out] = X[b, N_in] W (eq. forward), W^T read row by row.  With
// split_ok the product may split over K into the plan's partials region
// (small batches); otherwise it runs unsplit.
comera_status dense_forward(comera_ttm_plan_t p, int64_t b, const void *X, const float *const *G,
                            const float *const *D, void *Y, void *ws, bool split_ok, void *stream) {
    DenseBuild bd;
    int e = build_dense(p, G, D, ws, stream, bd, kWantWT | (p->reuse ? kWantW : 0));
    if (e) return COMERA_ERR_HIP;
    void *ev;
    timing_begin(p, COMERA_KERNEL_FWD, stream, &ev);
    GemmArgs g;
    g.dtype = p->s.act;
    g.a_kc = true;
    g.b_kc = true;
    g.out_bf16 = p->s.act == COMERA_BF16;
    g.A = X;
    g.B = bd.wt;
    g.C = Y;
    g.M = b;
    g.N = p->N_out;
    g.K = p->N_in;
    g.lda = p->N_in;
    g.ldb = p->N_in;
    g.rmap = remap_linear(p->N_out);
    g.cmap = remap_linear(1);
    if (split_ok && p->dense.part_elems > 0) {
        g.scratch = reinterpret_cast<float *>(at(ws, p->dense.part));
        g.scratch_elems = p->dense.part_elems;
        g.out_elems = b * p->N_out;
    }
    e = note_hip(launch_gemm(g, stream), "forward GEMM");
    timing_end(p, COMERA_KERNEL_FWD, stream, ev);
    return e ? COMERA_ERR_HIP : COMERA_OK;
}

// Scratch of comera_ttm_forward_noalloc: one array per GPU, taken when the
// library's code object is loaded on that GPU and held until the process
// ends.  Host code must never pass the array's name to a kernel (on the host
// it is only a stand-in for the symbol); scratch_address() returns this
// GPU's device address of it, looked up once per device with that device
// current.
constexpr size_t kNoAllocScratchBytes = size_t(COMERA_TTM_NOALLOC_SCRATCH_BYTES);
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_dev[kMaxDevices] = {};

int scratch_address(void **out) {
    *out = nullptr;
    if (launch_check_mode()) {   // host-only check: a placeholder, never dereferenced
        *out = reinterpret_cast<void *>(uintptr_t(1) << 40);
        return 0;
    }
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return int(e);
    if (dev < 0 || dev >= kMaxDevices) return int(hipErrorInvalidDevice);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return int(e);
        if (!ptr) return int(hipErrorInvalidSymbol);
        g_scratch_dev[dev] = ptr;
    }
    *out = g_scratch_dev[dev];
    return 0;
}

}  // namespace

extern "C" {

const char *comera_last_hip_error(void) { return g_last_hip_error; }

comera_status comera_ttm_forward(comera_ttm_plan_t p, int64_t b, const void *X, const float *const *G,
                                 const float *const *D, void *Y, void *ws, size_t ws_bytes, void *stream) {
    if (!p || b < 0 || b > p->batch) return COMERA_ERR_INVALID_ARG;
    if (b == 0) return COMERA_OK;
    if (!X || !Y) return COMERA_ERR_INVALID_ARG;
    const size_t esz = p->s.act == COMERA_BF16 ? 2 : 4;
    if (p->zero)
        return note_hip(launch_fill_zero(Y, size_t(b) * size_t(p->N_out) * esz, stream), "fill") ? COMERA_ERR_HIP
                                                                                                 : COMERA_OK;
    if (!G) return COMERA_ERR_INVALID_ARG;
    for (int k = 0; k < p->d; ++k)
        if (!G[k]) return COMERA_ERR_INVALID_ARG;
    if (!ws || ws_bytes < p->ws_bytes) return COMERA_ERR_WORKSPACE;
    if (p->chain) return chain_forward(p, b, X, G, D, Y, ws, stream);
    if (p->sweep.G > 0) return sweep_forward(p, b, X, G, D, Y, ws, stream);
    if (p->fp8) return fp8_forward(p, b, X, G, D, Y, ws, stream);
    return dense_forward(p, b, X, G, D, Y, ws, true, stream);
}

comera_status comera_ttm_forward_noalloc(comera_ttm_plan_t p, int64_t b, const void *X, const float *const *G,
                                         const float *const *D, void *Y, void *stream) {
    if (!p || b < 0 || b > p->batch) return COMERA_ERR_INVALID_ARG;
    if (b == 0) return COMERA_OK;
    if (!X || !Y) return COMERA_ERR_INVALID_ARG;
    const size_t esz = p->s.act == COMERA_BF16 ? 2 : 4;
    if (p->zero)
        return note_hip(launch_fill_zero(Y, size_t(b) * size_t(p->N_out) * esz, stream), "fill") ? COMERA_ERR_HIP
                                                                                                 : COMERA_OK;
    if (!G) return COMERA_ERR_INVALID_ARG;
    for (int k = 0; k < p->d; ++k)
        if (!G[k]) return COMERA_ERR_INVALID_ARG;
    if (p->chain || p->sweep.G > 0 || p->fp8 || p->reuse) return COMERA_ERR_UNSUPPORTED;
    // the unsplit forward of the dense order touches the folded cores, the
    // left chains, W, W^T and the 1.0 cell: every region before the dX partials
    if (p->dense.ones + sizeof(float) > kNoAllocScratchBytes) return COMERA_ERR_UNSUPPORTED;
    void *ws = nullptr;
    if (note_hip(scratch_address(&ws), "scratch address")) return COMERA_ERR_HIP;
    // no timing events: they would be allocations
    const bool timing = p->timing.on;
    p->timing.on = false;
    const comera_status st = dense_forward(p, b, X, G, D, Y, ws, false, stream);
    p->timing.on = timing;
    return st;
}

}  // extern "C"

namespace {

// Mixed-precision backward, up to dW: the codes of W (unless a forward call
// left them), of X^T (for dW, likewise) and of dY / dY^T, then dX =
// dY8 W8^T / (sdY sW).  Returns a HIP error code.
int fp8_backward(comera_ttm_plan_t p, int64_t b, const void *X, const void *dY, const DenseBuild &bd, void *dX,
                 bool want_grad, void *ws, void *stream) {
    const Fp8Layout &F = p->f8;
    float *sc = reinterpret_cast<float *>(at(ws, F.sc));
    float *pmax = reinterpret_cast<float *>(at(ws, F.pmax));
    int e = 0;
    if (!p->reuse) {
        if (dX)
            e = note_hip(launch_fp8_quant(bd.w, COMERA_F32, p->N_in, p->N_out, pmax, codes(ws, F.w8), F.nout_p,
                                          nullptr, 0, sc + kScW, nullptr, nullptr, nullptr, nullptr, stream),
                         "FP8 codes of W");
        if (!e && want_grad)
            e = note_hip(launch_fp8_quant(X, p->s.act, b, p->N_in, pmax, nullptr, 0, codes(ws, F.x8t), F.b_p,
                                          sc + kScX, nullptr, nullptr, nullptr, nullptr, stream),
                         "FP8 codes of X");
    }
    if (!e)
        e = note_hip(launch_fp8_quant(dY, p->s.act, b, p->N_out, pmax, dX ? codes(ws, F.dy8) : nullptr, F.nout_p,
                                      want_grad ? codes(ws, F.dy8t) : nullptr, F.b_p, sc + kScDY,
                                      dX ? sc + kScW : nullptr, sc + kScDX, want_grad ? sc + kScX : nullptr,
                                      sc + kScDW, stream),
                     "FP8 codes of dY");
    if (e || !dX) return e;
    void *ev;
    timing_begin(p, COMERA_KERNEL_DX, stream, &ev);
    GemmArgs g;
    g.dtype = kDtypeFp8;
    g.a_kc = true;
    g.b_kc = true;
    g.out_bf16 = p->s.act == COMERA_BF16;
    g.A = codes(ws, F.dy8);
    g.B = codes(ws, F.w8);
    g.C = dX;
    g.M = b;
    g.N = p->N_in;
    g.K = F.nout_p;
    g.lda = F.nout_p;
    g.ldb = F.nout_p;
    g.rmap = remap_linear(p->N_in);
    g.cmap = remap_linear(1);
    g.oscale = sc + kScDX;
    e = note_hip(launch_gemm(g, stream), "dX GEMM (FP8)");
    timing_end(p, COMERA_KERNEL_DX, stream, ev);
    return e;
}

comera_status backward_impl(comera_ttm_plan_t p, int64_t b, const void *X, const void *dY, const float *const *G,
                            const float *const *D, void *dX, float *const *dG, float *const *dD, void *ws,
                            size_t ws_bytes, void *stream) {
    if (!p || b < 0 || b > p->batch) return COMERA_ERR_INVALID_ARG;
    const int d = p->d;
    const size_t esz = p->s.act == COMERA_BF16 ? 2 : 4;
    bool want_dg = false, want_dd = false;
    if (dG)
        for (int k = 0; k < d; ++k) want_dg = want_dg || dG[k];
    if (dD)
        for (int k = 0; k + 1 < d; ++k) want_dd = want_dd || dD[k];
    if (!want_dd) dD = nullptr;
    // nothing flows when the batch is empty or a bond is fully masked (every
    // mask gradient is then zero too: an entry of the empty bond is declared
    // inactive, and any other entry's derivative is a layer with that bond)
    if (b == 0 || p->zero) {
        int e = 0;
        if (dX && b > 0) e = launch_fill_zero(dX, size_t(b) * size_t(p->N_in) * esz, stream);
        for (int k = 0; want_dg && k < d && !e; ++k)
            if (dG[k])
                e = launch_fill_zero(dG[k], sizeof(float) * size_t(p->s.r[k] * p->s.m[k] * p->s.n[k] * p->s.r[k + 1]),
                                     stream);
        for (int k = 0; want_dd && k + 1 < d && !e; ++k)
            if (dD[k]) e = launch_fill_zero(dD[k], sizeof(float) * size_t(p->s.r[k + 1]), stream);
        return note_hip(e, "fill") ? COMERA_ERR_HIP : COMERA_OK;
    }
    const bool want_grad = want_dg || want_dd;
    if (!dY || !G || (want_grad && !X)) return COMERA_ERR_INVALID_ARG;
    for (int k = 0; k < d; ++k)
        if (!G[k]) return COMERA_ERR_INVALID_ARG;
    if (!ws || ws_bytes < p->ws_bytes) return COMERA_ERR_WORKSPACE;
    if (p->chain) return chain_backward(p, b, X, dY, G, D, dX, want_dg ? dG : nullptr, dD, ws, stream);
    if (p->sweep.G > 0) return sweep_backward(p, b, X, dY, G, D, dX, want_dg ? dG : nullptr, dD, ws, stream);
    const DenseLayout &L = p->dense;
    DenseBuild bd;
    int e = 0;
    if (p->reuse)
        built_dense(p, ws, bd, p->fp8 ? kWantW : kWantWT | kWantW);
    else
        e = build_dense(p, G, D, ws, stream, bd, kWantW);
    if (e) return COMERA_ERR_HIP;
    if (p->fp8) {
        e = fp8_backward(p, b, X, dY, bd, dX, want_grad, ws, stream);
        if (e) return COMERA_ERR_HIP;
    }
    if (dX && !p->fp8) {
        // dX[b, N_in] = dY[b, N_out] W^T  (eq. back X)
        void *ev;
        timing_begin(p, COMERA_KERNEL_DX, stream, &ev);
        GemmArgs g;
        g.dtype = p->s.act;
        g.a_kc = true;
        g.b_kc = true;
        g.out_bf16 = p->s.act == COMERA_BF16;
        g.A = dY;
        g.B = bd.w;
        g.C = dX;
        g.M = b;
        g.N = p->N_in;
        g.K = p->N_out;
        g.lda = p->N_out;
        g.ldb = p->N_out;
        g.rmap = remap_linear(p->N_in);
        g.cmap = remap_linear(1);
        if (L.dx_splits == 1 && L.part_elems > 0) {
            g.scratch = reinterpret_cast<float *>(at(ws, L.part));
            g.scratch_elems = L.part_elems;
            g.out_elems = b * p->N_in;
        }
        if (L.dx_splits > 1) {
            g.C = at(ws, L.dx_part);
            g.splits = L.dx_splits;
            g.kchunk = L.dx_kchunk;
            g.split_stride = b * p->N_in;
        }
        e = note_hip(launch_gemm(g, stream), "dX GEMM");
        if (!e && L.dx_splits > 1)
            e = note_hip(launch_sum_splits(reinterpret_cast<const float *>(at(ws, L.dx_part)),
                                           reinterpret_cast<float *>(dX), b * p->N_in, L.dx_splits, stream),
                         "split sum");
        timing_end(p, COMERA_KERNEL_DX, stream, ev);
        if (e) return COMERA_ERR_HIP;
    }
    if (!want_grad) return COMERA_OK;
    // dW = X^T dY (split over tokens, fixed-order split sums); FP8: on the
    // transposed codes, K padded to whole 128-token tiles with zero codes
    float *dwp = nullptr;
    int splits = 0;
    {
        void *ev;
        timing_begin(p, COMERA_KERNEL_DW, stream, &ev);
        if (p->fp8) {
            const Fp8Layout &F = p->f8;
            e = dw_gemm(p, codes(ws, F.x8t), F.b_p, codes(ws, F.dy8t), F.b_p, (b + 127) / 128 * 128, ws, &dwp,
                        &splits, stream, reinterpret_cast<const float *>(at(ws, F.sc)) + kScDW);
        } else {
            e = dw_gemm(p, X, p->N_in, dY, p->N_out, b, ws, &dwp, &splits, stream);
        }
        timing_end(p, COMERA_KERNEL_DW, stream, ev);
        if (e) return COMERA_ERR_HIP;
    }
    bool want[kMaxCores];
    for (int k = 0; k < d; ++k) want[k] = (want_dg && dG[k]) || (dD && k + 1 < d && dD[k]);
    const float *part[kMaxCores];
    int nsplit[kMaxCores];
    e = project_cores(p, bd, dwp, splits, want, ws, part, nsplit, stream);
    if (e) return COMERA_ERR_HIP;
    CoreStrides st[kMaxCores];
    dense_strides(p, st);
    if (want_dg && expand_cores(p, part, nsplit, st, D, dG, stream)) return COMERA_ERR_HIP;
    return mask_grads(p, part, nsplit, st, G, dD, stream) ? COMERA_ERR_HIP : COMERA_OK;
}

}  // namespace

extern "C" {

comera_status comera_ttm_backward(comera_ttm_plan_t p, int64_t b, const void *X, const void *dY,
                                  const float *const *G, const float *const *D, void *dX, float *const *dG,
                                  void *ws, size_t ws_bytes, void *stream) {
    return backward_impl(p, b, X, dY, G, D, dX, dG, nullptr, ws, ws_bytes, stream);
}

comera_status comera_ttm_backward_masks(comera_ttm_plan_t p, int64_t b, const void *X, const void *dY,
                                        const float *const *G, const float *const *D, void *dX, float *const *dG,
                                        float *const *dD, void *ws, size_t ws_bytes, void *stream) {
    return backward_impl(p, b, X, dY, G, D, dX, dG, dD, ws, ws_bytes, stream);
}

comera_status comera_ttm_plan_set_reuse_forward(comera_ttm_plan_t p, int32_t enable) {
    if (!p) return COMERA_ERR_INVALID_ARG;
    p->reuse = enable != 0;
    return COMERA_OK;
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
