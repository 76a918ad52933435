// Sweep orders of a TTM layer (Prop. 4.1, Sec. 4.2): the cores are grouped,
// each group is contracted into one batch-free matrix W'_g (eq. TTM restricted
// to the group, with its outer bonds folded into its outer factors), and the
// activations pass through the groups one GEMM per group:
//   forward   Y = X W          right to left (last group first) or left to right
//   dX        dX = dY W^T      the mirror sweep over dY (eq. back X)
//   dG        the gradient of W'_g is the meet of the activation state and
//             the dY state at group g (eq. back Gi); it is projected onto the
//             group's own cores as for a dense layer.
// The backward call recomputes the group matrices and the activation states,
// or, when the plan reuses the forward's work, takes them from the workspace
// the forward call left.  Every product
// writes its output already permuted for the next one (mixed-radix epilogue).
#include <hip/hip_runtime.h>

#include <cstring>

#include "internal.h"

namespace comera {
namespace {

inline char *at(void *ws, size_t off) { return reinterpret_cast<char *>(ws) + off; }

comera_status status_of(int e) { return e ? COMERA_ERR_HIP : COMERA_OK; }

int64_t prod(const int64_t *v, int lo, int hi) {
    int64_t x = 1;
    for (int h = lo; h < hi; ++h) x *= v[h];
    return x;
}

Remap remap3(int64_t r1, int64_t r2, int64_t s0, int64_t s1, int64_t s2) {
    Remap r{};
    r.nd = 3;
    r.radix[1] = r1;
    r.radix[2] = r2;
    r.stride[0] = s0;
    r.stride[1] = s1;
    r.stride[2] = s2;
    return r;
}

Remap remap2(int64_t r1, int64_t s0, int64_t s1) {
    Remap r{};
    r.nd = 2;
    r.radix[1] = r1;
    r.stride[0] = s0;
    r.stride[1] = s1;
    return r;
}

// out[rm(r) + cm(c)] = sum_k A[r][k] W(k, c), W = W'_g [K][C] (b_kc false) or
// W'_g^T read from [C][K] (b_kc true); the output covers R x C consecutive
// elements, so a split over K can be summed elementwise
int step(const comera_ttm_plan_s *p, void *ws, const void *A, int64_t R, int64_t K, const void *W, bool b_kc,
         int64_t C, void *out, const Remap &rm, const Remap &cm, void *stream) {
    GemmArgs g;
    g.dtype = p->s.act;
    g.a_kc = true;
    g.b_kc = b_kc;
    g.out_bf16 = p->s.act == COMERA_BF16;
    g.A = A;
    g.B = W;
    g.C = out;
    g.M = R;
    g.N = C;
    g.K = K;
    g.lda = K;
    g.ldb = b_kc ? K : C;
    g.rmap = rm;
    g.cmap = cm;
    if (p->sweep.part_elems > 0) {
        g.scratch = reinterpret_cast<float *>(at(ws, p->sweep.part));
        g.scratch_elems = p->sweep.part_elems;
        g.out_elems = R * C;
    }
    return note_hip(launch_gemm(g, stream), b_kc ? "dY sweep GEMM" : "activation sweep GEMM");
}

struct Groups {
    DenseBuild bd[kMaxCores];
    void *ws[kMaxCores];
};

// fold every core into its group's layer, then build each W'_g [N'_in][N'_out]
int build_groups(const comera_ttm_plan_s *p, const float *const *G, const float *const *D, void *ws, Groups &gr,
                 void *stream) {
    const SweepLayout &L = p->sweep;
    float *dst[kMaxCores];
    for (int g = 0; g < L.G; ++g) {
        gr.ws[g] = at(ws, L.base[g]);
        dense_ptrs(p->sub[g].get(), gr.ws[g], gr.bd[g]);
        for (int k = L.s[g]; k <= L.e[g]; ++k) dst[k] = gr.bd[g].gc[k - L.s[g]];
    }
    if (int e = fold_cores(p, G, D, dst, L.st, stream)) return e;
    for (int g = 0; g < L.G; ++g)
        if (int e = build_chain(p->sub[g].get(), gr.ws[g], gr.bd[g], kWantW, stream)) return e;
    return 0;
}

// pointers of the groups an earlier forward call built (reuse)
void built_groups(const comera_ttm_plan_s *p, void *ws, Groups &gr) {
    const SweepLayout &L = p->sweep;
    for (int g = 0; g < L.G; ++g) {
        gr.ws[g] = at(ws, L.base[g]);
        built_dense(p->sub[g].get(), gr.ws[g], gr.bd[g], kWantW);
    }
}

// Activation sweep.  Right to left, step g maps Z_{g+1} (X for the last
// group) to Z_g (Y for g = 0); left to right, step g maps Z_g (X, or its
// per-token transpose, for g = 0) to Z_{g+1} (Y for the last group).  With
// all false only the intermediate states are written (steps producing Y are
// skipped).
int sweep_x(const comera_ttm_plan_s *p, int64_t b, const void *X0, void *Y, void *ws, const Groups &gr, bool all,
            void *stream) {
    const SweepLayout &L = p->sweep;
    const int G = L.G;
    if (L.dir == COMERA_ORDER_SWEEP_RL) {
        const void *in = X0;
        for (int g = G - 1; g >= 0; --g) {
            if (g == 0 && !all) break;
            void *out = g ? at(ws, L.z[g]) : Y;
            const int64_t T = prod(L.M, g + 1, G);
            const int64_t R = b * prod(L.N, 0, g) * T, K = L.N[g] * L.ae[g], C = L.as[g] * L.M[g];
            const int64_t Nn = g ? L.N[g - 1] : 1, A = L.as[g];
            // row (q, i, t), column (a, m) -> Z_g [(q, m, t)][(i, a)]
            const Remap rm = remap3(Nn, T, L.M[g] * T * Nn * A, A, Nn * A);
            const Remap cm = remap2(L.M[g], 1, T * Nn * A);
            if (int e = step(p, ws, in, R, K, gr.bd[g].w, false, C, out, rm, cm, stream)) return e;
            in = out;
        }
        return 0;
    }
    const void *in = X0;
    for (int g = 0; g < G; ++g) {
        const bool last = g == G - 1;
        if (last && !all) break;
        void *out = last ? Y : at(ws, L.z[g + 1]);
        const int64_t R = b * prod(L.M, 0, g) * prod(L.N, g + 1, G), K = L.as[g] * L.N[g], C = L.M[g] * L.ae[g];
        const int64_t Nn = last ? 1 : L.N[g + 1], A = L.ae[g], T = last ? 1 : prod(L.N, g + 2, G);
        // row (q, i, t), column (m, a) -> Z_{g+1} [(q, m, t)][(a, i)]
        const Remap rm = remap3(Nn, T, L.M[g] * T * A * Nn, 1, A * Nn);
        const Remap cm = remap2(A, T * A * Nn, Nn);
        if (int e = step(p, ws, in, R, K, gr.bd[g].w, false, C, out, rm, cm, stream)) return e;
        in = out;
    }
    return 0;
}

}  // namespace

comera_status sweep_forward(const comera_ttm_plan_s *p, int64_t b, const void *X, const float *const *G,
                            const float *const *D, void *Y, void *ws, void *stream) {
    const SweepLayout &L = p->sweep;
    const int esz = p->s.act == COMERA_BF16 ? 2 : 4;
    Groups gr;
    if (int e = build_groups(p, G, D, ws, gr, stream)) return status_of(e);
    const void *X0 = X;
    if (L.dir == COMERA_ORDER_SWEEP_LR && L.need_t) {
        if (int e = launch_permute_tokens(X, at(ws, L.tin), b, L.N[0], prod(L.N, 1, L.G), esz, stream))
            return status_of(note_hip(e, "transpose"));
        X0 = at(ws, L.tin);
    }
    void *ev;
    timing_begin(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_FWD, stream, &ev);
    int e = sweep_x(p, b, X0, Y, ws, gr, true, stream);
    timing_end(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_FWD, stream, ev);
    return status_of(e);
}

comera_status sweep_backward(const comera_ttm_plan_s *p, int64_t b, const void *X, const void *dY,
                             const float *const *G, const float *const *D, void *dX, float *const *dG,
                             float *const *dD, void *ws, void *stream) {
    const SweepLayout &L = p->sweep;
    const int NG = L.G;
    const int d = p->d;
    const int esz = p->s.act == COMERA_BF16 ? 2 : 4;
    const bool rl = L.dir == COMERA_ORDER_SWEEP_RL;
    // want_dg: some core or mask gradient is asked for (both come from the meets)
    bool want_dg = false;
    for (int k = 0; k < d; ++k) want_dg = want_dg || (dG && dG[k]) || (dD && k + 1 < d && dD[k]);
    // with reuse, the group layers, the transposed X (left to right) and the
    // activation states are the ones the forward call left in the workspace
    Groups gr;
    if (p->reuse)
        built_groups(p, ws, gr);
    else if (int e = build_groups(p, G, D, ws, gr, stream))
        return status_of(e);
    // inputs of the first step of each sweep (per-token transposes where the
    // first-swept factor is not the last one)
    const void *X0 = X, *H0 = dY;
    if (L.need_t) {
        if (rl) {
            if (int e = launch_permute_tokens(dY, at(ws, L.tin), b, L.M[0], prod(L.M, 1, NG), esz, stream))
                return status_of(note_hip(e, "transpose"));
            H0 = at(ws, L.tin);
        } else if (want_dg) {
            if (!p->reuse)
                if (int e = launch_permute_tokens(X, at(ws, L.tin), b, L.N[0], prod(L.N, 1, NG), esz, stream))
                    return status_of(note_hip(e, "transpose"));
            X0 = at(ws, L.tin);
        }
    }
    // activation states for the meets
    if (want_dg && !p->reuse)
        if (int e = sweep_x(p, b, X0, nullptr, ws, gr, false, stream)) return status_of(e);
    // dY sweep (the mirror direction); its last step writes dX
    {
        void *ev;
        timing_begin(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_DX, stream, &ev);
        if (rl) {
            const void *in = H0;
            for (int g = 0; g < NG; ++g) {
                const bool last = g == NG - 1;
                if (last && !dX) break;
                if (!last && !want_dg && !dX) break;
                void *out = last ? dX : at(ws, L.h[g + 1]);
                const int64_t R = b * prod(L.N, 0, g) * prod(L.M, g + 1, NG), K = L.as[g] * L.M[g],
                              C = L.N[g] * L.ae[g];
                const int64_t Mn = last ? 1 : L.M[g + 1], A = L.ae[g], T = last ? 1 : prod(L.M, g + 2, NG);
                // row (q, m, t), column (i, a) -> H_{g+1} [(q, i, t)][(a, m)]
                const Remap rm = remap3(Mn, T, L.N[g] * T * A * Mn, 1, A * Mn);
                const Remap cm = remap2(A, T * A * Mn, Mn);
                if (int e = step(p, ws, in, R, K, gr.bd[g].w, true, C, out, rm, cm, stream)) return status_of(e);
                in = out;
            }
        } else {
            const void *in = dY;
            for (int g = NG - 1; g >= 0; --g) {
                const bool first = g == 0;
                if (first && !dX) break;
                if (!first && !want_dg && !dX) break;
                void *out = first ? dX : at(ws, L.h[g - 1]);
                const int64_t T = prod(L.N, g + 1, NG);
                const int64_t R = b * prod(L.M, 0, g) * T, K = L.M[g] * L.ae[g], C = L.as[g] * L.N[g];
                const int64_t Mp = first ? 1 : L.M[g - 1], A = L.as[g];
                // row (q, m, t), column (a, i) -> H_{g-1} [(q, i, t)][(m, a)]
                const Remap rm = remap3(Mp, T, L.N[g] * T * Mp * A, A, Mp * A);
                const Remap cm = remap2(L.N[g], 1, T * Mp * A);
                if (int e = step(p, ws, in, R, K, gr.bd[g].w, true, C, out, rm, cm, stream)) return status_of(e);
                in = out;
            }
        }
        timing_end(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_DX, stream, ev);
    }
    if (!want_dg) return COMERA_OK;
    // meets: dW'_g = Z^T H over the token-like index, then the group's projections
    const float *part[kMaxCores];
    int nsplit[kMaxCores];
    void *ev;
    timing_begin(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_DW, stream, &ev);
    for (int g = 0; g < NG; ++g) {
        const comera_ttm_plan_s *sp = p->sub[g].get();
        const void *Za, *Hb;
        int64_t K;
        if (rl) {
            Za = g == NG - 1 ? X : at(ws, L.z[g + 1]);
            Hb = g == 0 ? H0 : at(ws, L.h[g]);
            K = b * prod(L.N, 0, g) * prod(L.M, g + 1, NG);
        } else {
            Za = g == 0 ? X0 : at(ws, L.z[g]);
            Hb = g == NG - 1 ? dY : at(ws, L.h[g]);
            K = b * prod(L.M, 0, g) * prod(L.N, g + 1, NG);
        }
        float *dwp = nullptr;
        int splits = 0;
        if (int e = dw_gemm(sp, Za, sp->N_in, Hb, sp->N_out, K, gr.ws[g], &dwp, &splits, stream))
            return status_of(e);
        bool want[kMaxCores];
        for (int j = 0; j < sp->d; ++j) {
            const int k = L.s[g] + j;
            want[j] = (dG && dG[k]) || (dD && k + 1 < d && dD[k]);
        }
        if (int e = project_cores(sp, gr.bd[g], dwp, splits, want, gr.ws[g], part + L.s[g], nsplit + L.s[g], stream))
            return status_of(e);
    }
    timing_end(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_DW, stream, ev);
    if (dG && expand_cores(p, part, nsplit, L.st, D, dG, stream)) return COMERA_ERR_HIP;
    return status_of(mask_grads(p, part, nsplit, L.st, G, dD, stream));
}

}  // namespace comera
