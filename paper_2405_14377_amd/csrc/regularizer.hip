// Gradients of the early-stage regularisers (eq. pretrain-rank), added in
// place to the loss gradients that comera_ttm_backward(_masks) returned:
//   dG_k += 2 beta G_k                                    (beta ||G||^2)
//   dD_k[c] += gamma sign(D_k[c]) (left_k + right_k)       (gamma S^(D))
// where S^ is the layer size with every ||D_k||_0 relaxed to ||D_k||_1 and
// s_j = m_j n_j is the entries of core j per pair of rank indices: bond k
// (between cores k and k+1) enters core k's term, s_k for the first core
// else s_k ||D_{k-1}||_1, and core k+1's term, s_{k+1} for the last core
// else s_{k+1} ||D_{k+1}||_1.  sign(0) = 0.
//
// Two small launches: a grid-stride update of every core gradient, and one
// workgroup that forms the l1 norms of the masks in a fixed order (thread t
// sums entries t, t + 256, ... then a fixed tree) and updates dD, so the
// result is bitwise reproducible.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "internal.h"

namespace {

constexpr int kMax = COMERA_MAX_CORES;

struct RegArgs {
    int d;
    int64_t size[kMax];        // entries of core k
    int64_t rk[kMax + 1];      // ranks
    float s[kMax];             // m_k n_k
    const float *G[kMax];
    const float *D[kMax];
    float *dG[kMax];
    float *dD[kMax];
    float two_beta, gamma;
};

__global__ __launch_bounds__(256) void reg_core_kernel(RegArgs a) {
    const int k = blockIdx.y;
    float *out = a.dG[k];
    if (!out) return;
    const float *G = a.G[k];
    const int64_t n = a.size[k];
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256)
        out[i] = out[i] + a.two_beta * G[i];
}

__global__ __launch_bounds__(256) void reg_mask_kernel(RegArgs a) {
    __shared__ float red[256];
    __shared__ float norm[kMax];
    const int t = threadIdx.x;
    for (int k = 0; k + 1 < a.d; ++k) {
        const int64_t r = a.rk[k + 1];
        float v = 0.f;
        for (int64_t c = t; c < r; c += 256) v += fabsf(a.D[k][c]);
        red[t] = v;
        __syncthreads();
        for (int w = 128; w > 0; w >>= 1) {
            if (t < w) red[t] += red[t + w];
            __syncthreads();
        }
        if (t == 0) norm[k] = red[0];
        __syncthreads();
    }
    for (int k = 0; k + 1 < a.d; ++k) {
        float *out = a.dD[k];
        if (!out) continue;
        const float left = k == 0 ? a.s[k] : a.s[k] * norm[k - 1];
        const float right = k + 2 == a.d ? a.s[k + 1] : a.s[k + 1] * norm[k + 1];
        const float coef = a.gamma * (left + right);
        for (int64_t c = t; c < a.rk[k + 1]; c += 256) {
            const float x = a.D[k][c];
            const float sg = x > 0.f ? 1.f : (x < 0.f ? -1.f : 0.f);
            out[c] = out[c] + sg * coef;
        }
    }
}

}  // namespace

extern "C" comera_status comera_ttm_regularizer_grads(const comera_ttm_shape *s, float gamma, float beta,
                                                      const float *const *G, const float *const *D,
                                                      float *const *dG, float *const *dD, void *stream) {
    if (!s || s->d < 1 || s->d > kMax || s->r[0] != 1 || s->r[s->d] != 1) return COMERA_ERR_INVALID_ARG;
    if (!(gamma >= 0.f) || !(beta >= 0.f) || !std::isfinite(gamma) || !std::isfinite(beta))
        return COMERA_ERR_INVALID_ARG;
    RegArgs a{};
    a.d = s->d;
    a.two_beta = 2.f * beta;
    a.gamma = gamma;
    int64_t mx = 0;
    for (int k = 0; k < s->d; ++k) {
        if (s->n[k] < 1 || s->m[k] < 1 || s->r[k] < 1 || s->r[k + 1] < 1) return COMERA_ERR_INVALID_ARG;
        const double sz = double(s->r[k]) * double(s->m[k]) * double(s->n[k]) * double(s->r[k + 1]);
        if (sz > 2147483647.0) return COMERA_ERR_UNSUPPORTED;
        a.size[k] = int64_t(sz);
        a.s[k] = float(s->m[k] * s->n[k]);
        a.dG[k] = dG ? dG[k] : nullptr;
        a.G[k] = G ? G[k] : nullptr;
        if (a.dG[k] && !a.G[k]) return COMERA_ERR_INVALID_ARG;
        if (a.dG[k]) mx = std::max<int64_t>(mx, a.size[k]);
    }
    for (int k = 0; k <= s->d; ++k) a.rk[k] = s->r[k];
    bool any_dD = false;
    for (int k = 0; k + 1 < s->d; ++k) {
        a.D[k] = D ? D[k] : nullptr;
        a.dD[k] = dD ? dD[k] : nullptr;
        any_dD = any_dD || a.dD[k];
    }
    if (any_dD)   // the size term needs every mask
        for (int k = 0; k + 1 < s->d; ++k)
            if (!a.D[k]) return COMERA_ERR_INVALID_ARG;
    hipStream_t st = hipStream_t(stream);
    if (mx > 0) {
        const unsigned gx = unsigned(std::min<int64_t>((mx + 255) / 256, 1024));
        COMERA_LAUNCH(reg_core_kernel, dim3(gx, unsigned(s->d)), dim3(256), 0, st, a);
        if (comera::note_hip(comera::launch_status(), "regulariser: core terms")) return COMERA_ERR_HIP;
    }
    if (any_dD) {
        COMERA_LAUNCH(reg_mask_kernel, dim3(1), dim3(256), 0, st, a);
        if (comera::note_hip(comera::launch_status(), "regulariser: mask terms")) return COMERA_ERR_HIP;
    }
    return COMERA_OK;
}
