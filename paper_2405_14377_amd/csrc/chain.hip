// Fused per-token sweep of a TTM layer through its single cores, right to
// left (Prop. 4.1 with every core its own group, the activation swept from
// the last core), with every intermediate state in LDS (Sec. 4.2, eq. path-Y
// for the forward, eq. path-U1 / path-gX for dX and eq. back Gi for the core
// gradients).  For one token the states are
//   S_d = X[b] as [I_<=d],   S_{k-1}[I_<k][a_{k-1}][j_k][J_>k]
//       = sum_{i_k, a_k} S_k[I_<k][i_k][a_k][J_>k] G~_k[a_{k-1}, j_k, i_k, a_k]
// down to S_0 = Y[b] as [J], and the dY sweep runs the other way through the
// same layouts,
//   H_0 = dY[b],   H_k[I_<k][i_k][a_k][J_>k]
//       = sum_{a_{k-1}, j_k} H_{k-1}[I_<k][a_{k-1}][j_k][J_>k] G~_k[a_{k-1}, j_k, i_k, a_k]
// up to H_d = dX[b]; the gradient of the masked core k is the meet of the
// two states that enter it,
//   dG~_k[a_{k-1}, j_k, i_k, a_k] = sum_b sum_{I_<k, J_>k} H_{k-1}[.. a_{k-1} j_k ..] S_k[.. i_k a_k ..].
// Each contraction is a small matrix product -- rows (token, I_<k, J_>k),
// contraction (i_k, a_k) or (a_{k-1}, j_k), columns the other pair -- whose
// operands are affine in the row and column indices, run on
// v_mfma_f32_32x32x2f32 straight out of LDS (fp32 throughout; bf16
// activations are widened on load and rounded once on store).  Bond ranks
// are the plan's compacted ones; the cores are folded with their masks and
// compacted while they are staged.
//
// Launches: the forward is one kernel; the backward is one kernel (it
// recomputes the forward states, which is cheaper than storing them), which
// writes one partial of every dG~_k per workgroup, then the shared expand
// kernel (fixed-order sum of the partials, unfold, masks).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>

#include "internal.h"

namespace comera {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return uint16_t((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

// out(row, col) = sum_k A(row, k) B(k, col) for row < R, col < C, k < K:
//   A(row, k) = sA[ar(row) + ak(k)],  B(k, col) = sB[bk(k) + bc(col)]
// (ar, bc evaluated once per tile and lane; ak, bk once per product).  Each
// wave takes 32 x 32 output tiles in turn; lane l feeds row / column l % 32
// and contraction slot l / 32 of every v_mfma_f32_32x32x2f32 and receives
// rows (v / 4) 8 + (l / 32) 4 + v % 4, column l % 32 of the tile.
template <class AR, class AK, class BK, class BC, class ST>
__device__ __forceinline__ void lds_mm(int R, int C, int K, const float *sA, AR ar, AK ak, const float *sB, BK bk,
                                       BC bc, ST st) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int l32 = lane & 31, slot = lane >> 5;
    const int tr = (R + 31) >> 5, tc = (C + 31) >> 5;
    for (int tile = wave; tile < tr * tc; tile += nw) {
        const int r0 = (tile / tc) << 5, c0 = (tile % tc) << 5;
        const int row = r0 + l32, col = c0 + l32;
        const bool rok = row < R, cok = col < C;
        const int abase = rok ? ar(row) : 0, bbase = cok ? bc(col) : 0;
        f32x16 acc;
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = 0.f;
        int k = 0;
        for (; k + 16 <= K; k += 16) {
            float av[8], bv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int kk = k + 2 * u + slot;
                av[u] = rok ? sA[abase + ak(kk)] : 0.f;
                bv[u] = cok ? sB[bk(kk) + bbase] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av[u], bv[u], acc, 0, 0, 0);
        }
        for (; k < K; k += 2) {
            const int kk = k + slot;
            const bool kok = kk < K;
            const float av = (rok && kok) ? sA[abase + ak(kk)] : 0.f;
            const float bv = (cok && kok) ? sB[bk(kk) + bbase] : 0.f;
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc, 0, 0, 0);
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int r = r0 + ((v >> 2) << 3) + (slot << 2) + (v & 3);
            if (r < R && cok) st(r, col, acc[v]);
        }
    }
}

// Stage the folded, compacted cores into LDS: element (a', j, i, a) of core
// k is G_k[amap(a'), j, i, amap(a)] D_k[amap(a)] (compacted ranks rc), at
// cm[k] + c K_k + kk (c = a' m_k + j, kk = i rc_{k+1} + a; the layout the dX
// step reads, c-major) and / or km[k] + kk C_k + c (k-major, the layout the
// forward step reads).
__device__ void stage_cores(const ChainArgs &a, float *sm, bool want_c, bool want_k) {
    for (int k = 0; k < a.d; ++k) {
        const int rl = a.rc[k], rr = a.rc[k + 1], m = a.m[k], n = a.n[k];
        const int K = n * rr, C = rl * m, total = C * K;
        const float *G = a.G[k];
        const float *D = (k < a.d - 1) ? a.D[k] : nullptr;
        for (int o = threadIdx.x; o < total; o += blockDim.x) {
            const int c = o / K, kk = o - c * K;
            const int al = c / m, j = c - al * m, i = kk / rr, ar = kk - i * rr;
            const int fa = k == 0 ? 0 : a.amap[k][al];
            const int fc = k == a.d - 1 ? 0 : a.amap[k + 1][ar];
            float v = G[((int64_t(fa) * m + j) * n + i) * a.r[k + 1] + fc];
            if (D) v *= D[fc];
            if (want_c) sm[a.cm[k] + o] = v;
            if (want_k) sm[a.km[k] + kk * C + c] = v;
        }
    }
}

// activation rows t0 .. t0 + nt - 1 of a [b][width] tensor into dst[t][width]
// (fp32; rows past nt zero-filled up to TB)
__device__ void load_rows(const ChainArgs &a, const void *src, int64_t t0, int nt, int width, float *dst) {
    const int total = a.TB * width;
    for (int o = threadIdx.x; o < total; o += blockDim.x) {
        const int t = o / width, e = o - t * width;
        float v = 0.f;
        if (t < nt) {
            const int64_t g = (t0 + t) * int64_t(width) + e;
            v = a.act_bf16 ? bf16_to_f32(reinterpret_cast<const uint16_t *>(src)[g])
                           : reinterpret_cast<const float *>(src)[g];
        }
        dst[o] = v;
    }
}

__device__ void store_rows(const ChainArgs &a, void *out, int64_t t0, int nt, int width, const float *srcl) {
    const int total = nt * width;
    for (int o = threadIdx.x; o < total; o += blockDim.x) {
        const int64_t g = t0 * int64_t(width) + o;
        if (a.act_bf16)
            reinterpret_cast<uint16_t *>(out)[g] = f32_to_bf16_rne(srcl[o]);
        else
            reinterpret_cast<float *>(out)[g] = srcl[o];
    }
}

// Forward step of core k (0-based in the code: core k maps S_{k+1} to S_k,
// the state indices being those above): rows (t, I_<k, J_>k), contraction
// kk = (i_k, a_{k+1}), columns c = (a_k, j_k).
__device__ void step_fwd(const ChainArgs &a, int k, const float *sm, const float *in, float *out) {
    const int M = a.Mg[k], NI = a.Nl[k];
    const int K = a.n[k] * a.rc[k + 1], C = a.rc[k] * a.m[k];
    const int sin = a.ssz[k + 1], sout = a.ssz[k];
    const int R = a.TB * NI * M;
    const float *Bk = sm + a.km[k];
    auto rowin = [=](int row) {
        const int q = row / M, J = row - q * M, t = q / NI, I = q - t * NI;
        return t * sin + I * K * M + J;
    };
    float *o = out;
    lds_mm(R, C, K, in, rowin, [=](int kk) { return kk * M; }, Bk, [=](int kk) { return kk * C; },
           [](int c) { return c; }, [=](int row, int c, float v) {
               const int q = row / M, J = row - q * M, t = q / NI, I = q - t * NI;
               o[t * sout + I * C * M + J + c * M] = v;
           });
}

// dX step k: H_k (rows, contraction c = (a_{k-1}, j_k)) -> H_{k+1}
// (columns kk = (i_k, a_k)); same row structure as the forward step
__device__ void step_bwd(const ChainArgs &a, int k, const float *sm, const float *in, float *out) {
    const int M = a.Mg[k], NI = a.Nl[k];
    const int K = a.n[k] * a.rc[k + 1], C = a.rc[k] * a.m[k];
    const int sin = a.ssz[k], sout = a.ssz[k + 1];
    const int R = a.TB * NI * M;
    const float *Bc = sm + a.cm[k];
    auto rowin = [=](int row) {
        const int q = row / M, J = row - q * M, t = q / NI, I = q - t * NI;
        return t * sin + I * C * M + J;
    };
    float *o = out;
    lds_mm(R, K, C, in, rowin, [=](int c) { return c * M; }, Bc, [=](int c) { return c * K; },
           [](int kk) { return kk; }, [=](int row, int kk, float v) {
               const int q = row / M, J = row - q * M, t = q / NI, I = q - t * NI;
               o[t * sout + I * K * M + J + kk * M] = v;
           });
}

// Meet of core k: part[c K + kk] (+)= sum_(t, I, J) H_k(t, I, c, J) S_{k+1}(t, I, kk, J)
__device__ void meet(const ChainArgs &a, int k, const float *h, const float *s, int *tab, float *part, bool add) {
    const int M = a.Mg[k], NI = a.Nl[k];
    const int K = a.n[k] * a.rc[k + 1], C = a.rc[k] * a.m[k];
    const int Q = a.TB * NI * M;
    for (int q = threadIdx.x; q < Q; q += blockDim.x) {
        const int p = q / M, J = q - p * M, t = p / NI, I = p - t * NI;
        tab[2 * q] = t * a.ssz[k] + I * C * M + J;
        tab[2 * q + 1] = t * a.ssz[k + 1] + I * K * M + J;
    }
    __syncthreads();
    lds_mm(C, K, Q, h, [=](int c) { return c * M; }, [=](int q) { return tab[2 * q]; }, s,
           [=](int q) { return tab[2 * q + 1]; }, [=](int kk) { return kk * M; }, [=](int c, int kk, float v) {
               float *dst = part + int64_t(c) * K + kk;
               *dst = add ? *dst + v : v;
           });
    __syncthreads();
}

__global__ __launch_bounds__(256) void chain_fwd_kernel(ChainArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sm[];
    stage_cores(a, sm, false, true);
    float *buf0 = sm + a.st0, *buf1 = sm + a.st1;
    for (int64_t g = blockIdx.x; g * a.TB < a.b; g += gridDim.x) {
        const int64_t t0 = g * a.TB;
        const int nt = int(min<int64_t>(a.TB, a.b - t0));
        __syncthreads();
        load_rows(a, a.X, t0, nt, a.ssz[a.d], buf0);
        __syncthreads();
        float *in = buf0, *out = buf1;
        for (int k = a.d - 1; k >= 0; --k) {
            step_fwd(a, k, sm, in, out);
            __syncthreads();
            float *tmp = in;
            in = out;
            out = tmp;
        }
        store_rows(a, a.Y, t0, nt, a.ssz[0], in);
    }
}

__global__ __launch_bounds__(256) void chain_bwd_kernel(ChainArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sm[];
    stage_cores(a, sm, true, a.d > 1);
    int *tab = reinterpret_cast<int *>(sm + a.tab);
    bool first = true;
    for (int64_t g = blockIdx.x; g * a.TB < a.b; g += gridDim.x) {
        const int64_t t0 = g * a.TB;
        const int nt = int(min<int64_t>(a.TB, a.b - t0));
        __syncthreads();
        // S_d = X, then S_{d-1} .. S_1 (every state kept for the meets)
        load_rows(a, a.X, t0, nt, a.ssz[a.d], sm + a.sk[a.d]);
        __syncthreads();
        for (int k = a.d - 1; k >= 1; --k) {
            step_fwd(a, k, sm, sm + a.sk[k + 1], sm + a.sk[k]);
            __syncthreads();
        }
        // H_0 = dY, then per core: meet, then the dX step
        float *hin = sm + a.st0, *hout = sm + a.st1;
        load_rows(a, a.dY, t0, nt, a.ssz[0], hin);
        __syncthreads();
        for (int k = 0; k < a.d; ++k) {
            if (a.want[k]) {
                // this workgroup's partial of core k: [grid][rc_k m_k n_k rc_{k+1}] from poff[k]
                const int64_t cs = int64_t(a.rc[k]) * a.m[k] * a.n[k] * a.rc[k + 1];
                meet(a, k, hin, sm + a.sk[k + 1], tab, a.part + a.poff[k] + int64_t(blockIdx.x) * cs, !first);
            }
            if (k == a.d - 1 && !a.dX) break;
            step_bwd(a, k, sm, hin, hout);
            __syncthreads();
            float *tmp = hin;
            hin = hout;
            hout = tmp;
        }
        if (a.dX) store_rows(a, a.dX, t0, nt, a.ssz[a.d], hin);
        first = false;
    }
}

}  // namespace

bool chain_fits(ChainArgs &a, int64_t b, bool backward, int TB) {
    const int d = a.d;
    a.TB = TB;
    // per-token state sizes (the same for S_k and H_k): N_<=k rc_k M_>k
    int64_t Nl = 1;
    for (int k = 0; k < d; ++k) {
        a.Nl[k] = int(Nl);
        Nl *= a.n[k];
    }
    int64_t Mg = 1;
    for (int k = d - 1; k >= 0; --k) {
        a.Mg[k] = int(Mg);
        Mg *= a.m[k];
    }
    int64_t big = 0;
    for (int k = 0; k <= d; ++k) {
        const int64_t nl = k == 0 ? 1 : int64_t(a.Nl[k - 1]) * a.n[k - 1];
        const int64_t mg = k == d ? 1 : int64_t(a.Mg[k]) * a.m[k];
        const int64_t s = nl * a.rc[k] * mg;
        if (s > (1 << 20)) return false;
        a.ssz[k] = int(s);
        big = std::max(big, s);
    }
    int64_t off = 0;
    for (int k = 0; k < d; ++k) {
        const int64_t cs = int64_t(a.rc[k]) * a.m[k] * a.n[k] * a.rc[k + 1];
        if (backward) {
            a.cm[k] = int(off);
            off += cs;
        }
        if (!backward || d > 1) {
            a.km[k] = int(off);
            off += cs;
        }
    }
    a.st0 = int(off);
    off += TB * big;
    a.st1 = int(off);
    off += TB * big;
    if (backward) {
        for (int k = 1; k <= d; ++k) {
            a.sk[k] = int(off);
            off += TB * int64_t(a.ssz[k]);
        }
        int64_t q = 0;
        for (int k = 0; k < d; ++k) q = std::max<int64_t>(q, int64_t(TB) * a.Nl[k] * a.Mg[k]);
        a.tab = int(off);
        off += 2 * q;
    }
    a.lds_bytes = size_t(off) * 4;
    a.b = b;
    return a.lds_bytes <= size_t(160 * 1024);
}

int launch_chain(const ChainArgs &a, bool backward, int grid, void *stream) {
    if (a.b <= 0) return 0;
    const void *kern = backward ? reinterpret_cast<const void *>(chain_bwd_kernel)
                                : reinterpret_cast<const void *>(chain_fwd_kernel);
    if (!launch_check_mode()) {
        // both kernels take up to the whole LDS of a CU
        static const int set_f = int(hipFuncSetAttribute(reinterpret_cast<const void *>(chain_fwd_kernel),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024));
        static const int set_b = int(hipFuncSetAttribute(reinterpret_cast<const void *>(chain_bwd_kernel),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024));
        if (set_f) return set_f;
        if (set_b) return set_b;
    }
    (void)kern;
    if (backward)
        COMERA_LAUNCH(chain_bwd_kernel, dim3(unsigned(grid)), dim3(256), a.lds_bytes, hipStream_t(stream), a);
    else
        COMERA_LAUNCH(chain_fwd_kernel, dim3(unsigned(grid)), dim3(256), a.lds_bytes, hipStream_t(stream), a);
    return launch_status();
}

}  // namespace comera

namespace comera {

namespace {
constexpr int kChainGridF = 2048;   // forward workgroups at most (each loops over token groups)
constexpr int kChainGridB = 512;    // backward workgroups at most (= core-gradient partials)
}

bool layout_chain(const comera_ttm_plan_s *p, ChainLayout &L) {
    L = ChainLayout();
    if (p->zero) return false;
    const int d = p->d;
    ChainArgs a;
    std::memset(&a, 0, sizeof(a));
    a.d = d;
    a.act_bf16 = p->s.act == COMERA_BF16 ? 1 : 0;
    for (int k = 0; k <= d; ++k) {
        a.r[k] = int(p->s.r[k]);
        a.rc[k] = int(p->rho[k]);
        if (a.rc[k] > kChainMaxRank) return false;
    }
    for (int k = 0; k < d; ++k) {
        a.m[k] = int(p->s.m[k]);
        a.n[k] = int(p->s.n[k]);
    }
    // compacted entry -> full index of every inner bond (identity when the
    // plan does not compact); full indices must fit a byte
    for (int k = 1; k < d; ++k) {
        int x = 0;
        for (int full = 0; full < a.r[k] && x < a.rc[k]; ++full) {
            const bool on = !p->compacted || ((p->act[k].w[full >> 6] >> (full & 63)) & 1ull);
            if (!on) continue;
            if (full > 255) return false;
            a.amap[k][x++] = uint8_t(full);
        }
        if (x != a.rc[k]) return false;
    }
    const int64_t b = std::max<int64_t>(p->batch, 1);
    // forward: one token per workgroup while that gives enough workgroups,
    // else up to four
    L.fa = a;
    int tbf = 0;
    for (int tb : {4, 2, 1}) {
        if (b <= 1024 && tb > 1) continue;
        if (chain_fits(L.fa, b, false, tb)) {
            tbf = tb;
            break;
        }
    }
    if (!tbf) return false;
    L.grid_f = int(std::min<int64_t>((b + tbf - 1) / tbf, kChainGridF));
    L.ba = a;
    if (!chain_fits(L.ba, b, true, 1)) return false;
    L.grid_b = int(std::min<int64_t>(b, kChainGridB));
    size_t off = 0;
    for (int k = 0; k < d; ++k) {
        const int64_t cs = int64_t(a.rc[k]) * a.m[k] * a.n[k] * a.rc[k + 1];
        L.ba.poff[k] = int64_t(off / 4);
        off = (off + size_t(L.grid_b) * size_t(cs) * 4 + 255) / 256 * 256;
    }
    L.part = 0;
    L.total = off;
    return true;
}

comera_status chain_forward(const comera_ttm_plan_s *p, int64_t b, const void *X, const float *const *G,
                            const float *const *D, void *Y, void *ws, void *stream) {
    (void)ws;
    ChainArgs a = p->ch.fa;
    for (int k = 0; k < p->d; ++k) {
        a.G[k] = G[k];
        a.D[k] = (D && k < p->d - 1) ? D[k] : nullptr;
    }
    a.X = X;
    a.Y = Y;
    a.b = b;
    const int grid = int(std::min<int64_t>((b + a.TB - 1) / a.TB, p->ch.grid_f));
    void *ev;
    timing_begin(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_FWD, stream, &ev);
    const int e = note_hip(launch_chain(a, false, grid, stream), "fused sweep forward");
    timing_end(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_FWD, stream, ev);
    return e ? COMERA_ERR_HIP : COMERA_OK;
}

comera_status chain_backward(const comera_ttm_plan_s *p, int64_t b, const void *X, const void *dY,
                             const float *const *G, const float *const *D, void *dX, float *const *dG,
                             float *const *dD, void *ws, void *stream) {
    const int d = p->d;
    ChainArgs a = p->ch.ba;
    bool any = dX != nullptr;
    for (int k = 0; k < d; ++k) {
        a.G[k] = G[k];
        a.D[k] = (D && k < d - 1) ? D[k] : nullptr;
        a.want[k] = ((dG && dG[k]) || (dD && k + 1 < d && dD[k])) ? 1 : 0;
        any = any || a.want[k];
    }
    if (!any) return COMERA_OK;
    a.X = X;
    a.dY = dY;
    a.dX = dX;
    a.b = b;
    a.part = reinterpret_cast<float *>(reinterpret_cast<char *>(ws) + p->ch.part);
    const int grid = int(std::min<int64_t>((b + a.TB - 1) / a.TB, p->ch.grid_b));
    void *ev;
    timing_begin(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_DX, stream, &ev);
    int e = note_hip(launch_chain(a, true, grid, stream), "fused sweep backward");
    timing_end(const_cast<comera_ttm_plan_s *>(p), COMERA_KERNEL_DX, stream, ev);
    if (e) return COMERA_ERR_HIP;
    const float *part[kMaxCores];
    int nsplit[kMaxCores];
    CoreStrides st[kMaxCores];
    for (int k = 0; k < d; ++k) {
        part[k] = a.part + a.poff[k];
        nsplit[k] = grid;
        st[k] = core_strides(a.rc[k], a.m[k], a.n[k], a.rc[k + 1], false);
    }
    if (dG && expand_cores(p, part, nsplit, st, D, dG, stream)) return COMERA_ERR_HIP;
    return mask_grads(p, part, nsplit, st, G, dD, stream) ? COMERA_ERR_HIP : COMERA_OK;
}

}  // namespace comera
