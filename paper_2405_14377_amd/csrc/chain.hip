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


__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return uint16_t((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

// floor(x / d) for 0 <= x < 2^22 and d >= 1, with inv = 1.0f / d: the
// float product is within one of the quotient (x is exact in fp32 and the
// relative error of inv x stays below 2^-23), so two integer tests fix it.
// Integer division proper is a long VALU sequence; the index arithmetic of
// these kernels divides per element.
struct Div {
    int d;
    float inv;
};
__device__ __forceinline__ Div mkdiv(int d) { return Div{d, 1.0f / float(d)}; }
__device__ __forceinline__ int udiv(int x, Div v) {
    int q = int(float(x) * v.inv);
    q += (q + 1) * v.d <= x ? 1 : 0;
    q -= q * v.d > x ? 1 : 0;
    return q;
}

// out(row, col) = sum_k A(row, k) B(k, col) for row < R, col < C, k < K:
//   A(row, k) = sA[ar(row) + ak(k)],  B(k, col) = sB[bk(k) + bc(col)]
// (ar, bc evaluated once per tile and lane; ak, bk once per product).  The
// workgroup's waves take 16 x 16 output tiles in turn (many small tiles, so
// that the 16 waves of a workgroup hide each other's LDS latency); lane
// l = 16 q + r feeds row / column r and contraction slot q of every
// v_mfma_f32_16x16x4f32 and receives rows 4 q + v, column r of the tile.
typedef float f32x4 __attribute__((ext_vector_type(4)));
template <class AR, class AK, class BK, class BC, class ST>
__device__ __forceinline__ void lds_mm(int R, int C, int K, const float *sA, AR ar, AK ak, const float *sB, BK bk,
                                       BC bc, ST st) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int r16 = lane & 15, q = lane >> 4;
    const int tr = (R + 15) >> 4, tc = (C + 15) >> 4;
    for (int tile = wave; tile < tr * tc; tile += nw) {
        const int tq = tile / tc;
        const int r0 = tq << 4, c0 = (tile - tq * tc) << 4;
        const int row = r0 + r16, col = c0 + r16;
        const bool rok = row < R, cok = col < C;
        const int abase = rok ? ar(row) : 0, bbase = cok ? bc(col) : 0;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        int k = 0;
        for (; k + 32 <= K; k += 32) {
            float av[8], bv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int kk = k + 4 * u + q;
                av[u] = rok ? sA[abase + ak(kk)] : 0.f;
                bv[u] = cok ? sB[bk(kk) + bbase] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u], bv[u], acc, 0, 0, 0);
        }
        for (; k < K; k += 4) {
            const int kk = k + q;
            const bool kok = kk < K;
            const float av = (rok && kok) ? sA[abase + ak(kk)] : 0.f;
            const float bv = (cok && kok) ? sB[bk(kk) + bbase] : 0.f;
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int r = r0 + 4 * q + v;
            if (r < R && cok) st(r, col, acc[v]);
        }
    }
}

// Stage the folded, compacted cores into LDS: element (a', j, i, a) of core
// k is G_k[amap(a'), j, i, amap(a)] D_k[amap(a)] (compacted ranks rc), at
// cm[k] + c cp[k] + kk (c = a' m_k + j, kk = i rc_{k+1} + a; the layout the
// dX step reads, c-major) and / or km[k] + kk kp[k] + c (k-major, the layout
// the forward step reads); the pitches are padded to 16 mod 64 floats so
// that the four contraction slots of an MFMA read different LDS banks.
// Every core gets its own block of waves (wave0[k] .. wave0[k + 1], sized by
// the host in proportion to the core), so all cores load in the same round
// trip (a kernel starts with cold caches and TLBs); in its block, thread t
// owns column kk = t mod K (i, a and the mask factor computed once) and rows
// c = t / K + P u (P = block threads / K), (a', j) advanced without integer
// division; kU rows' loads are in flight at once.  The index maps are read
// first only when the plan compacts its ranks.
constexpr int kU = 8;
constexpr int kChainThreads = 1024;   // 16 waves per workgroup
__device__ void stage_cores(const ChainArgs &a, float *sm, int *smap, bool want_c, bool want_k) {
    if (a.compacted) {
        for (int i = threadIdx.x; i < (a.d + 1) * kChainMaxRank; i += blockDim.x)
            smap[i] = a.amap[i / kChainMaxRank][i % kChainMaxRank];
        __syncthreads();
    }
    const int w = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
    int k = 0;
    while (k + 1 < a.d && w >= a.wave0[k + 1]) ++k;
    const int nt = (a.wave0[k + 1] - a.wave0[k]) * 64, t = int(threadIdx.x) - a.wave0[k] * 64;
    const int rr = a.rc[k + 1], m = a.m[k], n = a.n[k], rfull = a.r[k + 1];
    const int K = n * rr, C = a.rc[k] * m;
    const float *G = a.G[k];
    const float *D = (k < a.d - 1) ? a.D[k] : nullptr;
    const bool first = k == 0, last = k == a.d - 1;
    float *dcm = sm + a.cm[k], *dkm = sm + a.km[k];
    const int cp = a.cp[k], kp = a.kp[k];
    for (int kb = 0; kb < K; kb += nt) {
        const bool narrow = K - kb < nt;
        const int kw = narrow ? K - kb : nt;           // columns of this pass
        const int kk = kb + t % kw, c0 = t / kw, P = nt / kw;
        if (c0 >= P || kk >= K) continue;
        const int i = kk / rr, ar = kk - i * rr;
        const int fc = last ? 0 : (a.compacted ? smap[(k + 1) * kChainMaxRank + ar] : ar);
        const float dfac = D ? D[fc] : 1.f;
        const int64_t col = int64_t(i) * rfull + fc;
        const int dj = P % m, dal = P / m;
        int c = c0, al = c0 / m, j = c0 - al * m;
        while (c < C) {
            float v[kU];
            int cs[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                cs[u] = c;
                v[u] = 0.f;
                if (c < C) {
                    const int fa = first ? 0 : (a.compacted ? smap[k * kChainMaxRank + al] : al);
                    v[u] = G[(int64_t(fa) * m + j) * int64_t(n) * rfull + col];
                }
                c += P;
                j += dj;
                al += dal;
                if (j >= m) {
                    j -= m;
                    ++al;
                }
            }
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                if (cs[u] < C) {
                    const float x = v[u] * dfac;
                    if (want_c) dcm[cs[u] * cp + kk] = x;
                    if (want_k) dkm[kk * kp + cs[u]] = x;
                }
            }
        }
    }
}

// activation rows t0 .. t0 + nt - 1 of a [b][width] tensor into dst[t][width]
// (fp32; rows past nt zero-filled up to TB), kU loads in flight per thread
template <typename T>
__device__ void load_rows_t(const ChainArgs &a, const T *src, int64_t t0, int nt, int width, float *dst) {
    const int total = a.TB * width;
    const Div dw = mkdiv(width);
    for (int base = threadIdx.x; base < total; base += blockDim.x * kU) {
        // 32-bit registers for both types (a 16-bit load into half a
        // register would wait for the previous contents)
        uint32_t v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int o = base + u * int(blockDim.x);
            const int t = udiv(o, dw), e = o - t * width;
            const bool ok = o < total && t < nt;
            // every lane loads (element 0 of the first row when outside), then selects
            const int64_t g = ok ? (t0 + t) * int64_t(width) + e : 0;
            uint32_t x;
            if constexpr (sizeof(T) == 2)
                x = uint32_t(src[g]) << 16;
            else
                x = __float_as_uint(src[g]);
            v[u] = ok ? x : 0u;
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int o = base + u * int(blockDim.x);
            if (o < total) dst[o] = __uint_as_float(v[u]);
        }
    }
}

// The first token group's rows, loaded into registers before the cores are
// staged (two elements per thread at most; larger groups return false and are
// loaded by load_rows), so that both wait for one memory round trip.
struct RowPrefetch {
    uint32_t v[2];
    bool on;
};
template <typename T>
__device__ __forceinline__ void prefetch_rows_t(const ChainArgs &a, const T *src, int nt, int width, RowPrefetch &pf) {
    const Div dw = mkdiv(width);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int o = int(threadIdx.x) + u * int(blockDim.x);
        const int t = udiv(o, dw), e = o - t * width;
        const bool ok = o < a.TB * width && t < nt;
        const int64_t g = ok ? int64_t(t) * width + e : 0;
        uint32_t x;
        if constexpr (sizeof(T) == 2)
            x = uint32_t(src[g]) << 16;
        else
            x = __float_as_uint(src[g]);
        pf.v[u] = ok ? x : 0u;
    }
}
__device__ __forceinline__ void prefetch_rows(const ChainArgs &a, const void *src, int64_t t0, int nt, int width,
                                              RowPrefetch &pf) {
    pf.on = a.TB * width <= 2 * int(blockDim.x);
    if (!pf.on) return;
    if (a.act_bf16)
        prefetch_rows_t(a, reinterpret_cast<const uint16_t *>(src) + t0 * int64_t(width), nt, width, pf);
    else
        prefetch_rows_t(a, reinterpret_cast<const float *>(src) + t0 * int64_t(width), nt, width, pf);
}
__device__ __forceinline__ void store_prefetch(const ChainArgs &a, int width, const RowPrefetch &pf, float *dst) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int o = int(threadIdx.x) + u * int(blockDim.x);
        if (o < a.TB * width) dst[o] = __uint_as_float(pf.v[u]);
    }
}

__device__ void load_rows(const ChainArgs &a, const void *src, int64_t t0, int nt, int width, float *dst) {
    if (a.act_bf16)
        load_rows_t(a, reinterpret_cast<const uint16_t *>(src), t0, nt, width, dst);
    else
        load_rows_t(a, reinterpret_cast<const float *>(src), t0, nt, width, dst);
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
    const Div dM = mkdiv(M), dN = mkdiv(NI);
    auto rowin = [=](int row) {
        const int q = udiv(row, dM), J = row - q * M, t = udiv(q, dN), I = q - t * NI;
        return t * sin + I * K * M + J;
    };
    float *o = out;
    const int kp = a.kp[k];
    lds_mm(R, C, K, in, rowin, [=](int kk) { return kk * M; }, Bk, [=](int kk) { return kk * kp; },
           [](int c) { return c; }, [=](int row, int c, float v) {
               const int q = udiv(row, dM), J = row - q * M, t = udiv(q, dN), I = q - t * NI;
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
    const Div dM = mkdiv(M), dN = mkdiv(NI);
    auto rowin = [=](int row) {
        const int q = udiv(row, dM), J = row - q * M, t = udiv(q, dN), I = q - t * NI;
        return t * sin + I * C * M + J;
    };
    float *o = out;
    const int cp = a.cp[k];
    lds_mm(R, K, C, in, rowin, [=](int c) { return c * M; }, Bc, [=](int c) { return c * cp; },
           [](int kk) { return kk; }, [=](int row, int kk, float v) {
               const int q = udiv(row, dM), J = row - q * M, t = udiv(q, dN), I = q - t * NI;
               o[t * sout + I * K * M + J + kk * M] = v;
           });
}

// Meet of core k: part[c K + kk] (+)= sum_(t, I, J) H_k(t, I, c, J) S_{k+1}(t, I, kk, J)
__device__ void meet(const ChainArgs &a, int k, const float *h, const float *s, int *tab, float *part, bool add) {
    const int M = a.Mg[k], NI = a.Nl[k];
    const int K = a.n[k] * a.rc[k + 1], C = a.rc[k] * a.m[k];
    const int Q = a.TB * NI * M;
    const Div dM = mkdiv(M), dN = mkdiv(NI);
    for (int q = threadIdx.x; q < Q; q += blockDim.x) {
        const int p = udiv(q, dM), J = q - p * M, t = udiv(p, dN), I = p - t * NI;
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

__global__ __launch_bounds__(kChainThreads) void chain_fwd_kernel(ChainArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sm[];
    RowPrefetch pf;
    {
        const int64_t t0 = int64_t(blockIdx.x) * a.TB;
        prefetch_rows(a, a.X, t0, int(min<int64_t>(a.TB, a.b - t0)), a.ssz[a.d], pf);
    }
    stage_cores(a, sm, reinterpret_cast<int *>(sm + a.smap), false, true);
    float *buf0 = sm + a.st0, *buf1 = sm + a.st1;
    for (int64_t g = blockIdx.x; g * a.TB < a.b; g += gridDim.x) {
        const int64_t t0 = g * a.TB;
        const int nt = int(min<int64_t>(a.TB, a.b - t0));
        __syncthreads();
        if (g == blockIdx.x && pf.on)
            store_prefetch(a, a.ssz[a.d], pf, buf0);
        else
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

__global__ __launch_bounds__(kChainThreads) void chain_bwd_kernel(ChainArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sm[];
    RowPrefetch px, py;
    {
        const int64_t t0 = int64_t(blockIdx.x) * a.TB;
        const int nt0 = int(min<int64_t>(a.TB, a.b - t0));
        prefetch_rows(a, a.X, t0, nt0, a.ssz[a.d], px);
        prefetch_rows(a, a.dY, t0, nt0, a.ssz[0], py);
    }
    stage_cores(a, sm, reinterpret_cast<int *>(sm + a.smap), true, a.d > 1);
    int *tab = reinterpret_cast<int *>(sm + a.tab);
    bool first = true;
    for (int64_t g = blockIdx.x; g * a.TB < a.b; g += gridDim.x) {
        const int64_t t0 = g * a.TB;
        const int nt = int(min<int64_t>(a.TB, a.b - t0));
        const bool pre = g == blockIdx.x;
        __syncthreads();
        // S_d = X, then S_{d-1} .. S_1 (every state kept for the meets)
        if (pre && px.on)
            store_prefetch(a, a.ssz[a.d], px, sm + a.sk[a.d]);
        else
            load_rows(a, a.X, t0, nt, a.ssz[a.d], sm + a.sk[a.d]);
        __syncthreads();
        for (int k = a.d - 1; k >= 1; --k) {
            step_fwd(a, k, sm, sm + a.sk[k + 1], sm + a.sk[k]);
            __syncthreads();
        }
        // H_0 = dY, then per core: meet, then the dX step
        float *hin = sm + a.st0, *hout = sm + a.st1;
        if (pre && py.on)
            store_prefetch(a, a.ssz[0], py, hin);
        else
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
        if (s * TB >= (1 << 22)) return false;   // index arithmetic (udiv) stays below 2^22
        a.ssz[k] = int(s);
        big = std::max(big, s);
    }
    // LDS row pitches of the two core copies: 16 mod 64 floats
    auto pitch = [](int x) { return x + ((16 - x % 64) + 64) % 64; };
    int64_t off = 0, cst = 0;
    for (int k = 0; k < d; ++k) {
        const int K = a.n[k] * a.rc[k + 1], C = a.rc[k] * a.m[k];
        const int64_t cs = int64_t(C) * K;
        a.cstart[k] = int(cst);
        cst += cs;
        a.cp[k] = pitch(K);
        a.kp[k] = pitch(C);
        if (backward) {
            a.cm[k] = int(off);
            off += int64_t(C) * a.cp[k];
        }
        if (!backward || d > 1) {
            a.km[k] = int(off);
            off += int64_t(K) * a.kp[k];
        }
    }
    a.cstart[d] = int(cst);
    // waves of the staging pass per core, in proportion to the core sizes
    {
        const int waves = kChainThreads / 64;
        int given = 0;
        for (int k = 0; k < d; ++k) {
            const int64_t cs = int64_t(a.cstart[k + 1]) - a.cstart[k];
            int wk = std::max(1, int(cs * (waves - d) / std::max<int64_t>(cst, 1)) + 1);
            if (k == d - 1) wk = waves - given;
            wk = std::max(1, std::min(wk, waves - given - (d - 1 - k)));
            a.wave0[k] = given;
            given += wk;
        }
        a.wave0[d] = waves;
    }
    a.smap = int(off);
    off += (d + 1) * kChainMaxRank;
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
    return a.lds_bytes + 1024 <= size_t(160 * 1024);
}

int launch_chain(const ChainArgs &a, bool backward, int grid, void *stream) {
    if (a.b <= 0) return 0;
    const void *kern = backward ? reinterpret_cast<const void *>(chain_bwd_kernel)
                                : reinterpret_cast<const void *>(chain_fwd_kernel);
    if (!launch_check_mode()) {
        // both kernels take up to the whole LDS of a CU
        static const int set_f = int(hipFuncSetAttribute(reinterpret_cast<const void *>(chain_fwd_kernel),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, 159 * 1024));
        static const int set_b = int(hipFuncSetAttribute(reinterpret_cast<const void *>(chain_bwd_kernel),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, 159 * 1024));
        if (set_f) return set_f;
        if (set_b) return set_b;
    }
    (void)kern;
    if (backward)
        COMERA_LAUNCH(chain_bwd_kernel, dim3(unsigned(grid)), dim3(kChainThreads), a.lds_bytes, hipStream_t(stream),
                      a);
    else
        COMERA_LAUNCH(chain_fwd_kernel, dim3(unsigned(grid)), dim3(kChainThreads), a.lds_bytes, hipStream_t(stream),
                      a);
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
    a.compacted = p->compacted ? 1 : 0;
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
