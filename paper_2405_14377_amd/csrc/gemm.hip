// MFMA GEMM for gfx950 with a remapped epilogue.
//
//   C[off(m, n)] = sum_k Aop(m, k) * Bop(k, n)        (fp32 accumulation)
//   Aop(m, k) = A_KC ? A[m * lda + k] : A[k * lda + m]
//   Bop(k, n) = B_KC ? B[n * ldb + k] : B[k * ldb + n]
//   off(m, n) = split * split_stride + rmap(m) + cmap(n)
//
// rmap / cmap write an index in mixed radix and sum its digits times
// strides, which lets one kernel write plain row-major results, the rebuilt W
// straight from an interleaved core product, and the blocked intermediates of
// the gradient projections.
//
// Four waves per workgroup; each wave owns a WM x WN block made of 32 x 32
// MFMA tiles (bf16: v_mfma_f32_32x32x16_bf16, fp32: v_mfma_f32_32x32x2f32).
// Both operand tiles are staged in LDS as rows of 64 bytes of K (k
// contiguous), double buffered; operands whose k is strided in memory are
// transposed in registers on the way in.  Lanes read 16-byte vectors from
// LDS; the k slots fed to successive MFMAs are one fixed permutation of the
// tile's k range, shared by A and B, so the sum is unchanged.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "internal.h"

namespace comera {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int PITCH = 80;  // bytes per LDS row: 64 data + 16 pad (conflict-free 16 B reads)

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return uint16_t((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

template <typename T>
struct GemmCfg;
template <>
struct GemmCfg<uint16_t> {
    static constexpr int KT = 32;
    static constexpr int E = 8;
};
template <>
struct GemmCfg<float> {
    static constexpr int KT = 16;
    static constexpr int E = 4;
};

template <typename T>
__device__ __forceinline__ uint4 pack_elems(const T (&v)[GemmCfg<T>::E]) {
    uint4 r;
    if constexpr (sizeof(T) == 2) {
        r.x = uint32_t(v[0]) | (uint32_t(v[1]) << 16);
        r.y = uint32_t(v[2]) | (uint32_t(v[3]) << 16);
        r.z = uint32_t(v[4]) | (uint32_t(v[5]) << 16);
        r.w = uint32_t(v[6]) | (uint32_t(v[7]) << 16);
    } else {
        r.x = __float_as_uint(v[0]);
        r.y = __float_as_uint(v[1]);
        r.z = __float_as_uint(v[2]);
        r.w = __float_as_uint(v[3]);
    }
    return r;
}

// 16 bytes = E consecutive k of one row of a K-contiguous operand
template <typename T>
__device__ __forceinline__ uint4 load_kc(const T *__restrict__ p, int64_t ld, int64_t row, int64_t R, int64_t k,
                                         int64_t kend, bool vec) {
    constexpr int E = GemmCfg<T>::E;
    if (vec && row < R && k + E <= kend) return *reinterpret_cast<const uint4 *>(p + row * ld + k);
    T v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = (row < R && k + e < kend) ? p[row * ld + k + e] : T(0);
    return pack_elems<T>(v);
}

// 16 bytes = E consecutive rows at one k of an M-contiguous operand
template <typename T>
__device__ __forceinline__ uint4 load_mc(const T *__restrict__ p, int64_t ld, int64_t row, int64_t R, int64_t k,
                                         int64_t kend, bool vec) {
    constexpr int E = GemmCfg<T>::E;
    if (vec && k < kend && row + E <= R) return *reinterpret_cast<const uint4 *>(p + k * ld + row);
    T v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = (k < kend && row + e < R) ? p[k * ld + row + e] : T(0);
    return pack_elems<T>(v);
}

// Global -> registers -> LDS for one operand tile of RT rows x KT k.
template <typename T, bool KC, int RT>
struct TileLoader {
    static constexpr int E = GemmCfg<T>::E;
    static constexpr int NCH = KC ? (4 * RT + 255) / 256 : 1;
    uint4 v[2];

    __device__ __forceinline__ void load(const T *__restrict__ p, int64_t ld, int64_t r0, int64_t R, int64_t k0,
                                         int64_t kend, bool vec, int tid) {
        if constexpr (KC) {
#pragma unroll
            for (int j = 0; j < NCH; ++j) {
                const int c = tid + 256 * j;
                if (c < 4 * RT) v[j] = load_kc<T>(p, ld, r0 + (c >> 2), R, k0 + (c & 3) * E, kend, vec);
            }
        } else if (tid < 2 * RT) {
            if constexpr (sizeof(T) == 2) {
                const int kp = tid & 15, mg = tid >> 4;
                v[0] = load_mc<T>(p, ld, r0 + 8 * mg, R, k0 + 2 * kp, kend, vec);
                v[1] = load_mc<T>(p, ld, r0 + 8 * mg, R, k0 + 2 * kp + 1, kend, vec);
            } else {
                const int kp = tid & 7, mg = tid >> 3;
                v[0] = load_mc<T>(p, ld, r0 + 4 * mg, R, k0 + 2 * kp, kend, vec);
                v[1] = load_mc<T>(p, ld, r0 + 4 * mg, R, k0 + 2 * kp + 1, kend, vec);
            }
        }
    }

    __device__ __forceinline__ void store(char *lds, int tid) const {
        if constexpr (KC) {
#pragma unroll
            for (int j = 0; j < NCH; ++j) {
                const int c = tid + 256 * j;
                if (c < 4 * RT) *reinterpret_cast<uint4 *>(lds + (c >> 2) * PITCH + (c & 3) * 16) = v[j];
            }
        } else if (tid < 2 * RT) {
            const uint32_t a[4] = {v[0].x, v[0].y, v[0].z, v[0].w};
            const uint32_t b[4] = {v[1].x, v[1].y, v[1].z, v[1].w};
            if constexpr (sizeof(T) == 2) {
                const int kp = tid & 15, mg = tid >> 4;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t lo = (a[e >> 1] >> ((e & 1) * 16)) & 0xffffu;
                    const uint32_t hi = (b[e >> 1] >> ((e & 1) * 16)) & 0xffffu;
                    *reinterpret_cast<uint32_t *>(lds + (8 * mg + e) * PITCH + kp * 4) = lo | (hi << 16);
                }
            } else {
                const int kp = tid & 7, mg = tid >> 3;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    uint2 w;
                    w.x = a[e];
                    w.y = b[e];
                    *reinterpret_cast<uint2 *>(lds + (4 * mg + e) * PITCH + kp * 8) = w;
                }
            }
        }
    }
};

__device__ __forceinline__ int64_t remap(const Remap &r, int64_t idx) {
    int64_t off = 0;
    for (int t = r.nd - 1; t >= 1; --t) {
        const int64_t q = idx / r.radix[t];
        off += (idx - q * r.radix[t]) * r.stride[t];
        idx = q;
    }
    return off + idx * r.stride[0];
}

struct GemmParams {
    const void *A, *B;
    void *C;
    int64_t M, N, K, lda, ldb, kchunk, split_stride;
    Remap rmap, cmap;
    int vec_a, vec_b;
};

template <typename T, bool A_KC, bool B_KC, bool OUT_BF16, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void gemm_kernel(GemmParams p) {
    constexpr int KT = GemmCfg<T>::KT;
    constexpr int WAVES_N = BN / WN;
    constexpr int TM = WM / 32, TN = WN / 32;
    static_assert((BM / WM) * (BN / WN) == 4, "four waves per workgroup");
    __shared__ __attribute__((aligned(16))) char sA[2][BM * PITCH];
    __shared__ __attribute__((aligned(16))) char sB[2][BN * PITCH];
    __shared__ int64_t roff[BM];
    __shared__ int64_t coff[BN];

    const T *__restrict__ A = reinterpret_cast<const T *>(p.A);
    const T *__restrict__ B = reinterpret_cast<const T *>(p.B);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int64_t m0 = int64_t(blockIdx.y) * BM, n0 = int64_t(blockIdx.x) * BN;
    const int64_t kbeg = int64_t(blockIdx.z) * p.kchunk;
    const int64_t kend = min(p.K, kbeg + p.kchunk);
    const int ntiles = kend > kbeg ? int((kend - kbeg + KT - 1) / KT) : 0;

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    TileLoader<T, A_KC, BM> la;
    TileLoader<T, B_KC, BN> lb;
    if (ntiles > 0) {
        la.load(A, p.lda, m0, p.M, kbeg, kend, p.vec_a, tid);
        lb.load(B, p.ldb, n0, p.N, kbeg, kend, p.vec_b, tid);
    }
    for (int i = tid; i < BM; i += 256) roff[i] = m0 + i < p.M ? remap(p.rmap, m0 + i) : int64_t(-1);
    for (int i = tid; i < BN; i += 256) coff[i] = n0 + i < p.N ? remap(p.cmap, n0 + i) : int64_t(-1);
    if (ntiles > 0) {
        la.store(sA[0], tid);
        lb.store(sB[0], tid);
    }
    __syncthreads();

    const int lr = lane & 31, lh = lane >> 5;
    for (int kt = 0; kt < ntiles; ++kt) {
        const int cur = kt & 1;
        const bool more = kt + 1 < ntiles;
        if (more) {
            la.load(A, p.lda, m0, p.M, kbeg + int64_t(kt + 1) * KT, kend, p.vec_a, tid);
            lb.load(B, p.ldb, n0, p.N, kbeg + int64_t(kt + 1) * KT, kend, p.vec_b, tid);
        }
        const char *a_s = sA[cur];
        const char *b_s = sB[cur];
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                bf16x8 av[TM], bv[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    av[i] = *reinterpret_cast<const bf16x8 *>(a_s + (wm * WM + i * 32 + lr) * PITCH + ks * 32 + lh * 16);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    bv[j] = *reinterpret_cast<const bf16x8 *>(b_s + (wn * WN + j * 32 + lr) * PITCH + ks * 32 + lh * 16);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
            }
        } else {
#pragma unroll
            for (int kq = 0; kq < 2; ++kq) {
                f32x4 av[TM], bv[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    av[i] = *reinterpret_cast<const f32x4 *>(a_s + (wm * WM + i * 32 + lr) * PITCH + kq * 32 + lh * 16);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    bv[j] = *reinterpret_cast<const f32x4 *>(b_s + (wn * WN + j * 32 + lr) * PITCH + kq * 32 + lh * 16);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int i = 0; i < TM; ++i)
#pragma unroll
                        for (int j = 0; j < TN; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][e], bv[j][e], acc[i][j], 0, 0, 0);
            }
        }
        if (more) {
            la.store(sA[cur ^ 1], tid);
            lb.store(sB[cur ^ 1], tid);
        }
        __syncthreads();
    }

    // 32x32 accumulator layout: element v of lane l is row (v/4)*8 + (l/32)*4 + v%4, column l%32
    const int64_t zoff = int64_t(blockIdx.z) * p.split_stride;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int64_t co = coff[wn * WN + j * 32 + lr];
        if (co < 0) continue;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t ro = roff[wm * WM + i * 32 + (v >> 2) * 8 + lh * 4 + (v & 3)];
                if (ro < 0) continue;
                if constexpr (OUT_BF16)
                    reinterpret_cast<uint16_t *>(p.C)[zoff + ro + co] = f32_to_bf16_rne(acc[i][j][v]);
                else
                    reinterpret_cast<float *>(p.C)[zoff + ro + co] = acc[i][j][v];
            }
    }
}

enum TileId { T128x128 = 0, T64x64 = 1, T128x32 = 2, T32x128 = 3, T128x64 = 4, T64x128 = 5 };

template <typename T, bool AK, bool BK, bool OB>
int launch_t(const GemmArgs &g, const GemmParams &p, int tile, void *stream) {
    auto go = [&](auto kern, int bm, int bn) {
        dim3 grid(unsigned((g.N + bn - 1) / bn), unsigned((g.M + bm - 1) / bm), unsigned(g.splits));
        hipLaunchKernelGGL(kern, grid, dim3(256), 0, hipStream_t(stream), p);
        return int(hipGetLastError());
    };
    switch (tile) {
        case T128x128: return go(gemm_kernel<T, AK, BK, OB, 128, 128, 64, 64>, 128, 128);
        case T64x64: return go(gemm_kernel<T, AK, BK, OB, 64, 64, 32, 32>, 64, 64);
        case T128x32: return go(gemm_kernel<T, AK, BK, OB, 128, 32, 32, 32>, 128, 32);
        case T32x128: return go(gemm_kernel<T, AK, BK, OB, 32, 128, 32, 32>, 32, 128);
        case T128x64: return go(gemm_kernel<T, AK, BK, OB, 128, 64, 64, 32>, 128, 64);
        case T64x128: return go(gemm_kernel<T, AK, BK, OB, 64, 128, 32, 64>, 64, 128);
    }
    return int(hipErrorInvalidValue);
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Tile shape: the largest tile that still gives about one workgroup per CU;
// skinny products use the matching skinny tile.
int pick_tile(int64_t M, int64_t N, int splits) {
    if (N <= 32) return T128x32;
    if (M <= 32) return T32x128;
    if (N <= 64) return T128x64;
    if (M <= 64) return T64x128;
    const int64_t big = ceil_div(M, 128) * ceil_div(N, 128) * splits;
    if (big >= 240) return T128x128;
    const int64_t mid = ceil_div(M, 64) * ceil_div(N, 128) * splits;
    if (mid >= 240) return M >= N ? T128x64 : T64x128;
    return T64x64;
}

}  // namespace

Remap remap_linear(int64_t stride) {
    Remap r{};
    r.nd = 1;
    r.stride[0] = stride;
    return r;
}

int launch_gemm(const GemmArgs &g, void *stream) {
    if (g.M <= 0 || g.N <= 0) return 0;
    GemmParams p;
    p.A = g.A;
    p.B = g.B;
    p.C = g.C;
    p.M = g.M;
    p.N = g.N;
    p.K = g.K;
    p.lda = g.lda;
    p.ldb = g.ldb;
    p.kchunk = g.kchunk > 0 ? g.kchunk : std::max<int64_t>(g.K, 1);
    p.split_stride = g.split_stride;
    p.rmap = g.rmap;
    p.cmap = g.cmap;
    const int E = g.dtype == COMERA_BF16 ? 8 : 4;
    auto aligned = [&](const void *ptr, int64_t ld) {
        return (reinterpret_cast<uintptr_t>(ptr) % 16 == 0) && (ld % E == 0);
    };
    p.vec_a = aligned(g.A, g.lda);
    p.vec_b = aligned(g.B, g.ldb);
    GemmArgs gg = g;
    if (gg.splits < 1) gg.splits = 1;
    const int tile = g.tile >= 0 ? g.tile : pick_tile(g.M, g.N, gg.splits);
#define COMERA_GEMM_CASE(T, AK, BK, OB) \
    if (g.a_kc == AK && g.b_kc == BK && g.out_bf16 == OB) return launch_t<T, AK, BK, OB>(gg, p, tile, stream);
    if (g.dtype == COMERA_BF16) {
        COMERA_GEMM_CASE(uint16_t, true, false, true)
        COMERA_GEMM_CASE(uint16_t, true, true, true)
        COMERA_GEMM_CASE(uint16_t, false, false, false)
    } else {
        COMERA_GEMM_CASE(float, true, false, false)
        COMERA_GEMM_CASE(float, true, false, true)
        COMERA_GEMM_CASE(float, true, true, false)
        COMERA_GEMM_CASE(float, false, false, false)
    }
#undef COMERA_GEMM_CASE
    return int(hipErrorInvalidValue);
}

int chain_gemm(const float *P, const float *Gc, void *out, bool out_bf16, int64_t NI, int64_t NJ, int A, int nx,
               int ny, int C, void *stream) {
    GemmArgs g;
    g.dtype = COMERA_F32;
    g.a_kc = true;
    g.b_kc = false;
    g.out_bf16 = out_bf16;
    g.A = P;
    g.B = Gc;
    g.C = out;
    g.M = NI * NJ;
    g.N = int64_t(nx) * ny * C;
    g.K = A;
    g.lda = A;
    g.ldb = g.N;
    g.rmap.nd = 2;
    g.rmap.radix[1] = NJ;
    g.rmap.stride[0] = int64_t(nx) * NJ * ny * C;
    g.rmap.stride[1] = int64_t(ny) * C;
    g.cmap.nd = 3;
    g.cmap.radix[1] = ny;
    g.cmap.radix[2] = C;
    g.cmap.stride[0] = NJ * ny * C;
    g.cmap.stride[1] = C;
    g.cmap.stride[2] = 1;
    return launch_gemm(g, stream);
}

int split_for(int64_t M, int64_t N, int64_t K) {
    const int64_t tiles = std::max<int64_t>(1, ceil_div(M, 64) * ceil_div(N, 64));
    int64_t sp = std::max<int64_t>(1, ceil_div(512, tiles));
    sp = std::min<int64_t>(sp, std::max<int64_t>(1, K / 256));
    return int(std::min<int64_t>(sp, 1024));
}

int adjoint_gemm(const float *En, const float *Gc, float *out, int64_t NI, int64_t NJ, int A, int nx, int ny, int C,
                 int nxp, int nyp, int splits, float *scratch, void *stream) {
    GemmArgs g;
    g.dtype = COMERA_F32;
    g.a_kc = true;
    g.b_kc = true;
    g.A = En;
    g.B = Gc;
    g.C = out;
    g.M = NI * NJ;
    g.N = A;
    g.K = int64_t(nx) * ny * C;
    g.lda = g.K;
    g.ldb = g.K;
    const int64_t NJp = NJ / nyp;
    g.rmap.nd = 4;
    g.rmap.radix[1] = nxp;
    g.rmap.radix[2] = NJp;
    g.rmap.radix[3] = nyp;
    g.rmap.stride[0] = NJp * nxp * nyp * A;
    g.rmap.stride[1] = int64_t(nyp) * A;
    g.rmap.stride[2] = int64_t(nxp) * nyp * A;
    g.rmap.stride[3] = A;
    g.cmap = remap_linear(1);
    if (splits > 1 && scratch) {
        g.C = scratch;
        g.splits = splits;
        g.kchunk = (g.K + splits - 1) / splits;
        g.split_stride = g.M * g.N;
        int e = launch_gemm(g, stream);
        if (e) return e;
        return launch_sum_splits(scratch, out, g.M * g.N, splits, stream);
    }
    return launch_gemm(g, stream);
}

int meet_gemm(const float *P, const float *En, float *part, int64_t NI, int64_t NJ, int A, int nx, int ny, int C,
              int splits, void *stream) {
    GemmArgs g;
    g.dtype = COMERA_F32;
    g.a_kc = false;
    g.b_kc = false;
    g.A = P;
    g.B = En;
    g.C = part;
    g.M = A;
    g.N = int64_t(nx) * ny * C;
    g.K = NI * NJ;
    g.lda = A;
    g.ldb = g.N;
    g.rmap = remap_linear(g.N);
    g.cmap = remap_linear(1);
    g.splits = std::max(1, splits);
    g.kchunk = (g.K + g.splits - 1) / g.splits;
    g.split_stride = g.M * g.N;
    return launch_gemm(g, stream);
}

}  // namespace comera
