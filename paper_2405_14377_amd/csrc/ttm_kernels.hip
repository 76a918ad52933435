// HIP kernels (gfx950) for the dense contraction order of a TTM layer:
//   fold      masked, rank-compacted core copies (eq. Wcompress)
//   chain     left-to-right core products P_k and the rebuilt W (eq. TTM)
//   gemm      MFMA products Y = X W, dX = dY W^T, dW = X^T dY (Sec. 4.2)
//   adjoint   right environments E_k = dW contracted with cores k..d-1
//   meet      core gradients from P_k and E_{k+1} (eq. back Gi)
//   expand    compacted gradients back to the full core layout
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "internal.h"

namespace comera {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return uint16_t((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// index of the idx-th set bit of a 256-bit set
__device__ int select_bit(const BondBits &b, int idx) {
    for (int w = 0; w < 4; ++w) {
        int c = __popcll(b.w[w]);
        if (idx < c) {
            uint64_t x = b.w[w];
            for (int t = 0; t < idx; ++t) x &= x - 1;
            return w * 64 + __builtin_ctzll(x);
        }
        idx -= c;
    }
    return -1;
}

// rank of bit a among set bits (number of set bits below a); -1 if a is not set
__device__ int rank_bit(const BondBits &b, int a) {
    if (a >= 256) return -1;
    if (!((b.w[a >> 6] >> (a & 63)) & 1ull)) return -1;
    int r = 0;
    for (int w = 0; w < (a >> 6); ++w) r += __popcll(b.w[w]);
    uint64_t low = (a & 63) ? (b.w[a >> 6] & ((1ull << (a & 63)) - 1)) : 0ull;
    return r + __popcll(low);
}

// ---------------------------------------------------------------- fold / expand
__global__ void fold_kernel(FoldArgs a) {
    const int k = blockIdx.y;
    if (k >= a.nfold) return;
    const int rl = a.rc[k], rr = a.rc[k + 1], m = a.m[k], n = a.n[k];
    const int64_t total = int64_t(rl) * m * n * rr;
    const float *G = a.G[k];
    const float *D = (k < a.d - 1) ? a.D[k] : nullptr;
    for (int64_t o = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; o < total;
         o += int64_t(gridDim.x) * blockDim.x) {
        int c = int(o % rr);
        int64_t t = o / rr;
        int mn = int(t % (int64_t(m) * n));
        int al = int(t / (int64_t(m) * n));
        int fa = al, fc = c;
        if (a.compacted) {
            fa = (k == 0) ? 0 : select_bit(a.act[k], al);
            fc = (k == a.d - 1) ? 0 : select_bit(a.act[k + 1], c);
        }
        float v = G[(int64_t(fa) * m * n + mn) * a.r[k + 1] + fc];
        if (D) v *= D[fc];
        a.Gc[k][o] = v;
    }
}

__global__ void expand_kernel(ExpandArgs a) {
    const int k = blockIdx.y;
    if (k >= a.d || !a.dG[k]) return;
    const int rl = a.r[k], rr = a.r[k + 1], m = a.m[k], n = a.n[k];
    const int crl = a.rc[k], crr = a.rc[k + 1];
    const int64_t total = int64_t(rl) * m * n * rr;
    const int64_t csize = int64_t(crl) * m * n * crr;
    const float *D = (k < a.d - 1) ? a.D[k] : nullptr;
    for (int64_t o = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; o < total;
         o += int64_t(gridDim.x) * blockDim.x) {
        int c = int(o % rr);
        int64_t t = o / rr;
        int mn = int(t % (int64_t(m) * n));
        int al = int(t / (int64_t(m) * n));
        int ca = al, cc = c;
        if (a.compacted) {
            ca = (k == 0) ? 0 : rank_bit(a.act[k], al);
            cc = (k == a.d - 1) ? 0 : rank_bit(a.act[k + 1], c);
        }
        float v = 0.f;
        if (ca >= 0 && cc >= 0) {
            const int64_t ci = (int64_t(ca) * m * n + mn) * crr + cc;
            for (int s = 0; s < a.splits[k]; ++s) v += a.part[k][s * csize + ci];
            if (D) v *= D[c];
        }
        a.dG[k][o] = v;
    }
}

// ---------------------------------------------------------------- core chains
// Core G has layout [A][p1][p2][C].  x is axis `xaxis` (1 or 2) with size nx,
// y is the other axis with size ny.
__device__ __forceinline__ int64_t core_off(int a, int x, int y, int c, int p1, int p2, int C, int xaxis) {
    return xaxis == 2 ? ((int64_t(a) * p1 + y) * p2 + x) * C + c : ((int64_t(a) * p1 + x) * p2 + y) * C + c;
}

__global__ void chain_kernel(const float *__restrict__ P, const float *__restrict__ G, float *__restrict__ out,
                             uint16_t *__restrict__ out_bf16, int64_t NX, int64_t NY, int A, int p1, int p2,
                             int C, int xaxis) {
    const int nx = xaxis == 2 ? p2 : p1, ny = xaxis == 2 ? p1 : p2;
    const int64_t rowlen = NY * ny;
    const int64_t total = NX * nx * rowlen * C;
    for (int64_t o = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; o < total;
         o += int64_t(gridDim.x) * blockDim.x) {
        int c = int(o % C);
        int64_t t = o / C;
        int64_t Yy = t % rowlen, Xx = t / rowlen;
        int64_t Y = Yy / ny, X = Xx / nx;
        int y = int(Yy % ny), x = int(Xx % nx);
        float acc = 0.f;
        if (P) {
            const float *pr = P + (X * NY + Y) * A;
            for (int a = 0; a < A; ++a) acc += pr[a] * G[core_off(a, x, y, c, p1, p2, C, xaxis)];
        } else {
            acc = G[core_off(0, x, y, c, p1, p2, C, xaxis)];
        }
        if (out_bf16) out_bf16[o] = f32_to_bf16_rne(acc);
        else out[o] = acc;
    }
}

// thread per output; used when the reduction (nx*ny*C) is short
__global__ void adjoint_small_kernel(const float *__restrict__ E, const float *__restrict__ G,
                                     float *__restrict__ out, int64_t NX, int64_t NY, int A, int p1, int p2,
                                     int C, int xaxis) {
    const int nx = xaxis == 2 ? p2 : p1, ny = xaxis == 2 ? p1 : p2;
    const int64_t total = NX * NY * A;
    const int64_t rowlen = NY * ny;
    for (int64_t o = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; o < total;
         o += int64_t(gridDim.x) * blockDim.x) {
        int a = int(o % A);
        int64_t t = o / A;
        int64_t Y = t % NY, X = t / NY;
        float acc = 0.f;
        for (int x = 0; x < nx; ++x)
            for (int y = 0; y < ny; ++y) {
                const float *er = E + ((X * nx + x) * rowlen + Y * ny + y) * C;
                for (int c = 0; c < C; ++c) acc += er[c] * G[core_off(a, x, y, c, p1, p2, C, xaxis)];
            }
        out[o] = acc;
    }
}

// one wave per (X, Y); lanes split the (x, y, c) reduction
__global__ __launch_bounds__(256) void adjoint_wave_kernel(const float *__restrict__ E, const float *__restrict__ G,
                                                           float *__restrict__ out, int64_t NX, int64_t NY, int A,
                                                           int p1, int p2, int C, int xaxis) {
    const int nx = xaxis == 2 ? p2 : p1, ny = xaxis == 2 ? p1 : p2;
    const int lane = threadIdx.x & 63;
    const int64_t pair = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (pair >= NX * NY) return;
    const int64_t Y = pair % NY, X = pair / NY;
    const int64_t rowlen = NY * ny;
    const int nterm = nx * ny * C;
    for (int a = 0; a < A; ++a) {
        float acc = 0.f;
        for (int t = lane; t < nterm; t += 64) {
            int c = t % C;
            int xy = t / C;
            int y = xy % ny, x = xy / ny;
            acc += E[((X * nx + x) * rowlen + Y * ny + y) * C + c] * G[core_off(a, x, y, c, p1, p2, C, xaxis)];
        }
        for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
        if (lane == 0) out[pair * A + a] = acc;
    }
}

__global__ void meet_kernel(const float *__restrict__ P, const float *__restrict__ E, float *__restrict__ part,
                            int64_t NX, int64_t NY, int A, int p1, int p2, int C, int xaxis, int64_t chunk) {
    const int nx = xaxis == 2 ? p2 : p1, ny = xaxis == 2 ? p1 : p2;
    const int64_t outs = int64_t(A) * p1 * p2 * C;
    const int64_t XY = NX * NY;
    const int s = blockIdx.y;
    const int64_t beg = s * chunk, end = min(XY, beg + chunk);
    const int64_t rowlen = NY * ny;
    for (int64_t o = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; o < outs;
         o += int64_t(gridDim.x) * blockDim.x) {
        int c = int(o % C);
        int64_t t = o / C;
        int q2 = int(t % p2);
        t /= p2;
        int q1 = int(t % p1);
        int a = int(t / p1);
        int x = xaxis == 2 ? q2 : q1, y = xaxis == 2 ? q1 : q2;
        float acc = 0.f;
        for (int64_t xy = beg; xy < end; ++xy) {
            int64_t X = xy / NY, Y = xy % NY;
            float pv = P ? P[xy * A + a] : 1.f;
            acc += pv * E[((X * nx + x) * rowlen + Y * ny + y) * C + c];
        }
        part[s * outs + o] = acc;
    }
}

__global__ void sum_splits_kernel(const float *__restrict__ part, float *__restrict__ out, int64_t n, int splits) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x) {
        float v = 0.f;
        for (int s = 0; s < splits; ++s) v += part[s * n + i];
        out[i] = v;
    }
}

__global__ void fill_zero_kernel(uint32_t *p, int64_t n) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        p[i] = 0u;
}

// ---------------------------------------------------------------- MFMA GEMM
// C[m, n] = sum_k Aop(m, k) * Bop(k, n), fp32 accumulation.
//   Aop(m, k) = A_KC ? A[m * lda + k] : A[k * lda + m]
//   Bop(k, n) = B_KC ? B[n * ldb + k] : B[k * ldb + n]
// Workgroup tile 128 x 128, four waves of 64 x 64, each a 2 x 2 block of
// 32 x 32 MFMA tiles.  Both operand tiles are staged in LDS as rows of K
// (k contiguous), double buffered; operands whose k is strided in memory are
// transposed in registers on the way in.  Lanes read 16-byte vectors: the
// k-slots they feed to successive MFMAs are a fixed permutation of the tile's
// k range, the same for A and B, so the sum is unchanged.
// blockIdx.z selects a split of K; split s writes C + s * c_split_stride.
constexpr int BM = 128;
constexpr int BN = 128;
constexpr int PITCH = 80;  // bytes per LDS row: 64 data + 16 pad (conflict-free 16 B reads)

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
__device__ __forceinline__ T ld_elem(const T *p, int64_t i) {
    return p[i];
}

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

// Load 16 bytes = E consecutive elements starting at (row, k) of a
// K-contiguous operand; out-of-range elements read as zero.
template <typename T>
__device__ __forceinline__ uint4 load_kc(const T *__restrict__ p, int64_t ld, int64_t row, int64_t R, int64_t k,
                                         int64_t kend, bool vec) {
    constexpr int E = GemmCfg<T>::E;
    if (vec && row < R && k + E <= kend) return *reinterpret_cast<const uint4 *>(p + row * ld + k);
    T v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = (row < R && k + e < kend) ? ld_elem(p, row * ld + k + e) : T(0);
    return pack_elems<T>(v);
}

// Load 16 bytes = E consecutive rows at one k of an M-contiguous operand.
template <typename T>
__device__ __forceinline__ uint4 load_mc(const T *__restrict__ p, int64_t ld, int64_t row, int64_t R, int64_t k,
                                         int64_t kend, bool vec) {
    constexpr int E = GemmCfg<T>::E;
    if (vec && k < kend && row + E <= R) return *reinterpret_cast<const uint4 *>(p + k * ld + row);
    T v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = (k < kend && row + e < R) ? ld_elem(p, k * ld + row + e) : T(0);
    return pack_elems<T>(v);
}

template <typename T, bool KC>
struct TileLoader {
    uint4 v[2];
    // global -> registers for rows [r0, r0 + 128), k in [k0, k0 + KT)
    __device__ __forceinline__ void load(const T *__restrict__ p, int64_t ld, int64_t r0, int64_t R, int64_t k0,
                                         int64_t kend, bool vec, int tid) {
        constexpr int E = GemmCfg<T>::E;
        if constexpr (KC) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                int c = tid + 256 * j;
                int row = c >> 2, kc = c & 3;
                v[j] = load_kc<T>(p, ld, r0 + row, R, k0 + kc * E, kend, vec);
            }
        } else {
            if constexpr (sizeof(T) == 2) {
                int kp = tid & 15, mg = tid >> 4;
                v[0] = load_mc<T>(p, ld, r0 + 8 * mg, R, k0 + 2 * kp, kend, vec);
                v[1] = load_mc<T>(p, ld, r0 + 8 * mg, R, k0 + 2 * kp + 1, kend, vec);
            } else {
                int kp = tid & 7, mg = tid >> 3;
                v[0] = load_mc<T>(p, ld, r0 + 4 * mg, R, k0 + 2 * kp, kend, vec);
                v[1] = load_mc<T>(p, ld, r0 + 4 * mg, R, k0 + 2 * kp + 1, kend, vec);
            }
        }
    }
    // registers -> LDS tile [128 rows][KT k] (k contiguous, PITCH bytes per row)
    __device__ __forceinline__ void store(char *lds, int tid) const {
        if constexpr (KC) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                int c = tid + 256 * j;
                int row = c >> 2, kc = c & 3;
                *reinterpret_cast<uint4 *>(lds + row * PITCH + kc * 16) = v[j];
            }
        } else {
            const uint32_t a[4] = {v[0].x, v[0].y, v[0].z, v[0].w};
            const uint32_t b[4] = {v[1].x, v[1].y, v[1].z, v[1].w};
            if constexpr (sizeof(T) == 2) {
                int kp = tid & 15, mg = tid >> 4;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    uint32_t lo = (a[e >> 1] >> ((e & 1) * 16)) & 0xffffu;
                    uint32_t hi = (b[e >> 1] >> ((e & 1) * 16)) & 0xffffu;
                    *reinterpret_cast<uint32_t *>(lds + (8 * mg + e) * PITCH + kp * 4) = lo | (hi << 16);
                }
            } else {
                int kp = tid & 7, mg = tid >> 3;
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

template <typename T, bool A_KC, bool B_KC, bool OUT_BF16>
__global__ __launch_bounds__(256) void gemm_kernel(const T *__restrict__ A, const T *__restrict__ B,
                                                   void *__restrict__ Cv, int64_t M, int64_t N, int64_t K,
                                                   int64_t lda, int64_t ldb, int64_t ldc, int64_t kchunk,
                                                   int64_t c_split_stride, int vec_a, int vec_b) {
    constexpr int KT = GemmCfg<T>::KT;
    __shared__ __attribute__((aligned(16))) char smem[2][2][BM * PITCH];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = int64_t(blockIdx.y) * BM, n0 = int64_t(blockIdx.x) * BN;
    const int64_t kbeg = int64_t(blockIdx.z) * kchunk;
    const int64_t kend = min(K, kbeg + kchunk);
    const int ntiles = kend > kbeg ? int((kend - kbeg + KT - 1) / KT) : 0;

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    TileLoader<T, A_KC> la;
    TileLoader<T, B_KC> lb;
    if (ntiles > 0) {
        la.load(A, lda, m0, M, kbeg, kend, vec_a, tid);
        lb.load(B, ldb, n0, N, kbeg, kend, vec_b, tid);
        la.store(smem[0][0], tid);
        lb.store(smem[0][1], tid);
    }
    __syncthreads();

    const int lr = lane & 31, lh = lane >> 5;
    for (int kt = 0; kt < ntiles; ++kt) {
        const int cur = kt & 1;
        const bool more = kt + 1 < ntiles;
        if (more) {
            la.load(A, lda, m0, M, kbeg + int64_t(kt + 1) * KT, kend, vec_a, tid);
            lb.load(B, ldb, n0, N, kbeg + int64_t(kt + 1) * KT, kend, vec_b, tid);
        }
        const char *sa = smem[cur][0];
        const char *sb = smem[cur][1];
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                bf16x8 av[2], bv[2];
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    av[i] = *reinterpret_cast<const bf16x8 *>(sa + (wm * 64 + i * 32 + lr) * PITCH + ks * 32 + lh * 16);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bv[j] = *reinterpret_cast<const bf16x8 *>(sb + (wn * 64 + j * 32 + lr) * PITCH + ks * 32 + lh * 16);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
            }
        } else {
#pragma unroll
            for (int kq = 0; kq < 2; ++kq) {
                f32x4 av[2], bv[2];
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    av[i] = *reinterpret_cast<const f32x4 *>(sa + (wm * 64 + i * 32 + lr) * PITCH + kq * 32 + lh * 16);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bv[j] = *reinterpret_cast<const f32x4 *>(sb + (wn * 64 + j * 32 + lr) * PITCH + kq * 32 + lh * 16);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int i = 0; i < 2; ++i)
#pragma unroll
                        for (int j = 0; j < 2; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][e], bv[j][e], acc[i][j], 0, 0, 0);
            }
        }
        if (more) {
            la.store(smem[cur ^ 1][0], tid);
            lb.store(smem[cur ^ 1][1], tid);
        }
        __syncthreads();
    }

    // epilogue: 32x32 accumulator layout, element v of lane l holds
    // row (v / 4) * 8 + (l / 32) * 4 + v % 4, column l % 32
    const int64_t coff = int64_t(blockIdx.z) * c_split_stride;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + wn * 64 + j * 32 + lr;
            if (col >= N) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = m0 + wm * 64 + i * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
                if (row < M) {
                    if constexpr (OUT_BF16)
                        reinterpret_cast<uint16_t *>(Cv)[coff + row * ldc + col] = f32_to_bf16_rne(acc[i][j][v]);
                    else
                        reinterpret_cast<float *>(Cv)[coff + row * ldc + col] = acc[i][j][v];
                }
            }
        }
}

inline int grid_for(int64_t n, int threads = 256, int64_t cap = 65536) {
    int64_t g = (n + threads - 1) / threads;
    return int(std::max<int64_t>(1, std::min<int64_t>(g, cap)));
}

template <typename T, bool AK, bool BK, bool OB>
int launch_gemm_t(const void *A, const void *B, void *C, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb,
                  int64_t ldc, int splits, int64_t kchunk, void *stream) {
    constexpr int E = GemmCfg<T>::E;
    auto aligned = [](const void *p, int64_t ld) {
        return (reinterpret_cast<uintptr_t>(p) % 16 == 0) && (ld % E == 0);
    };
    dim3 grid(unsigned((N + BN - 1) / BN), unsigned((M + BM - 1) / BM), unsigned(splits));
    hipLaunchKernelGGL((gemm_kernel<T, AK, BK, OB>), grid, dim3(256), 0, hipStream_t(stream),
                       reinterpret_cast<const T *>(A), reinterpret_cast<const T *>(B), C, M, N, K, lda, ldb, ldc,
                       kchunk, splits > 1 ? M * ldc : int64_t(0), int(aligned(A, lda)), int(aligned(B, ldb)));
    return int(hipGetLastError());
}

}  // namespace

int launch_fold(const FoldArgs &a, void *stream) {
    int64_t mx = 1;
    for (int k = 0; k < a.nfold; ++k) mx = std::max<int64_t>(mx, int64_t(a.rc[k]) * a.m[k] * a.n[k] * a.rc[k + 1]);
    if (a.nfold <= 0) return 0;
    dim3 grid(grid_for(mx), a.nfold);
    hipLaunchKernelGGL(fold_kernel, grid, dim3(256), 0, hipStream_t(stream), a);
    return int(hipGetLastError());
}

int launch_expand(const ExpandArgs &a, void *stream) {
    int64_t mx = 1;
    for (int k = 0; k < a.d; ++k) mx = std::max<int64_t>(mx, int64_t(a.r[k]) * a.m[k] * a.n[k] * a.r[k + 1]);
    dim3 grid(grid_for(mx), a.d);
    hipLaunchKernelGGL(expand_kernel, grid, dim3(256), 0, hipStream_t(stream), a);
    return int(hipGetLastError());
}

int launch_chain(const float *P, const float *G, float *out, uint16_t *out_bf16, int64_t NX, int64_t NY, int A,
                 int p1, int p2, int C, int xaxis, void *stream) {
    int64_t total = NX * NY * int64_t(p1) * p2 * C;
    hipLaunchKernelGGL(chain_kernel, dim3(grid_for(total)), dim3(256), 0, hipStream_t(stream), P, G, out, out_bf16,
                       NX, NY, A, p1, p2, C, xaxis);
    return int(hipGetLastError());
}

int launch_adjoint(const float *E, const float *G, float *out, int64_t NX, int64_t NY, int A, int p1, int p2, int C,
                   int xaxis, void *stream) {
    int64_t nterm = int64_t(p1) * p2 * C;
    if (nterm <= 256) {
        hipLaunchKernelGGL(adjoint_small_kernel, dim3(grid_for(NX * NY * A)), dim3(256), 0, hipStream_t(stream), E, G,
                           out, NX, NY, A, p1, p2, C, xaxis);
    } else {
        int64_t blocks = (NX * NY + 3) / 4;
        hipLaunchKernelGGL(adjoint_wave_kernel, dim3(unsigned(blocks)), dim3(256), 0, hipStream_t(stream), E, G, out,
                           NX, NY, A, p1, p2, C, xaxis);
    }
    return int(hipGetLastError());
}

int launch_meet(const float *P, const float *E, float *part, int64_t NX, int64_t NY, int A, int p1, int p2, int C,
                int xaxis, int splits, void *stream) {
    int64_t outs = int64_t(A) * p1 * p2 * C;
    int64_t XY = NX * NY;
    int64_t chunk = (XY + splits - 1) / splits;
    dim3 grid(grid_for(outs), unsigned(splits));
    hipLaunchKernelGGL(meet_kernel, grid, dim3(256), 0, hipStream_t(stream), P, E, part, NX, NY, A, p1, p2, C, xaxis,
                       chunk);
    return int(hipGetLastError());
}

int launch_sum_splits(const float *part, float *out, int64_t n, int splits, void *stream) {
    hipLaunchKernelGGL(sum_splits_kernel, dim3(grid_for(n)), dim3(256), 0, hipStream_t(stream), part, out, n, splits);
    return int(hipGetLastError());
}

int launch_fill_zero(void *ptr, size_t bytes, void *stream) {
    if (bytes == 0) return 0;
    int64_t n = int64_t(bytes / 4);
    hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(n)), dim3(256), 0, hipStream_t(stream),
                       reinterpret_cast<uint32_t *>(ptr), n);
    return int(hipGetLastError());
}

int launch_gemm(int dtype, bool a_kc, bool b_kc, bool out_bf16, const void *A, const void *B, void *C, int64_t M,
                int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc, int splits, int64_t kchunk,
                void *stream) {
    if (M <= 0 || N <= 0) return 0;
    if (splits < 1) splits = 1;
    if (kchunk <= 0) kchunk = K;
#define COMERA_GEMM_CASE(T, AK, BK, OB)                                                                        \
    if (a_kc == AK && b_kc == BK && out_bf16 == OB)                                                           \
        return launch_gemm_t<T, AK, BK, OB>(A, B, C, M, N, K, lda, ldb, ldc, splits, kchunk, stream);
    if (dtype == COMERA_BF16) {
        COMERA_GEMM_CASE(uint16_t, true, false, true)
        COMERA_GEMM_CASE(uint16_t, true, true, true)
        COMERA_GEMM_CASE(uint16_t, false, false, false)
    } else {
        COMERA_GEMM_CASE(float, true, false, false)
        COMERA_GEMM_CASE(float, true, true, false)
        COMERA_GEMM_CASE(float, false, false, false)
    }
#undef COMERA_GEMM_CASE
    return int(hipErrorInvalidValue);
}

}  // namespace comera
