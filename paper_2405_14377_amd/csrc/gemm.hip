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
// Four or eight waves per workgroup; each wave owns a WM x WN block made of
// 32 x 32 MFMA tiles (bf16: v_mfma_f32_32x32x16_bf16, fp32:
// v_mfma_f32_32x32x2f32, FP8 E4M3: v_mfma_scale_f32_32x32x64_f8f6f4 with
// unit block scales).  Both operand tiles are staged in LDS as rows of K
// (k contiguous), double buffered; operands whose k is strided in memory are
// transposed in registers on the way in.  A general kernel (64-byte K rows,
// bounds-checked loads) handles any shape; a fast kernel takes over when all
// accesses are in bounds by construction, and writes outputs whose 16-byte
// column pieces are contiguous through an LDS-staged tile (the fast kernel's
// bf16 products take the operands in the order B, A so that each lane ends
// with four consecutive columns of one row, converted to bf16 two at a time
// by the hardware's packed round-to-nearest-even).  Lanes read
// 16-byte vectors from LDS; the k slots fed to successive MFMAs are one fixed
// permutation of the tile's k range, shared by A and B, so the sum is
// unchanged.
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

// two floats -> two bf16 (round to nearest even) in one dword, a low; one
// v_cvt_pk_bf16_f32 on gfx950
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
    const f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
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
// FP8 (OCP E4M3) operands: fast kernel only
template <>
struct GemmCfg<uint8_t> {
    static constexpr int KT = 64;
    static constexpr int E = 16;
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
    int stage_c;   // fast kernel: row-major output staged through LDS (see epilogue_lds)
    int gw;   // tile-order group width in column tiles (see tile_of)
    uint32_t tx, ty;   // column tiles, row tiles (the grid is one-dimensional)
    const float *oscale;   // device scalar multiplying every result, or null
};

// Workgroup -> (split, row tile, column tile).  The dispatcher deals
// consecutive workgroup ids round-robin to the 8 XCDs, each with its own L2.
// The linear id is first turned into an XCD-major order (each XCD gets one
// contiguous range), and that order walks the tiles in groups of gw column
// tiles, row by row inside a group, so one XCD covers a compact block of the
// output and fetches each operand row into its L2 about once.
struct TileIdx {
    int64_t z, row, col;
};
__device__ __forceinline__ TileIdx tile_of(const GemmParams &p) {
    constexpr uint32_t kXcds = 8;
    const uint32_t nx = p.tx, ny = p.ty;
    const uint32_t per = nx * ny;
    const uint32_t total = gridDim.x;
    const uint32_t lin = blockIdx.x;
    const uint32_t x = lin % kXcds, i = lin / kXcds;
    const uint32_t q = total / kXcds, rem = total % kXcds;
    const uint32_t id = x * q + min(x, rem) + i;
    TileIdx t;
    t.z = id / per;
    const uint32_t tt = id % per;
    const uint32_t gw = p.gw > 0 ? min(uint32_t(p.gw), nx) : nx;
    const uint32_t g = tt / (gw * ny), r = tt % (gw * ny);
    const uint32_t w = min(gw, nx - g * gw);
    t.row = r / w;
    t.col = g * gw + r % w;
    return t;
}

// Write the accumulators: 32x32 layout, element v of lane l is row
// (v/4)*8 + (l/32)*4 + v%4 and column l%32; with SWAP (operands given to the
// MFMA in the order B, A) the transpose: row l%32, column (v/4)*8 + (l/32)*4 + v%4.
template <bool OUT_BF16, int TM, int TN, int WM, int WN, bool SWAP = false>
__device__ __forceinline__ void epilogue(const GemmParams &p, const f32x16 (&acc)[TM][TN], const int64_t *roff,
                                         const int64_t *coff, int wm, int wn, int lr, int lh) {
    const int64_t zoff = tile_of(p).z * p.split_stride;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int ra = (v >> 2) * 8 + lh * 4 + (v & 3);
                const int rl = wm * WM + i * 32 + (SWAP ? lr : ra);
                const int cl = wn * WN + j * 32 + (SWAP ? ra : lr);
                const int64_t ro = roff[rl], co = coff[cl];
                if (ro < 0 || co < 0) continue;
                if constexpr (OUT_BF16)
                    reinterpret_cast<uint16_t *>(p.C)[zoff + ro + co] = f32_to_bf16_rne(acc[i][j][v]);
                else
                    reinterpret_cast<float *>(p.C)[zoff + ro + co] = acc[i][j][v];
            }
}

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
    const TileIdx ti = tile_of(p);
    const int64_t m0 = ti.row * BM, n0 = ti.col * BN;
    const int64_t kbeg = ti.z * p.kchunk;
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

    epilogue<OUT_BF16, TM, TN, WM, WN>(p, acc, roff, coff, wm, wn, lr, lh);
}

// ---------------------------------------------------------------- fast path
// Used when every 16-byte operand access is in bounds by construction: rows
// aligned to 16 bytes, the K range of each split a multiple of the K tile,
// and (for operands whose rows are contiguous in memory) the row count a
// multiple of the 16-byte group.  Each thread computes its byte offsets
// once; a K step only moves a wave-uniform base pointer, so the loop body is
// loads, LDS traffic and MFMAs.  Rows past the end are clamped to the last
// row (their results are never stored).  LDS rows hold 64 or 128 bytes of K
// plus 16 bytes of padding; 128-byte rows (144-byte pitch) measure free of
// LDS bank conflicts on gfx950, 64-byte rows are kept for the operands
// transposed on the way in, where they load faster.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// KTB = bytes of K per LDS row (64 or 128), FP = KTB + 16 = LDS row pitch;
// NT threads share the loads
template <typename T, bool KC, int RT, int KTB, int NT = 256>
struct FastLoader {
    static constexpr int FP = KTB + 16;
    static constexpr int E = GemmCfg<T>::E;
    static constexpr int KT = KTB / int(sizeof(T));
    static constexpr int CPR = KTB / 16;
    static constexpr int NKC = (RT * CPR + NT - 1) / NT;
    static constexpr int KP = KT / 2;
    static constexpr int MG = sizeof(T) == 2 ? 8 : 4;
    static constexpr int NMB = (KP * (RT / MG) + NT - 1) / NT;
    static constexpr int NV = KC ? NKC : 2 * NMB;
    u32x4 v[NV];
    uint32_t off[NV];

    __device__ __forceinline__ void setup(int64_t ld, int64_t r0, int64_t R, int tid) {
        if constexpr (KC) {
#pragma unroll
            for (int j = 0; j < NKC; ++j) {
                const int c = min(tid + NT * j, RT * CPR - 1);
                const int64_t row = min(r0 + c / CPR, R - 1);
                off[j] = uint32_t((row * ld + (c % CPR) * E) * int64_t(sizeof(T)));
            }
        } else {
#pragma unroll
            for (int j = 0; j < NMB; ++j) {
                const int id = min(tid + NT * j, KP * (RT / MG) - 1);
                const int kp = id % KP, mg = id / KP;
                const int64_t row = min(r0 + MG * mg, R - MG);
                off[2 * j] = uint32_t(((2 * kp) * ld + row) * int64_t(sizeof(T)));
                off[2 * j + 1] = uint32_t(((2 * kp + 1) * ld + row) * int64_t(sizeof(T)));
            }
        }
    }
    __device__ __forceinline__ void load(const char *__restrict__ base) {
#pragma unroll
        for (int j = 0; j < NV; ++j) v[j] = *reinterpret_cast<const u32x4 *>(base + off[j]);
    }
    __device__ __forceinline__ void store(char *lds, int tid) const {
        if constexpr (KC) {
#pragma unroll
            for (int j = 0; j < NKC; ++j) {
                const int c = tid + NT * j;
                if (RT * CPR % NT == 0 || c < RT * CPR)
                    *reinterpret_cast<u32x4 *>(lds + (c / CPR) * FP + (c % CPR) * 16) = v[j];
            }
        } else {
#pragma unroll
            for (int j = 0; j < NMB; ++j) {
                const int id = tid + NT * j;
                if (KP * (RT / MG) % NT == 0 || id < KP * (RT / MG)) {
                    const int kp = id % KP, mg = id / KP;
                    if constexpr (sizeof(T) == 2) {
                        // element e of the two k rows -> one dword (k even low, k odd high)
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
                            const uint32_t w = __builtin_amdgcn_perm(v[2 * j + 1][e >> 1], v[2 * j][e >> 1], sel);
                            *reinterpret_cast<uint32_t *>(lds + (8 * mg + e) * FP + kp * 4) = w;
                        }
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            u32x2 w;
                            w[0] = v[2 * j][e];
                            w[1] = v[2 * j + 1][e];
                            *reinterpret_cast<u32x2 *>(lds + (4 * mg + e) * FP + kp * 8) = w;
                        }
                    }
                }
            }
        }
    }
};

// LDS of the fast kernel before the row / column offset tables: the two
// operand buffers, or, for eight-wave tiles (one workgroup per CU anyway),
// the staged output tile when that is larger and still fits the 160 KB of
// a CU.
constexpr size_t kLdsPerCu = 160 * 1024;
template <int BM, int BN, int KTB, int NT, bool OB>
constexpr size_t fast_main_lds() {
    const size_t ops = size_t(2) * (BM + BN) * (KTB + 16);
    const size_t stg = size_t(BM) * (BN * (OB ? 2 : 4) + 16);
    const size_t tables = size_t(BM + BN) * sizeof(int64_t);
    return (NT == 512 && stg > ops && stg + tables <= kLdsPerCu) ? stg : ops;
}
template <int BM, int BN, int KTB, int NT, bool OB>
constexpr bool fast_stage_fits() {
    return size_t(BM) * (BN * (OB ? 2 : 4) + 16) <= fast_main_lds<BM, BN, KTB, NT, OB>();
}

// Output through LDS: the accumulators are written into a BM x BN tile in
// LDS (16 bytes of padding per row), then every thread stores 16-byte
// pieces of its rows, so the output leaves as contiguous segments instead
// of 2- or 4-byte scattered stores.  Requires (p.stage_c) that every piece
// of 16 bytes / element size consecutive columns starting at a multiple of
// that count is contiguous and aligned in memory: unit innermost column
// stride, an innermost column radix that the piece divides, every other
// stride, N and the split stride multiples of the piece, and C 16-byte
// aligned.  Offsets come from the row and column tables (-1 = outside).
template <bool OUT_BF16, int TM, int TN, int WM, int WN, int BM, int BN, int NT, bool SWAP = false>
__device__ __forceinline__ void epilogue_lds(const GemmParams &p, const f32x16 (&acc)[TM][TN], char *stage,
                                             const int64_t *roff, const int64_t *coff, int wm, int wn, int lr,
                                             int lh, int tid) {
    constexpr int OESZ = OUT_BF16 ? 2 : 4;
    constexpr int CP = BN * OESZ + 16;
    constexpr int PIECES = BN * OESZ / 16;
    if constexpr (SWAP) {
        // four consecutive columns per lane and group g: one 8- or 16-byte write
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int row = wm * WM + i * 32 + lr;
                    const int col = wn * WN + j * 32 + g * 8 + lh * 4;
                    if constexpr (OUT_BF16) {
                        u32x2 w;
                        w[0] = pack2_bf16(acc[i][j][4 * g], acc[i][j][4 * g + 1]);
                        w[1] = pack2_bf16(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
                        *reinterpret_cast<u32x2 *>(stage + row * CP + col * 2) = w;
                    } else {
                        f32x4 w;
                        w[0] = acc[i][j][4 * g];
                        w[1] = acc[i][j][4 * g + 1];
                        w[2] = acc[i][j][4 * g + 2];
                        w[3] = acc[i][j][4 * g + 3];
                        *reinterpret_cast<f32x4 *>(stage + row * CP + col * 4) = w;
                    }
                }
    } else {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = wm * WM + i * 32 + (v >> 2) * 8 + lh * 4 + (v & 3);
                    const int col = wn * WN + j * 32 + lr;
                    if constexpr (OUT_BF16)
                        *reinterpret_cast<uint16_t *>(stage + row * CP + col * 2) = f32_to_bf16_rne(acc[i][j][v]);
                    else
                        *reinterpret_cast<float *>(stage + row * CP + col * 4) = acc[i][j][v];
                }
    }
    __syncthreads();
    const int64_t zoff = tile_of(p).z * p.split_stride;
    for (int id = tid; id < BM * PIECES; id += NT) {
        const int r = id / PIECES, c = id % PIECES;
        const int64_t ro = roff[r], co = coff[c * (16 / OESZ)];
        if (ro >= 0 && co >= 0)
            *reinterpret_cast<u32x4 *>(reinterpret_cast<char *>(p.C) + (zoff + ro + co) * OESZ) =
                *reinterpret_cast<const u32x4 *>(stage + r * CP + c * 16);
    }
}

// PF = register stages of global prefetch: 1 keeps the next K tile in
// registers while the current one is multiplied; 2 keeps two (the loads of
// tile kt + 2 are issued before tile kt is multiplied), for tiles whose K
// step is short against the load latency.
template <typename T, bool A_KC, bool B_KC, bool OUT_BF16, int BM, int BN, int WM, int WN, int KTB, int NT = 256,
          int PF = 1>
__global__ __launch_bounds__(NT) void gemm_fast_kernel(GemmParams p) {
    constexpr int FP = KTB + 16;
    constexpr int KT = KTB / int(sizeof(T));
    constexpr int WAVES_N = BN / WN;
    constexpr int TM = WM / 32, TN = WN / 32;
    static_assert((BM / WM) * (BN / WN) * 64 == NT, "one wave per WM x WN block");
    static_assert(PF == 1 || PF == 2, "prefetch depth");
    extern __shared__ __attribute__((aligned(16))) char smem[];
    char *sA0 = smem;
    char *sA1 = smem + BM * FP;
    char *sB0 = smem + 2 * BM * FP;
    char *sB1 = sB0 + BN * FP;
    int64_t *roff = reinterpret_cast<int64_t *>(smem + fast_main_lds<BM, BN, KTB, NT, OUT_BF16>());
    int64_t *coff = roff + BM;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const TileIdx ti = tile_of(p);
    const int64_t m0 = ti.row * BM, n0 = ti.col * BN;
    const int64_t kbeg = ti.z * p.kchunk;
    const int64_t kend = min(p.K, kbeg + p.kchunk);
    const int ntiles = kend > kbeg ? int((kend - kbeg) / KT) : 0;
    const char *abase = reinterpret_cast<const char *>(p.A) + (A_KC ? kbeg : kbeg * p.lda) * int64_t(sizeof(T));
    const char *bbase = reinterpret_cast<const char *>(p.B) + (B_KC ? kbeg : kbeg * p.ldb) * int64_t(sizeof(T));
    const int64_t astep = (A_KC ? KT : int64_t(KT) * p.lda) * int64_t(sizeof(T));
    const int64_t bstep = (B_KC ? KT : int64_t(KT) * p.ldb) * int64_t(sizeof(T));

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    FastLoader<T, A_KC, BM, KTB, NT> la;
    FastLoader<T, B_KC, BN, KTB, NT> lb;
    la.setup(p.lda, m0, p.M, tid);
    lb.setup(p.ldb, n0, p.N, tid);
    if (ntiles > 0) {
        la.load(abase);
        lb.load(bbase);
    }
    for (int i = tid; i < BM; i += NT) roff[i] = m0 + i < p.M ? remap(p.rmap, m0 + i) : int64_t(-1);
    for (int i = tid; i < BN; i += NT) coff[i] = n0 + i < p.N ? remap(p.cmap, n0 + i) : int64_t(-1);
    if (ntiles > 0) {
        la.store(sA0, tid);
        lb.store(sB0, tid);
    }

    const int lr = lane & 31, lh = lane >> 5;
    const int aoff = (wm * WM + lr) * FP + lh * 16, boff = (wn * WN + lr) * FP + lh * 16;
    // acc += the product of the K tile in LDS buffer cur
    auto mma = [&](int cur) {
        const char *a_s = (cur ? sA1 : sA0) + aoff;
        const char *b_s = (cur ? sB1 : sB0) + boff;
        if constexpr (sizeof(T) == 1) {
            // FP8 E4M3 x E4M3 (v_mfma_scale_f32_32x32x64_f8f6f4, unit block
            // scales 127 = 2^0): of each 64-byte k step, lane (lr, lh) supplies
            // bytes 16 lh .. 16 lh + 15 and 32 + 16 lh .. 32 + 16 lh + 15 of its
            // row (a_s, b_s already point 16 lh bytes in), the same k slots for
            // A and B.
#pragma unroll
            for (int ks = 0; ks < KT / 64; ++ks) {
                i32x8 bv[TN];
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const u32x4 lo = *reinterpret_cast<const u32x4 *>(b_s + j * 32 * FP + ks * 64);
                    const u32x4 hi = *reinterpret_cast<const u32x4 *>(b_s + j * 32 * FP + ks * 64 + 32);
                    bv[j] = __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                }
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const u32x4 lo = *reinterpret_cast<const u32x4 *>(a_s + i * 32 * FP + ks * 64);
                    const u32x4 hi = *reinterpret_cast<const u32x4 *>(a_s + i * 32 * FP + ks * 64 + 32);
                    const i32x8 av = __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv[j], acc[i][j], 0, 0, 0,
                                                                                    127, 0, 127);
                }
            }
        } else if constexpr (sizeof(T) == 2) {
            // the wave in its product phase goes first at the issue arbiter,
            // so the other wave's loads and LDS traffic fill the gaps (a few
            // per cent on the large bf16 products)
            __builtin_amdgcn_s_setprio(3);
#pragma unroll
            for (int ks = 0; ks < KT / 16; ++ks) {
                bf16x8 av[TM], bv[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) av[i] = *reinterpret_cast<const bf16x8 *>(a_s + i * 32 * FP + ks * 32);
#pragma unroll
                for (int j = 0; j < TN; ++j) bv[j] = *reinterpret_cast<const bf16x8 *>(b_s + j * 32 * FP + ks * 32);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv[j], av[i], acc[i][j], 0, 0, 0);
            }
            if constexpr (TM == 4 && TN == 2 && KT == 64) {
                // eight-wave tiles: the operands of step ks + 1 are read
                // from LDS between the products of step ks (one read per
                // product) instead of in one block (measured 2-7 % faster)
                __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
                for (int r = 0; r < 3; ++r) {
#pragma unroll
                    for (int t = 0; t < 6; ++t) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    }
                    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
            }
            __builtin_amdgcn_s_setprio(0);
        } else {
#pragma unroll
            for (int kq = 0; kq < KT / 8; ++kq) {
                f32x4 av[TM], bv[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) av[i] = *reinterpret_cast<const f32x4 *>(a_s + i * 32 * FP + kq * 32);
#pragma unroll
                for (int j = 0; j < TN; ++j) bv[j] = *reinterpret_cast<const f32x4 *>(b_s + j * 32 * FP + kq * 32);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int i = 0; i < TM; ++i)
#pragma unroll
                        for (int j = 0; j < TN; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][e], bv[j][e], acc[i][j], 0, 0, 0);
            }
        }
    };

    if constexpr (PF == 1) {
        __syncthreads();
        for (int kt = 0; kt < ntiles; ++kt) {
            const int cur = kt & 1;
            const bool more = kt + 1 < ntiles;
            if (more) {
                abase += astep;
                bbase += bstep;
                la.load(abase);
                lb.load(bbase);
            }
            mma(cur);
            if (more) {
                la.store(cur ? sA0 : sA1, tid);
                lb.store(cur ? sB0 : sB1, tid);
            }
            __syncthreads();
        }
    } else {
        // tile 0 is in buffer 0; tile 1 waits in la / lb, tile t + 2 is
        // loaded into the other register set while tile t is multiplied
        FastLoader<T, A_KC, BM, KTB, NT> la2;
        FastLoader<T, B_KC, BN, KTB, NT> lb2;
        la2.setup(p.lda, m0, p.M, tid);
        lb2.setup(p.ldb, n0, p.N, tid);
        if (ntiles > 1) {
            abase += astep;
            bbase += bstep;
            la.load(abase);
            lb.load(bbase);
        }
        __syncthreads();
        for (int kt = 0; kt < ntiles; kt += 2) {
            // buffer 0 holds tile kt, la / lb hold tile kt + 1
            if (kt + 2 < ntiles) {
                abase += astep;
                bbase += bstep;
                la2.load(abase);
                lb2.load(bbase);
            }
            mma(0);
            if (kt + 1 < ntiles) {
                la.store(sA1, tid);
                lb.store(sB1, tid);
            }
            __syncthreads();
            if (kt + 1 >= ntiles) break;
            // buffer 1 holds tile kt + 1, la2 / lb2 hold tile kt + 2
            if (kt + 3 < ntiles) {
                abase += astep;
                bbase += bstep;
                la.load(abase);
                lb.load(bbase);
            }
            mma(1);
            if (kt + 2 < ntiles) {
                la2.store(sA0, tid);
                lb2.store(sB0, tid);
            }
            __syncthreads();
        }
    }
    if (p.oscale) {
        const float sc = *p.oscale;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] *= sc;
    }
    // bf16 products take the operands swapped (B, A): each lane holds four
    // consecutive columns of one row
    constexpr bool SWAP = sizeof(T) == 2;
    if constexpr (fast_stage_fits<BM, BN, KTB, NT, OUT_BF16>()) {
        if (p.stage_c) {
            __syncthreads();   // every wave is done with the operand buffers
            epilogue_lds<OUT_BF16, TM, TN, WM, WN, BM, BN, NT, SWAP>(p, acc, smem, roff, coff, wm, wn, lr, lh, tid);
            return;
        }
    }
    epilogue<OUT_BF16, TM, TN, WM, WN, SWAP>(p, acc, roff, coff, wm, wn, lr, lh);
}

enum TileId { T128x128 = 0, T64x64 = 1, T128x32 = 2, T32x128 = 3, T128x64 = 4, T64x128 = 5 };

// Group width for tile_of: split the XCDs that share one split's tiles
// into p row blocks x q column blocks, choosing the split that fetches the
// fewest operand bytes (A is fetched once per column block, B once per row
// block).
int choose_gw(const GemmArgs &g, int bm, int bn, int splits) {
    const int64_t nx = (g.N + bn - 1) / bn, ny = (g.M + bm - 1) / bm;
    const int per_slice = splits >= 8 ? 1 : 8 / splits;
    int best_q = 1;
    double best = -1.0;
    for (int q = 1; q <= per_slice; q *= 2) {
        const int pr = per_slice / q;
        if (q > nx || pr > ny) continue;
        const double cost = double(q) * double(g.M) + double(pr) * double(g.N);
        if (best < 0 || cost < best) {
            best = cost;
            best_q = q;
        }
    }
    return int((nx + best_q - 1) / best_q);
}

// One-dimensional grid over (split, row tile, column tile); 0 when the tile
// count does not fit 31 bits.
dim3 tile_grid(const GemmArgs &g, int bm, int bn, GemmParams &q) {
    const int64_t tx = (g.N + bn - 1) / bn, ty = (g.M + bm - 1) / bm;
    const int64_t total = tx * ty * int64_t(g.splits);
    if (total <= 0 || total >= (int64_t(1) << 31)) return dim3(0, 1, 1);
    q.tx = uint32_t(tx);
    q.ty = uint32_t(ty);
    return dim3(static_cast<unsigned>(total), 1, 1);
}

// ---------------------------------------------------------------- DMA path
// bf16 products whose operands are both K-contiguous (KC: forward, dX) or
// both M/N-contiguous (MN: dW = X^T dY), 256 x 256 tiles of eight waves
// (128 x 64 each; KC also 256 x 192 tiles of waves of 64 x 96), K stages of
// 64 in two LDS slots.  The operand tiles go
// from global memory straight into LDS (global_load_lds_dwordx4: lane l of a
// wave writes 16 bytes at the instruction's LDS base + 16 l), so they take no
// registers and no LDS store instructions, and the loads of stage kt + 1 fly
// while stage kt is multiplied.  LDS rows carry no padding; 16-byte chunks
// are placed by an XOR swizzle instead (gfx950's LDS serves 16 or 32 lanes
// at a time from 64 four-byte banks):
//  - KC: rows of 128 bytes = 64 k of one m; chunk c of row r at c ^ ((r / 2)
//    & 7), so the sixteen rows sixteen consecutive lanes read fall in sixteen
//    different groups of four banks;
//  - MN: rows of 512 bytes = 256 m of one k; chunk c of row k at
//    c ^ (4 (k & 3)).  The MFMA wants eight consecutive k of one m per lane:
//    ds_read_b64_tr_b16 hands lane i of each 16-lane group element i % 4 of
//    the 8-byte reads of lanes i / 4 + 4 e (e = 0..3); with lane j of the
//    group reading 4 m at row k0 + j / 4, column m0 + 4 (j % 4), lane i gets
//    m0 + i at k0 .. k0 + 3, and a second read at k0 + 4 the rest.  The two
//    slots are separate LDS arrays addressed by name (the K loop runs in
//    pairs of stages), so the compiler sees that the loads in flight into one
//    slot do not feed the reads of the other.
typedef __attribute__((address_space(3))) void lds_void_t;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

constexpr int kDmaKT = 64;                      // k per stage
constexpr int kDmaOpB = 256 * kDmaKT * 2;       // one operand tile (32 KB)
constexpr int kDmaStageB = 2 * kDmaOpB;         // A and B of one stage

template <bool OUT_BF16>
constexpr size_t dma_main_lds() {
    // operand slots, or (when larger and within the CU) the staged bf16 tile
    const size_t ops = size_t(2) * kDmaStageB;
    const size_t stg = OUT_BF16 ? size_t(256) * (256 * 2 + 16) : 0;
    return stg > ops ? stg : ops;
}

// Loads of one stage (KC or MN) into the LDS slot sa (A) / sa + kDmaOpB (B):
// instruction j of wave w fills bytes 1024 (4 w + j) .. + 1023 of an operand
// tile.  KC: row 8 (4 w + j) + l / 8, position l % 8.  MN: k row
// 2 (4 w + j) + l / 32, position l % 32.  Rows / columns past the operand
// are clamped (their results are never stored).
template <bool MN, int IPB = 4, int ESZ = 2>
__device__ __forceinline__ void dma_offsets(const GemmParams &p, int64_t m0, int64_t n0, int wave, int lane,
                                            uint32_t (&aoffs)[4], uint32_t (&boffs)[IPB]) {
    static_assert(!MN || (IPB == 4 && ESZ == 2), "the dW tile is 256 wide, bf16");
    if constexpr (!MN) {
        // B tiles of 64 IPB rows (256 or 192): IPB instructions per wave
#pragma unroll
        for (int j = 0; j < IPB; ++j) {
            const int row = (wave * IPB + j) * 8 + (lane >> 3);
            const int c = (lane & 7) ^ ((row >> 1) & 7);
            const int64_t gb = min(n0 + row, p.N - 1);
            boffs[j] = uint32_t(gb * p.ldb * ESZ + c * 16);
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if constexpr (!MN) {
            const int row = (wave * 4 + j) * 8 + (lane >> 3);
            const int c = (lane & 7) ^ ((row >> 1) & 7);
            const int64_t ga = min(m0 + row, p.M - 1);
            aoffs[j] = uint32_t(ga * p.lda * ESZ + c * 16);
        } else {
            const int kr = (wave * 4 + j) * 2 + (lane >> 5);
            const int c = (lane & 31) ^ (4 * (kr & 3));
            const int64_t ga = min(m0 + 8 * c, p.M - 8), gb = min(n0 + 8 * c, p.N - 8);
            aoffs[j] = uint32_t((kr * p.lda + ga) * ESZ);
            boffs[j] = uint32_t((kr * p.ldb + gb) * ESZ);
        }
    }
}

template <int IPB = 4>
__device__ __forceinline__ void dma_issue(char *st, const char *ga, const char *gb, const uint32_t (&aoffs)[4],
                                          const uint32_t (&boffs)[IPB], int wave) {
    char *sa = st + wave * 4 * 1024;
    char *sb = st + kDmaOpB + wave * IPB * 1024;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void *>(ga + aoffs[j]), (lds_void_t *)(sa + j * 1024),
                                         16, 0, 0);
        if (j < IPB)
            __builtin_amdgcn_global_load_lds(reinterpret_cast<const void *>(gb + boffs[j]),
                                             (lds_void_t *)(sb + j * 1024), 16, 0, 0);
    }
}

// acc += the products of one stage in LDS slot st.  KC: lane (lr, lh) of k
// step ks takes logical chunk 2 ks + lh of its row (kpos).  MN: per 32-row
// block, two transposed 8-byte reads (k rows 16 ks + 8 lh + j / 4 and + 4).
template <bool MN, int TM, int TN, bool FP8 = false>
__device__ __forceinline__ void dma_mma(f32x16 (&acc)[TM][TN], const char *st, const uint32_t (&aaddr)[TM],
                                        const uint32_t (&baddr)[TN], const uint32_t (&kpos)[4]) {
    if constexpr (FP8) {
        // FP8 E4M3 (KC, 128 k per 128-byte row): k step ks of 64 takes
        // chunks 4 ks + lh and 4 ks + 2 + lh of the lane's row (positions
        // kpos[2 ks], kpos[2 ks + 1]), the k slots of the register-staged FP8
        // tile; unit block scales (127 = 2^0), the tensor scales applied in
        // the epilogue
        auto read8 = [&](uint32_t addr, int ks) -> i32x8 {
            const u32x4 lo = *reinterpret_cast<const u32x4 *>(st + addr + kpos[2 * ks]);
            const u32x4 hi = *reinterpret_cast<const u32x4 *>(st + addr + kpos[2 * ks + 1]);
            return __builtin_bit_cast(i32x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        };
        __builtin_amdgcn_s_setprio(3);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            i32x8 av[TM], bv[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) av[i] = read8(aaddr[i], ks);
#pragma unroll
            for (int j = 0; j < TN; ++j) bv[j] = read8(baddr[j], ks);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(bv[j], av[i], acc[i][j], 0, 0, 0, 127,
                                                                                0, 127);
        }
        // the operands of step 1 are read between the products of step 0
        constexpr int NR = TM + TN, NM = TM * TN;
        __builtin_amdgcn_sched_group_barrier(0x100, NR * 2, 0);
#pragma unroll
        for (int t = 0; t < NR; ++t) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
        __builtin_amdgcn_s_setprio(0);
        return;
    }
    constexpr int RPS = MN ? 2 : 1;   // LDS reads per operand block and k step
    auto read_op = [&](uint32_t addr, int ks) -> bf16x8 {
        if constexpr (!MN) {
            return *reinterpret_cast<const bf16x8 *>(st + addr + kpos[ks]);
        } else {
            const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)(st + addr + ks * 16 * 512));
            const s16x4 hi =
                __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)(st + addr + ks * 16 * 512 + 4 * 512));
            return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        }
    };
    __builtin_amdgcn_s_setprio(3);
#pragma unroll
    for (int ks = 0; ks < kDmaKT / 16; ++ks) {
        bf16x8 av[TM], bv[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) av[i] = read_op(aaddr[i], ks);
#pragma unroll
        for (int j = 0; j < TN; ++j) bv[j] = read_op(baddr[j], ks);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bv[j], av[i], acc[i][j], 0, 0, 0);
    }
    // the operands of step ks + 1 are read between the products of step ks
    constexpr int NR = TM + TN, NM = TM * TN;
    static_assert(NM >= NR, "more products than operand reads per k step");
    __builtin_amdgcn_sched_group_barrier(0x100, NR * RPS, 0);
#pragma unroll
    for (int r = 0; r < kDmaKT / 16 - 1; ++r) {
#pragma unroll
        for (int t = 0; t < NR; ++t) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, RPS, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
    __builtin_amdgcn_s_setprio(0);
}

// vmcnt(0): this wave's part of the stage about to be read has landed in
// LDS; the barrier then covers every wave's part, and every wave is done
// with the slot refilled next (it held the previous stage).  A plain
// barrier: a workgroup fence would also wait for nothing more here, and the
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void dma_stage_barrier() {
    __builtin_amdgcn_s_waitcnt(0x0F70);
    asm volatile("s_barrier" ::: "memory");
}

// BN = 256: waves of 128 x 64; BN = 192 (products whose 256 x 256 tiles
// would leave CUs idle, e.g. N = 768): waves of 64 x 96, B tiles of 192 rows.
// FP8: E4M3 codes, the same 128-byte K rows (128 k per stage).
template <bool OUT_BF16, int BN = 256, bool FP8 = false>
__global__ __launch_bounds__(512) void gemm_dma_kernel(GemmParams p) {
    static_assert(BN == 256 || BN == 192, "tile width");
    constexpr int ESZ = FP8 ? 1 : 2;
    constexpr int BM = 256, WM = BN == 256 ? 128 : 64, WN = BN == 256 ? 64 : 96, NT = 512, KT = 128 / ESZ;
    constexpr int IPB = BN / 64;   // B-operand load instructions per wave
    constexpr int TM = WM / 32, TN = WN / 32, WAVES_N = BN / WN;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    int64_t *roff = reinterpret_cast<int64_t *>(smem + dma_main_lds<OUT_BF16>());
    int64_t *coff = roff + BM;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const TileIdx ti = tile_of(p);
    const int64_t m0 = ti.row * BM, n0 = ti.col * BN;
    // split z covers k in [z kchunk, (z + 1) kchunk) (whole stages)
    const int64_t k0 = ti.z * p.kchunk, k1 = min(p.K, k0 + p.kchunk);
    const int ntiles = k1 > k0 ? int((k1 - k0) / KT) : 0;
    const char *abase = reinterpret_cast<const char *>(p.A) + k0 * ESZ;
    const char *bbase = reinterpret_cast<const char *>(p.B) + k0 * ESZ;
    constexpr int64_t kstep = KT * ESZ;
    uint32_t aoffs[4], boffs[IPB];
    dma_offsets<false, IPB, ESZ>(p, m0, n0, wave, lane, aoffs, boffs);

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    if (ntiles > 0) dma_issue<IPB>(smem, abase, bbase, aoffs, boffs, wave);
    for (int i = tid; i < BM; i += NT) roff[i] = m0 + i < p.M ? remap(p.rmap, m0 + i) : int64_t(-1);
    for (int i = tid; i < BN; i += NT) coff[i] = n0 + i < p.N ? remap(p.cmap, n0 + i) : int64_t(-1);

    const int lr = lane & 31, lh = lane >> 5;
    // every row a lane reads has the swizzle of row lr (rows start at
    // multiples of 32)
    uint32_t kpos[4], aaddr[TM], baddr[TN];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) kpos[ks] = uint32_t(((2 * ks + lh) ^ ((lr >> 1) & 7)) * 16);
#pragma unroll
    for (int i = 0; i < TM; ++i) aaddr[i] = uint32_t((wm * WM + i * 32 + lr) * 128);
#pragma unroll
    for (int j = 0; j < TN; ++j) baddr[j] = uint32_t(kDmaOpB + (wn * WN + j * 32 + lr) * 128);

    for (int kt = 0; kt < ntiles; ++kt) {
        dma_stage_barrier();
        if (kt + 1 < ntiles)
            dma_issue<IPB>(smem + ((kt + 1) & 1) * kDmaStageB, abase + (kt + 1) * kstep, bbase + (kt + 1) * kstep, aoffs,
                      boffs, wave);
        dma_mma<false, TM, TN, FP8>(acc, smem + (kt & 1) * kDmaStageB, aaddr, baddr, kpos);
    }
    __syncthreads();   // every wave is done with the operand slots
    if (p.oscale) {
        const float sc = *p.oscale;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] *= sc;
    }
    if constexpr (OUT_BF16) {
        if (p.stage_c) {
            epilogue_lds<OUT_BF16, TM, TN, WM, WN, BM, BN, NT, true>(p, acc, smem, roff, coff, wm, wn, lr, lh, tid);
            return;
        }
    }
    epilogue<OUT_BF16, TM, TN, WM, WN, true>(p, acc, roff, coff, wm, wn, lr, lh);
}

// Persistent form of the K-contiguous bf16 (and FP8) product for plain
// row-major bf16 outputs C[m * ldc + n]: one workgroup per CU walks its
// tiles, the loads of a tile's first stage fly while the previous tile's
// last stage is multiplied, and the finished tile leaves through per-wave
// staging in the slot of that last stage (8 KB per wave: 64 rows of 128
// bytes, 16-byte chunks XOR-swizzled by row, written and read back in two
// halves of the wave's 128 x 64 block).  Of the 16 sixteen-byte pieces a
// lane then owns, 12 are stored at once and the last 4 are held in
// registers and stored one per stage during the next tile's first four
// stages, each after that stage's loads.  Vector memory operations of a
// wave complete in issue order (gfx9 counts loads and stores on one
// counter), so the wait for a stage's loads names the number of stores
// issued after them and does not wait for those.  The FP8 form stores all
// 16 at once: its MFMA operands take the registers (holding would spill).
constexpr int kPersHold = 4;   // bf16: 16-byte pieces per lane held into the next tile
template <bool FP8>
constexpr int pers_hold() {
    return FP8 ? 0 : kPersHold;
}

__device__ __forceinline__ void pers_tile(const GemmParams &p, uint32_t id, int64_t &row, int64_t &col) {
    const uint32_t nx = p.tx, ny = p.ty;
    const uint32_t gw = p.gw > 0 ? min(uint32_t(p.gw), nx) : nx;
    const uint32_t g = id / (gw * ny), r = id % (gw * ny);
    const uint32_t w = min(gw, nx - g * gw);
    row = r / w;
    col = g * gw + r % w;
}

// vmcnt(n) for the n used here (0, 1, NOW), no wait on the other counters,
// then the workgroup barrier
template <int NOW>
__device__ __forceinline__ void pers_wait(int n) {
    static_assert(NOW > 1 && NOW < 64, "vmcnt range");
    if (n == 0) __builtin_amdgcn_s_waitcnt(0x0F70);
    else if (n == 1) __builtin_amdgcn_s_waitcnt(0x0F71);
    else __builtin_amdgcn_s_waitcnt(0x0F70 | (NOW & 15) | ((NOW >> 4) << 14));
    asm volatile("s_barrier" ::: "memory");
}

// FP8: E4M3 codes in the same 128-byte K rows (128 k per stage), the
// tensor scales applied before the bf16 conversion.
template <bool FP8>
__global__ __launch_bounds__(512) void gemm_dma_pers_kernel(GemmParams p) {
    constexpr int kPersHold = pers_hold<FP8>(), kPersNow = 16 - kPersHold;
    static_assert(kPersHold <= 8, "held pieces come from the second half");
    constexpr int ESZ = FP8 ? 1 : 2, OESZ = 2, BM = 256, BN = 256, WM = 128, WN = 64, KT = 128 / ESZ, IPB = 4;
    constexpr int TM = WM / 32, TN = WN / 32, WAVES_N = BN / WN;
    constexpr int64_t kstep = KT * ESZ;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int lr = lane & 31, lh = lane >> 5;
    const uint32_t ntile = p.tx * p.ty, G = gridDim.x;
    // workgroup b runs on XCD b % 8; round i of XCD x takes the ids
    // i G + x (G / 8) .. + G / 8 - 1 of the grouped order
    const uint32_t per_x = G / 8;
    const uint32_t base = (blockIdx.x % 8) * per_x + blockIdx.x / 8;
    if (base >= ntile) return;
    const int nst = int(p.K / KT);
    const int64_t ldc = p.rmap.stride[0];
    const char *A0 = reinterpret_cast<const char *>(p.A);
    const char *B0 = reinterpret_cast<const char *>(p.B);
    char *C0 = reinterpret_cast<char *>(p.C);

    uint32_t kpos[4], aaddr[TM], baddr[TN];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) kpos[ks] = uint32_t(((2 * ks + lh) ^ ((lr >> 1) & 7)) * 16);
#pragma unroll
    for (int i = 0; i < TM; ++i) aaddr[i] = uint32_t((wm * WM + i * 32 + lr) * 128);
#pragma unroll
    for (int j = 0; j < TN; ++j) baddr[j] = uint32_t(kDmaOpB + (wn * WN + j * 32 + lr) * 128);

    uint32_t id = base;
    int64_t row, col;
    pers_tile(p, id, row, col);
    uint32_t aoffs[4], boffs[IPB];
    dma_offsets<false, IPB, ESZ>(p, row * BM, col * BN, wave, lane, aoffs, boffs);
    dma_issue<IPB>(smem, A0, B0, aoffs, boffs, wave);
    int s0 = 0;               // slot of the current tile's stage 0
    int after0 = 0;           // stores issued after the current tile's stage-0 loads (0 or kPersNow)
    bool held = false;        // pieces of the previous tile waiting in hv
    bool held_full = false;   // ... all of them inside the output
    u32x4 hv[kPersHold > 0 ? kPersHold : 1];
    char *hbase = C0;         // the lane's first held piece
    int64_t hm = 0, hn = 0;   // its row and column
    // lane's piece q of a half block: row 8 q + lane / 8, columns 8 (lane % 8) .. + 7
    const int prow = lane >> 3, pcol = 8 * (lane & 7);
    const int64_t rstep = 8 * ldc * OESZ;   // bytes between pieces q and q + 1
    for (;;) {
        f32x16 acc[TM][TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
        const uint32_t nid = id + G;
        const bool has_next = nid < ntile;
        int64_t nrow = row, ncol = col;
        if (has_next) pers_tile(p, nid, nrow, ncol);
        const int hone = held && held_full ? 1 : 0;
        // the first stages store the held pieces, one per stage after its loads
#pragma unroll
        for (int kt = 0; kt < kPersHold; ++kt) {
            pers_wait<kPersNow>(kt == 0 ? after0 : hone);
            const int sl = (s0 + kt) & 1;
            dma_issue<IPB>(smem + (sl ^ 1) * kDmaStageB, A0 + (kt + 1) * kstep, B0 + (kt + 1) * kstep, aoffs, boffs,
                           wave);
            if (held && (held_full || (hm + 8 * kt < p.M && hn < p.N)))
                *reinterpret_cast<u32x4 *>(hbase + kt * rstep) = hv[kt];
            dma_mma<false, TM, TN, FP8>(acc, smem + sl * kDmaStageB, aaddr, baddr, kpos);
        }
        for (int kt = kPersHold; kt < nst; ++kt) {
            pers_wait<kPersNow>(kt == 0 ? after0 : kt == kPersHold ? hone : 0);
            const int sl = (s0 + kt) & 1;
            if (kt + 1 < nst) {
                dma_issue<IPB>(smem + (sl ^ 1) * kDmaStageB, A0 + (kt + 1) * kstep, B0 + (kt + 1) * kstep, aoffs,
                               boffs, wave);
            } else if (has_next) {
                dma_offsets<false, IPB, ESZ>(p, nrow * BM, ncol * BN, wave, lane, aoffs, boffs);
                dma_issue<IPB>(smem + (sl ^ 1) * kDmaStageB, A0, B0, aoffs, boffs, wave);
            }
            dma_mma<false, TM, TN, FP8>(acc, smem + sl * kDmaStageB, aaddr, baddr, kpos);
        }
        if (FP8 && p.oscale) {
            const float sc = *p.oscale;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v) acc[i][j][v] *= sc;
        }
        // every wave is done with the last stage's slot: it becomes the
        // staging area (no wait for the next tile's loads in flight)
        __builtin_amdgcn_s_waitcnt(0xC07F);
        asm volatile("s_barrier" ::: "memory");
        const int ls = (s0 + nst - 1) & 1;
        char *st = smem + ls * kDmaStageB + wave * 8192;
        const int64_t m0 = row * BM + wm * WM + prow, n0 = col * BN + wn * WN + pcol;
        const bool full = row * BM + BM <= p.M && col * BN + BN <= p.N;
        char *cb = C0 + (m0 * ldc + n0) * OESZ;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int i = 2 * half + ii;
                        const int lrow = ii * 32 + lr, ch = j * 4 + g;
                        u32x2 w;
                        w[0] = pack2_bf16(acc[i][j][4 * g], acc[i][j][4 * g + 1]);
                        w[1] = pack2_bf16(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
                        *reinterpret_cast<u32x2 *>(st + lrow * 128 + ((ch ^ (lrow & 7)) * 16) + lh * 8) = w;
                    }
            // pieces q of this half: all of the upper half and the first
            // 8 - kPersHold of the lower half now, the rest held
            constexpr int NOW = 8 - kPersHold;
            u32x4 v[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int lrow = 8 * q + prow;
                const u32x4 x = *reinterpret_cast<const u32x4 *>(st + lrow * 128 + (((lane & 7) ^ (lrow & 7)) * 16));
                if (half == 1 && q >= NOW)
                    hv[q - NOW] = x;
                else
                    v[q] = x;
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                if (half == 1 && q >= NOW) break;
                if (full || (m0 + 64 * half + 8 * q < p.M && n0 < p.N))
                    *reinterpret_cast<u32x4 *>(cb + (8 * half + q) * rstep) = v[q];
            }
        }
        // this wave's staging reads have returned before any wave passes the
        // next barrier (the slot is refilled after it)
        __builtin_amdgcn_s_waitcnt(0xC07F);
        held = true;
        held_full = full;
        hm = m0 + 64 + 8 * (8 - kPersHold);
        hn = n0;
        hbase = cb + (8 + 8 - kPersHold) * rstep;
        if (!has_next) break;
        after0 = full ? kPersNow : 0;
        s0 = (s0 + nst) & 1;
        id = nid;
        row = nrow;
        col = ncol;
    }
    // the last tile's held pieces
#pragma unroll
    for (int q = 0; q < kPersHold; ++q)
        if (held_full || (hm + 8 * q < p.M && hn < p.N)) *reinterpret_cast<u32x4 *>(hbase + q * rstep) = hv[q];
}

// MN operands (dW): two named LDS slots, each also holding a quarter of the
// output tile (64 rows) on its way out
constexpr int kDmaMnSlotB = 64 * (256 * 4 + 16);   // >= kDmaStageB, one fp32 quarter tile

template <bool OUT_BF16>
__global__ __launch_bounds__(512) void gemm_dma_mn_kernel(GemmParams p) {
    static_assert(kDmaMnSlotB >= kDmaStageB, "slot size");
    constexpr int BM = 256, BN = 256, WM = 128, WN = 64, NT = 512, KT = kDmaKT;
    constexpr int TM = WM / 32, TN = WN / 32, WAVES_N = BN / WN;
    constexpr int ESZ = int(sizeof(uint16_t));
    __shared__ __attribute__((aligned(16))) char slot0[kDmaMnSlotB];
    __shared__ __attribute__((aligned(16))) char slot1[kDmaMnSlotB];
    __shared__ int64_t roff[BM], coff[BN];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const TileIdx ti = tile_of(p);
    const int64_t m0 = ti.row * BM, n0 = ti.col * BN;
    const int64_t kbeg = ti.z * p.kchunk;
    const int64_t kend = min(p.K, kbeg + p.kchunk);
    const int ntiles = kend > kbeg ? int((kend - kbeg) / KT) : 0;
    const char *abase = reinterpret_cast<const char *>(p.A) + kbeg * p.lda * ESZ;
    const char *bbase = reinterpret_cast<const char *>(p.B) + kbeg * p.ldb * ESZ;
    const int64_t astep = KT * p.lda * ESZ, bstep = KT * p.ldb * ESZ;
    uint32_t aoffs[4], boffs[4];
    dma_offsets<true, 4>(p, m0, n0, wave, lane, aoffs, boffs);

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    if (ntiles > 0) dma_issue<4>(slot0, abase, bbase, aoffs, boffs, wave);
    for (int i = tid; i < BM; i += NT) roff[i] = m0 + i < p.M ? remap(p.rmap, m0 + i) : int64_t(-1);
    for (int i = tid; i < BN; i += NT) coff[i] = n0 + i < p.N ? remap(p.cmap, n0 + i) : int64_t(-1);

    const int lr = lane & 31, lh = lane >> 5;
    const int g1 = (lane >> 4) & 1, jj = lane & 15, q = jj >> 2;
    const int krow = 8 * lh + q;   // (krow & 3) == q for every k step and half
    uint32_t kpos[4] = {0, 0, 0, 0}, aaddr[TM], baddr[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int m = wm * WM + i * 32 + 16 * g1 + 4 * (jj & 3);
        aaddr[i] = uint32_t(krow * 512 + (((m >> 3) ^ (4 * q)) * 16) + (m & 7) * 2);
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int n = wn * WN + j * 32 + 16 * g1 + 4 * (jj & 3);
        baddr[j] = uint32_t(kDmaOpB + krow * 512 + (((n >> 3) ^ (4 * q)) * 16) + (n & 7) * 2);
    }

    for (int kt = 0; kt < ntiles; kt += 2) {
        dma_stage_barrier();
        if (kt + 1 < ntiles) dma_issue<4>(slot1, abase + (kt + 1) * astep, bbase + (kt + 1) * bstep, aoffs, boffs, wave);
        dma_mma<true, TM, TN>(acc, slot0, aaddr, baddr, kpos);
        if (kt + 1 >= ntiles) break;
        dma_stage_barrier();
        if (kt + 2 < ntiles) dma_issue<4>(slot0, abase + (kt + 2) * astep, bbase + (kt + 2) * bstep, aoffs, boffs, wave);
        dma_mma<true, TM, TN>(acc, slot1, aaddr, baddr, kpos);
    }
    __syncthreads();   // every wave is done with the operand slots
    if (p.oscale) {
        const float sc = *p.oscale;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] *= sc;
    }
    if (!p.stage_c) {
        epilogue<OUT_BF16, TM, TN, WM, WN, true>(p, acc, roff, coff, wm, wn, lr, lh);
        return;
    }
    // a quarter of the rows (two 32-row blocks of one wm) at a time through slot0
    constexpr int OESZ = OUT_BF16 ? 2 : 4;
    constexpr int CP = BN * OESZ + 16, PIECES = BN * OESZ / 16;
    const int64_t zoff = ti.z * p.split_stride;
#pragma unroll
    for (int qr = 0; qr < 4; ++qr) {
        if (wm == qr / 2) {
#pragma unroll
            for (int i = 2 * (qr % 2); i < 2 * (qr % 2) + 2; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        char *dst = slot0 + ((i % 2) * 32 + lr) * CP + (wn * WN + j * 32 + g * 8 + lh * 4) * OESZ;
                        if constexpr (OUT_BF16) {
                            u32x2 w;
                            w[0] = pack2_bf16(acc[i][j][4 * g], acc[i][j][4 * g + 1]);
                            w[1] = pack2_bf16(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
                            *reinterpret_cast<u32x2 *>(dst) = w;
                        } else {
                            f32x4 w;
                            w[0] = acc[i][j][4 * g];
                            w[1] = acc[i][j][4 * g + 1];
                            w[2] = acc[i][j][4 * g + 2];
                            w[3] = acc[i][j][4 * g + 3];
                            *reinterpret_cast<f32x4 *>(dst) = w;
                        }
                    }
        }
        __syncthreads();
        for (int id = tid; id < 64 * PIECES; id += NT) {
            const int r = id / PIECES, c = id % PIECES;
            const int64_t ro = roff[qr * 64 + r], co = coff[c * (16 / OESZ)];
            if (ro >= 0 && co >= 0)
                *reinterpret_cast<u32x4 *>(reinterpret_cast<char *>(p.C) + (zoff + ro + co) * OESZ) =
                    *reinterpret_cast<const u32x4 *>(slot0 + r * CP + c * 16);
        }
        __syncthreads();
    }
}

// fp32 dW = X^T dY (operands M/N-contiguous) on the straight-to-LDS path:
// 128 x 128 tiles of four waves (64 x 64 each, v_mfma_f32_32x32x2f32), K
// stages of 32 k rows in two LDS slots of 32 KB (two workgroups per CU),
// split over K by the grid (split z covers k in [z kchunk, (z + 1) kchunk)).
// A k row of a tile is 128 m (512 bytes) loaded as 16-byte chunks, chunk c at
// position c ^ (8 (k & 1)), so that the two k rows one MFMA reads (the two
// lane halves) fall on different banks; lane (lr, lh) reads element m = lr of
// k row 2 s + lh, no transposition needed for 4-byte elements.  Columns past
// M / N are clamped (their results are never stored).  Measured against the
// register-staged 128 x 128 fp32 tile: 197 against 210 us on 768 x 3072 x
// 4096 (its register transposes are what this saves); the K-contiguous form
// of the same kernel was slower than the register-staged tile (192 against
// 181 us on 4096 x 3072 x 768) and is not kept.
constexpr int kD32KT = 32;                  // k per stage
constexpr int kD32Op = 128 * kD32KT * 4;    // one operand tile (16 KB)
constexpr int kD32Stage = 2 * kD32Op;       // A and B of one stage

__global__ __launch_bounds__(256) void gemm_dma32_kernel(GemmParams p) {
    constexpr int BM = 128, BN = 128, WM = 64, WN = 64, TM = 2, TN = 2, NT = 256;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    int64_t *roff = reinterpret_cast<int64_t *>(smem + 2 * kD32Stage);
    int64_t *coff = roff + BM;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const TileIdx ti = tile_of(p);
    const int64_t m0 = ti.row * BM, n0 = ti.col * BN;
    const int64_t k0 = ti.z * p.kchunk, k1 = min(p.K, k0 + p.kchunk);
    const int ntiles = k1 > k0 ? int((k1 - k0) / kD32KT) : 0;
    const char *abase = reinterpret_cast<const char *>(p.A);
    const char *bbase = reinterpret_cast<const char *>(p.B);
    // byte offsets of this thread's four chunks of A and of B in one stage
    uint32_t aoffs[4], boffs[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int kr = (wave * 4 + j) * 2 + (lane >> 5);
        const int c = (lane & 31) ^ (8 * (kr & 1));
        const int64_t ga = min(m0 + 4 * c, p.M - 4), gb = min(n0 + 4 * c, p.N - 4);
        aoffs[j] = uint32_t((kr * p.lda + ga) * 4);
        boffs[j] = uint32_t((kr * p.ldb + gb) * 4);
    }
    abase += k0 * p.lda * 4;
    bbase += k0 * p.ldb * 4;
    const int64_t astep = int64_t(kD32KT) * p.lda * 4, bstep = int64_t(kD32KT) * p.ldb * 4;
    auto issue = [&](char *st, int kt) {
        char *sa = st + wave * 4 * 1024, *sb = st + kD32Op + wave * 4 * 1024;
        const char *ga = abase + kt * astep, *gb = bbase + kt * bstep;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            __builtin_amdgcn_global_load_lds(reinterpret_cast<const void *>(ga + aoffs[j]),
                                             (lds_void_t *)(sa + j * 1024), 16, 0, 0);
            __builtin_amdgcn_global_load_lds(reinterpret_cast<const void *>(gb + boffs[j]),
                                             (lds_void_t *)(sb + j * 1024), 16, 0, 0);
        }
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    if (ntiles > 0) issue(smem, 0);
    for (int i = tid; i < BM; i += NT) roff[i] = m0 + i < p.M ? remap(p.rmap, m0 + i) : int64_t(-1);
    for (int i = tid; i < BN; i += NT) coff[i] = n0 + i < p.N ? remap(p.cmap, n0 + i) : int64_t(-1);

    const int lr = lane & 31, lh = lane >> 5;
    for (int kt = 0; kt < ntiles; ++kt) {
        dma_stage_barrier();
        if (kt + 1 < ntiles) issue(smem + ((kt + 1) & 1) * kD32Stage, kt + 1);
        const char *st = smem + (kt & 1) * kD32Stage;
        // k rows of 512 bytes; lane (lr, lh) reads m = lr of k row 2 s + lh
        const float *fa = reinterpret_cast<const float *>(st), *fb = reinterpret_cast<const float *>(st + kD32Op);
#pragma unroll
        for (int s = 0; s < kD32KT / 2; ++s) {
            const int kr = 2 * s + lh, sw = 32 * (kr & 1);
            f32x2_t av, bv;   // (block 0, block 1)
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                const int ma = wm * WM + i * 32 + lr, nb = wn * WN + i * 32 + lr;
                av[i] = fa[kr * 128 + (ma ^ sw)];
                bv[i] = fb[kr * 128 + (nb ^ sw)];
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(bv[j], av[i], acc[i][j], 0, 0, 0);
        }
    }
    epilogue<false, TM, TN, WM, WN, true>(p, acc, roff, coff, wm, wn, lr, lh);
}

int launch_dma32(const GemmArgs &g, const GemmParams &p, void *stream) {
    constexpr size_t lds = size_t(2) * kD32Stage + size_t(256) * sizeof(int64_t);
    static_assert(lds <= kLdsPerCu, "LDS of one workgroup");
    auto kern = gemm_dma32_kernel;
    if (!launch_check_mode()) {
        static const int set = int(hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)));
        if (set) return set;
    }
    GemmParams q = p;
    const dim3 grid = tile_grid(g, 128, 128, q);
    if (!grid.x) return int(hipErrorInvalidConfiguration);
    q.gw = choose_gw(g, 128, 128, g.splits);
    COMERA_LAUNCH_NAMED("gemm_dma32_kernel", kern, grid, dim3(256), lds, hipStream_t(stream), q);
    return launch_status();
}

template <bool OB, bool MN, int BN = 256, bool FP8 = false>
int launch_dma(const GemmArgs &g, const GemmParams &p, void *stream) {
    static_assert(!MN || (BN == 256 && !FP8), "the dW tile is 256 wide, bf16");
    constexpr size_t lds = MN ? 0 : dma_main_lds<OB>() + size_t(512) * sizeof(int64_t);
    static_assert(lds <= kLdsPerCu, "LDS of one workgroup");
    auto kern = MN ? gemm_dma_mn_kernel<OB> : gemm_dma_kernel<OB, BN, FP8>;
    if (!MN && !launch_check_mode()) {
        static const int set = int(hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)));
        if (set) return set;
    }
    GemmParams q = p;
    const dim3 grid = tile_grid(g, 256, BN, q);
    if (!grid.x) return int(hipErrorInvalidConfiguration);
    q.gw = choose_gw(g, 256, BN, g.splits);
    COMERA_LAUNCH_NAMED("gemm_dma_kernel", kern, grid, dim3(512), lds, hipStream_t(stream), q);
    return launch_status();
}

// The persistent product: bf16 or FP8 K-contiguous operands, one split, K a
// whole number of stages (64 k bf16, 128 FP8) with more stages than held
// pieces, output bf16 C[m * ldc + n] (16-byte pieces aligned), an output
// scale only for FP8.
bool pers_ok(const GemmArgs &g) {
    const bool fp8 = g.dtype == kDtypeFp8;
    if ((g.dtype != COMERA_BF16 && !fp8) || !g.a_kc || !g.b_kc || !g.out_bf16 || g.splits != 1) return false;
    if (g.oscale && !fp8) return false;
    const int64_t kt = fp8 ? 128 : 64;   // k per stage
    if (g.K % kt != 0 || g.K / kt <= (fp8 ? 1 : kPersHold)) return false;
    if (g.rmap.nd != 1 || g.cmap.nd != 1 || g.cmap.stride[0] != 1) return false;
    if (g.N % 8 != 0 || g.rmap.stride[0] % 8 != 0 || reinterpret_cast<uintptr_t>(g.C) % 16 != 0) return false;
    if (reinterpret_cast<uintptr_t>(g.A) % 16 != 0 || reinterpret_cast<uintptr_t>(g.B) % 16 != 0) return false;
    const int64_t e16 = fp8 ? 16 : 8;   // elements per 16-byte chunk
    if (g.lda % e16 != 0 || g.ldb % e16 != 0) return false;
    return true;
}

template <bool FP8>
int launch_dma_pers(const GemmArgs &g, const GemmParams &p, void *stream) {
    constexpr size_t lds = size_t(2) * kDmaStageB;
    static_assert(lds <= kLdsPerCu, "LDS of one workgroup");
    if (!launch_check_mode()) {
        static const int set = int(hipFuncSetAttribute(reinterpret_cast<const void *>(gemm_dma_pers_kernel<FP8>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)));
        if (set) return set;
    }
    GemmParams q = p;
    const dim3 tiles = tile_grid(g, 256, 256, q);
    if (!tiles.x) return int(hipErrorInvalidConfiguration);
    if (tiles.x < 256) return int(hipErrorInvalidValue);   // whole rounds of 256 workgroups, 32 per XCD
    // groups of four column tiles: a round's 32 tiles of one XCD then span
    // eight row tiles x four column tiles, whose operands (6 MB on
    // 65536 x 4096 x 1024) sit closer to the XCD's 4 MB L2 than two whole
    // rows of tiles (9 MB); measured 0.565 against 0.581 ms there, and level
    // on products four column tiles wide
    q.gw = int(std::min<uint32_t>(4u, q.tx));
    const unsigned grid = 256;
    COMERA_LAUNCH_NAMED("gemm_dma_pers_kernel", gemm_dma_pers_kernel<FP8>, dim3(grid), dim3(512), lds,
                        hipStream_t(stream), q);
    return launch_status();
}

template <typename T, bool AK, bool BK, bool OB>
int launch_t(const GemmArgs &g, const GemmParams &p, int tile, void *stream) {
    auto go = [&](auto kern, int bm, int bn) {
        GemmParams q = p;
        const dim3 grid = tile_grid(g, bm, bn, q);
        if (!grid.x) return int(hipErrorInvalidConfiguration);
        q.gw = choose_gw(g, bm, bn, g.splits);
        COMERA_LAUNCH_NAMED("gemm_kernel", kern, grid, dim3(256), 0, hipStream_t(stream), q);
        return launch_status();
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


// Fast-path tiles: {BM, BN, K bytes per LDS row}.
enum FastId {
    F128x128_128 = 0, F128x64_128, F64x128_128, F128x128_64, F256x128_64,
    // bf16 only, eight waves: 256 x 256 (waves of 128 x 64), 256 x 128 (64 x 64)
    F256x256_128w8, F256x128_128w8,
    // bf16 and FP8, eight waves of 128 x 64 on 64-byte K rows with two
    // register stages of prefetch (FP8: the operands of two 64-byte steps
    // per stage would not fit the registers of a wave beside its
    // accumulators)
    F256x256_64w8,
    // bf16, straight-to-LDS loads (gemm_dma_kernel, gemm_dma_mn_kernel)
    F256x256_dma,
    // bf16, K-contiguous operands, straight-to-LDS loads, 256 x 192 tiles
    F256x192_dma,
    // fp32, M/N-contiguous operands, straight-to-LDS loads (gemm_dma32_kernel),
    // 128 x 128 tiles
    F128x128_dma32,
    // bf16 or FP8, K-contiguous operands, plain bf16 output: the persistent
    // form of F256x256_dma (gemm_dma_pers_kernel)
    F256x256_pers
};

template <typename T, bool AK, bool BK, bool OB, int BM, int BN, int WM, int WN, int KTB, int NT = 256, int PF = 1>
int go_fast(const GemmArgs &g, const GemmParams &p, void *stream) {
    constexpr size_t lds = fast_main_lds<BM, BN, KTB, NT, OB>() + size_t(BM + BN) * sizeof(int64_t);
    static_assert(lds <= kLdsPerCu, "LDS of one workgroup");
    auto kern = gemm_fast_kernel<T, AK, BK, OB, BM, BN, WM, WN, KTB, NT, PF>;
    // above the default 64 KB of dynamic LDS: raise the limit once per kernel
    if (!launch_check_mode()) {
        static const int set = int(hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)));
        if (set) return set;
    }
    GemmParams q = p;
    const dim3 grid = tile_grid(g, BM, BN, q);
    if (!grid.x) return int(hipErrorInvalidConfiguration);
    q.gw = choose_gw(g, BM, BN, g.splits);
    COMERA_LAUNCH_NAMED("gemm_fast_kernel", kern, grid, dim3(NT), lds, hipStream_t(stream), q);
    return launch_status();
}

template <typename T, bool AK, bool BK, bool OB>
int launch_fast(const GemmArgs &g, const GemmParams &p, int id, void *stream) {
    switch (id) {
        case F128x128_128: return go_fast<T, AK, BK, OB, 128, 128, 64, 64, 128>(g, p, stream);
        case F128x64_128: return go_fast<T, AK, BK, OB, 128, 64, 64, 32, 128>(g, p, stream);
        case F64x128_128: return go_fast<T, AK, BK, OB, 64, 128, 32, 64, 128>(g, p, stream);
        case F128x128_64: return go_fast<T, AK, BK, OB, 128, 128, 64, 64, 64>(g, p, stream);
        case F256x128_64: return go_fast<T, AK, BK, OB, 256, 128, 128, 64, 64>(g, p, stream);
    }
    if constexpr (sizeof(T) == 2) {
        switch (id) {
            case F256x256_128w8: return go_fast<T, AK, BK, OB, 256, 256, 128, 64, 128, 512>(g, p, stream);
            case F256x128_128w8: return go_fast<T, AK, BK, OB, 256, 128, 64, 64, 128, 512>(g, p, stream);
        }
    }
    if constexpr (sizeof(T) <= 2) {
        if (id == F256x256_64w8) return go_fast<T, AK, BK, OB, 256, 256, 128, 64, 64, 512, 2>(g, p, stream);
    }
    return int(hipErrorInvalidValue);
}

// Tile for the fast path (measured on the layer shapes): operands that are
// both K-contiguous take 128-byte K rows; products with a transposed operand
// take 64-byte rows.  Returns -1 when the product is too small to fill the
// chip with these tiles (the general kernel's smaller tiles do better).
int pick_fast(const GemmArgs &g, int splits) {
    // transposed operands with a side of 64 or less (the meets of the paper's
    // TT layout) stream the token rows: these tiles would mostly compute
    // padding, the general kernel's 32-wide skinny tiles do better (the
    // sweep steps of that layout are measured on its 1024 -> 4096 shape)
    if (!g.a_kc && !g.b_kc && (g.M <= 64 || g.N <= 64) && g.dtype != kDtypeFp8) return -1;
    // K-contiguous operands with a side of 64 or less: the tile whose short
    // side is 64
    if (g.a_kc && g.b_kc && std::min(g.M, g.N) <= 64 && g.dtype != kDtypeFp8)
        return g.N <= 64 ? F128x64_128 : F64x128_128;
    const int64_t t128 = ceil_div(g.M, 128) * ceil_div(g.N, 128) * splits;
    const int64_t t256 = ceil_div(g.M, 256) * ceil_div(g.N, 256) * splits;
    // bf16: 256 x 256 tiles of eight waves once they give two or more
    // workgroups per CU (transposed operands, split over K: half a wave of
    // workgroups is enough)
    // FP8 codes (always K-contiguous) on the straight-to-LDS tile from half a
    // wave of tiles
    if (g.dtype == kDtypeFp8 && g.a_kc && g.b_kc && t256 >= 256 && splits == 1 && pers_ok(g)) return F256x256_pers;
    if (g.dtype == kDtypeFp8 && g.a_kc && g.b_kc && t256 >= 128) return F256x256_dma;
    if (g.dtype == kDtypeFp8 && t256 >= 512) return F256x256_64w8;
    // bf16 256 x 256 tiles with straight-to-LDS operand loads: K-contiguous
    // unsplit products from half a wave of tiles (below that the smaller
    // tiles fill more CUs), M/N-contiguous ones (dW) from an eighth: their
    // transposing loads are what the DMA form saves (measured on the layer
    // shapes)
    if (g.dtype == COMERA_BF16 && g.a_kc && g.b_kc && splits == 1 && t256 >= 128) {
        // 256 x 192 tiles where 256 x 256 ones leave CUs idle in the last
        // round: rounds of 256 tiles, the narrower tile doing 3/4 of the
        // work (and measured about 10 % slower per flop); e.g. N = 768
        // fills the chip once with 192-wide tiles (16384 x 768 x 768:
        // 26.8 -> 23.9 us), not with 256-wide ones
        const int64_t t192 = ceil_div(g.M, 256) * ceil_div(g.N, 192);
        const int64_t r256 = ceil_div(t256, 256), r192 = ceil_div(t192, 256);
        if (double(r192) * 0.75 * 1.1 < double(r256)) return F256x192_dma;
        // whole rounds of 256 tiles and a plain bf16 output: the persistent
        // form, whose tile epilogues overlap the next tiles' loads and
        // products (65536 x 4096 x 1024: 0.614 -> 0.583 ms, 16384 x 3072 x
        // 768: 0.094 -> 0.085 ms)
        if (t256 >= 256 && pers_ok(g)) return F256x256_pers;
        return F256x256_dma;
    }
    if (g.dtype == COMERA_BF16 && !g.a_kc && !g.b_kc && t256 >= 32) return F256x256_dma;
    if ((g.dtype == COMERA_BF16 || g.dtype == kDtypeFp8) && g.a_kc == g.b_kc && t256 >= (g.a_kc ? 512 : 128))
        return F256x256_128w8;
    if (g.a_kc && g.b_kc) {
        // fp32 tiles of 128 x 128 fit three workgroups per CU with 64-byte rows
        if (g.dtype == COMERA_F32 && t128 >= 240) return F128x128_64;
        if (t128 >= 512) return F128x128_128;
        const int64_t t64 = ceil_div(g.M, g.M >= g.N ? 128 : 64) * ceil_div(g.N, g.M >= g.N ? 64 : 128) * splits;
        if (t64 >= 240) return g.M >= g.N ? F128x64_128 : F64x128_128;
        return -1;
    }
    if (!g.a_kc && !g.b_kc) {
        if (g.dtype == COMERA_F32 && t128 >= 240) return F128x128_dma32;
        if (ceil_div(g.M, 256) * ceil_div(g.N, 128) * splits >= 480) return F256x128_64;
        return t128 >= 240 ? F128x128_64 : -1;
    }
    return t128 >= 240 ? F128x128_64 : -1;
}

// Whether every 16-byte access of the fast kernel stays inside the operand:
// 16-byte aligned rows, whole K tiles in every split, row groups that divide
// the row count of transposed operands, and byte offsets within 32 bits.
bool fast_ok_k(const GemmArgs &g, int64_t kchunk, int ktb) {
    const int64_t sz = g.dtype == COMERA_BF16 ? 2 : (g.dtype == kDtypeFp8 ? 1 : 4);
    const int64_t kt = ktb / sz;
    return g.K % kt == 0 && kchunk % kt == 0;
}

bool fast_ok(const GemmArgs &g, int64_t kchunk, int ktb) {
    const int64_t sz = g.dtype == COMERA_BF16 ? 2 : (g.dtype == kDtypeFp8 ? 1 : 4);
    const int64_t kt = ktb / sz;
    if (g.K % kt || kchunk % kt) return false;
    auto op_ok = [&](const void *ptr, int64_t ld, bool kc, int64_t R) {
        if (reinterpret_cast<uintptr_t>(ptr) % 16 || (ld * sz) % 16) return false;
        if (kc) return R * ld * sz < (int64_t(1) << 32);
        return R % (16 / sz) == 0 && (kt * ld + R) * sz < (int64_t(1) << 32);
    };
    return op_ok(g.A, g.lda, g.a_kc, g.M) && op_ok(g.B, g.ldb, g.b_kc, g.N);
}
}  // namespace

int gemm_auto_splits(int64_t M, int64_t N, int64_t K) {
    const int64_t tiles = ceil_div(M, 64) * ceil_div(N, 64);
    // a side of 64 or less with a long K streams the other operand through a
    // few hundred 128-row tiles: split K until about 1024 workgroups load at once
    if (std::min(M, N) <= 64 && K >= 2048) {
        const int64_t t = ceil_div(std::max(M, N), 128);
        if (t < 1024) return int(std::max<int64_t>(1, std::min<int64_t>(ceil_div(1024, t), std::min<int64_t>(K / 512, 8))));
        return 1;
    }
    if (tiles >= 256 || K < 128) return 1;
    int64_t s = ceil_div(1024, tiles);
    s = std::min<int64_t>(s, K / 64);
    s = std::min<int64_t>(s, 32);
    return int(std::max<int64_t>(s, 1));
}

Remap remap_linear(int64_t stride) {
    Remap r{};
    r.nd = 1;
    r.stride[0] = stride;
    return r;
}

int launch_gemm(const GemmArgs &g, void *stream) {
    if (g.M <= 0 || g.N <= 0) return 0;
    if (g.splits <= 1 && g.scratch && g.out_elems > 0 && g.dtype != kDtypeFp8) {
        int s = gemm_auto_splits(g.M, g.N, g.K);
        while (s > 1 && int64_t(s) * g.out_elems > g.scratch_elems) --s;
        if (s > 1) {
            GemmArgs h = g;
            h.scratch = nullptr;
            h.C = g.scratch;
            h.out_bf16 = false;
            h.kchunk = (ceil_div(g.K, s) + 31) / 32 * 32;
            h.splits = int(ceil_div(g.K, h.kchunk));
            h.split_stride = g.out_elems;
            if (int e = launch_gemm(h, stream)) return e;
            return g.out_bf16 ? launch_sum_splits_bf16(g.scratch, g.C, g.out_elems, h.splits, stream)
                              : launch_sum_splits(g.scratch, reinterpret_cast<float *>(g.C), g.out_elems, h.splits,
                                                  stream);
        }
    }
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
    const int esz = g.dtype == COMERA_BF16 ? 2 : (g.dtype == kDtypeFp8 ? 1 : 4);
    const int E = 16 / esz;
    auto aligned = [&](const void *ptr, int64_t ld) {
        return (reinterpret_cast<uintptr_t>(ptr) % 16 == 0) && (ld % E == 0);
    };
    p.vec_a = aligned(g.A, g.lda);
    p.vec_b = aligned(g.B, g.ldb);
    {
        // pieces of V consecutive output columns must be contiguous and
        // aligned; digits of radix 1 (always 0) do not matter
        const int64_t V = g.out_bf16 ? 8 : 4;   // elements per 16-byte piece
        auto live = [](const Remap &r, int k) { return k == 0 || r.radix[k] > 1; };
        bool ok = g.rmap.nd >= 1 && g.cmap.nd >= 1 && g.N % V == 0 && g.split_stride % V == 0 &&
                  reinterpret_cast<uintptr_t>(g.C) % 16 == 0;
        for (int k = 0; k < g.rmap.nd; ++k) ok = ok && (!live(g.rmap, k) || g.rmap.stride[k] % V == 0);
        int in = g.cmap.nd - 1;                  // innermost live column digit
        while (in > 0 && !live(g.cmap, in)) --in;
        for (int k = 0; k < in; ++k) ok = ok && (!live(g.cmap, k) || g.cmap.stride[k] % V == 0);
        ok = ok && in >= 0 && g.cmap.stride[in] == 1 && (in == 0 || g.cmap.radix[in] % V == 0);
        p.stage_c = ok ? 1 : 0;
    }
    p.gw = 0;
    p.oscale = g.oscale;
    GemmArgs gg = g;
    if (gg.splits < 1) gg.splits = 1;
    // fast path: K chunk rounded up to whole K tiles (later splits may get
    // fewer tiles or none; an empty split writes zeros)
    int fast = g.fast >= 0 ? g.fast : (g.fast == -1 && g.tile < 0 ? pick_fast(gg, gg.splits) : -1);
    GemmParams pf = p;
    // the fp32 straight-to-LDS tile writes fp32 results of M/N-contiguous
    // operands only (otherwise: the register-staged tile)
    if (fast == F128x128_dma32 && (g.out_bf16 || g.a_kc || g.b_kc)) fast = F128x128_64;
    if (fast == F128x128_dma32 && (g.dtype != COMERA_F32 || g.oscale)) fast = -1;
    if (fast >= 0) {
        const int ktb = (fast == F128x128_64 || fast == F256x128_64 || fast == F256x256_64w8) ? 64 : 128;
        if (fast >= F256x256_128w8 && fast != F128x128_dma32 && g.dtype == COMERA_F32) fast = -1;

        const int64_t kt = ktb / esz;
        pf.kchunk = ceil_div(p.kchunk, kt) * kt;
        if (!fast_ok(gg, pf.kchunk, ktb)) {
            // a K that is a multiple of the 64-byte K row but not of the
            // 128-byte one keeps a fast 128 x 128 tile on 64-byte rows
            const bool was32 = fast == F128x128_dma32;
            fast = -1;
            // fp32: the register-staged 128 x 128 tile on 64-byte rows
            if (was32 && fast_ok_k(gg, p.kchunk, 64)) {
                fast = F128x128_64;
                pf.kchunk = ceil_div(p.kchunk, 16) * 16;
                if (!fast_ok(gg, pf.kchunk, 64)) fast = -1;
            }
            if (ktb == 128 && g.dtype != COMERA_F32 && (fast_ok_k(gg, p.kchunk, 64))) {
                fast = F128x128_64;
                pf.kchunk = ceil_div(p.kchunk, 64 / esz) * (64 / esz);
                if (!fast_ok(gg, pf.kchunk, 64)) fast = -1;
            }
        }
    }
    const int tile = g.tile >= 0 ? g.tile : pick_tile(g.M, g.N, gg.splits);
#define COMERA_GEMM_CASE(T, AK, BK, OB)                                                    \
    if (g.a_kc == AK && g.b_kc == BK && g.out_bf16 == OB) {                                \
        if (fast >= 0) return launch_fast<T, AK, BK, OB>(gg, pf, fast, stream);           \
        return launch_t<T, AK, BK, OB>(gg, p, tile, stream);                               \
    }
    if (fast == F256x256_pers) {
        if (!pers_ok(gg)) return int(hipErrorInvalidValue);
        return g.dtype == kDtypeFp8 ? launch_dma_pers<true>(gg, pf, stream) : launch_dma_pers<false>(gg, pf, stream);
    }
    if (fast == F128x128_dma32) return launch_dma32(gg, pf, stream);
    if (fast == F256x192_dma) {
        if (g.dtype != COMERA_BF16 || !g.a_kc || !g.b_kc) return int(hipErrorInvalidValue);
        return g.out_bf16 ? launch_dma<true, false, 192>(gg, pf, stream) : launch_dma<false, false, 192>(gg, pf, stream);
    }
    if (fast == F256x256_dma && g.dtype == kDtypeFp8) {
        if (!g.a_kc || !g.b_kc) return int(hipErrorInvalidValue);
        return g.out_bf16 ? launch_dma<true, false, 256, true>(gg, pf, stream)
                          : launch_dma<false, false, 256, true>(gg, pf, stream);
    }
    if (fast == F256x256_dma) {
        if (g.dtype != COMERA_BF16 || g.a_kc != g.b_kc) return int(hipErrorInvalidValue);
        if (g.a_kc) return g.out_bf16 ? launch_dma<true, false>(gg, pf, stream) : launch_dma<false, false>(gg, pf, stream);
        return g.out_bf16 ? launch_dma<true, true>(gg, pf, stream) : launch_dma<false, true>(gg, pf, stream);
    }
    if (g.dtype == kDtypeFp8) {
        // FP8 operands: K-contiguous fast tiles only (the caller pads K);
        // products too small for the measured choice take the smallest tile
        if (!g.a_kc || !g.b_kc) return int(hipErrorInvalidValue);
        if (fast < 0 && g.fast == -1) {
            fast = g.M <= 64 ? F64x128_128 : (g.N <= 64 ? F128x64_128 : F128x128_128);
            pf.kchunk = ceil_div(p.kchunk, 128) * 128;
            if (!fast_ok(gg, pf.kchunk, 128)) fast = -1;
        }
        if (fast < 0) return int(hipErrorInvalidValue);
        if (g.out_bf16) return launch_fast<uint8_t, true, true, true>(gg, pf, fast, stream);
        return launch_fast<uint8_t, true, true, false>(gg, pf, fast, stream);
    }
    if (g.dtype == COMERA_BF16) {
        COMERA_GEMM_CASE(uint16_t, true, false, true)
        COMERA_GEMM_CASE(uint16_t, true, true, true)
        COMERA_GEMM_CASE(uint16_t, true, false, false)
        COMERA_GEMM_CASE(uint16_t, true, true, false)
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
               int ny, int C, void *stream, int layout) {
    const bool transpose = layout == kChainT;
    if (transpose && C != 1) return int(hipErrorInvalidValue);
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
    g.cmap.nd = 3;
    g.cmap.radix[1] = ny;
    g.cmap.radix[2] = C;
    if (layout == kChainRankMajor) {
        const int64_t ncol = NJ * ny;   // length of one (J y) run
        g.rmap.stride[0] = int64_t(nx) * C * ncol;
        g.rmap.stride[1] = ny;
        g.cmap.stride[0] = C * ncol;
        g.cmap.stride[1] = 1;
        g.cmap.stride[2] = ncol;
    } else if (!transpose) {
        g.rmap.stride[0] = int64_t(nx) * NJ * ny * C;
        g.rmap.stride[1] = int64_t(ny) * C;
        g.cmap.stride[0] = NJ * ny * C;
        g.cmap.stride[1] = C;
        g.cmap.stride[2] = 1;
    } else {
        const int64_t rows_in = NI * nx;  // length of one (J y) row of the output
        g.rmap.stride[0] = nx;
        g.rmap.stride[1] = int64_t(ny) * rows_in;
        g.cmap.stride[0] = 1;
        g.cmap.stride[1] = rows_in;
        g.cmap.stride[2] = 0;
    }
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
