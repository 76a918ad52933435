// Fused projection of the core gradients (eq. back Gi, dense order).
//
// dG_k = <dW, dW/dG_k> is computed right to left: E_d = dW (blocked as
// [(I_<, J_<)][(x, y)]), and for k = d-1 .. 1 one step reads E_{k+1} once
// and produces both
//   the right environment E_k[(I, J)][a] = sum_c E_{k+1}[(I, J)][c] G~_k[a][c]
//   the core gradient     dG~_k[a][c]    = sum_(I, J) P_k[(I, J)][a] E_{k+1}[(I, J)][c]
// with c = (x, y, c') over the modes of core k.  A workgroup owns a tile of
// RT rows x CT columns of E_{k+1} in LDS (the incoming split slices summed in
// slice order while loading), the matching slices of G~_k and P_k, and
// writes one adjoint partial per column chunk and one meet partial per row
// chunk.  The partials are summed in a fixed order by the next step (adjoint)
// and by the expand kernel (meet), so results are bitwise reproducible.
//
// The contractions are small (rank <= 64) and read operands that the step
// fetched once into LDS; they run on MFMA in 16 x 16 output tiles (a rank of
// 45 pads to 48, not 64), one tile per wave at a time, with the operands
// zero-padded in LDS so that no read is guarded.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "internal.h"

namespace comera {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kProjMaxA = 64;
constexpr size_t kProjLds = 80 * 1024;    // dynamic LDS of a projection workgroup
constexpr size_t kWtileLds = 64 * 1024;   // of a W-tile workgroup
constexpr int kProjThreadsMax = 1024;  // threads per projection workgroup (large tiles)

// Offset of flat index idx under a mixed-radix remap, with the index and the
// radices below 2^32 (launch_proj checks): 32-bit divisions instead of the
// emulated 64-bit ones
__device__ __forceinline__ int64_t remap_off32(const Remap &r, uint32_t idx) {
    int64_t off = 0;
    for (int t = r.nd - 1; t >= 1; --t) {
        const uint32_t rad = uint32_t(r.radix[t]);
        const uint32_t q = idx / rad;
        off += int64_t(idx - q * rad) * r.stride[t];
        idx = q;
    }
    return off + int64_t(idx) * r.stride[0];
}

// Position (r, c) of element tid + k T of a row-major index space of width
// w, stepped by T without a division per step: (dr, dc) = (T / w, T % w).
struct Walk {
    int r, c;
    __device__ __forceinline__ Walk(int tid, int w) : r(tid / w), c(tid - (tid / w) * w) {}
    __device__ __forceinline__ void step(int w, int dr, int dc) {
        c += dc;
        r += dr;
        if (c >= w) {
            c -= w;
            ++r;
        }
    }
};

__host__ __device__ inline int round4(int x) { return (x + 3) & ~3; }

__host__ __device__ inline int round16(int x) { return (x + 15) & ~15; }

// LDS floats of a projection workgroup: the E tile [R16][C16 + 4], the core
// slice [A16][C16 + 4], the left-chain slice transposed [A16][R16 + 4] (R16,
// C16, A16: RT, CT, A rounded up to 16; zero past the data, so that the
// products read whole 16-deep blocks) and the adjoint row-offset table (RT
// int64, kept 16-byte aligned).  Row pitches of 4 mod 16 floats keep the
// 16-byte reads of 16 consecutive rows on distinct banks.
__host__ __device__ inline size_t proj_lds_floats(int RT, int CT, int A) {
    const int R16 = round16(RT), C16 = round16(CT), A16 = round16(A);
    return size_t(R16) * (C16 + 4) + size_t(A16) * (C16 + 4) + size_t(A16) * (R16 + 4) + size_t(round4(2 * RT));
}

// One 16 x 16 output tile over nb 16-deep blocks of K.  A operand rows
// start at pa (k contiguous: one 16-byte read per block); the B operand
// starts at pb, k contiguous as well (ROWB) or k along rows of pitch pe
// (four single reads per block).  Whole groups of NG blocks read all their
// operands before the first of their products (the order is pinned: the
// compiler would otherwise move each read down to its product and wait for
// it there); the remaining blocks go one at a time.
template <bool ROWB, int NG>
__device__ __forceinline__ f32x4 proj_tile(const float *pa, const float *pb, int nb, int pe) {
    constexpr int RB = ROWB ? 1 : 4;   // LDS reads of one B block
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    auto read = [&](int g, f32x4 &x, f32x4 &y) {
        x = *reinterpret_cast<const f32x4 *>(pa + 16 * g);
        if constexpr (ROWB) {
            y = *reinterpret_cast<const f32x4 *>(pb + 16 * g);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) y[j] = pb[(16 * g + j) * pe];
        }
    };
    int g0 = 0;
    for (; g0 + NG <= nb; g0 += NG) {
        f32x4 x[NG], y[NG];
#pragma unroll
        for (int b = 0; b < NG; ++b) read(g0 + b, x[b], y[b]);
#pragma unroll
        for (int b = 0; b < NG; ++b)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(x[b][j], y[b][j], acc, 0, 0, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, NG * (1 + RB), 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 4 * NG, 0);
    }
    for (; g0 < nb; ++g0) {
        f32x4 x, y;
        read(g0, x, y);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(x[j], y[j], acc, 0, 0, 0);
    }
    return acc;
}

// Two 1024-thread workgroups per CU: eight waves per SIMD, <= 64 registers.
template <int kProjThreads>
__global__ __launch_bounds__(kProjThreads, kProjThreads == 1024 ? 8 : 1) void proj_kernel(ProjArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int RT = a.RT, CT = a.CT, A = a.A;
    const int R16 = round16(RT), C16 = round16(CT), A16 = round16(A);
    const int pe = C16 + 4, pt = R16 + 4;
    float *En_s = sm;                    // [R16][pe]
    float *Gc_s = En_s + R16 * pe;       // [A16][pe]
    float *Pt_s = Gc_s + A16 * pe;       // [A16][pt]: P_k transposed
    int64_t *roff_s = reinterpret_cast<int64_t *>(Pt_s + A16 * pt);   // [RT] remapped adjoint rows
    const int tid = threadIdx.x;
    constexpr int T = kProjThreads;
    const int64_t r0 = int64_t(blockIdx.y) * RT, c0 = int64_t(blockIdx.x) * CT;
    const int nr = int(min<int64_t>(RT, a.rows - r0)), nc = int(min<int64_t>(CT, a.cols - c0));
    if (a.Gc)
        for (int r = tid; r < nr; r += T) roff_s[r] = remap_off32(a.rmap, uint32_t(r0 + r));

    // Every load below comes from an in-bounds address (the tile corner for
    // positions past the data) and is then replaced by 0 where it lies
    // outside, so that the loads are issued unconditionally; positions are
    // stepped with Walk rather than divided out per element.
    //
    // E_{k+1} tile, split slices summed in slice order; zero padding.  Each
    // thread keeps four float4 loads in flight before adding them (one
    // vector of four slices with 1024 threads, two with 256), so that two
    // 1024-thread workgroups fit on a CU.
    const bool vec = (a.cols % 4 == 0) && (CT % 4 == 0) && (a.in_stride % 4 == 0) &&
                     (reinterpret_cast<uintptr_t>(a.En) % 16 == 0);
    const float *etile = a.En + r0 * a.cols + c0;
    if (vec) {
        constexpr int JV = T == 1024 ? 1 : 2, SS = 4;
        const int q4 = C16 / 4, n4 = R16 * q4;
        const int dr = T / q4, dc = T - dr * q4;
        Walk w(tid, q4);
        for (int jb = 0; jb * T < n4; jb += JV) {
            float4 v[JV];
            int ri[JV], ci[JV];
            bool ok[JV];
            const float *src[JV];
#pragma unroll
            for (int j = 0; j < JV; ++j) {
                ri[j] = w.r;
                ci[j] = 4 * w.c;
                ok[j] = ri[j] < nr && ci[j] < nc;
                src[j] = etile + (ok[j] ? int64_t(ri[j]) * a.cols + ci[j] : 0);
                v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
                w.step(q4, dr, dc);
            }
            for (int s0 = 0; s0 < a.nin; s0 += SS) {
                float4 x[SS][JV];
#pragma unroll
                for (int ss = 0; ss < SS; ++ss) {
                    const int64_t so = int64_t(min(s0 + ss, a.nin - 1)) * a.in_stride;
#pragma unroll
                    for (int j = 0; j < JV; ++j) x[ss][j] = *reinterpret_cast<const float4 *>(src[j] + so);
                }
#pragma unroll
                for (int ss = 0; ss < SS; ++ss) {
                    if (s0 + ss >= a.nin) break;
#pragma unroll
                    for (int j = 0; j < JV; ++j) {
                        v[j].x += x[ss][j].x;
                        v[j].y += x[ss][j].y;
                        v[j].z += x[ss][j].z;
                        v[j].w += x[ss][j].w;
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < JV; ++j) {
                if (ri[j] >= R16) break;
                *reinterpret_cast<float4 *>(En_s + ri[j] * pe + ci[j]) =
                    ok[j] ? v[j] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    } else {
        Walk w(tid, C16);
        const int dr = T / C16, dc = T - dr * C16;
        for (; w.r < R16; w.step(C16, dr, dc)) {
            const bool ok = w.r < nr && w.c < nc;
            const float *src = etile + (ok ? int64_t(w.r) * a.cols + w.c : 0);
            float v = 0.f;
            for (int s = 0; s < a.nin; ++s) v += src[s * a.in_stride];
            En_s[w.r * pe + w.c] = ok ? v : 0.f;
        }
    }
    // core and left-chain slices: every thread issues its loads before its
    // stores; the core slice as float4 where the E tile is (nc is then a
    // multiple of 4)
    if (a.Gc && vec && (reinterpret_cast<uintptr_t>(a.Gc) % 16 == 0)) {
        const int q4 = C16 / 4;
        const int dr = T / q4, dc = T - dr * q4;
        Walk w(tid, q4);
        const float *gtile = a.Gc + c0;
        while (w.r < A16) {
            float4 v[4];
            int ro[4], co[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                ro[u] = w.r;
                co[u] = 4 * w.c;
                const bool ok = ro[u] < A && co[u] < nc;
                v[u] = *reinterpret_cast<const float4 *>(gtile + (ok ? int64_t(ro[u]) * a.cols + co[u] : 0));
                if (!ok) v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                w.step(q4, dr, dc);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (ro[u] < A16) *reinterpret_cast<float4 *>(Gc_s + ro[u] * pe + co[u]) = v[u];
        }
    } else if (a.Gc) {
        const int dr = T / C16, dc = T - dr * C16;
        Walk w(tid, C16);
        const float *gtile = a.Gc + c0;
        while (w.r < A16) {
            float v[4];
            int ro[4], co[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                ro[u] = w.r;
                co[u] = w.c;
                const bool ok = ro[u] < A && co[u] < nc;
                v[u] = gtile[ok ? int64_t(ro[u]) * a.cols + co[u] : 0];
                if (!ok) v[u] = 0.f;
                w.step(C16, dr, dc);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (ro[u] < A16) Gc_s[ro[u] * pe + co[u]] = v[u];
        }
    }
    if (a.P) {
        // P_k [r][a] read along a, stored transposed
        const int dr = T / A16, dc = T - dr * A16;
        Walk w(tid, A16);
        const float *ptile = a.P + r0 * A;
        while (w.r < R16) {
            float v[4];
            int ro[4], co[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                ro[u] = w.r;
                co[u] = w.c;
                const bool ok = ro[u] < nr && co[u] < A;
                v[u] = ptile[ok ? ro[u] * A + co[u] : 0];
                if (!ok) v[u] = 0.f;
                w.step(A16, dr, dc);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (ro[u] < R16) Pt_s[co[u] * pt + ro[u]] = v[u];
        }
    }
    __syncthreads();

    // Both products on MFMA (v_mfma_f32_16x16x4f32) in 16 x 16 output tiles:
    //   adjoint tiles (rows x a), K = the C16 columns,
    //   meet tiles    (a x columns), K = the R16 rows.
    // Lane l = 16 q + i supplies A[i][s] and B[s][i] of k slot s = q and
    // receives rows 4 q + v (v = 0..3), column i.  In the 16-deep block g of
    // K, product j of the block gives slot q the k index 16 g + 4 q + j, so a
    // lane's four values along a contiguous k run are one 16-byte read.
    // Adjoint: A = E_{k+1} rows, B = G~ rows (k = column, contiguous).  Meet:
    // A = P_k^T rows (k = row, contiguous), B = E_{k+1} columns (k = row).
    // Tiles are dealt round-robin to the waves.
    // blocks per operand group: 1024-thread workgroups have 64 registers
    constexpr int NG = T == 1024 ? 2 : 4;
    // the wave index as a scalar: tile choice and loop bounds stay uniform
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, lq = lane >> 4;
    const int ta_m = R16 / 16, ta_n = A16 / 16;
    const int nadj = a.Gc ? ta_m * ta_n : 0;
    const int tm_n = C16 / 16;
    const int nmeet = a.P ? ta_n * tm_n : 0;
    for (int t = wave; t < nadj + nmeet; t += kProjThreads / 64) {
        if (t < nadj) {
            const int mt = t / ta_n, nt = t - mt * ta_n;
            const f32x4 acc = proj_tile<true, NG>(En_s + (mt * 16 + li) * pe + 4 * lq,
                                              Gc_s + (nt * 16 + li) * pe + 4 * lq, C16 / 16, pe);
            float *dst = a.Eout + int64_t(blockIdx.x) * a.out_stride;
            const int al = nt * 16 + li;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int r = mt * 16 + 4 * lq + v;
                if (r < nr && al < A) dst[roff_s[r] + al] = acc[v];
            }
        } else {
            const int u0 = t - nadj;
            const int mt = u0 / tm_n, nt = u0 - mt * tm_n;
            const f32x4 acc = proj_tile<false, NG>(Pt_s + (mt * 16 + li) * pt + 4 * lq,
                                               En_s + (4 * lq) * pe + nt * 16 + li, R16 / 16, pe);
            float *dst = a.part + int64_t(blockIdx.y) * A * a.cols;
            const int c = nt * 16 + li;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int al = mt * 16 + 4 * lq + v;
                if (al < A && c < nc) dst[int64_t(al) * a.cols + c0 + c] = acc[v];
            }
        }
    }
}

// ---------------------------------------------------------------- chain step
// One inner step of the batch-free chain (eq. TTM, read left to right): with
// the left chain P = P_k [I][J][a] and the folded core G [a][x][y][c],
//   P_{k+1}[(I x)][(J y)][c] = sum_a P[I][J][a] G[a][x][y][c],
// a product with rows (I, J), columns (x, y, c) and the rank as its short
// contraction.  A workgroup owns 64 rows x 64 columns: the P rows and the
// G columns (transposed) are staged in LDS zero-padded to 16-deep blocks of
// the rank, and each wave forms one 16-row block across the four 16-column
// blocks on v_mfma_f32_16x16x4f32, one 16-byte read per operand and block
// (the k order of the projection kernel).  The interleaved output offsets
// of the tile's rows and columns are taken apart once, into LDS.
constexpr int kLcRows = 64, kLcCols = 64;

__global__ __launch_bounds__(256) void lchain_kernel(LChainArgs a) {
    __shared__ __attribute__((aligned(16))) float Ps[kLcRows * (kProjMaxA + 4)];
    __shared__ __attribute__((aligned(16))) float Gt[kLcCols * (kProjMaxA + 4)];
    __shared__ int64_t roff[kLcRows], coff[kLcCols];
    const int A = a.A, A16 = round16(A), pa = A16 + 4;
    const int64_t rows = a.NI * a.NJ, cols = int64_t(a.nx) * a.ny * a.C;
    const int64_t r0 = int64_t(blockIdx.y) * kLcRows, c0 = int64_t(blockIdx.x) * kLcCols;
    const int nr = int(min<int64_t>(kLcRows, rows - r0)), nc = int(min<int64_t>(kLcCols, cols - c0));
    const int tid = threadIdx.x;
    const int64_t orow = int64_t(a.nx) * a.NJ * a.ny * a.C;   // stride of I in the output
    const int64_t ox = a.NJ * a.ny * a.C;                     // stride of x
    if (tid < kLcRows) {
        // rows below 2^32 (launch_lchain checks)
        const uint32_t r = uint32_t(r0 + tid), nj = uint32_t(a.NJ);
        const uint32_t I = r / nj, J = r - I * nj;
        roff[tid] = int64_t(I) * orow + int64_t(J) * a.ny * a.C;
    } else if (tid < kLcRows + kLcCols) {
        const int t = tid - kLcRows;
        const uint32_t col = uint32_t(c0 + t), C = uint32_t(a.C), ny = uint32_t(a.ny);
        const uint32_t q = col / C, c = col - q * C;
        const uint32_t x = q / ny, y = q - x * ny;
        coff[t] = int64_t(x) * ox + int64_t(y) * a.C + c;
    }
    // P rows (contiguous: 64 A floats from row r0) and G columns, loads
    // from in-bounds addresses then zero outside
    {
        const float *pt = a.P + r0 * A;
        const int dr = 256 / A16, dc = 256 - dr * A16;
        Walk w(tid, A16);
        while (w.r < kLcRows) {
            float v[4];
            int ro[4], co[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                ro[u] = w.r;
                co[u] = w.c;
                const bool ok = ro[u] < nr && co[u] < A;
                v[u] = pt[ok ? ro[u] * A + co[u] : 0];
                if (!ok) v[u] = 0.f;
                w.step(A16, dr, dc);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (ro[u] < kLcRows) Ps[ro[u] * pa + co[u]] = v[u];
        }
    }
    {
        const float *gt = a.G + c0;
        constexpr int dr = 256 / kLcCols, dc = 0;
        Walk w(tid, kLcCols);
        while (w.r < A16) {
            float v[4];
            int ro[4], co[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                ro[u] = w.r;
                co[u] = w.c;
                const bool ok = ro[u] < A && co[u] < nc;
                v[u] = gt[ok ? int64_t(ro[u]) * cols + co[u] : 0];
                if (!ok) v[u] = 0.f;
                w.step(kLcCols, dr, dc);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (ro[u] < A16) Gt[co[u] * pa + ro[u]] = v[u];
        }
    }
    __syncthreads();
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, lq = lane >> 4;
    f32x4 acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    const float *pa_ = Ps + (wave * 16 + li) * pa + 4 * lq;
    const float *pb_ = Gt + li * pa + 4 * lq;
    for (int g = 0; g < A16 / 16; ++g) {
        const f32x4 x = *reinterpret_cast<const f32x4 *>(pa_ + 16 * g);
        f32x4 y[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) y[t] = *reinterpret_cast<const f32x4 *>(pb_ + t * 16 * pa + 16 * g);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(x[j], y[t][j], acc[t], 0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int col = t * 16 + li;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = wave * 16 + 4 * lq + v;
            if (row < nr && col < nc) a.out[roff[row] + coff[col]] = acc[t][v];
        }
    }
}

// ---------------------------------------------------------------- W build
// Last step of the batch-free chain (eq. TTM): with the left chain
// P = P_{d-1} [I][J][a] and the folded last core G [a][x][y] (x = i_{d-1},
// y = j_{d-1}),
//   W[(I x)][(J y)] = sum_a P[I][J][a] G[a][x][y]
// written as W [N_in][N_out], as W^T [N_out][N_in], or both, fp32 or bf16.
// A workgroup owns QI values of I and QJ values of J, i.e. a tile of
// (QI nx) x (QJ ny) entries of W: it stages its P slice (rank-major) and G in
// LDS, computes the tile as a [QI QJ] x [nx ny] product with 4 x 4 register
// blocks, keeps it in LDS and writes it out in each requested layout,
// consecutive threads on consecutive addresses.  Loads and stores move four
// entries per thread where the addresses allow it (16-byte pieces), else one.
// The kernel is latency-bound (a few KB per workgroup, one pass): on the
// 768 x 3072 layer (rank 30, 12 x 12 last core) the four-entry paths and
// tiles of 36 x 96 entries take it from 18.5 to 10 us.
__device__ __forceinline__ uint16_t to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return uint16_t((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

// LDS floats of a W tile workgroup: P^T [A][NP4], G [A][NC4], tile [TI][TJ + 1]
__host__ __device__ inline size_t wtile_lds_floats(int A, int QI, int QJ, int nx, int ny) {
    const int NP4 = round4(QI * QJ), NC4 = round4(nx * ny);
    return size_t(A) * NP4 + size_t(A) * NC4 + size_t(QI * nx) * (QJ * ny + 1);
}

__device__ __forceinline__ void put_w(void *out, bool bf, int64_t off, float v) {
    if (bf)
        reinterpret_cast<uint16_t *>(out)[off] = to_bf16_rne(v);
    else
        reinterpret_cast<float *>(out)[off] = v;
}

__global__ __launch_bounds__(256) void wtile_kernel(WBuildArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sw[];
    const int A = a.A, nx = a.nx, ny = a.ny, QI = a.QI, QJ = a.QJ;
    const int NP = QI * QJ, NC = nx * ny;
    const int NP4 = round4(NP), NC4 = round4(NC);
    const int TI = QI * nx, TJ = QJ * ny, tp = TJ + 1;
    float *Pt = sw;                 // [A][NP4], pair p = qi * QJ + qj
    float *Gs = Pt + A * NP4;       // [A][NC4], column c = x * ny + y
    float *tile = Gs + A * NC4;     // [TI][tp]
    const int64_t I0 = int64_t(blockIdx.y) * QI, J0 = int64_t(blockIdx.x) * QJ;
    const int nI = int(min<int64_t>(QI, a.NI - I0)), nJ = int(min<int64_t>(QJ, a.NJ - J0));
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // Every integer division below is per thread or per item, never per
    // element: a wave64 instruction occupies its SIMD for four cycles, and a
    // division is a few dozen of them.
    const bool vP = ((a.NJ * A) % 4 == 0) && ((J0 * A) % 4 == 0) && ((int64_t(nJ) * A) % 4 == 0) &&
                    ((reinterpret_cast<uintptr_t>(a.P) & 15) == 0);
    const bool vG = (NC % 4 == 0) && ((reinterpret_cast<uintptr_t>(a.G) & 15) == 0);
    if (vP && vG) {
        // P slice: nI runs of nJ A consecutive floats; G: A NC consecutive
        // floats (NC4 == NC); both as float4, all loads before any store.
        // Pairs outside the slice stay unset: their products are computed
        // but never stored.
        const int rowf = nJ * A / 4, npf = nI * rowf, ngf = A * NC / 4;
        constexpr int U = 8;
        float4 v[U];
        // the address is selected first and every load is issued
        // unconditionally (in bounds: past the end it reads G's first
        // vector), so the loads do not wait for each other under branches
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int f = tid + u * 256;
            const int qi = f < npf ? f / rowf : 0, e = f - qi * rowf;
            const float4 *src = f < npf ? reinterpret_cast<const float4 *>(a.P + ((I0 + qi) * a.NJ + J0) * A) + e
                                        : reinterpret_cast<const float4 *>(a.G) + (f < npf + ngf ? f - npf : 0);
            v[u] = *src;
        }
        auto put_p = [&](int f, float4 w) {
            const int qi = f / rowf, e = 4 * (f - qi * rowf);
            int qj = e / A, al = e - qj * A;
            const float x[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                Pt[al * NP4 + qi * QJ + qj] = x[k];
                if (++al == A) {
                    al = 0;
                    ++qj;
                }
            }
        };
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int f = tid + u * 256;
            if (f < npf) put_p(f, v[u]);
            else if (f < npf + ngf) reinterpret_cast<float4 *>(Gs)[f - npf] = v[u];
        }
        // anything beyond U loads per thread (large ranks or cores)
        for (int f = tid + U * 256; f < npf + ngf; f += 256) {
            if (f < npf) {
                const int qi = f / rowf;
                put_p(f, reinterpret_cast<const float4 *>(a.P + ((I0 + qi) * a.NJ + J0) * A)[f - qi * rowf]);
            } else {
                reinterpret_cast<float4 *>(Gs)[f - npf] = reinterpret_cast<const float4 *>(a.G)[f - npf];
            }
        }
    } else {
        // P slice: thread t loads rank entries al = t % A, t % A + ... of the
        // pairs p = t / A + 256 / A * i (coalesced runs of A floats per pair);
        // G: consecutive floats.  All loads are issued before any store.
        constexpr int U = 24;
        float v[U];
        const int pa0 = tid % A, pp0 = tid / A, pstep = 256 / A;     // A <= 64
        const int np_t = (tid < pstep * A && pp0 < NP4) ? (NP4 - pp0 + pstep - 1) / pstep : 0;
        const int ng_t = (A * NC4 - tid + 255) / 256;
        int qi = pp0 / QJ, qj = pp0 - (pp0 / QJ) * QJ;
        const int dqi = pstep / QJ, dqj = pstep - dqi * QJ;
        // addresses selected first, loads unconditional (an in-bounds
        // element when outside), zero selected afterwards
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float *src = a.G;
            bool ok = false;
            if (u < np_t) {
                const int p = pp0 + u * pstep;
                ok = p < NP && qi < nI && qj < nJ;
                if (ok) src = a.P + ((I0 + qi) * a.NJ + J0 + qj) * A + pa0;
                qi += dqi;
                qj += dqj;
                if (qj >= QJ) {
                    qj -= QJ;
                    ++qi;
                }
            } else if (u - np_t < ng_t) {
                const int g = tid + (u - np_t) * 256;
                const int al = g / NC4, c = g - al * NC4;
                ok = c < NC;
                if (ok) src = a.G + al * NC + c;
            }
            const float x = *src;
            v[u] = ok ? x : 0.f;
        }
        for (int u = 0; u < U; ++u) {
            if (u < np_t) {
                Pt[pa0 * NP4 + pp0 + u * pstep] = v[u];
            } else if (u - np_t < ng_t) {
                const int g = tid + (u - np_t) * 256;
                Gs[g] = v[u];
            }
        }
        // anything beyond U loads per thread (large ranks or cores)
        for (int u = U; u < np_t; ++u) {
            const int p = pp0 + u * pstep;
            const int q1 = p / QJ, q2 = p - (p / QJ) * QJ;
            Pt[pa0 * NP4 + p] = (p < NP && q1 < nI && q2 < nJ) ? a.P[((I0 + q1) * a.NJ + J0 + q2) * A + pa0] : 0.f;
        }
        for (int u = max(0, U - np_t); u < ng_t; ++u) {
            const int g = tid + u * 256;
            const int al = g / NC4, c = g - al * NC4;
            Gs[g] = c < NC ? a.G[al * NC + c] : 0.f;
        }
    }
    __syncthreads();
    const int npb = NP4 / 4, ncb = NC4 / 4;
    for (int w = tid; w < npb * ncb; w += 256) {
        const int pb = w / ncb, cb = w - pb * ncb;
        float acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
        const float *pp = Pt + pb * 4, *gp = Gs + cb * 4;
#pragma unroll 4
        for (int al = 0; al < A; ++al) {
            const float4 pv = *reinterpret_cast<const float4 *>(pp + al * NP4);
            const float4 gv = *reinterpret_cast<const float4 *>(gp + al * NC4);
            const float pa[4] = {pv.x, pv.y, pv.z, pv.w}, ga[4] = {gv.x, gv.y, gv.z, gv.w};
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] += pa[i] * ga[j];
        }
        // tile offsets of the four pairs and the four columns
        int roff[4], coff[4];
        {
            int p = pb * 4, q1 = p / QJ, q2 = p - q1 * QJ;
            int c = cb * 4, x = c / ny, y = c - x * ny;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                roff[i] = (p + i < NP) ? q1 * nx * tp + q2 * ny : -1;
                coff[i] = (c + i < NC) ? x * tp + y : -1;
                if (++q2 == QJ) {
                    q2 = 0;
                    ++q1;
                }
                if (++y == ny) {
                    y = 0;
                    ++x;
                }
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (roff[i] >= 0 && coff[j] >= 0) tile[roff[i] + coff[j]] = acc[i][j];
    }
    __syncthreads();
    const bool bf = a.out_bf16 != 0;
    const int ri = nI * nx, rj = nJ * ny;
    const int64_t Nin = a.NI * nx, Nout = a.NJ * ny;
    const int64_t i0 = I0 * nx, j0 = J0 * ny;
    const uintptr_t al_need = bf ? 7 : 15;
    const bool v4 = (rj % 4 == 0) && (ri % 4 == 0) && (Nout % 4 == 0) && (Nin % 4 == 0) && (j0 % 4 == 0) &&
                    (i0 % 4 == 0) && ((reinterpret_cast<uintptr_t>(a.out) & al_need) == 0) &&
                    ((reinterpret_cast<uintptr_t>(a.out_t) & al_need) == 0);
    if (v4) {
        // four consecutive entries per thread over the tile flattened in
        // the output's row order, so one wave covers several short rows
        auto put4 = [&](void *out, int64_t off, float x0, float x1, float x2, float x3) {
            if (bf) {
                uint2 u;
                u.x = uint32_t(to_bf16_rne(x0)) | (uint32_t(to_bf16_rne(x1)) << 16);
                u.y = uint32_t(to_bf16_rne(x2)) | (uint32_t(to_bf16_rne(x3)) << 16);
                *reinterpret_cast<uint2 *>(reinterpret_cast<uint16_t *>(out) + off) = u;
            } else {
                *reinterpret_cast<float4 *>(reinterpret_cast<float *>(out) + off) = make_float4(x0, x1, x2, x3);
            }
        };
        if (a.out) {
            const int q4 = rj / 4, tot = ri * q4;
            for (int t = tid; t < tot; t += 256) {
                const int r = t / q4, c = 4 * (t - r * q4);
                const float *e = tile + r * tp + c;
                put4(a.out, (i0 + r) * Nout + j0 + c, e[0], e[1], e[2], e[3]);
            }
        }
        if (a.out_t) {
            const int q4 = ri / 4, tot = rj * q4;
            for (int t = tid; t < tot; t += 256) {
                const int c = t / q4, r = 4 * (t - c * q4);
                const float *e = tile + r * tp + c;
                put4(a.out_t, (j0 + c) * Nin + i0 + r, e[0], e[tp], e[2 * tp], e[3 * tp]);
            }
        }
        return;
    }
    // one output row per wave at a time, lanes on consecutive addresses
    if (a.out)       // W [N_in][N_out]: rows i, runs of rj consecutive j
        for (int r = wave; r < ri; r += 4) {
            const int64_t base = (i0 + r) * Nout + j0;
            for (int c = lane; c < rj; c += 64) put_w(a.out, bf, base + c, tile[r * tp + c]);
        }
    if (a.out_t)     // W^T [N_out][N_in]: rows j, runs of ri consecutive i
        for (int c = wave; c < rj; c += 4) {
            const int64_t base = (j0 + c) * Nin + i0;
            for (int r = lane; r < ri; r += 64) put_w(a.out_t, bf, base + r, tile[r * tp + c]);
        }
}

}  // namespace

bool proj_supported(int A) { return A >= 1 && A <= kProjMaxA; }

void proj_tiles(int64_t rows, int64_t cols, int A, int &RT, int &CT) {
    // whole column ranges up to 256; wider steps in chunks of 64 (measured
    // faster than 128 on the 2048 x 1440 rank-45 step)
    CT = int(cols <= 256 ? cols : 64);
    // 128-row tiles where they still give 256 workgroups (fewer meet
    // partials; measured faster on the 65536-row step of the 1024<->4096
    // pair), else 64; halved while the grid holds fewer than 160 workgroups
    // (a tile over many dW slices is a long load: 192 workgroups of 32 rows
    // beat 384 of 16 on the 6144-row, 26-slice step of the 768x768 layer)
    RT = (rows >= 256 * 128 && proj_lds_floats(128, CT, A) * sizeof(float) <= kProjLds) ? 128 : 64;
    while (proj_lds_floats(RT, CT, A) * sizeof(float) > kProjLds && CT > 32) CT = (CT + 1) / 2;
    while (proj_lds_floats(RT, CT, A) * sizeof(float) > kProjLds && RT > 8) RT /= 2;
    const int64_t nct = (cols + CT - 1) / CT;
    while (RT > 8 && ((rows + RT - 1) / RT) * nct < 160) RT /= 2;
}

bool wbuild_tiles(int64_t NI, int64_t NJ, int A, int nx, int ny, int &QI, int &QJ) {
    if (A < 1 || A > kProjMaxA || NI < 1 || NJ < 1) return false;
    // tiles of about 32 x 96 entries of W (more workgroups than square
    // tiles, rows of 96+ entries in W); halved while a workgroup would hold
    // more LDS than allowed
    int qi = int(std::min<int64_t>(NI, std::max(1, (32 + nx - 1) / nx)));
    int qj = int(std::min<int64_t>(NJ, std::max(1, (96 + ny - 1) / ny)));
    while (wtile_lds_floats(A, qi, qj, nx, ny) * sizeof(float) > kWtileLds && (qi > 1 || qj > 1)) {
        if (qj >= qi && qj > 1) qj = (qj + 1) / 2;
        else qi = (qi + 1) / 2;
    }
    if (wtile_lds_floats(A, qi, qj, nx, ny) * sizeof(float) > kWtileLds) return false;
    QI = qi;
    QJ = qj;
    return true;
}

int launch_wbuild(const WBuildArgs &a, void *stream) {
    if (a.NI <= 0 || a.NJ <= 0 || (!a.out && !a.out_t)) return 0;
    const size_t lds = wtile_lds_floats(a.A, a.QI, a.QJ, a.nx, a.ny) * sizeof(float);
    if (lds > kWtileLds || a.QI < 1 || a.QJ < 1) return int(hipErrorInvalidValue);
    if (!launch_check_mode()) {
        static const int set = int(hipFuncSetAttribute(reinterpret_cast<const void *>(wtile_kernel),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(kWtileLds)));
        if (set) return set;
    }
    const int64_t gx = (a.NJ + a.QJ - 1) / a.QJ, gy = (a.NI + a.QI - 1) / a.QI;
    if (gx >= (int64_t(1) << 31) || gy > 65535) return int(hipErrorInvalidValue);
    COMERA_LAUNCH(wtile_kernel, dim3(unsigned(gx), unsigned(gy)), dim3(256), lds, hipStream_t(stream), a);
    return launch_status();
}

int launch_proj(const ProjArgs &a, void *stream) {
    if (a.rows <= 0 || a.cols <= 0) return 0;
    if (!proj_supported(a.A) || a.RT % 4 || a.CT < 1 || a.nin < 1) return int(hipErrorInvalidValue);
    // row offsets are taken apart in 32 bits
    if (a.Gc) {
        if (a.rows >= (int64_t(1) << 32)) return int(hipErrorInvalidValue);
        for (int t = 1; t < a.rmap.nd; ++t)
            if (a.rmap.radix[t] < 1 || a.rmap.radix[t] >= (int64_t(1) << 32)) return int(hipErrorInvalidValue);
    }
    const size_t lds = proj_lds_floats(a.RT, a.CT, a.A) * sizeof(float);
    if (lds > kProjLds) return int(hipErrorInvalidValue);
    dim3 grid(unsigned((a.cols + a.CT - 1) / a.CT), unsigned((a.rows + a.RT - 1) / a.RT));
    // 1024 threads when the tile load is large (many loads in flight per CU),
    // else 256 (several workgroups per CU)
    if (!launch_check_mode()) {
        static const int set = int(hipFuncSetAttribute(reinterpret_cast<const void *>(proj_kernel<kProjThreadsMax>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(kProjLds))) |
                               int(hipFuncSetAttribute(reinterpret_cast<const void *>(proj_kernel<256>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, int(kProjLds)));
        if (set) return set;
    }
    const int64_t loads4 = int64_t(a.RT) * ((a.CT + 3) / 4) * std::max(1, a.nin);
    if (loads4 >= 4096)
        COMERA_LAUNCH((proj_kernel<kProjThreadsMax>), grid, dim3(kProjThreadsMax), lds, hipStream_t(stream), a);
    else
        COMERA_LAUNCH((proj_kernel<256>), grid, dim3(256), lds, hipStream_t(stream), a);
    return launch_status();
}

bool lchain_supported(int A) { return A >= 1 && A <= kProjMaxA; }

int launch_lchain(const LChainArgs &a, void *stream) {
    const int64_t rows = a.NI * a.NJ, cols = int64_t(a.nx) * a.ny * a.C;
    if (rows <= 0 || cols <= 0) return 0;
    if (!lchain_supported(a.A) || rows >= (int64_t(1) << 32) || cols >= (int64_t(1) << 32))
        return int(hipErrorInvalidValue);
    const int64_t gx = (cols + kLcCols - 1) / kLcCols, gy = (rows + kLcRows - 1) / kLcRows;
    if (gx >= (int64_t(1) << 31) || gy > 65535) return int(hipErrorInvalidValue);
    COMERA_LAUNCH(lchain_kernel, dim3(unsigned(gx), unsigned(gy)), dim3(256), 0, hipStream_t(stream), a);
    return launch_status();
}

}  // namespace comera
