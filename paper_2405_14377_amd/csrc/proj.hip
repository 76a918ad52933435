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
// fetched once into LDS; they run on MFMA, one 32 x 32 output tile per wave
// at a time.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "internal.h"

namespace comera {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kProjMaxA = 64;
constexpr size_t kProjLds = 64 * 1024;
constexpr int kProjThreadsMax = 1024;  // threads per projection workgroup (large tiles)

__device__ __forceinline__ int64_t remap_off(const Remap &r, int64_t idx) {
    int64_t off = 0;
    for (int t = r.nd - 1; t >= 1; --t) {
        const int64_t q = idx / r.radix[t];
        off += (idx - q * r.radix[t]) * r.stride[t];
        idx = q;
    }
    return off + idx * r.stride[0];
}

__host__ __device__ inline int round4(int x) { return (x + 3) & ~3; }

// LDS floats of a projection workgroup: E tile, core slice, left-chain
// slice (row pitches padded by 4 floats) and the adjoint row-offset table
// (RT int64, kept 16-byte aligned)
__host__ __device__ inline size_t proj_lds_floats(int RT, int CT, int A) {
    const int CT4 = round4(CT), A4 = round4(A);
    return size_t(RT) * (CT4 + 4) + size_t(A4) * (CT4 + 4) + size_t(RT) * (A4 + 4) + size_t(round4(2 * RT));
}

template <int kProjThreads>
__global__ __launch_bounds__(kProjThreads) void proj_kernel(ProjArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int RT = a.RT, CT = a.CT, A = a.A;
    const int CT4 = round4(CT), A4 = round4(A);
    const int pe = CT4 + 4, pp = A4 + 4;
    float *En_s = sm;                    // [RT][pe]
    float *Gc_s = En_s + RT * pe;        // [A4][pe]
    float *P_s = Gc_s + A4 * pe;         // [RT][pp]
    int64_t *roff_s = reinterpret_cast<int64_t *>(P_s + RT * pp);   // [RT] remapped adjoint rows
    const int tid = threadIdx.x;
    const int64_t r0 = int64_t(blockIdx.y) * RT, c0 = int64_t(blockIdx.x) * CT;
    const int nr = int(min<int64_t>(RT, a.rows - r0)), nc = int(min<int64_t>(CT, a.cols - c0));
    if (a.Gc)
        for (int r = tid; r < nr; r += kProjThreads) roff_s[r] = remap_off(a.rmap, r0 + r);

    // E_{k+1} tile, split slices summed in slice order; zero padding.  Each
    // thread keeps 4 x 4 float4 loads (four vectors of four slices) in
    // flight before adding them.
    const bool vec = (a.cols % 4 == 0) && (CT % 4 == 0) && (a.in_stride % 4 == 0) &&
                     (reinterpret_cast<uintptr_t>(a.En) % 16 == 0);
    if (vec) {
        const int q4 = CT4 / 4, n4 = RT * q4;
        for (int jb = 0; jb * kProjThreads < n4; jb += 4) {
            float4 v[4];
            int ri[4], ci[4];
            bool ok[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int i = tid + kProjThreads * (jb + j);
                ri[j] = i / q4;
                ci[j] = (i - ri[j] * q4) * 4;
                ok[j] = i < n4 && ri[j] < nr && ci[j] < nc;
                v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
            }
            for (int s0 = 0; s0 < a.nin; s0 += 4) {
                float4 x[4][4];
#pragma unroll
                for (int ss = 0; ss < 4; ++ss)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        x[ss][j] = (ok[j] && s0 + ss < a.nin)
                                       ? *reinterpret_cast<const float4 *>(a.En + (s0 + ss) * a.in_stride +
                                                                           (r0 + ri[j]) * a.cols + c0 + ci[j])
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int ss = 0; ss < 4; ++ss)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        v[j].x += x[ss][j].x;
                        v[j].y += x[ss][j].y;
                        v[j].z += x[ss][j].z;
                        v[j].w += x[ss][j].w;
                    }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int i = tid + kProjThreads * (jb + j);
                if (i < n4) *reinterpret_cast<float4 *>(En_s + ri[j] * pe + ci[j]) = v[j];
            }
        }
    } else {
        for (int i = tid; i < RT * CT4; i += kProjThreads) {
            const int r = i / CT4, c = i - r * CT4;
            float v = 0.f;
            if (r < nr && c < nc)
                for (int s = 0; s < a.nin; ++s) v += a.En[s * a.in_stride + (r0 + r) * a.cols + c0 + c];
            En_s[r * pe + c] = v;
        }
    }
    // core and left-chain slices: every thread issues its loads before its stores
    if (a.Gc)
        for (int i0 = tid; i0 < A4 * CT4; i0 += kProjThreads * 4) {
            float v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + u * kProjThreads;
                const int al = i / CT4, c = i - al * CT4;
                v[u] = (i < A4 * CT4 && al < A && c < nc) ? a.Gc[int64_t(al) * a.cols + c0 + c] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + u * kProjThreads;
                const int al = i / CT4, c = i - al * CT4;
                if (i < A4 * CT4) Gc_s[al * pe + c] = v[u];
            }
        }
    if (a.P)
        for (int i0 = tid; i0 < RT * A4; i0 += kProjThreads * 4) {
            float v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + u * kProjThreads;
                const int r = i / A4, al = i - r * A4;
                v[u] = (i < RT * A4 && r < nr && al < A) ? a.P[(r0 + r) * A + al] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + u * kProjThreads;
                const int r = i / A4, al = i - r * A4;
                if (i < RT * A4) P_s[r * pp + al] = v[u];
            }
        }
    __syncthreads();

    // Both products on MFMA (v_mfma_f32_32x32x2f32) in 32 x 32 output tiles:
    //   adjoint tiles (rows x a), K = the CT4 columns,
    //   meet tiles    (a x columns), K = the RT rows.
    // Lane l supplies A[l % 32][k0 + l / 32] and B[k0 + l / 32][l % 32];
    // accumulator v of lane l is row 8 (v / 4) + 4 (l / 32) + v % 4, column
    // l % 32.  Tiles are dealt round-robin to the waves.
    const int lane = tid & 63, wave = tid >> 6;
    const int li = lane & 31, lk = lane >> 5;
    const int ta_m = (RT + 31) / 32, ta_n = (A + 31) / 32;
    const int nadj = a.Gc ? ta_m * ta_n : 0;
    const int tm_n = (CT4 + 31) / 32;
    const int nmeet = a.P ? ta_n * tm_n : 0;
    for (int t = wave; t < nadj + nmeet; t += kProjThreads / 64) {
        f32x16 acc;
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = 0.f;
        if (t < nadj) {
            const int mt = t / ta_n, nt = t - mt * ta_n;
            const int ra = mt * 32 + li, gb = nt * 32 + li;
            const float *pa = En_s + min(ra, RT - 1) * pe + lk;
            const float *pb = Gc_s + min(gb, A4 - 1) * pe + lk;
            const bool va = ra < RT, vb = gb < A4;
            for (int k = 0; k < CT4; k += 8) {
                float x[4], y[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    x[u] = va ? pa[k + 2 * u] : 0.f;
                    y[u] = vb ? pb[k + 2 * u] : 0.f;
                }
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (k + 2 * u < CT4) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x[u], y[u], acc, 0, 0, 0);
            }
            float *dst = a.Eout + int64_t(blockIdx.x) * a.out_stride;
            const int al = nt * 32 + li;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int r = mt * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
                if (r < nr && al < A) dst[roff_s[r] + al] = acc[v];
            }
        } else {
            const int u0 = t - nadj;
            const int mt = u0 / tm_n, nt = u0 - mt * tm_n;
            const int am = mt * 32 + li, cn = nt * 32 + li;
            const bool va = am < A4, vb = cn < CT4;
            const float *pa = P_s + lk * pp + min(am, A4 - 1);
            const float *pb = En_s + lk * pe + min(cn, CT4 - 1);
            for (int r = 0; r < RT; r += 8) {
                float x[4], y[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int rr = min(r + 2 * u, RT - 2);
                    x[u] = va ? pa[rr * pp] : 0.f;
                    y[u] = vb ? pb[rr * pe] : 0.f;
                }
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (r + 2 * u < RT) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x[u], y[u], acc, 0, 0, 0);
            }
            float *dst = a.part + int64_t(blockIdx.y) * A * a.cols;
            const int c = nt * 32 + li;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int al = mt * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
                if (al < A && c < nc) dst[int64_t(al) * a.cols + c0 + c] = acc[v];
            }
        }
    }
}

// ---------------------------------------------------------------- W build
// Last step of the batch-free chain (eq. TTM): with the left chain
// P = P_{d-1} [I][J][a] and the folded last core G [a][x][y] (x = i_{d-1},
// y = j_{d-1}),
//   W[(I x)][(J y)] = sum_a P[I][J][a] G[a][x][y]
// written as W [N_in][N_out] or as W^T [N_out][N_in], fp32 or bf16.  A
// workgroup owns one value of the outer index of the output rows (J for W^T,
// I for W) and a block of QB values of the inner one; consecutive threads
// write consecutive output columns.
__device__ __forceinline__ uint16_t to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return uint16_t((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

// G is staged as [a][q][o] with o (the output-row digit) padded to a multiple
// of 4, so every thread reads float4 runs of G for its (Q, q) column.
template <bool TR>
__global__ __launch_bounds__(256) void wbuild_kernel(WBuildArgs a) {
    extern __shared__ __attribute__((aligned(16))) float sw[];
    const int64_t NQ = TR ? a.NI : a.NJ;
    const int no = TR ? a.ny : a.nx, nq = TR ? a.nx : a.ny;
    const int NO4 = round4(no);
    const int A = a.A, QB = a.QB;
    const int gsz = A * nq * NO4;
    float *G_s = sw;
    float *P_s = sw + gsz;
    const int64_t O = blockIdx.x;
    const int64_t Q0 = int64_t(blockIdx.y) * QB;
    const int nQ = int(min<int64_t>(QB, NQ - Q0));
    stage_lds<8>(G_s, gsz, threadIdx.x, 256, [&](int i) {
        const int o = i % NO4, t = i / NO4;
        const int q = t % nq, al = t / nq;
        const int x = TR ? q : o, y = TR ? o : q;
        return o < no ? a.G[(al * a.nx + x) * a.ny + y] : 0.f;
    });
    stage_lds<8>(P_s, nQ * A, threadIdx.x, 256, [&](int i) {
        const int ql = i / A, al = i - ql * A;
        const int64_t I = TR ? Q0 + ql : O, J = TR ? O : Q0 + ql;
        return a.P[(I * a.NJ + J) * A + al];
    });
    __syncthreads();
    const int64_t rowlen = NQ * nq;
    for (int item = threadIdx.x; item < nQ * nq; item += 256) {
        const int ql = item / nq, q = item - ql * nq;
        const int64_t col = (Q0 + ql) * nq + q;
        const float *pr = P_s + ql * A;
        for (int o0 = 0; o0 < NO4; o0 += 16) {
            const int n4 = min(4, (NO4 - o0) / 4);
            float acc[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) acc[j] = 0.f;
            const float *gq = G_s + q * NO4 + o0;
            for (int al = 0; al < A; ++al) {
                const float p = pr[al];
                const float *g = gq + al * nq * NO4;
#pragma unroll
                for (int j4 = 0; j4 < 4; ++j4) {
                    if (j4 < n4) {
                        const float4 g4 = *reinterpret_cast<const float4 *>(g + 4 * j4);
                        acc[4 * j4 + 0] += p * g4.x;
                        acc[4 * j4 + 1] += p * g4.y;
                        acc[4 * j4 + 2] += p * g4.z;
                        acc[4 * j4 + 3] += p * g4.w;
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                if (o0 + j >= no) break;
                const int64_t off = (O * no + o0 + j) * rowlen + col;
                if (a.out_bf16)
                    reinterpret_cast<uint16_t *>(a.out)[off] = to_bf16_rne(acc[j]);
                else
                    reinterpret_cast<float *>(a.out)[off] = acc[j];
            }
        }
    }
}

}  // namespace

bool proj_supported(int A) { return A >= 1 && A <= kProjMaxA; }

void proj_tiles(int64_t rows, int64_t cols, int A, int &RT, int &CT) {
    CT = int(cols <= 256 ? cols : 128);
    RT = 64;
    while (proj_lds_floats(RT, CT, A) * sizeof(float) > kProjLds && CT > 32) CT = (CT + 1) / 2;
    while (proj_lds_floats(RT, CT, A) * sizeof(float) > kProjLds && RT > 8) RT /= 2;
    const int64_t nct = (cols + CT - 1) / CT;
    while (RT > 8 && ((rows + RT - 1) / RT) * nct < 256) RT /= 2;
}

bool wbuild_tiles(int64_t NI, int64_t NJ, int A, int nx, int ny, bool transpose, int &QB) {
    if (A < 1 || A > kProjMaxA) return false;
    const int64_t NQ = transpose ? NI : NJ;
    const int nq = transpose ? nx : ny;
    const int no = transpose ? ny : nx;
    const size_t g = size_t(A) * nq * round4(no);
    // about 256 output columns per workgroup: several workgroups per CU hide
    // the staging latency better than fewer, larger ones (measured); blocks of
    // equal size
    int64_t qb = std::max<int64_t>(1, std::min<int64_t>(NQ, 256 / std::max(1, nq)));
    const int64_t nblk = (NQ + qb - 1) / qb;
    qb = (NQ + nblk - 1) / nblk;
    while (qb > 1 && (g + size_t(qb) * A) * sizeof(float) > kProjLds) qb /= 2;
    if ((g + size_t(qb) * A) * sizeof(float) > kProjLds) return false;
    QB = int(qb);
    return true;
}

int launch_wbuild(const WBuildArgs &a, void *stream) {
    const int64_t NO = a.transpose ? a.NJ : a.NI, NQ = a.transpose ? a.NI : a.NJ;
    if (NO <= 0 || NQ <= 0) return 0;
    const int no = a.transpose ? a.ny : a.nx, nq = a.transpose ? a.nx : a.ny;
    const size_t lds = (size_t(a.A) * nq * round4(no) + size_t(a.QB) * a.A) * sizeof(float);
    if (lds > kProjLds || a.QB < 1) return int(hipErrorInvalidValue);
    dim3 grid(unsigned(NO), unsigned((NQ + a.QB - 1) / a.QB));
    if (a.transpose)
        hipLaunchKernelGGL(wbuild_kernel<true>, grid, dim3(256), lds, hipStream_t(stream), a);
    else
        hipLaunchKernelGGL(wbuild_kernel<false>, grid, dim3(256), lds, hipStream_t(stream), a);
    return int(hipGetLastError());
}

int launch_proj(const ProjArgs &a, void *stream) {
    if (a.rows <= 0 || a.cols <= 0) return 0;
    if (!proj_supported(a.A) || a.RT % 4 || a.CT < 1) return int(hipErrorInvalidValue);
    const size_t lds = proj_lds_floats(a.RT, a.CT, a.A) * sizeof(float);
    if (lds > kProjLds) return int(hipErrorInvalidValue);
    dim3 grid(unsigned((a.cols + a.CT - 1) / a.CT), unsigned((a.rows + a.RT - 1) / a.RT));
    // 1024 threads when the tile load is large (many loads in flight per CU),
    // else 256 (several workgroups per CU)
    const int64_t loads4 = int64_t(a.RT) * ((a.CT + 3) / 4) * std::max(1, a.nin);
    if (loads4 > 4096)
        hipLaunchKernelGGL((proj_kernel<kProjThreadsMax>), grid, dim3(kProjThreadsMax), lds, hipStream_t(stream), a);
    else
        hipLaunchKernelGGL((proj_kernel<256>), grid, dim3(256), lds, hipStream_t(stream), a);
    return int(hipGetLastError());
}

}  // namespace comera
