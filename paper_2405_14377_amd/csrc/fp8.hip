// FP8 (OCP E4M3) operands for the batch products of the mixed-precision
// layer (the contractions with the batch dimension run in FP8, the batch-free
// core contractions in fp32).  Per tensor: a power-of-two scale s = 2^e, e
// the largest integer with amax * s <= 448, clamped to [-60, 60] (s = 1 for
// amax == 0), then x * s rounded to E4M3 (nearest, ties to the even code,
// saturating at 448).  x * s is exact in fp32, so the codes depend only on
// the fp32 values; the clamp keeps s and 1 / (s s') finite and nonzero in
// fp32.
//
//   amax_vec_kernel       max |x| per workgroup with 16-byte loads (no
//                         atomics, no clearing); amax_partial_kernel for
//                         unaligned x
//   quant_vec_kernel      max of the partials -> s; codes of x (row-major,
//                         rows padded with zero codes to ldq) and / or of
//                         x^T (rows padded with zero codes to ldt), 128 x 128
//                         tiles; workgroup 0 also writes s and the products
//                         1 / (s * s_partner) that scale GEMM results;
//                         quant_kernel does the same for shapes the 16-byte
//                         path does not cover
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "internal.h"

namespace comera {
namespace {

constexpr int kAmaxBlocks = 512;   // partial maxima per tensor
static_assert(kAmaxBlocks * sizeof(float) <= COMERA_FP8_QUANTIZE_WS_BYTES, "scratch of comera_fp8_quantize");

__device__ __forceinline__ float load_act(const void *x, int dtype, int64_t i) {
    if (dtype == COMERA_BF16) return __uint_as_float(uint32_t(reinterpret_cast<const uint16_t *>(x)[i]) << 16);
    return reinterpret_cast<const float *>(x)[i];
}

__device__ __forceinline__ float wave_max(float v) {
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

__global__ __launch_bounds__(256) void amax_partial_kernel(const void *__restrict__ x, int dtype, int64_t n,
                                                           float *__restrict__ pmax) {
    __shared__ float red[4];
    float m = 0.f;
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256)
        m = fmaxf(m, fabsf(load_act(x, dtype, i)));
    m = wave_max(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) pmax[blockIdx.x] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// |x| of the V elements in a 16-byte chunk (V = 4 fp32 or 8 bf16)
template <int V>
__device__ __forceinline__ float chunk_absmax(const u32x4 v) {
    float m = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        if constexpr (V == 4) {
            m = fmaxf(m, fabsf(__uint_as_float(v[w])));
        } else {
            m = fmaxf(m, fabsf(__uint_as_float(v[w] << 16)));
            m = fmaxf(m, fabsf(__uint_as_float(v[w] & 0xFFFF0000u)));
        }
    }
    return m;
}

// The same maxima with 16-byte loads, four in flight per thread; x 16-byte
// aligned.  Elements past the last whole chunk are taken by workgroup 0.
constexpr int kAmaxThreads = 1024;   // 512 workgroups of 16 waves fill every SIMD
template <int V>
__global__ __launch_bounds__(kAmaxThreads) void amax_vec_kernel(const void *__restrict__ x, int dtype, int64_t n,
                                                                float *__restrict__ pmax) {
    __shared__ float red[kAmaxThreads / 64];
    const u32x4 *xv = reinterpret_cast<const u32x4 *>(x);
    const int64_t nv = n / V;
    // one contiguous range of 16-byte chunks per workgroup, walked with
    // eight loads in flight per thread
    const int64_t per = (nv + gridDim.x - 1) / gridDim.x;
    const int64_t b1 = min(nv, (int64_t(blockIdx.x) + 1) * per);
    int64_t i = int64_t(blockIdx.x) * per + threadIdx.x;
    float m = 0.f;
    for (; i + 7 * kAmaxThreads < b1; i += 8 * kAmaxThreads) {
        u32x4 a[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) a[u] = xv[i + u * kAmaxThreads];
#pragma unroll
        for (int u = 0; u < 8; ++u) m = fmaxf(m, chunk_absmax<V>(a[u]));
    }
    for (; i < b1; i += kAmaxThreads) m = fmaxf(m, chunk_absmax<V>(xv[i]));
    if (blockIdx.x == 0)
        for (int64_t j = nv * V + threadIdx.x; j < n; j += kAmaxThreads) m = fmaxf(m, fabsf(load_act(x, dtype, j)));
    m = wave_max(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        float r = red[0];
        for (int w = 1; w < kAmaxThreads / 64; ++w) r = fmaxf(r, red[w]);
        pmax[blockIdx.x] = r;
    }
}

// largest power of two s with amax * s <= 448 (448 = 0.875 * 2^9), the
// exponent clamped to [-60, 60]; 1 for amax == 0
__device__ __forceinline__ float pow2_scale(float amax) {
    if (!(amax > 0.f) || !isfinite(amax)) return 1.f;
    int k;
    const float f = frexpf(amax, &k);
    int e = f <= 0.875f ? 9 - k : 8 - k;
    e = max(-60, min(e, 60));
    return ldexpf(1.f, e);
}

// E4M3 code of v (|v| <= 448 expected; larger magnitudes saturate)
__device__ __forceinline__ uint8_t e4m3_rne(float v) {
    const uint32_t u = __float_as_uint(v);
    const uint32_t sign = (u >> 24) & 0x80u;
    const float a = fabsf(v);
    uint32_t code;
    if (!(a >= 0.015625f)) {                       // below 2^-6: subnormal steps of 2^-9 (exact scaling)
        code = uint32_t(rintf(a * 512.f));          // 0 .. 8 (8 is the smallest normal, code 0x08)
    } else {
        const uint32_t ua = __float_as_uint(a);
        int E = int((ua >> 23) & 0xFFu) - 127;
        const uint32_t frac = ua & 0x7FFFFFu;
        uint32_t m = frac >> 20;
        const uint32_t rem = frac & 0xFFFFFu;
        if (rem > 0x80000u || (rem == 0x80000u && (m & 1u))) ++m;
        if (m == 8u) {
            m = 0u;
            ++E;
        }
        const int eb = E + 7;
        code = (eb > 15 || (eb == 15 && m == 7u)) ? 0x7Eu : (uint32_t(eb) << 3) | m;
    }
    return uint8_t(code | sign);
}

// Four floats -> four E4M3 codes in one dword (byte k from value k):
// gfx950's packed conversion (v_cvt_pk_fp8_f32, round to nearest even) after
// clamping to +-448, which gives the codes of e4m3_rne for every finite
// input (compared on the GPU over a 2^-14-step grid of every binade up to
// 448, the ties between codes, the subnormal steps and 2^20 random values)
__device__ __forceinline__ uint32_t e4m3_pk4(float a, float b, float c, float d) {
    a = __builtin_amdgcn_fmed3f(a, -448.f, 448.f);
    b = __builtin_amdgcn_fmed3f(b, -448.f, 448.f);
    c = __builtin_amdgcn_fmed3f(c, -448.f, 448.f);
    d = __builtin_amdgcn_fmed3f(d, -448.f, 448.f);
    const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
    return uint32_t(__builtin_amdgcn_cvt_pk_fp8_f32(c, d, lo, true));
}

// Tiles of 64 rows x 64 columns over x [R][C]: q[r][c] for c < ldq (if q;
// zero codes for c >= C) and qt[c][r] for r < ldt (if qt; zero codes for
// r >= R).  The grid covers ceil(R' / 64) x ceil(C' / 64) tiles with
// R' = max(R, ldt if qt), C' = max(C, ldq if q).
__global__ __launch_bounds__(256) void quant_kernel(const void *__restrict__ x, int dtype, int64_t R, int64_t C,
                                                    const float *__restrict__ pmax, int nb, uint8_t *__restrict__ q,
                                                    int64_t ldq, uint8_t *__restrict__ qt, int64_t ldt,
                                                    float *__restrict__ s_out, const float *pa, float *oa,
                                                    const float *pb, float *ob) {
    __shared__ float red[4];
    __shared__ uint8_t tile[64][65];
    const int tid = threadIdx.x;
    float m = 0.f;
    for (int i = tid; i < nb; i += 256) m = fmaxf(m, pmax[i]);
    m = wave_max(m);
    if ((tid & 63) == 0) red[tid >> 6] = m;
    __syncthreads();
    const float s = pow2_scale(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])));
    if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) {
        if (s_out) s_out[0] = s;
        if (pa && oa) *oa = 1.f / (s * *pa);
        if (pb && ob) *ob = 1.f / (s * *pb);
    }
    const int64_t r0 = int64_t(blockIdx.x) * 64, c0 = int64_t(blockIdx.y) * 64;
    // thread t: column t % 64 of rows t / 64 + 4 i
    const int cc = tid & 63, rr0 = tid >> 6;
#pragma unroll 4
    for (int i = 0; i < 16; ++i) {
        const int rr = rr0 + 4 * i;
        const int64_t r = r0 + rr, c = c0 + cc;
        const bool ok = r < R && c < C;
        const float v = load_act(x, dtype, ok ? r * C + c : 0);
        const uint8_t code = ok ? e4m3_rne(v * s) : uint8_t(0);
        tile[rr][cc] = code;
        if (q && r < R && c < ldq) q[r * ldq + c] = code;
    }
    if (!qt) return;
    __syncthreads();
    // transposed: row c of qt holds the codes of rows r0 .. r0 + 63
#pragma unroll 4
    for (int i = 0; i < 16; ++i) {
        const int ccl = rr0 + 4 * i;        // column within the tile = row of qt
        const int rrl = cc;                 // row within the tile = column of qt
        const int64_t c = c0 + ccl, r = r0 + rrl;
        if (c < C && r < ldt) qt[c * ldt + r] = tile[rrl][ccl];
    }
}

// quant_kernel with 16-byte loads (V elements per chunk) over tiles of
// 128 rows x 128 columns: V-byte stores of q (128-byte row segments) and
// 16-byte stores of qt through a transposed LDS tile (128-byte segments).
// A thread takes one chunk column of four consecutive rows at a time, so
// the codes of one column in those rows form one dword of the transposed
// tile; its 16-byte pieces are XOR-swizzled by row (piece p of row c at
// p ^ ((c / 8) & 7)), which spreads those dword writes over the banks.
// Requires x 16-byte aligned, C % V == 0, q (if any) V-byte aligned with
// ldq % V == 0, qt (if any) 16-byte aligned with ldt % 16 == 0: every chunk
// then lies wholly inside or wholly outside each bound.  The grid covers
// ceil(R' / 128) x ceil(C' / 128) tiles.
constexpr int kQT = 128;
template <int V>
__global__ __launch_bounds__(256) void quant_vec_kernel(const void *__restrict__ x, int64_t R, int64_t C,
                                                        const float *__restrict__ pmax, int nb, uint8_t *__restrict__ q,
                                                        int64_t ldq, uint8_t *__restrict__ qt, int64_t ldt,
                                                        float *__restrict__ s_out, const float *pa, float *oa,
                                                        const float *pb, float *ob) {
    constexpr int CPR = kQT / V;             // chunks per tile row
    constexpr int RG = 256 / CPR;            // four-row groups per pass
    constexpr int NG = kQT / (4 * RG);       // passes
    constexpr int ESZ = 16 / V;              // bytes per element
    __shared__ float red[4];
    __shared__ __attribute__((aligned(16))) uint8_t tt[kQT][kQT];   // tt[c][r], 16-byte pieces swizzled
    const int tid = threadIdx.x;
    const int ch = tid % CPR, rg = tid / CPR;
    const int64_t r0 = int64_t(blockIdx.x) * kQT, c0 = int64_t(blockIdx.y) * kQT;
    const int64_t c = c0 + int64_t(ch) * V;
    const char *xb = reinterpret_cast<const char *>(x);
    // every load of the tile first (addresses in bounds; zero selected after)
    u32x4 v[NG][4];
#pragma unroll
    for (int gi = 0; gi < NG; ++gi)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t r = r0 + gi * 4 * RG + 4 * rg + j;
            const bool ok = r < R && c < C;
            v[gi][j] = *reinterpret_cast<const u32x4 *>(xb + (ok ? r * C + c : 0) * ESZ);
            if (!ok) v[gi][j] = u32x4{0u, 0u, 0u, 0u};
        }
    float m = 0.f;
    for (int i = tid; i < nb; i += 256) m = fmaxf(m, pmax[i]);
    m = wave_max(m);
    if ((tid & 63) == 0) red[tid >> 6] = m;
    __syncthreads();
    const float s = pow2_scale(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])));
    if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) {
        if (s_out) s_out[0] = s;
        if (pa && oa) *oa = 1.f / (s * *pa);
        if (pb && ob) *ob = 1.f / (s * *pb);
    }
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
        uint32_t w[4][V / 4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float f[V];
#pragma unroll
            for (int e = 0; e < V; ++e) {
                if constexpr (V == 4) f[e] = __uint_as_float(v[gi][j][e]) * s;
                else f[e] = __uint_as_float((e & 1) ? (v[gi][j][e >> 1] & 0xFFFF0000u) : (v[gi][j][e >> 1] << 16)) * s;
            }
#pragma unroll
            for (int k = 0; k < V / 4; ++k) w[j][k] = e4m3_pk4(f[4 * k], f[4 * k + 1], f[4 * k + 2], f[4 * k + 3]);
            const int64_t r = r0 + gi * 4 * RG + 4 * rg + j;
            if (q && r < R && c < ldq) {
                if constexpr (V == 4) *reinterpret_cast<uint32_t *>(q + r * ldq + c) = w[j][0];
                else *reinterpret_cast<uint2 *>(q + r * ldq + c) = make_uint2(w[j][0], w[j][1]);
            }
        }
        if (qt) {
            // column ch V + e, rows gi 4 RG + 4 rg .. + 3: one dword
            const int rl = gi * 4 * RG + 4 * rg;
#pragma unroll
            for (int e = 0; e < V; ++e) {
                const int cc = ch * V + e, sh = 8 * (e & 3);
                const uint32_t d = ((w[0][e >> 2] >> sh) & 0xFFu) | (((w[1][e >> 2] >> sh) & 0xFFu) << 8) |
                                   (((w[2][e >> 2] >> sh) & 0xFFu) << 16) | (((w[3][e >> 2] >> sh) & 0xFFu) << 24);
                const int piece = (rl >> 4) ^ ((cc >> 3) & 7);
                *reinterpret_cast<uint32_t *>(&tt[cc][piece * 16 + (rl & 15)]) = d;
            }
        }
    }
    if (!qt) return;
    __syncthreads();
    // qt rows c0 .. c0 + 127, bytes r0 .. r0 + 127: 8 pieces of 16 bytes per row
#pragma unroll
    for (int i = 0; i < kQT * 8 / 256; ++i) {
        const int id = tid + 256 * i;
        const int cc = id >> 3, part = id & 7;
        const int64_t cq = c0 + cc, r = r0 + part * 16;
        if (cq < C && r < ldt)
            *reinterpret_cast<u32x4 *>(qt + cq * ldt + r) =
                *reinterpret_cast<const u32x4 *>(&tt[cc][(part ^ ((cc >> 3) & 7)) * 16]);
    }
}

}  // namespace

int fp8_amax_blocks() { return kAmaxBlocks; }

int launch_fp8_quant(const void *x, int dtype, int64_t R, int64_t C, float *pmax, uint8_t *q, int64_t ldq,
                     uint8_t *qt, int64_t ldt, float *s_out, const float *pa, float *oa, const float *pb, float *ob,
                     void *stream) {
    if (R <= 0 || C <= 0) return 0;
    if ((q && ldq < C) || (qt && ldt < R)) return int(hipErrorInvalidValue);
    const int64_t n = R * C;
    const int V = dtype == COMERA_BF16 ? 8 : 4;
    auto al = [](const void *ptr, int a) { return reinterpret_cast<uintptr_t>(ptr) % uintptr_t(a) == 0; };
    const bool xa = al(x, 16);
    int nb;
    if (xa) {
        // at least four 16-byte loads per thread
        const int64_t per = int64_t(kAmaxThreads) * 4;
        nb = int(std::min<int64_t>(kAmaxBlocks, std::max<int64_t>(1, (n / V + per - 1) / per)));
        if (V == 8)
            COMERA_LAUNCH(amax_vec_kernel<8>, dim3(nb), dim3(kAmaxThreads), 0, hipStream_t(stream), x, dtype, n,
                               pmax);
        else
            COMERA_LAUNCH(amax_vec_kernel<4>, dim3(nb), dim3(kAmaxThreads), 0, hipStream_t(stream), x, dtype, n,
                               pmax);
    } else {
        nb = int(std::min<int64_t>(kAmaxBlocks, (n + 255) / 256));
        COMERA_LAUNCH(amax_partial_kernel, dim3(nb), dim3(256), 0, hipStream_t(stream), x, dtype, n, pmax);
    }
    if (int e = launch_status()) return e;
    const int64_t rows = qt ? std::max<int64_t>(R, ldt) : R;
    const int64_t cols = q ? std::max<int64_t>(C, ldq) : C;
    const bool vec = xa && C % V == 0 && (!q || (al(q, V) && ldq % V == 0)) && (!qt || (al(qt, 16) && ldt % 16 == 0));
    const int tile = vec ? kQT : 64;
    const int64_t gx = (rows + tile - 1) / tile, gy = (cols + tile - 1) / tile;
    if (gx > 2147483647 || gy > 65535) return int(hipErrorInvalidValue);
    const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>(gy), 1);
    if (vec && V == 8)
        COMERA_LAUNCH(quant_vec_kernel<8>, grid, dim3(256), 0, hipStream_t(stream), x, R, C, pmax, nb, q, ldq,
                           qt, ldt, s_out, pa, oa, pb, ob);
    else if (vec)
        COMERA_LAUNCH(quant_vec_kernel<4>, grid, dim3(256), 0, hipStream_t(stream), x, R, C, pmax, nb, q, ldq,
                           qt, ldt, s_out, pa, oa, pb, ob);
    else
        COMERA_LAUNCH(quant_kernel, grid, dim3(256), 0, hipStream_t(stream), x, dtype, R, C, pmax, nb, q, ldq,
                           qt, ldt, s_out, pa, oa, pb, ob);
    return launch_status();
}

}  // namespace comera

extern "C" {

comera_status comera_fp8_quantize(const void *x, int32_t dtype, int64_t rows, int64_t cols, uint8_t *q, int64_t ldq,
                                  uint8_t *qt, int64_t ldt, float *scale, void *ws, size_t ws_bytes, void *stream) {
    if (rows < 0 || cols < 0 || (dtype != COMERA_F32 && dtype != COMERA_BF16)) return COMERA_ERR_INVALID_ARG;
    if (rows == 0 || cols == 0) return COMERA_OK;
    if (!x || !scale || (!q && !qt)) return COMERA_ERR_INVALID_ARG;
    if ((q && ldq < cols) || (qt && ldt < rows)) return COMERA_ERR_INVALID_ARG;
    if (!ws || ws_bytes < size_t(COMERA_FP8_QUANTIZE_WS_BYTES)) return COMERA_ERR_WORKSPACE;
    const int64_t tr = qt ? std::max(rows, ldt) : rows, tc = q ? std::max(cols, ldq) : cols;
    if ((tr + 63) / 64 > 2147483647 || (tc + 63) / 64 > 65535) return COMERA_ERR_UNSUPPORTED;
    const int e = comera::launch_fp8_quant(x, dtype, rows, cols, reinterpret_cast<float *>(ws), q, ldq, qt, ldt, scale,
                                           nullptr, nullptr, nullptr, nullptr, stream);
    return comera::note_hip(e, "FP8 quantisation") ? COMERA_ERR_HIP : COMERA_OK;
}

}  // extern "C"
