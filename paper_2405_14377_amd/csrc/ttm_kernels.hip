// Elementwise HIP kernels (gfx950) around the core contractions:
//   fold      masked, rank-compacted core copies (eq. Wcompress)
//   expand    compacted core gradients back to the full core layout, with
//             the fixed-order sum of split partials and the mask factor
//   sum       fixed-order sum of split-K partials
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
// threads of a fold workgroup (a constant, not blockDim, which would be one
// more memory round trip)
constexpr int kFoldThreads = 256;

// Map of a compacted bond's entries to full ones, built in LDS by 256
// threads at once: thread t owns full entry t and, when it is active, writes
// t at its rank (the set bits below it).  Compaction only happens for ranks
// up to 256; bonds 0 and d (rank 1) map the identity.  Uncompacted plans
// (ranks up to 4096) do not read the map.
__device__ __forceinline__ void bond_map(const FoldArgs &a, int bond, int *map) {
    const int t = threadIdx.x;
    if (!a.compacted) return;
    if (bond == 0 || bond == a.d) {
        map[t] = t;
        return;
    }
    // the four words by uniform (scalar) loads, then picked per lane
    const BondBits b = a.act[bond];
    const int w = t >> 6, bit = t & 63;
    const int c1 = __popcll(b.w[0]), c2 = c1 + __popcll(b.w[1]), c3 = c2 + __popcll(b.w[2]);
    const uint64_t word = w == 0 ? b.w[0] : w == 1 ? b.w[1] : w == 2 ? b.w[2] : b.w[3];
    const int below = w == 0 ? 0 : w == 1 ? c1 : w == 2 ? c2 : c3;
    if ((word >> bit) & 1) map[below + __popcll(word & ((uint64_t(1) << bit) - 1))] = t;
}

__global__ __launch_bounds__(kFoldThreads) void fold_kernel(FoldArgs a) {
    __shared__ int map_l[256], map_r[256];
    const int k = blockIdx.y;
    if (k >= a.nfold) return;
    // bonds on either side of core k
    bond_map(a, k, map_l);
    bond_map(a, k + 1, map_r);
    __syncthreads();
    const int rl = a.rc[k], rr = a.rc[k + 1], m = a.m[k], n = a.n[k];
    const int total = rl * m * n * rr;     // core sizes are far below 2^31 (host checks)
    const float *G = a.G[k];
    const float *D = (k < a.d - 1) ? a.D[k] : nullptr;
    const CoreStrides st = a.st[k];
    for (int o = blockIdx.x * kFoldThreads + threadIdx.x; o < total; o += gridDim.x * kFoldThreads) {
        // compacted element o = (al, jm, in, c)
        const int c = o % rr;
        int t = o / rr;
        const int in = t % n;
        t /= n;
        const int jm = t % m;
        const int al = t / m;
        const int fa = a.compacted ? map_l[al] : al, fc = a.compacted ? map_r[c] : c;
        float v = G[((fa * m + jm) * n + in) * a.r[k + 1] + fc];
        if (D) v *= D[fc];
        a.Gc[k][al * st.sa + jm * st.sm + in * st.sn + c * st.sc] = v;
    }
}

// Workgroup of NT threads = (NT / G) outputs x G split groups (G = 1 .. 8
// per core, about eight splits per group; up to 64 for a core in more than
// 512 partials, so that a thread still waits for only a few rounds of loads):
// group g sums the splits [g S / G, (g + 1) S / G) in order, then group 0
// adds the G group sums in order.  One flattened grid covers all cores
// (a.blk0[k] = first block of core k).  The result does not depend on the
// launch shape other than G.  NT = 256 while every core has G <= 8, else
// 1024 (the many-split cores then still get a few hundred workgroups).
constexpr int kExpandMaxGroups = 64;
template <int NT>
__global__ __launch_bounds__(NT) void expand_kernel(ExpandArgs a) {
    __shared__ float red[NT + kExpandMaxGroups];   // [G][no + 1]
    int k = 0;
    while (k + 1 < a.d && int(blockIdx.x) >= a.blk0[k + 1]) ++k;
    if (!a.dG[k]) return;
    const int G = a.groups[k], no = NT / G;
    const int rl = a.r[k], rr = a.r[k + 1], m = a.m[k], n = a.n[k];
    const int crl = a.rc[k], crr = a.rc[k + 1];
    const int tot32 = rl * m * n * rr;     // core sizes are far below 2^31 (host checks)
    const int64_t csize = int64_t(crl) * m * n * crr;
    const int mn_ = m * n;
    const float *D = (k < a.d - 1) ? a.D[k] : nullptr;
    const int lo = threadIdx.x % no, g = threadIdx.x / no;
    const int S = a.splits[k];
    const int s0 = int(int64_t(g) * S / G), s1 = int(int64_t(g + 1) * S / G);
    const float *part = a.part[k];
    const int o = (int(blockIdx.x) - a.blk0[k]) * no + lo;
    int ci = -1;
    if (o < tot32) {
        const int c = o % rr;
        const int t = o / rr;
        const int mn = t % mn_;
        const int al = t / mn_;
        int ca = al, cc = c;
        if (a.compacted) {
            ca = (k == 0) ? 0 : rank_bit(a.act[k], al);
            cc = (k == a.d - 1) ? 0 : rank_bit(a.act[k + 1], c);
        }
        if (ca >= 0 && cc >= 0) {
            const int jm = mn / n, in = mn % n;
            const CoreStrides st = a.st[k];
            ci = ca * st.sa + jm * st.sm + in * st.sn + cc * st.sc;
        }
    }
    float v = 0.f;
    if (ci >= 0) {
        int s = s0;
        for (; s + 8 <= s1; s += 8) {
            float x[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) x[u] = part[(s + u) * csize + ci];
#pragma unroll
            for (int u = 0; u < 8; ++u) v += x[u];
        }
        for (; s < s1; ++s) v += part[s * csize + ci];
    }
    red[g * (no + 1) + lo] = v;
    __syncthreads();
    if (g == 0 && o < tot32) {
        float t = red[lo];
        for (int gg = 1; gg < G; ++gg) t += red[gg * (no + 1) + lo];
        if (ci < 0) t = 0.f;
        else if (D) t *= D[o % rr];
        a.dG[k][o] = t;
    }
}

// Mask gradients (chain rule through eq. Wcompress): with dG~_k the gradient
// of the masked core G~_k = G_k D_k (the sum of the compacted partials),
//   dD_k[c] = sum_{a, m, n} dG~_k[a, m, n, c] G_k[a, m, n, c].
// One workgroup per (bond k, entry c): thread t sums the elements t, t + 256,
// ... in that order (each from its split partials in split order), then a
// fixed-shape tree adds the 256 thread sums, so the result is bitwise
// reproducible.  Entries dropped by the compaction (declared inactive) get 0.
__global__ __launch_bounds__(256) void mask_grad_kernel(MaskGradArgs a) {
    __shared__ float red[256];
    int k = 0;
    while (k + 1 < a.d - 1 && int(blockIdx.x) >= a.blk0[k + 1]) ++k;
    float *out = a.dD[k];
    if (!out) return;
    const int c = int(blockIdx.x) - a.blk0[k];
    const int rl = a.r[k], rr = a.r[k + 1], m = a.m[k], n = a.n[k];
    const int cc = a.compacted ? rank_bit(a.act[k + 1], c) : c;
    if (cc < 0) {
        if (threadIdx.x == 0) out[c] = 0.f;
        return;
    }
    const int64_t csize = int64_t(a.rc[k]) * m * n * a.rc[k + 1];
    const CoreStrides st = a.st[k];
    const float *part = a.part[k];
    const float *G = a.G[k];
    const int S = a.splits[k];
    const int mn_ = m * n;
    float v = 0.f;
    for (int e = threadIdx.x; e < rl * mn_; e += 256) {
        const int al = e / mn_, mn = e - al * mn_;
        const int ca = (a.compacted && k > 0) ? rank_bit(a.act[k], al) : al;
        if (ca < 0) continue;   // inactive left slice: G~_{k-1} is zero there, so is dG~_k
        const int jm = mn / n, in = mn - jm * n;
        const int64_t ci = int64_t(ca) * st.sa + jm * st.sm + in * st.sn + int64_t(cc) * st.sc;
        float g = 0.f;
        for (int s = 0; s < S; ++s) g += part[s * csize + ci];
        v += g * G[int64_t(e) * rr + c];
    }
    red[threadIdx.x] = v;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (int(threadIdx.x) < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[c] = red[0];
}

// sum of the split partials in split order, eight loads in flight
__device__ __forceinline__ float split_sum(const float *__restrict__ part, int64_t n, int64_t i, int splits) {
    float v = 0.f;
    int s = 0;
    for (; s + 8 <= splits; s += 8) {
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = part[(s + u) * n + i];
#pragma unroll
        for (int u = 0; u < 8; ++u) v += x[u];
    }
    float x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = part[int64_t(s + u < splits ? s + u : 0) * n + i];
#pragma unroll
    for (int u = 0; u < 8; ++u)
        if (s + u < splits) v += x[u];
    return v;
}

__global__ void sum_splits_kernel(const float *__restrict__ part, float *__restrict__ out, int64_t n, int splits) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        out[i] = split_sum(part, n, i, splits);
}

__global__ void sum_splits_bf16_kernel(const float *__restrict__ part, uint16_t *__restrict__ out, int64_t n,
                                       int splits) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        out[i] = f32_to_bf16_rne(split_sum(part, n, i, splits));
}

// out[t][j][i] = in[t][i][j] (i < M, j < Tn) through a 32 x 33 LDS tile; the
// workgroups stride over (token, row tile, column tile).
template <typename T>
__global__ __launch_bounds__(256) void permute_kernel(const T *__restrict__ in, T *__restrict__ out, int64_t b, int M,
                                                      int Tn, int64_t tiles_m, int64_t tiles_t) {
    __shared__ T tile[32][33];
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    const int64_t per = tiles_m * tiles_t, total = b * per;
    for (int64_t id = blockIdx.x; id < total; id += gridDim.x) {
        const int64_t t = id / per, r = id % per;
        const int i0 = int(r / tiles_t) * 32, j0 = int(r % tiles_t) * 32;
        const T *src = in + t * int64_t(M) * Tn;
        T *dst = out + t * int64_t(M) * Tn;
        for (int y = ty; y < 32; y += 8) {
            const int i = i0 + y, j = j0 + tx;
            if (i < M && j < Tn) tile[y][tx] = src[int64_t(i) * Tn + j];
        }
        __syncthreads();
        for (int y = ty; y < 32; y += 8) {
            const int j = j0 + y, i = i0 + tx;
            if (i < M && j < Tn) dst[int64_t(j) * M + i] = tile[tx][y];
        }
        __syncthreads();
    }
}

__global__ void fill_one_kernel(float *p) { *p = 1.0f; }

__global__ void fill_zero_kernel(uint32_t *p, int64_t n) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        p[i] = 0u;
}

inline int grid_for(int64_t n, int threads = 256, int64_t cap = 65536) {
    int64_t g = (n + threads - 1) / threads;
    return int(std::max<int64_t>(1, std::min<int64_t>(g, cap)));
}

}  // namespace

CoreStrides core_strides(int A, int m, int n, int C, bool swap) {
    (void)A;
    CoreStrides s;
    s.sc = 1;
    if (swap) {
        s.sm = C;
        s.sn = m * C;
    } else {
        s.sn = C;
        s.sm = n * C;
    }
    s.sa = m * n * C;
    return s;
}

int launch_fold(const FoldArgs &a, void *stream) {
    int64_t mx = 1;
    for (int k = 0; k < a.nfold; ++k) mx = std::max<int64_t>(mx, int64_t(a.rc[k]) * a.m[k] * a.n[k] * a.rc[k + 1]);
    if (a.nfold <= 0) return 0;
    // compacted bonds index a 256-entry map (one entry per thread)
    if (a.compacted)
        for (int k = 0; k <= a.d; ++k)
            if (a.r[k] > 256) return int(hipErrorInvalidValue);
    dim3 grid(grid_for(mx), a.nfold);
    COMERA_LAUNCH(fold_kernel, grid, dim3(kFoldThreads), 0, hipStream_t(stream), a);
    return launch_status();
}

int launch_expand(const ExpandArgs &a_in, void *stream) {
    ExpandArgs a = a_in;
    int gmax = 1;
    for (int k = 0; k < a.d; ++k) {
        // up to 8 groups; up to 64 for cores in more than 512 partials
        // (measured: 8 groups of 256 threads are faster up to 256 partials)
        const int gcap = a.splits[k] > 512 ? kExpandMaxGroups : 8;
        int G = 1;
        while (G < gcap && G * 8 < a.splits[k]) G *= 2;
        a.groups[k] = G;
        if (a.dG[k]) gmax = std::max(gmax, G);
    }
    const int nt = gmax <= 8 ? 256 : 1024;
    int blocks = 0;
    for (int k = 0; k < a.d; ++k) {
        a.blk0[k] = blocks;
        const int64_t total = a.dG[k] ? int64_t(a.r[k]) * a.m[k] * a.n[k] * a.r[k + 1] : 0;
        const int no = nt / a.groups[k];
        blocks += int((total + no - 1) / no);
    }
    for (int k = a.d; k < kMaxCores; ++k) a.blk0[k] = blocks;
    if (blocks == 0) return 0;
    if (nt == 256)
        COMERA_LAUNCH_NAMED("expand_kernel", expand_kernel<256>, dim3(unsigned(blocks)), dim3(256), 0, hipStream_t(stream), a);
    else
        COMERA_LAUNCH_NAMED("expand_kernel", expand_kernel<1024>, dim3(unsigned(blocks)), dim3(1024), 0, hipStream_t(stream), a);
    return launch_status();
}

int launch_mask_grad(const MaskGradArgs &a_in, void *stream) {
    MaskGradArgs a = a_in;
    int blocks = 0;
    for (int k = 0; k + 1 < a.d; ++k) {
        a.blk0[k] = blocks;
        blocks += a.dD[k] ? a.r[k + 1] : 0;
    }
    for (int k = std::max(0, a.d - 1); k < kMaxCores; ++k) a.blk0[k] = blocks;
    if (blocks == 0) return 0;
    COMERA_LAUNCH(mask_grad_kernel, dim3(unsigned(blocks)), dim3(256), 0, hipStream_t(stream), a);
    return launch_status();
}

int launch_sum_splits(const float *part, float *out, int64_t n, int splits, void *stream) {
    COMERA_LAUNCH(sum_splits_kernel, dim3(grid_for(n)), dim3(256), 0, hipStream_t(stream), part, out, n, splits);
    return launch_status();
}

int launch_permute_tokens(const void *in, void *out, int64_t b, int64_t M, int64_t T, int esz, void *stream) {
    if (b <= 0 || M <= 0 || T <= 0) return 0;
    const int64_t tm = (M + 31) / 32, tt = (T + 31) / 32;
    const int64_t total = b * tm * tt;
    const unsigned grid = unsigned(std::min<int64_t>(total, 16384));
    if (esz == 2)
        COMERA_LAUNCH(permute_kernel<uint16_t>, dim3(grid), dim3(256), 0, hipStream_t(stream),
                           reinterpret_cast<const uint16_t *>(in), reinterpret_cast<uint16_t *>(out), b, int(M),
                           int(T), tm, tt);
    else
        COMERA_LAUNCH(permute_kernel<float>, dim3(grid), dim3(256), 0, hipStream_t(stream),
                           reinterpret_cast<const float *>(in), reinterpret_cast<float *>(out), b, int(M), int(T),
                           tm, tt);
    return launch_status();
}

int launch_sum_splits_bf16(const float *part, void *out, int64_t n, int splits, void *stream) {
    COMERA_LAUNCH(sum_splits_bf16_kernel, dim3(grid_for(n)), dim3(256), 0, hipStream_t(stream), part,
                       reinterpret_cast<uint16_t *>(out), n, splits);
    return launch_status();
}

int launch_fill_one(float *ptr, void *stream) {
    COMERA_LAUNCH(fill_one_kernel, dim3(1), dim3(1), 0, hipStream_t(stream), ptr);
    return launch_status();
}

int launch_fill_zero(void *ptr, size_t bytes, void *stream) {
    if (bytes == 0) return 0;
    int64_t n = int64_t(bytes / 4);
    COMERA_LAUNCH(fill_zero_kernel, dim3(grid_for(n)), dim3(256), 0, hipStream_t(stream),
                       reinterpret_cast<uint32_t *>(ptr), n);
    return launch_status();
}

}  // namespace comera
