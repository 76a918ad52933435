// HIP kernels (gfx950) for the TTM embedding table of Sec. 4.1.
//
// The table T[V, E] is never formed.  The cores before the last one are
// contracted into a prefix table A[Vp, Ep, R] over every value of the leading
// digits (eq. emb_A1 generalised to d-1 cores); a row is then
//   T[id, (ep, es)] = sum_a A[vp, ep, a] * G_last[a, vs, es]
// with vp = id / v_last and vs = id % v_last (eq. emb_unique with the last
// core as the suffix table).
//
// Backward (the paper states only the lookup; the gradients follow from its
// linearity).  Tokens are grouped by id with a stable LSD radix sort; the dY
// rows of each id are summed in token order into S[p], p = the sorted
// position of the id's first token (runs longer than a chunk are summed
// chunk by chunk, the chunk sums added in chunk order).  Then, per prefix vp
// and its ids u (in id order),
//   dA[vp, ep, a]      = sum_u sum_es S_u[ep, es] G_last[a, vs_u, es]
//   dG_last[a, vs, es] = sum_u sum_ep A[vp, ep, a] S_u[ep, es]
// and dA is projected onto the prefix cores exactly like dW is for a linear
// layer.  Every sum runs in a fixed order, so results are bitwise
// reproducible.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "embed_internal.h"

namespace comera {
namespace {

constexpr int kMaxEs = 16;          // columns of the last core per register pass
constexpr int kBlk = 1024;          // keys per radix workgroup (256 threads x 4)
constexpr int kSub = kBlk / 256;
constexpr int kGlVp = 4;            // prefixes per dG_last workgroup (= partial)
constexpr size_t kEmbLds = 64 * 1024;

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int lane = threadIdx.x & 63;
    return lane ? ((~0ull) >> (64 - lane)) : 0ull;
}

__device__ __forceinline__ int64_t wave_uniform64(int64_t v) {
    const int lo = __builtin_amdgcn_readfirstlane(int(uint64_t(v) & 0xffffffffu));
    const int hi = __builtin_amdgcn_readfirstlane(int(uint64_t(v) >> 32));
    return int64_t((uint64_t(uint32_t(hi)) << 32) | uint32_t(lo));
}

// First index in sorted keys[lo, hi) with keys[i] >= key, found by the whole
// wave: each round probes 64 evenly spaced positions.
__device__ int wave_lower_bound(const uint32_t *__restrict__ keys, int lo, int hi, uint32_t key) {
    const int lane = threadIdx.x & 63;
    while (hi > lo) {
        const int step = (hi - lo + 63) / 64;
        const int probe = lo + lane * step;
        const bool less = probe < hi && keys[probe] < key;
        const int cnt = __popcll(__ballot(less));
        if (cnt == 0) return lo;
        const int nlo = lo + (cnt - 1) * step + 1;
        const int nhi = min(hi, lo + cnt * step);
        lo = nlo;
        hi = nhi;
    }
    return lo;
}

// ---------------------------------------------------------------- forward rows
// One wave per token.  Lane ep loads its prefix row A[vp, ep, :] into
// registers (with the rank-major table, a wave reads 64 consecutive floats
// per rank), the wave copies the slice G_last[:, vs, :] (R x Es floats) into
// its own LDS region, all loads issued before any store; the slice is read
// back as broadcast 16-byte LDS reads and every lane writes Es consecutive
// outputs.  A element (vp, ep, a) sits at vp Ep R + ep sE + a sR.
__device__ __forceinline__ void wave_sync_lds() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int RMAX, int NJ4>
__global__ __launch_bounds__(256) void embed_rows_kernel(const int64_t *__restrict__ ids, int64_t n_tokens,
                                                         int64_t V, const float *__restrict__ Apre,
                                                         const float *__restrict__ Gs, float *__restrict__ Y, int Ep,
                                                         int R, int Vs, int Es, int sE, int sR,
                                                         int *__restrict__ err_flag) {
    constexpr int ES4 = 4 * NJ4;
    __shared__ __attribute__((aligned(16))) float gsl[4][RMAX * ES4];   // per wave: [RMAX][ES4], zero padded
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t t = int64_t(blockIdx.x) * 4 + wave;
    if (t >= n_tokens) return;
    const int64_t id = wave_uniform64(ids[t]);
    const int E = Ep * Es;
    float *yrow = Y + t * E;
    if (id < 0 || id >= V) {
        if (lane == 0 && err_flag) *err_flag = 1;
        for (int o = lane; o < E; o += 64) yrow[o] = 0.f;
        return;
    }
    const uint32_t vp = uint32_t(id) / uint32_t(Vs);        // ids are below 2^31
    const int vs = int(uint32_t(id) - vp * uint32_t(Vs));
    float *gw = gsl[wave];
    for (int ep0 = 0; ep0 < Ep; ep0 += 64) {
        const int ep = ep0 + lane;
        const int epc = min(ep, Ep - 1);
        float av[RMAX];
        const float *ar = Apre ? Apre + int64_t(vp) * Ep * R + int64_t(epc) * sE : nullptr;
#pragma unroll
        for (int a = 0; a < RMAX; ++a) av[a] = ar ? ar[int64_t(min(a, R - 1)) * sR] : 1.f;
        if (ep0 == 0)
            stage_lds<(RMAX * ES4 + 63) / 64>(gw, RMAX * ES4, lane, 64, [&](int i) {
                const int a = i / ES4, es = i - a * ES4;
                return (a < R && es < Es) ? Gs[(int64_t(a) * Vs + vs) * Es + es] : 0.f;
            });
        wave_sync_lds();
        float acc[ES4];
#pragma unroll
        for (int j = 0; j < ES4; ++j) acc[j] = 0.f;
        // rows a >= R of the slice are zero, so the products for a >= R vanish
#pragma unroll
        for (int a = 0; a < RMAX; ++a) {
#pragma unroll
            for (int j4 = 0; j4 < NJ4; ++j4) {
                const float4 g4 = *reinterpret_cast<const float4 *>(gw + a * ES4 + 4 * j4);
                acc[4 * j4 + 0] += av[a] * g4.x;
                acc[4 * j4 + 1] += av[a] * g4.y;
                acc[4 * j4 + 2] += av[a] * g4.z;
                acc[4 * j4 + 3] += av[a] * g4.w;
            }
        }
        if (ep < Ep) {
            float *yr = yrow + int64_t(ep) * Es;
            if (Es == ES4 && (reinterpret_cast<uintptr_t>(yr) & 15) == 0) {
#pragma unroll
                for (int j = 0; j < ES4; j += 4)
                    *reinterpret_cast<float4 *>(yr + j) = make_float4(acc[j], acc[j + 1], acc[j + 2], acc[j + 3]);
            } else {
#pragma unroll
                for (int j = 0; j < ES4; ++j)
                    if (j < Es) yr[j] = acc[j];
            }
        }
    }
}

// Rows on MFMA (v_mfma_f32_16x16x4f32), one wave per token: the row is the
// product out[ep][es] = sum_a A[vp, ep, a] G_last[a, vs, es], an
// (Ep x R) x (R x Es) product with Ep = 16 NT, R <= 4 NS, Es <= 16.  Lane
// l = 16 q + r supplies A[16 t + r][4 s + q] and B[4 s + q][r] and receives
// rows 4 q + v, column r of each 16 x 16 output tile t; the tile goes
// through the wave's LDS region so that the row is written with 16-byte
// stores.
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int NT, int NS>
__global__ __launch_bounds__(256) void embed_rows_mfma_kernel(const int64_t *__restrict__ ids, int64_t n_tokens,
                                                              int64_t V, const float *__restrict__ Apre,
                                                              const float *__restrict__ Gs, float *__restrict__ Y,
                                                              int R, int Vs, int Es, int sE, int sR,
                                                              int *__restrict__ err_flag) {
    constexpr int Ep = 16 * NT;
    __shared__ __attribute__((aligned(16))) float rowbuf[4][Ep * 16];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t t = int64_t(blockIdx.x) * 4 + wave;
    if (t >= n_tokens) return;
    const int64_t id = wave_uniform64(ids[t]);
    const int E = Ep * Es;
    float *yrow = Y + t * E;
    if (id < 0 || id >= V) {
        if (lane == 0 && err_flag) *err_flag = 1;
        for (int o = lane; o < E; o += 64) yrow[o] = 0.f;
        return;
    }
    const uint32_t vp = uint32_t(id) / uint32_t(Vs);        // ids are below 2^31
    const int vs = int(uint32_t(id) - vp * uint32_t(Vs));
    const int r = lane & 15, q = lane >> 4;
    // operands, every load issued before the first product
    float av[NT][NS], bv[NS];
    const float *ar = Apre ? Apre + int64_t(vp) * Ep * R : nullptr;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const int a = 4 * s + q;
        const bool ok = a < R;
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
            av[tt][s] = ok ? (ar ? ar[int64_t(16 * tt + r) * sE + int64_t(a) * sR] : 1.f) : 0.f;
        bv[s] = (ok && r < Es) ? Gs[(int64_t(a) * Vs + vs) * Es + r] : 0.f;
    }
    f32x4 acc[NT];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
        acc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s) acc[tt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[tt][s], bv[s], acc[tt], 0, 0, 0);
    }
    // tile -> LDS as out[ep][es] (pitch Es), then whole-row stores
    float *rb = rowbuf[wave];
    if (r < Es)
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int v = 0; v < 4; ++v) rb[(16 * tt + 4 * q + v) * Es + r] = acc[tt][v];
    wave_sync_lds();
    if ((E & 3) == 0 && (reinterpret_cast<uintptr_t>(yrow) & 15) == 0) {
        for (int o = 4 * lane; o < E; o += 256)
            *reinterpret_cast<float4 *>(yrow + o) = *reinterpret_cast<const float4 *>(rb + o);
    } else {
        for (int o = lane; o < E; o += 64) yrow[o] = rb[o];
    }
}

// ---------------------------------------------------------------- prefix table
// Prefix table of a three-core table (eq. emb_A1): for prefix (z0, z1),
//   A[(z0, z1)][a2][(e0, e1)] = sum_{a1} G~0[0][z0][e0][a1] G~1[a1][z1][e1][a2]
// with the masks folded on the fly (G~0 = G0 D0 on a1, G~1 = G1 D1 on a2),
// stored rank-major.  Workgroup (z1, block of kTabZ values of z0): the
// block's G~0 rows are staged in LDS; thread (a2, e1) holds the column
// G~1[:, z1, e1, a2] in registers and forms the kTabZ x e0 entries at its
// (a2, e1) position; the block's kTabZ tables go out through LDS as
// contiguous rows.  The workgroups of z0 block 0 also write the folded G~1
// slice to gc1 ([r1][v1][e1][r2]) and those of z1 = 0 the folded G~0 rows to
// gc0 ([v0][e0][r1]): the backward's prefix-core projections read them.
constexpr int kTabZ = 2;
template <int R1MAX>
__global__ __launch_bounds__(256) void embed_table_kernel(const float *__restrict__ G0, const float *__restrict__ D0,
                                                          const float *__restrict__ G1, const float *__restrict__ D1,
                                                          float *__restrict__ A, float *__restrict__ gc0,
                                                          float *__restrict__ gc1, int v0, int v1, int e0, int e1,
                                                          int r1, int r2) {
    extern __shared__ __attribute__((aligned(16))) float tl[];
    const int z1 = blockIdx.x, zb = blockIdx.y * kTabZ;
    const int nz = min(kTabZ, v0 - zb);
    const int Ep = e0 * e1;
    constexpr int r1p = R1MAX;                         // row pitch: the products below read whole rows
    float *g0s = tl;                                   // [kTabZ][e0][r1p], zero past r1
    float *out = g0s + kTabZ * e0 * r1p;               // [kTabZ][r2][Ep]
    // the block's folded G~0 rows (and their copy in gc0 from z1 = 0)
    for (int i = threadIdx.x; i < nz * e0 * r1p; i += blockDim.x) {
        const int zl = i / (e0 * r1p), rem = i - zl * e0 * r1p, ee = rem / r1p, a1 = rem - ee * r1p;
        const int a1c = min(a1, r1 - 1);
        float v = G0[(int64_t(zb + zl) * e0 + ee) * r1 + a1c] * (D0 ? D0[a1c] : 1.f);
        v = a1 < r1 ? v : 0.f;
        if (a1 < r1 && z1 == 0) gc0[(int64_t(zb + zl) * e0 + ee) * r1 + a1] = v;
        g0s[i] = v;
    }
    __syncthreads();
    for (int p = threadIdx.x; p < r2 * e1; p += blockDim.x) {
        // consecutive threads take consecutive e1 (consecutive LDS words of the staged table)
        const int a2 = p / e1, ee1 = p - a2 * e1;
        const float dm = D1 ? D1[a2] : 1.f;
        // unconditional loads (index clamped into the core), then a select:
        // loads under a branch would each wait for their round trip
        float col[R1MAX];
#pragma unroll
        for (int a1 = 0; a1 < R1MAX; ++a1) {
            const float g = G1[((int64_t(min(a1, r1 - 1)) * v1 + z1) * e1 + ee1) * r2 + a2];
            col[a1] = a1 < r1 ? g * dm : 0.f;
        }
        if (blockIdx.y == 0)
#pragma unroll
            for (int a1 = 0; a1 < R1MAX; ++a1)
                if (a1 < r1) gc1[((int64_t(a1) * v1 + z1) * e1 + ee1) * r2 + a2] = col[a1];
        // four (z0, e0) entries at a time: independent accumulators, so the
        // FMAs of one wave do not wait on each other
        const int nrow = nz * e0;
        for (int r0 = 0; r0 < nrow; r0 += 4) {
            float acc[4];
#pragma unroll
            for (int h = 0; h < 4; ++h) acc[h] = 0.f;
#pragma unroll
            for (int q = 0; q < R1MAX / 4; ++q) {
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    const int row = min(r0 + h, nrow - 1);
                    const float4 g = reinterpret_cast<const float4 *>(g0s + row * r1p)[q];
                    acc[h] += g.x * col[4 * q] + g.y * col[4 * q + 1] + g.z * col[4 * q + 2] + g.w * col[4 * q + 3];
                }
            }
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const int row = r0 + h;
                if (row < nrow) {
                    const int zl = row / e0, ee0 = row - zl * e0;
                    out[(zl * r2 + a2) * Ep + ee0 * e1 + ee1] = acc[h];
                }
            }
        }
    }
    __syncthreads();
    // every table row (r2 x Ep floats) of a prefix is contiguous
    const int per = r2 * Ep;
    for (int zl = 0; zl < nz; ++zl) {
        float *dst = A + (int64_t(zb + zl) * v1 + z1) * per;
        for (int i = threadIdx.x; i < per; i += blockDim.x) dst[i] = out[zl * per + i];
    }
}

// ---------------------------------------------------------------- radix sort
// Stable LSD radix sort of (key, token) pairs, 8-bit digits, kBlk keys per
// workgroup.  Keys are the ids; out-of-range ids get the key V and sort last.
// Every pass takes the per-workgroup digit histograms of its own input order.
__device__ __forceinline__ uint32_t key_of(const int64_t *ids, int i, int64_t V) {
    const int64_t id = ids[i];
    return (id >= 0 && id < V) ? uint32_t(id) : uint32_t(V);
}

// Workgroups b < nblk take the digit histogram of their kBlk keys (pass 0
// reads the ids and also counts out-of-range ones); the others clear
// headpos[0 .. nclear) to -1 and zero[0 .. nzero) to 0.0f.
__global__ __launch_bounds__(256) void radix_hist_kernel(const int64_t *__restrict__ ids, const uint32_t *kin, int n,
                                                         int64_t V, int shift, int nblk, int *__restrict__ hist,
                                                         int *__restrict__ bad_out, int *err_flag,
                                                         int *__restrict__ headpos, int64_t nclear,
                                                         float *__restrict__ zero, int64_t nzero) {
    __shared__ int h[256];
    __shared__ int bad_s;
    const int b = blockIdx.x;
    if (b >= nblk) {
        const int64_t stride = int64_t(gridDim.x - nblk) * 256;
        const int64_t i0 = int64_t(b - nblk) * 256 + threadIdx.x;
        for (int64_t i = i0; i < nclear; i += stride) headpos[i] = -1;
        for (int64_t i = i0; i < nzero; i += stride) zero[i] = 0.f;
        return;
    }
    h[threadIdx.x] = 0;
    if (threadIdx.x == 0) bad_s = 0;
    __syncthreads();
    int bad = 0;
    for (int j = 0; j < kSub; ++j) {
        const int i = b * kBlk + j * 256 + threadIdx.x;
        if (i < n) {
            const uint32_t key = kin ? kin[i] : key_of(ids, i, V);
            bad += key == uint32_t(V);
            atomicAdd(&h[(key >> shift) & 255u], 1);
        }
    }
    if (bad) atomicAdd(&bad_s, bad);
    __syncthreads();
    hist[threadIdx.x * nblk + b] = h[threadIdx.x];
    if (threadIdx.x == 0 && bad_out) {
        bad_out[b] = bad_s;
        if (bad_s && err_flag) *err_flag = 1;
    }
}

// Exclusive scan of hist[256 * nblk] in place (digit-major order); with
// bad != null also meta[0] = n - (number of out-of-range ids).
__global__ __launch_bounds__(1024) void radix_scan_kernel(int *hist, int nblk, const int *bad, int n, int *meta) {
    __shared__ int wsum[17];
    __shared__ int carry;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int total = 256 * nblk;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int base = 0; base < total; base += 1024) {
        const int i = base + threadIdx.x;
        const int v = i < total ? hist[i] : 0;
        int x = v;
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        if (lane == 63) wsum[w] = x;
        __syncthreads();
        if (threadIdx.x == 0) {
            int run = 0;
            for (int k = 0; k < 16; ++k) {
                const int c = wsum[k];
                wsum[k] = run;
                run += c;
            }
            wsum[16] = run;
        }
        __syncthreads();
        if (i < total) hist[i] = carry + wsum[w] + x - v;
        __syncthreads();
        if (threadIdx.x == 0) carry += wsum[16];
        __syncthreads();
    }
    if (threadIdx.x == 0 && bad) {
        int nb = 0;
        for (int b = 0; b < nblk; ++b) nb += bad[b];
        meta[0] = n - nb;
    }
}

// With scan != 0 (few blocks) the workgroup derives its own digit offsets
// from the raw histograms: offs[dg][b] = sum of all counts of digits below
// dg plus the counts of digit dg in blocks below b (and block 0 writes
// meta[0] = n - out-of-range ids when bad != null), so no scan kernel runs.
__global__ __launch_bounds__(256) void radix_scatter_kernel(const int64_t *__restrict__ ids, const uint32_t *kin,
                                                            const uint32_t *vin, int n, int64_t V, int shift, int nblk,
                                                            const int *__restrict__ offs, uint32_t *kout,
                                                            uint32_t *vout, int scan, const int *bad, int *meta) {
    __shared__ int wcount[kSub * 4][256];
    __shared__ int dbase[256];
    __shared__ int wsum[4];
    const int tid = threadIdx.x, w = tid >> 6;
    for (int i = tid; i < kSub * 4 * 256; i += 256) (&wcount[0][0])[i] = 0;
    const int b = blockIdx.x;
    if (scan) {
        // thread tid = digit: its total and its count in the blocks below b
        int tot = 0, below = 0;
        for (int bb = 0; bb < nblk; ++bb) {
            const int h = offs[tid * nblk + bb];
            tot += h;
            below += bb < b ? h : 0;
        }
        // exclusive scan of the digit totals (wave scans, then the four waves)
        const int lane = tid & 63;
        int x = tot;
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        if (lane == 63) wsum[w] = x;
        __syncthreads();
        int pre = 0;
        for (int ww = 0; ww < w; ++ww) pre += wsum[ww];
        dbase[tid] = pre + x - tot + below;
        if (b == 0 && tid == 0 && bad) {
            int nb = 0;
            for (int bb = 0; bb < nblk; ++bb) nb += bad[bb];
            meta[0] = n - nb;
        }
    }
    __syncthreads();
    uint32_t key[kSub], val[kSub], dg[kSub];
    int rank[kSub];
    bool valid[kSub];
#pragma unroll
    for (int j = 0; j < kSub; ++j) {
        const int i = b * kBlk + j * 256 + tid;
        valid[j] = i < n;
        key[j] = 0;
        val[j] = 0;
        if (valid[j]) {
            if (kin) {
                key[j] = kin[i];
                val[j] = vin[i];
            } else {
                key[j] = key_of(ids, i, V);
                val[j] = uint32_t(i);
            }
        }
        dg[j] = (key[j] >> shift) & 255u;
        uint64_t peers = __ballot(valid[j]);
        for (int bt = 0; bt < 8; ++bt) {
            const bool set = (dg[j] >> bt) & 1u;
            const uint64_t bb = __ballot(valid[j] && set);
            peers &= set ? bb : ~bb;
        }
        rank[j] = __popcll(peers & lanemask_lt());
        if (valid[j] && rank[j] == 0) wcount[j * 4 + w][dg[j]] = __popcll(peers);
    }
    __syncthreads();
    {
        int run = 0;
        for (int vw = 0; vw < kSub * 4; ++vw) {
            const int c = wcount[vw][tid];
            wcount[vw][tid] = run;
            run += c;
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kSub; ++j) {
        if (!valid[j]) continue;
        const int pos = (scan ? dbase[dg[j]] : offs[dg[j] * nblk + b]) + wcount[j * 4 + w][dg[j]] + rank[j];
        kout[pos] = key[j];
        vout[pos] = val[j];
    }
}

// ---------------------------------------------------------------- segment sums
// Chunk c covers sorted positions [c * kEmbedItem, (c + 1) * kEmbedItem).
// Each run of equal keys inside it is summed in position (= token) order.  A
// run that is a whole segment goes to S[head]; a run cut by the chunk's end
// goes to Plast[c]; a run cut by the chunk's start goes to Pfirst[c].  A head
// (first token of an id) inside the chunk records headpos[id].  Every dY row
// of the chunk is loaded once, all loads before the sums, 16 bytes per load
// when rows are 16-byte aligned.
__global__ __launch_bounds__(256) void embed_segsum_kernel(const float *__restrict__ dY, int E,
                                                           const int *__restrict__ meta,
                                                           const uint32_t *__restrict__ keys,
                                                           const uint32_t *__restrict__ vals, float *__restrict__ S,
                                                           float *__restrict__ Pfirst, float *__restrict__ Plast,
                                                           int *__restrict__ headpos) {
    __shared__ uint32_t sv[kEmbedItem];
    __shared__ int run_end[kEmbedItem];
    __shared__ int dst_kind[kEmbedItem];    // destination of the run closed at j: 0 S, 1 Pfirst, 2 Plast
    __shared__ int64_t dst_off[kEmbedItem]; // row offset (floats) in that buffer
    const int nv = meta[0];
    const int c = blockIdx.x;
    const int p0 = c * kEmbedItem;
    if (p0 >= nv) return;
    const int p1 = min(nv, p0 + kEmbedItem);
    const int len = p1 - p0;
    if (int(threadIdx.x) < len) {
        const int j = threadIdx.x;
        const uint32_t k = keys[p0 + j];
        sv[j] = vals[p0 + j];
        if (p0 + j == 0 || keys[p0 + j - 1] != k) headpos[k] = p0 + j;
        const bool end = j == len - 1 || keys[p0 + j + 1] != k;
        run_end[j] = end;
        if (end) {
            int r0 = j;
            while (r0 > 0 && keys[p0 + r0 - 1] == k) --r0;
            const bool cut_front = r0 == 0 && p0 > 0 && keys[p0 - 1] == k;
            const bool cut_back = j == len - 1 && p1 < nv && keys[p1] == k;
            dst_kind[j] = cut_front ? 1 : (cut_back ? 2 : 0);
            dst_off[j] = (cut_front || cut_back) ? int64_t(c) * E : int64_t(p0 + r0) * E;
        }
    }
    __syncthreads();
    auto dst_row = [&](int j) -> float * {
        const int kd = dst_kind[j];
        return (kd == 0 ? S : (kd == 1 ? Pfirst : Plast)) + dst_off[j];
    };
    if ((E & 3) == 0 && (reinterpret_cast<uintptr_t>(dY) & 15) == 0) {
        const int E4 = E >> 2;
        for (int col = threadIdx.x; col < E4; col += blockDim.x) {
            float4 x[kEmbedItem];
#pragma unroll
            for (int j = 0; j < kEmbedItem; ++j)
                x[j] = j < len ? reinterpret_cast<const float4 *>(dY + int64_t(sv[j]) * E)[col]
                               : make_float4(0.f, 0.f, 0.f, 0.f);
            float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int j = 0; j < kEmbedItem; ++j) {
                if (j < len) {
                    acc.x += x[j].x;
                    acc.y += x[j].y;
                    acc.z += x[j].z;
                    acc.w += x[j].w;
                    if (run_end[j]) {
                        reinterpret_cast<float4 *>(dst_row(j))[col] = acc;
                        acc = make_float4(0.f, 0.f, 0.f, 0.f);
                    }
                }
            }
        }
    } else {
        for (int col = threadIdx.x; col < E; col += blockDim.x) {
            float x[kEmbedItem];
#pragma unroll
            for (int j = 0; j < kEmbedItem; ++j) x[j] = j < len ? dY[int64_t(sv[j]) * E + col] : 0.f;
            float acc = 0.f;
#pragma unroll
            for (int j = 0; j < kEmbedItem; ++j) {
                if (j < len) {
                    acc += x[j];
                    if (run_end[j]) {
                        dst_row(j)[col] = acc;
                        acc = 0.f;
                    }
                }
            }
        }
    }
}

// A segment that starts in chunk c and runs past its end: S[head] =
// Plast[c] + Pfirst[c+1] + ... + Pfirst[cend-1].  Workgroup (c, column
// block) of 64 columns x 4 groups: group g sums a fixed quarter of that list
// in order (eight loads in flight), then the quarters are added in order.
__global__ __launch_bounds__(256) void embed_segfix_kernel(int E, const int *__restrict__ meta,
                                                           const uint32_t *__restrict__ keys,
                                                           const float *__restrict__ Pfirst,
                                                           const float *__restrict__ Plast, float *__restrict__ S) {
    __shared__ int info[2];
    __shared__ float red[4][64];
    const int nv = meta[0];
    const int c = blockIdx.x;
    const int p0 = c * kEmbedItem, p1 = min(nv, p0 + kEmbedItem);
    if (p0 >= nv || p1 >= nv) return;
    const uint32_t k = keys[p1 - 1];
    if (keys[p1] != k) return;                              // the last run ends inside the chunk
    if (threadIdx.x < 64) {
        const int head = wave_lower_bound(keys, p0 > 0 ? p0 - 1 : 0, p1, k);
        const int pend = wave_lower_bound(keys, p1, nv, k + 1);
        if (threadIdx.x == 0) {
            info[0] = head >= p0 ? head : -1;                // started in an earlier chunk: not ours
            info[1] = (pend - 1) / kEmbedItem + 1;
        }
    }
    __syncthreads();
    const int head = info[0];
    if (head < 0) return;
    const int cnt = info[1] - c;           // Plast[c] then Pfirst[c+1 .. cend-1]
    const int g = threadIdx.x >> 6, lc = threadIdx.x & 63;
    const int col = blockIdx.y * 64 + lc;
    const int colc = min(col, E - 1);
    const int i0 = int(int64_t(g) * cnt / 4), i1 = int(int64_t(g + 1) * cnt / 4);
    float acc = 0.f;
    for (int i = i0; i < i1; i += 8) {
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int ii = min(i + u, i1 - 1);
            x[u] = ii == 0 ? Plast[int64_t(c) * E + colc] : Pfirst[int64_t(c + ii) * E + colc];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (i + u < i1) acc += x[u];
    }
    red[g][lc] = acc;
    __syncthreads();
    if (g == 0 && col < E) S[int64_t(head) * E + col] = ((red[0][lc] + red[1][lc]) + red[2][lc]) + red[3][lc];
}

// ---------------------------------------------------------------- per prefix
// dA: one workgroup per prefix vp; its ids (at most Vs) come from headpos[],
// in id order.  For a batch of ids the S rows and G_last slices are staged
// in LDS; wave w and lane (q, g) = (lane % 16, lane / 16) accumulate
// dA[vp, ep, a] for ep = q + 16 w + 64 e and a = g + 4 i in registers:
//   dA[vp, ep, a] = sum_u sum_es S_u[ep, es] G_last[a, vs_u, es]
// Prefixes without ids exit at once (dA was cleared before the sort).
template <int NJ4>
__global__ __launch_bounds__(256) void embed_dapre_kernel(const int *__restrict__ headpos,
                                                          const float *__restrict__ S, const float *__restrict__ Gs,
                                                          int Ep, int R, int Vs, int Es, int vq, int eq, int nbmax,
                                                          float *__restrict__ dA) {
    constexpr int ES4 = 4 * NJ4;
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ int nid;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int vp = blockIdx.x;
    const int E = Ep * Es;
    float *G_s = lds;                                    // [nbmax][R][ES4]
    float *S_s = G_s + nbmax * R * ES4;                  // [nbmax][Ep][ES4]
    int *idl = reinterpret_cast<int *>(S_s + nbmax * Ep * ES4);   // [Vs] ids, then [Vs] heads
    int *hpl = idl + Vs;
    if (tid < 64) {
        int cnt = 0;
        for (int j0 = 0; j0 < Vs; j0 += 64) {
            const int j = j0 + lane;
            const int hp = j < Vs ? headpos[int64_t(vp) * Vs + j] : -1;
            const uint64_t m = __ballot(hp >= 0);
            if (hp >= 0) {
                const int slot = cnt + __popcll(m & lanemask_lt());
                idl[slot] = j;
                hpl[slot] = hp;
            }
            cnt += __popcll(m);
        }
        if (lane == 0) nid = cnt;
    }
    __syncthreads();
    const int ni = nid;
    if (ni == 0) return;
    const int q = lane & 15, g = lane >> 4;
    float acc[2][16];
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[e][i] = 0.f;
    for (int b0 = 0; b0 < ni; b0 += nbmax) {
        const int nb = min(nbmax, ni - b0);
        stage_lds<8>(G_s, nb * R * ES4, tid, 256, [&](int i) {
            const int u = i / (R * ES4), r = i - u * (R * ES4);
            const int a = r / ES4, es = r - a * ES4;
            return es < Es ? Gs[(int64_t(a) * Vs + idl[b0 + u]) * Es + es] : 0.f;
        });
        stage_lds<8>(S_s, nb * Ep * ES4, tid, 256, [&](int i) {
            const int u = i / (Ep * ES4), r = i - u * (Ep * ES4);
            const int ep = r / ES4, es = r - ep * ES4;
            return es < Es ? S[int64_t(hpl[b0 + u]) * E + ep * Es + es] : 0.f;
        });
        __syncthreads();
        for (int u = 0; u < nb; ++u) {
            const float *gu = G_s + u * R * ES4;
            const float *su = S_s + u * Ep * ES4;
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const int ep = q + 16 * wave + 64 * e;
                if (ep >= Ep) continue;
                float4 s4[NJ4];
#pragma unroll
                for (int j4 = 0; j4 < NJ4; ++j4) s4[j4] = *reinterpret_cast<const float4 *>(su + ep * ES4 + 4 * j4);
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int a = g + 4 * i;
                    if (a < R) {
                        float t = 0.f;
#pragma unroll
                        for (int j4 = 0; j4 < NJ4; ++j4) {
                            const float4 g4 = *reinterpret_cast<const float4 *>(gu + a * ES4 + 4 * j4);
                            t += s4[j4].x * g4.x;
                            t += s4[j4].y * g4.y;
                            t += s4[j4].z * g4.z;
                            t += s4[j4].w * g4.w;
                        }
                        acc[e][i] += t;
                    }
                }
            }
        }
        __syncthreads();
    }
    // dA[vp] written blocked for the prefix-core projections
    const int Vh = vp / vq, x = vp - Vh * vq;
    const int NEq = Ep / eq;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int ep = q + 16 * wave + 64 * e;
        if (ep >= Ep) continue;
        const int Eh = ep / eq, y = ep - Eh * eq;
        float *dst = dA + (((int64_t(Vh) * NEq + Eh) * vq + x) * eq + y) * R;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int a = g + 4 * i;
            if (a < R) dst[a] = acc[e][i];
        }
    }
}

// dG_last: workgroup (vs, chunk) sums, over the ids vp Vs + vs with vp in
// [kGlVp chunk, kGlVp (chunk + 1)) in vp order,
//   part[chunk][a][vs][es] = sum_u sum_ep A[vp_u, ep, a] S_u[ep, es]
// with A blocks (ranks padded to R4 = 4 ceil(R / 4)) and S rows of a batch
// of ids staged in LDS.  Thread item (a quad, es quad, ep eighth) keeps a
// 4 x 4 block of sums; the eight ep parts are added in order at the end.
// The expand kernel adds the chunk partials in order.
template <int NJ4>
__global__ __launch_bounds__(256) void embed_dglast_kernel(const int *__restrict__ headpos,
                                                           const float *__restrict__ S,
                                                           const float *__restrict__ Apre, int sE, int sR, int64_t Vp,
                                                           int Ep, int R, int Vs, int Es, int nbmax,
                                                           float *__restrict__ part) {
    constexpr int ES4 = 4 * NJ4;
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ int vpl[kGlVp], hpl[kGlVp];
    __shared__ int nid;
    const int tid = threadIdx.x, lane = tid & 63;
    const int vs = blockIdx.x, chunk = blockIdx.y;
    const int E = Ep * Es;
    const int R4 = (R + 3) & ~3, na4 = R4 / 4;
    float *A_s = lds;                                  // [nbmax][Ep][R4]
    float *S_s = A_s + nbmax * Ep * R4;                // [nbmax][Ep][ES4]
    float *red = S_s + nbmax * Ep * ES4;               // [8][R4][ES4] ep-part sums
    if (tid < 64) {
        const int64_t vp = int64_t(chunk) * kGlVp + lane;
        const int hp = (lane < kGlVp && vp < Vp) ? headpos[vp * Vs + vs] : -1;
        const uint64_t m = __ballot(hp >= 0);
        if (hp >= 0) {
            const int slot = __popcll(m & lanemask_lt());
            vpl[slot] = int(vp);
            hpl[slot] = hp;
        }
        if (lane == 0) nid = __popcll(m);
    }
    __syncthreads();
    const int ni = nid;
    const int items = na4 * NJ4 * 8;                    // (a quad, es quad, ep eighth)
    const bool act = tid < items;
    const int pe = tid & 7, rest = tid >> 3;
    const int aq = act ? rest / NJ4 : 0, jq = act ? rest - (rest / NJ4) * NJ4 : 0;
    const int ept = (Ep + 7) / 8;
    const int ep0 = pe * ept, ep1 = min(Ep, ep0 + ept);
    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
    for (int b0 = 0; b0 < ni; b0 += nbmax) {
        const int nb = min(nbmax, ni - b0);
        stage_lds<8>(A_s, nb * Ep * R4, tid, 256, [&](int i) {
            const int u = i / (Ep * R4), r = i - u * (Ep * R4);
            const int ep = r / R4, a = r - ep * R4;
            return a < R ? (Apre ? Apre[int64_t(vpl[b0 + u]) * Ep * R + int64_t(ep) * sE + int64_t(a) * sR] : 1.f)
                         : 0.f;
        });
        stage_lds<8>(S_s, nb * Ep * ES4, tid, 256, [&](int i) {
            const int u = i / (Ep * ES4), r = i - u * (Ep * ES4);
            const int ep = r / ES4, es = r - ep * ES4;
            return es < Es ? S[int64_t(hpl[b0 + u]) * E + ep * Es + es] : 0.f;
        });
        __syncthreads();
        if (act)
            for (int u = 0; u < nb; ++u) {
                const float *au = A_s + u * Ep * R4 + 4 * aq;
                const float *su = S_s + u * Ep * ES4 + 4 * jq;
                for (int ep = ep0; ep < ep1; ++ep) {
                    const float4 a4 = *reinterpret_cast<const float4 *>(au + ep * R4);
                    const float4 s4 = *reinterpret_cast<const float4 *>(su + ep * ES4);
                    const float av[4] = {a4.x, a4.y, a4.z, a4.w};
                    const float sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int j = 0; j < 4; ++j) acc[i][j] += av[i] * sv[j];
                }
            }
        __syncthreads();
    }
    if (act)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) red[(pe * R4 + 4 * aq + i) * ES4 + 4 * jq + j] = acc[i][j];
    __syncthreads();
    float *dst = part + int64_t(chunk) * R * Vs * Es;
    for (int o = tid; o < R * Es; o += 256) {
        const int a = o / Es, es = o - a * Es;
        float v = red[(0 * R4 + a) * ES4 + es];
#pragma unroll
        for (int p = 1; p < 8; ++p) v += red[(p * R4 + a) * ES4 + es];
        dst[(int64_t(a) * Vs + vs) * Es + es] = v;
    }
}

// MFMA forms of the two per-id contractions (v_mfma_f32_16x16x4f32; lane
// l = 16 q + r supplies A[row 16 t + r][k 4 s + q], B[k 4 s + q][col 16 c + r]
// and receives rows 4 q + v, column r of each 16 x 16 tile).  One wave owns
// one accumulator set and walks its ids in id order, so every sum keeps the
// fixed order of the LDS kernels above.
//
// dA: one workgroup per prefix vp (Ep = 16 NT, R <= 32, Es <= 4 NKS); its
// ids, in id order, are cut into four contiguous quarters, wave w sums
// quarter w, and the four partial sums are added in wave order:
//   dA[vp][ep][a] = sum_u sum_es S_u[ep][es] G_last[a][vs_u][es]
// The contraction index es runs in the order es = NKS q + k (k-th product,
// lane group q), so each lane reads NKS consecutive floats of S_u and of
// G_last.
template <int NT, int NKS>
__global__ __launch_bounds__(256) void embed_dapre_mfma_kernel(const int *__restrict__ headpos,
                                                               const float *__restrict__ S,
                                                               const float *__restrict__ Gs, int64_t Vp, int R,
                                                               int Vs, int Es, int vq, int eq,
                                                               float *__restrict__ dA) {
    constexpr int Ep = 16 * NT;
    __shared__ int vsl[1024], hpl[1024];
    __shared__ int nid;
    __shared__ float red[3][Ep][33];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t vp = blockIdx.x;
    const int r = lane & 15, q = lane >> 4;
    const int E = Ep * Es;
    if (wave == 0) {
        int cnt = 0;
        for (int j0 = 0; j0 < Vs; j0 += 64) {
            const int j = j0 + lane;
            const int hp = j < Vs ? headpos[vp * Vs + j] : -1;
            const uint64_t m = __ballot(hp >= 0);
            if (hp >= 0) {
                const int slot = cnt + __popcll(m & lanemask_lt());
                vsl[slot] = j;
                hpl[slot] = hp;
            }
            cnt += __popcll(m);
        }
        if (lane == 0) nid = cnt;
    }
    __syncthreads();
    const int ni = nid;
    if (ni == 0) return;               // no ids under this prefix: dA stays as cleared (0)
    const int u0 = (ni * wave) / 4, u1 = (ni * (wave + 1)) / 4;
    f32x4 acc[NT][2];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[t][c] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int u = u0; u < u1; ++u) {
        const int vs = vsl[u];
        const float *su = S + int64_t(hpl[u]) * E;
        float sa[NT][NKS], gb[2][NKS];
#pragma unroll
        for (int k = 0; k < NKS; ++k) {
            const int es = NKS * q + k;
#pragma unroll
            for (int t = 0; t < NT; ++t) sa[t][k] = es < Es ? su[(16 * t + r) * Es + es] : 0.f;
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int a = 16 * c + r;
                gb[c][k] = (es < Es && a < R) ? Gs[(int64_t(a) * Vs + vs) * Es + es] : 0.f;
            }
        }
#pragma unroll
        for (int k = 0; k < NKS; ++k)
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int c = 0; c < 2; ++c)
                    acc[t][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(sa[t][k], gb[c][k], acc[t][c], 0, 0, 0);
    }
    // waves 1..3 hand their sums to wave 0, which adds them in wave order
    for (int w = 1; w < 4; ++w) {
        if (wave == w)
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int v = 0; v < 4; ++v)
#pragma unroll
                    for (int c = 0; c < 2; ++c) red[w - 1][16 * t + 4 * q + v][16 * c + r] = acc[t][c][v];
    }
    __syncthreads();
    if (wave != 0) return;
    // dA[vp] written blocked for the prefix-core projections
    const int Vh = int(vp / vq), x = int(vp - int64_t(Vh) * vq);
    const int NEq = Ep / eq;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int ep = 16 * t + 4 * q + v;
            const int Eh = ep / eq, y = ep - Eh * eq;
            float *dst = dA + (((int64_t(Vh) * NEq + Eh) * vq + x) * eq + y) * R;
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int a = 16 * c + r;
                const float sum = ((acc[t][c][v] + red[0][ep][a]) + red[1][ep][a]) + red[2][ep][a];
                if (a < R) dst[a] = sum;
            }
        }
}

// dG_last: one wave per (vs, chunk of kGlVp prefixes) (Ep = 4 NKE, R <= 32,
// Es <= 16), over the ids vp Vs + vs of the chunk in vp order:
//   part[chunk][a][vs][es] = sum_u sum_ep A[vp_u, ep, a] S_u[ep][es]
template <int NKE>
__global__ __launch_bounds__(256) void embed_dglast_mfma_kernel(const int *__restrict__ headpos,
                                                                const float *__restrict__ S,
                                                                const float *__restrict__ Apre, int sE, int sR,
                                                                int64_t Vp, int R, int Vs, int Es, int nchunk,
                                                                float *__restrict__ part) {
    constexpr int Ep = 4 * NKE;
    const int lane = threadIdx.x & 63;
    const int wv = int(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (wv >= Vs * nchunk) return;
    const int vs = wv % Vs, chunk = wv / Vs;
    const int r = lane & 15, q = lane >> 4;
    const int E = Ep * Es;
    f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
    const int64_t vp0 = int64_t(chunk) * kGlVp;
    const int hp_l = (lane < kGlVp && vp0 + lane < Vp) ? headpos[(vp0 + lane) * Vs + vs] : -1;
    uint64_t m = __ballot(hp_l >= 0);
    while (m) {
        const int bit = __builtin_ctzll(m);
        m &= m - 1;
        const int64_t vp = vp0 + bit;
        const int hp = __shfl(hp_l, bit, 64);
        const float *su = S + int64_t(hp) * E;
        const float *ar = Apre ? Apre + vp * Ep * R : nullptr;
        // contraction index ep = NKE q + k for the k-th product: lane group q
        // reads NKE consecutive prefix-table entries per rank (16-byte loads
        // when the table is rank-major)
        float aa[2][NKE], sb[NKE];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int a = 16 * c + r;
            if (a < R && ar && sE == 1 && (NKE & 3) == 0) {
                const float4 *p4 = reinterpret_cast<const float4 *>(ar + int64_t(a) * sR + NKE * q);
#pragma unroll
                for (int k4 = 0; k4 < NKE / 4; ++k4) {
                    const float4 v = p4[k4];
                    aa[c][4 * k4] = v.x;
                    aa[c][4 * k4 + 1] = v.y;
                    aa[c][4 * k4 + 2] = v.z;
                    aa[c][4 * k4 + 3] = v.w;
                }
            } else {
#pragma unroll
                for (int k = 0; k < NKE; ++k)
                    aa[c][k] = a < R ? (ar ? ar[int64_t(NKE * q + k) * sE + int64_t(a) * sR] : 1.f) : 0.f;
            }
        }
#pragma unroll
        for (int k = 0; k < NKE; ++k) sb[k] = r < Es ? su[(NKE * q + k) * Es + r] : 0.f;
#pragma unroll
        for (int k = 0; k < NKE; ++k)
#pragma unroll
            for (int c = 0; c < 2; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(aa[c][k], sb[k], acc[c], 0, 0, 0);
    }
    float *dst = part + int64_t(chunk) * R * Vs * Es;
    if (r < Es)
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int a = 16 * c + 4 * q + v;
                if (a < R) dst[(int64_t(a) * Vs + vs) * Es + r] = acc[c][v];
            }
}

// d = 1: the table is the core itself; dG_0[0, v, e, 0] = S[headpos[v]][e].
__global__ __launch_bounds__(256) void embed_gather_kernel(const int *__restrict__ headpos,
                                                           const float *__restrict__ S, int64_t V, int E,
                                                           float *__restrict__ dG0) {
    const int64_t total = V * E;
    for (int64_t o = int64_t(blockIdx.x) * 256 + threadIdx.x; o < total; o += int64_t(gridDim.x) * 256) {
        const int64_t v = o / E;
        const int e = int(o - v * E);
        const int hp = headpos[v];
        dG0[o] = hp >= 0 ? S[int64_t(hp) * E + e] : 0.f;
    }
}

int es4_of(int Es) { return 4 * ((Es + 3) / 4); }

// ids staged per batch so that the LDS use stays within kEmbLds (0: too large)
int dapre_batch(int Ep, int R, int Vs, int Es) {
    const size_t per = sizeof(float) * size_t(R + Ep) * es4_of(Es);
    const size_t fixed = 2 * sizeof(int) * size_t(Vs);
    if (fixed + per > kEmbLds) return 0;
    return int(std::min<size_t>(8, (kEmbLds - fixed) / per));
}
size_t dapre_lds_bytes(int Ep, int R, int Vs, int Es, int nb) {
    return sizeof(float) * size_t(nb) * (R + Ep) * es4_of(Es) + 2 * sizeof(int) * size_t(Vs);
}

int dglast_batch(int Ep, int R, int Es) {
    const int R4 = (R + 3) & ~3;
    const size_t per = sizeof(float) * size_t(Ep) * (R4 + es4_of(Es));
    const size_t fixed = sizeof(float) * size_t(8) * R4 * es4_of(Es);
    if (fixed + per > kEmbLds) return 0;
    return int(std::min<size_t>(kGlVp, (kEmbLds - fixed) / per));
}
size_t dglast_lds_bytes(int Ep, int R, int Es, int nb) {
    const int R4 = (R + 3) & ~3;
    return sizeof(float) * (size_t(nb) * Ep * (R4 + es4_of(Es)) + size_t(8) * R4 * es4_of(Es));
}

const uint32_t *sorted_vals(const EmbedWs &w, int passes) { return (passes & 1) ? w.valsA : w.valsB; }

}  // namespace

bool embed_kernels_support(int64_t Ep, int R, int Vs, int Es, int d) {
    if (R < 1 || R > 64 || Es < 1 || Es > kMaxEs) return false;
    if (d == 1) return true;
    // dG_last items (a quad, es quad, ep eighth) must fit one workgroup
    return Ep <= 128 && Vs <= 1024 && dapre_batch(int(Ep), R, Vs, Es) > 0 && dglast_batch(int(Ep), R, Es) > 0 &&
           ((R + 3) / 4) * ((Es + 3) / 4) * 8 <= 256;
}

template <int RM>
void launch_rows_nj(int nj4, dim3 grid, void *stream, const int64_t *ids, int64_t n, int64_t V, const float *Apre,
                    const float *Gs, float *Y, int Ep, int R, int Vs, int Es, int sE, int sR, int *err_flag) {
    switch (nj4) {
        case 1: COMERA_LAUNCH((embed_rows_kernel<RM, 1>), grid, dim3(256), 0, hipStream_t(stream), ids, n, V, Apre, Gs, Y, Ep, R, Vs, Es, sE, sR, err_flag); break;
        case 2: COMERA_LAUNCH((embed_rows_kernel<RM, 2>), grid, dim3(256), 0, hipStream_t(stream), ids, n, V, Apre, Gs, Y, Ep, R, Vs, Es, sE, sR, err_flag); break;
        case 3: COMERA_LAUNCH((embed_rows_kernel<RM, 3>), grid, dim3(256), 0, hipStream_t(stream), ids, n, V, Apre, Gs, Y, Ep, R, Vs, Es, sE, sR, err_flag); break;
        default: COMERA_LAUNCH((embed_rows_kernel<RM, 4>), grid, dim3(256), 0, hipStream_t(stream), ids, n, V, Apre, Gs, Y, Ep, R, Vs, Es, sE, sR, err_flag); break;
    }
}

template <int NT>
void launch_rows_mfma(int ns, dim3 grid, void *stream, const int64_t *ids, int64_t n, int64_t V, const float *Apre,
                      const float *Gs, float *Y, int R, int Vs, int Es, int sE, int sR, int *err_flag) {
    switch (ns) {
        case 1: COMERA_LAUNCH((embed_rows_mfma_kernel<NT, 1>), grid, dim3(256), 0, hipStream_t(stream), ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
        case 2: COMERA_LAUNCH((embed_rows_mfma_kernel<NT, 2>), grid, dim3(256), 0, hipStream_t(stream), ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
        case 4: COMERA_LAUNCH((embed_rows_mfma_kernel<NT, 4>), grid, dim3(256), 0, hipStream_t(stream), ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
        default: COMERA_LAUNCH((embed_rows_mfma_kernel<NT, 8>), grid, dim3(256), 0, hipStream_t(stream), ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
    }
}

int launch_embed_rows(const int64_t *ids, int64_t n, int64_t V, const float *Apre, bool rank_major, const float *Gs,
                      float *Y, int Ep, int R, int Vs, int Es, int *err_flag, void *stream) {
    if (n <= 0) return 0;
    const dim3 grid(unsigned((n + 3) / 4));
    const int nj4 = (Es + 3) / 4;
    const int sE = rank_major ? 1 : R, sR = rank_major ? Ep : 1;
    // MFMA rows when the product fits 16 x 16 tiles: Ep a multiple of 16 up
    // to 128, Es <= 16, R <= 32
    if (Ep % 16 == 0 && Ep <= 128 && Es <= 16 && R <= 32) {
        const int ns = (R + 3) / 4 <= 1 ? 1 : ((R + 3) / 4 <= 2 ? 2 : ((R + 3) / 4 <= 4 ? 4 : 8));
        switch (Ep / 16) {
            case 1: launch_rows_mfma<1>(ns, grid, stream, ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
            case 2: launch_rows_mfma<2>(ns, grid, stream, ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
            case 3: launch_rows_mfma<3>(ns, grid, stream, ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
            case 4: launch_rows_mfma<4>(ns, grid, stream, ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
            case 5: launch_rows_mfma<5>(ns, grid, stream, ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
            case 6: launch_rows_mfma<6>(ns, grid, stream, ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
            case 7: launch_rows_mfma<7>(ns, grid, stream, ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
            default: launch_rows_mfma<8>(ns, grid, stream, ids, n, V, Apre, Gs, Y, R, Vs, Es, sE, sR, err_flag); break;
        }
        return launch_status();
    }
    if (R <= 8) launch_rows_nj<8>(nj4, grid, stream, ids, n, V, Apre, Gs, Y, Ep, R, Vs, Es, sE, sR, err_flag);
    else if (R <= 16) launch_rows_nj<16>(nj4, grid, stream, ids, n, V, Apre, Gs, Y, Ep, R, Vs, Es, sE, sR, err_flag);
    else if (R <= 32) launch_rows_nj<32>(nj4, grid, stream, ids, n, V, Apre, Gs, Y, Ep, R, Vs, Es, sE, sR, err_flag);
    else launch_rows_nj<64>(nj4, grid, stream, ids, n, V, Apre, Gs, Y, Ep, R, Vs, Es, sE, sR, err_flag);
    return launch_status();
}

const uint32_t *embed_sorted_keys(const EmbedWs &w, int passes) { return (passes & 1) ? w.keysA : w.keysB; }

int launch_embed_sort(const int64_t *ids, int n, int64_t V, int passes, const EmbedWs &w, int *err_flag,
                      int64_t nclear, float *zero, int64_t nzero, void *stream) {
    const int nblk = (n + kBlk - 1) / kBlk;
    int *bad = w.hist + 256 * nblk;
    const uint32_t *kin = nullptr, *vin = nullptr;
    uint32_t *kout = w.keysA, *vout = w.valsA;
    for (int p = 0; p < passes; ++p) {
        // pass 0 also clears the buffers, counts out-of-range ids and sets meta[0]
        const int nclr = p == 0 ? int(std::min<int64_t>(2048, std::max<int64_t>(1, (nclear + nzero + 4095) / 4096))) : 0;
        COMERA_LAUNCH(radix_hist_kernel, dim3(nblk + nclr), dim3(256), 0, hipStream_t(stream), ids, kin, n, V,
                           8 * p, nblk, w.hist, p == 0 ? bad : nullptr, err_flag, w.headpos, p == 0 ? nclear : 0,
                           zero, p == 0 ? nzero : 0);
        // up to 64 blocks, each scatter workgroup scans the histograms itself
        const int self_scan = nblk <= 64 ? 1 : 0;
        if (!self_scan)
            COMERA_LAUNCH(radix_scan_kernel, dim3(1), dim3(1024), 0, hipStream_t(stream), w.hist, nblk,
                               p == 0 ? bad : nullptr, n, w.meta);
        COMERA_LAUNCH(radix_scatter_kernel, dim3(nblk), dim3(256), 0, hipStream_t(stream), ids, kin, vin, n, V,
                           8 * p, nblk, w.hist, kout, vout, self_scan, p == 0 ? bad : nullptr, w.meta);
        kin = kout;
        vin = vout;
        kout = (kout == w.keysA) ? w.keysB : w.keysA;
        vout = (vout == w.valsA) ? w.valsB : w.valsA;
    }
    return launch_status();
}

int launch_embed_segsum(const float *dY, int E, int n, int passes, const EmbedWs &w, void *stream) {
    const int chunks = (n + kEmbedItem - 1) / kEmbedItem;
    const uint32_t *keys = embed_sorted_keys(w, passes), *vals = sorted_vals(w, passes);
    COMERA_LAUNCH(embed_segsum_kernel, dim3(chunks), dim3(256), 0, hipStream_t(stream), dY, E, w.meta, keys, vals,
                       w.S, w.Pfirst, w.Plast, w.headpos);
    if (int e = launch_status()) return e;
    COMERA_LAUNCH(embed_segfix_kernel, dim3(chunks, unsigned((E + 63) / 64)), dim3(256), 0, hipStream_t(stream),
                       E, w.meta, keys, w.Pfirst, w.Plast, w.S);
    return launch_status();
}

int launch_embed_dapre(const EmbedWs &w, const float *Gs, int64_t Vp, int Ep, int R, int Vs, int Es, int vq, int eq,
                       void *stream) {
    if (Ep % 16 == 0 && Ep <= 64 && R <= 32 && Es <= 16 && Vs <= 1024) {
        const dim3 grid(static_cast<unsigned>(Vp), 1, 1);
#define COMERA_DAPRE(NT, NK)                                                                                     \
    COMERA_LAUNCH((embed_dapre_mfma_kernel<NT, NK>), grid, dim3(256), 0, hipStream_t(stream), w.headpos, w.S, \
                       Gs, Vp, R, Vs, Es, vq, eq, w.dA)
        const int nk = (Es + 3) / 4;
        switch (Ep / 16) {
            case 1: if (nk <= 2) COMERA_DAPRE(1, 2); else COMERA_DAPRE(1, 4); break;
            case 2: if (nk <= 2) COMERA_DAPRE(2, 2); else COMERA_DAPRE(2, 4); break;
            case 3: if (nk <= 2) COMERA_DAPRE(3, 2); else if (nk == 3) COMERA_DAPRE(3, 3); else COMERA_DAPRE(3, 4); break;
            default: if (nk <= 2) COMERA_DAPRE(4, 2); else if (nk == 3) COMERA_DAPRE(4, 3); else COMERA_DAPRE(4, 4); break;
        }
#undef COMERA_DAPRE
        return launch_status();
    }
    const int nb = dapre_batch(Ep, R, Vs, Es);
    if (nb <= 0) return int(hipErrorInvalidValue);
    const size_t lds = dapre_lds_bytes(Ep, R, Vs, Es, nb);
    const dim3 grid(static_cast<unsigned>(Vp), 1, 1);
    switch ((Es + 3) / 4) {
        case 1: COMERA_LAUNCH((embed_dapre_kernel<1>), grid, dim3(256), lds, hipStream_t(stream), w.headpos, w.S, Gs, Ep, R, Vs, Es, vq, eq, nb, w.dA); break;
        case 2: COMERA_LAUNCH((embed_dapre_kernel<2>), grid, dim3(256), lds, hipStream_t(stream), w.headpos, w.S, Gs, Ep, R, Vs, Es, vq, eq, nb, w.dA); break;
        case 3: COMERA_LAUNCH((embed_dapre_kernel<3>), grid, dim3(256), lds, hipStream_t(stream), w.headpos, w.S, Gs, Ep, R, Vs, Es, vq, eq, nb, w.dA); break;
        default: COMERA_LAUNCH((embed_dapre_kernel<4>), grid, dim3(256), lds, hipStream_t(stream), w.headpos, w.S, Gs, Ep, R, Vs, Es, vq, eq, nb, w.dA); break;
    }
    return launch_status();
}

bool embed_table_supported(int r1, int e0) { return r1 >= 1 && r1 <= 64 && e0 >= 1; }

int launch_embed_table(const float *G0, const float *D0, const float *G1, const float *D1, float *A, float *gc0,
                       float *gc1, int v0, int v1, int e0, int e1, int r1, int r2, void *stream) {
    const int r1p = r1 <= 16 ? 16 : (r1 <= 32 ? 32 : 64);   // the kernel's R1MAX
    const size_t lds = sizeof(float) * (size_t(kTabZ) * e0 * r1p + size_t(kTabZ) * r2 * e0 * e1);
    if (!embed_table_supported(r1, e0) || lds > 64 * 1024) return int(hipErrorInvalidValue);
    const dim3 grid(unsigned(v1), unsigned((v0 + kTabZ - 1) / kTabZ));
    if (grid.y > 65535) return int(hipErrorInvalidValue);
    if (r1 <= 16)
        COMERA_LAUNCH((embed_table_kernel<16>), grid, dim3(256), lds, hipStream_t(stream), G0, D0, G1, D1, A, gc0, gc1,
                      v0, v1, e0, e1, r1, r2);
    else if (r1 <= 32)
        COMERA_LAUNCH((embed_table_kernel<32>), grid, dim3(256), lds, hipStream_t(stream), G0, D0, G1, D1, A, gc0, gc1,
                      v0, v1, e0, e1, r1, r2);
    else
        COMERA_LAUNCH((embed_table_kernel<64>), grid, dim3(256), lds, hipStream_t(stream), G0, D0, G1, D1, A, gc0, gc1,
                      v0, v1, e0, e1, r1, r2);
    return launch_status();
}

int embed_dglast_chunks(int64_t Vp) { return int((Vp + kGlVp - 1) / kGlVp); }

int launch_embed_dglast(const EmbedWs &w, const float *Apre, bool rank_major, int64_t Vp, int Ep, int R, int Vs,
                        int Es, void *stream) {
    const int sE = rank_major ? 1 : R, sR = rank_major ? Ep : 1;
    if (Ep % 16 == 0 && Ep <= 64 && R <= 32 && Es <= 16) {
        const int nchunk = embed_dglast_chunks(Vp);
        const dim3 grid(unsigned((int64_t(Vs) * nchunk + 3) / 4));
        switch (Ep / 16) {
            case 1: COMERA_LAUNCH((embed_dglast_mfma_kernel<4>), grid, dim3(256), 0, hipStream_t(stream), w.headpos, w.S, Apre, sE, sR, Vp, R, Vs, Es, nchunk, w.dglast_part); break;
            case 2: COMERA_LAUNCH((embed_dglast_mfma_kernel<8>), grid, dim3(256), 0, hipStream_t(stream), w.headpos, w.S, Apre, sE, sR, Vp, R, Vs, Es, nchunk, w.dglast_part); break;
            case 3: COMERA_LAUNCH((embed_dglast_mfma_kernel<12>), grid, dim3(256), 0, hipStream_t(stream), w.headpos, w.S, Apre, sE, sR, Vp, R, Vs, Es, nchunk, w.dglast_part); break;
            default: COMERA_LAUNCH((embed_dglast_mfma_kernel<16>), grid, dim3(256), 0, hipStream_t(stream), w.headpos, w.S, Apre, sE, sR, Vp, R, Vs, Es, nchunk, w.dglast_part); break;
        }
        return launch_status();
    }
    const int nb = dglast_batch(Ep, R, Es);
    if (nb <= 0) return int(hipErrorInvalidValue);
    const size_t lds = dglast_lds_bytes(Ep, R, Es, nb);
    const dim3 grid(unsigned(Vs), unsigned(embed_dglast_chunks(Vp)));
    switch ((Es + 3) / 4) {
        case 1: COMERA_LAUNCH((embed_dglast_kernel<1>), grid, dim3(256), lds, hipStream_t(stream), w.headpos, w.S, Apre, sE, sR, Vp, Ep, R, Vs, Es, nb, w.dglast_part); break;
        case 2: COMERA_LAUNCH((embed_dglast_kernel<2>), grid, dim3(256), lds, hipStream_t(stream), w.headpos, w.S, Apre, sE, sR, Vp, Ep, R, Vs, Es, nb, w.dglast_part); break;
        case 3: COMERA_LAUNCH((embed_dglast_kernel<3>), grid, dim3(256), lds, hipStream_t(stream), w.headpos, w.S, Apre, sE, sR, Vp, Ep, R, Vs, Es, nb, w.dglast_part); break;
        default: COMERA_LAUNCH((embed_dglast_kernel<4>), grid, dim3(256), lds, hipStream_t(stream), w.headpos, w.S, Apre, sE, sR, Vp, Ep, R, Vs, Es, nb, w.dglast_part); break;
    }
    return launch_status();
}

int launch_embed_gather(const EmbedWs &w, int64_t V, int E, float *dG0, void *stream) {
    const int64_t total = V * E;
    const int grid = int(std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 65536)));
    COMERA_LAUNCH(embed_gather_kernel, dim3(grid), dim3(256), 0, hipStream_t(stream), w.headpos, w.S, V, E, dG0);
    return launch_status();
}

}  // namespace comera
