// HIP kernels (gfx950) for the TTM embedding table of Sec. 4.1.
//
// The table T[V, E] is never formed.  The cores before the last one are
// contracted into a prefix table A[Vp, Ep, r] over every value of the leading
// digits (eq. emb_A1 generalised to d-1 cores); a row is then
//   T[id, (ep, es)] = sum_a A[vp, ep, a] * G_last[a, vs, es]
// with vp = id / v_last and vs = id % v_last (eq. emb_unique with the last
// core as the suffix table).
//
// Backward (the paper states only the lookup; the gradients follow from its
// linearity).  Tokens are grouped by id with a stable LSD radix sort; the dY
// rows of each id are summed in token order into S[p], p = the sorted
// position of the id's first token (long runs are cut into chunks whose
// partial sums are added in chunk order); then
//   dG_last[a, vs, es] = sum_ids sum_ep A[vp, ep, a] S[ep, es]
//   dA[vp, ep, a]      = sum_{ids in vp} sum_es S[ep, es] G_last[a, vs, es]
// and dA is projected onto the prefix cores exactly like dW is for a linear
// layer.  Every sum runs in a fixed order, so results are bitwise
// reproducible.
//
// The contraction kernels are wave-centric: one wave owns a token, a prefix
// or a (suffix digit, chunk) pair, keeps its accumulators in registers and
// never waits on a workgroup barrier; operands whose address is the same for
// the whole wave are read with scalar loads, and inner loops are unrolled
// with clamped (always valid) indices so that loads are issued in batches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "embed_internal.h"

namespace comera {
namespace {

constexpr int kMaxEs = 16;   // columns of the last core per register pass

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
// G_last is staged once per workgroup in LDS.  One wave per token: lane ep
// loads its prefix row A[vp, ep, :] into registers (all loads issued before
// the arithmetic) and accumulates T[id, ep, :] from LDS broadcast reads of
// G_last[:, vs, :].
__device__ __forceinline__ void stage_to_lds(float *dst, const float *__restrict__ src, int count) {
    if ((reinterpret_cast<uintptr_t>(src) & 15) == 0 && (count & 3) == 0) {
        const float4 *s4 = reinterpret_cast<const float4 *>(src);
        float4 *d4 = reinterpret_cast<float4 *>(dst);
        for (int i = threadIdx.x; i < count / 4; i += blockDim.x) d4[i] = s4[i];
    } else {
        for (int i = threadIdx.x; i < count; i += blockDim.x) dst[i] = src[i];
    }
}

template <int RMAX>
__global__ __launch_bounds__(256) void embed_rows_kernel(const int64_t *__restrict__ ids, int64_t n_tokens,
                                                         int64_t V, const float *__restrict__ Apre,
                                                         const float *__restrict__ Gs, float *__restrict__ Y, int Ep,
                                                         int R, int Vs, int Es, int *__restrict__ err_flag) {
    extern __shared__ float gs_s[];   // [R][Vs][Es]
    stage_to_lds(gs_s, Gs, R * Vs * Es);
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int64_t nw = int64_t(gridDim.x) * 4;
    const int E = Ep * Es;
    for (int64_t t = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6); t < n_tokens; t += nw) {
        const int64_t id = wave_uniform64(ids[t]);
        float *yrow = Y + t * E;
        if (id < 0 || id >= V) {
            if (lane == 0 && err_flag) *err_flag = 1;
            for (int o = lane; o < E; o += 64) yrow[o] = 0.f;
            continue;
        }
        const int64_t vp = id / Vs;
        const int vs = int(id - vp * Vs);
        for (int ep = lane; ep < Ep; ep += 64) {
            float av[RMAX];
            if (Apre) {
                const float *ar = Apre + (vp * Ep + ep) * R;
#pragma unroll
                for (int a = 0; a < RMAX; ++a) av[a] = ar[min(a, R - 1)];
            } else {
#pragma unroll
                for (int a = 0; a < RMAX; ++a) av[a] = 1.f;
            }
            __builtin_amdgcn_sched_barrier(0);
            for (int e0 = 0; e0 < Es; e0 += kMaxEs) {
                const int ne = min(kMaxEs, Es - e0);
                float acc[kMaxEs];
#pragma unroll
                for (int j = 0; j < kMaxEs; ++j) acc[j] = 0.f;
#pragma unroll
                for (int a = 0; a < RMAX; ++a) {
                    if (a < R) {
                        const float *g = gs_s + (a * Vs + vs) * Es + e0;
#pragma unroll
                        for (int j = 0; j < kMaxEs; ++j) acc[j] += av[a] * g[min(j, ne - 1)];
                    }
                }
                float *yr = yrow + int64_t(ep) * Es + e0;
                if (ne % 4 == 0 && (reinterpret_cast<uintptr_t>(yr) & 15) == 0) {
#pragma unroll
                    for (int j = 0; j < kMaxEs; j += 4)
                        if (j < ne) *reinterpret_cast<float4 *>(yr + j) = make_float4(acc[j], acc[j + 1], acc[j + 2], acc[j + 3]);
                } else {
#pragma unroll
                    for (int j = 0; j < kMaxEs; ++j)
                        if (j < ne) yr[j] = acc[j];
                }
            }
        }
    }
}

// ---------------------------------------------------------------- radix sort
// Stable LSD radix sort of (key, token) pairs, 8-bit digits, kBlk keys per
// workgroup.  Keys are the ids; out-of-range ids get the key V and sort last.
constexpr int kBlk = 1024;          // keys per workgroup (256 threads x 4)
constexpr int kSub = kBlk / 256;    // sub-tiles of 256 keys

__device__ __forceinline__ uint32_t key_of(const int64_t *ids, int i, int64_t V) {
    const int64_t id = ids[i];
    return (id >= 0 && id < V) ? uint32_t(id) : uint32_t(V);
}

__global__ __launch_bounds__(256) void radix_hist_kernel(const int64_t *__restrict__ ids, const uint32_t *kin, int n,
                                                         int64_t V, int shift, int nblk, int *__restrict__ hist,
                                                         int *err_flag) {
    __shared__ int h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int b = blockIdx.x;
    bool bad = false;
    for (int j = 0; j < kSub; ++j) {
        const int i = b * kBlk + j * 256 + threadIdx.x;
        if (i < n) {
            uint32_t key;
            if (kin) {
                key = kin[i];
            } else {
                key = key_of(ids, i, V);
                bad |= key == uint32_t(V);
            }
            atomicAdd(&h[(key >> shift) & 255u], 1);
        }
    }
    if (bad && err_flag) *err_flag = 1;
    __syncthreads();
    hist[threadIdx.x * nblk + b] = h[threadIdx.x];
}

// exclusive scan of hist[256 * nblk] in place (digit-major order)
__global__ __launch_bounds__(1024) void radix_scan_kernel(int *hist, int total) {
    __shared__ int wsum[17];
    __shared__ int carry;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
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
}

__global__ __launch_bounds__(256) void radix_scatter_kernel(const int64_t *__restrict__ ids, const uint32_t *kin,
                                                            const uint32_t *vin, int n, int64_t V, int shift, int nblk,
                                                            const int *__restrict__ offs, uint32_t *kout,
                                                            uint32_t *vout) {
    __shared__ int wcount[kSub * 4][256];
    const int tid = threadIdx.x, w = tid >> 6;
    for (int i = tid; i < kSub * 4 * 256; i += 256) (&wcount[0][0])[i] = 0;
    __syncthreads();
    const int b = blockIdx.x;
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
        const int pos = offs[dg[j] * nblk + b] + wcount[j * 4 + w][dg[j]] + rank[j];
        kout[pos] = key[j];
        vout[pos] = val[j];
    }
}

// number of in-range keys (position of the first key V) -> meta[0]
__global__ __launch_bounds__(64) void nvalid_kernel(const uint32_t *__restrict__ keys, int n, int64_t V, int *meta) {
    const int nv = wave_lower_bound(keys, 0, n, uint32_t(V));
    if (threadIdx.x == 0) meta[0] = nv;
}

// ---------------------------------------------------------------- segment sums
// Chunk c covers sorted positions [c * kEmbedItem, (c + 1) * kEmbedItem).
// Each run of equal keys inside it is summed in position (= token) order.  A
// run that is a whole segment goes to S[head]; a run cut by the chunk's end
// goes to Plast[c]; a run cut by the chunk's start goes to Pfirst[c].  Every
// dY row of the chunk is loaded once, all loads before the sums.
__global__ __launch_bounds__(256) void embed_segsum_kernel(const float *__restrict__ dY, int E,
                                                           const int *__restrict__ meta,
                                                           const uint32_t *__restrict__ keys,
                                                           const uint32_t *__restrict__ vals, float *__restrict__ S,
                                                           float *__restrict__ Pfirst, float *__restrict__ Plast) {
    __shared__ uint32_t sv[kEmbedItem];
    __shared__ int run_end[kEmbedItem];     // 1 if position j closes its run
    __shared__ float *dst_s[kEmbedItem];     // destination row of the run closed at j
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
        const bool end = j == len - 1 || keys[p0 + j + 1] != k;
        run_end[j] = end;
        if (end) {
            int r0 = j;
            while (r0 > 0 && keys[p0 + r0 - 1] == k) --r0;
            const bool cut_front = r0 == 0 && p0 > 0 && keys[p0 - 1] == k;
            const bool cut_back = j == len - 1 && p1 < nv && keys[p1] == k;
            dst_s[j] = cut_front ? Pfirst + int64_t(c) * E
                                 : (cut_back ? Plast + int64_t(c) * E : S + int64_t(p0 + r0) * E);
        }
    }
    __syncthreads();
    for (int col = threadIdx.x; col < E; col += blockDim.x) {
        float x[kEmbedItem];
#pragma unroll
        for (int j = 0; j < kEmbedItem; ++j) x[j] = j < len ? dY[int64_t(sv[j]) * E + col] : 0.f;
        __builtin_amdgcn_sched_barrier(0);
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < kEmbedItem; ++j) {
            if (j < len) {
                acc += x[j];
                if (run_end[j]) {
                    dst_s[j][col] = acc;
                    acc = 0.f;
                }
            }
        }
    }
}

// A segment that starts in chunk c and runs past its end: S[head] =
// Plast[c] + Pfirst[c+1] + ... + Pfirst[cend-1].  The four waves each sum a
// fixed quarter of that list (four interleaved partial sums each); the
// quarters are then added in order.
__global__ __launch_bounds__(256) void embed_segfix_kernel(int E, const int *__restrict__ meta,
                                                           const uint32_t *__restrict__ keys,
                                                           const float *__restrict__ Pfirst,
                                                           const float *__restrict__ Plast, float *__restrict__ S) {
    extern __shared__ float part_s[];   // [4][E]
    __shared__ int info[2];
    const int nv = meta[0];
    const int c = blockIdx.x;
    const int p0 = c * kEmbedItem, p1 = min(nv, p0 + kEmbedItem);
    if (p0 >= nv || p1 >= nv) return;
    const uint32_t k = keys[p1 - 1];
    if (keys[p1] != k) return;                              // the last run ends inside the chunk
    if (threadIdx.x < 64) {
        // head of the last run, and the end of its segment
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
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int i0 = int(int64_t(w) * cnt / 4), i1 = int(int64_t(w + 1) * cnt / 4);
    for (int col = lane; col < E; col += 64) {
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        for (int i = i0; i < i1; i += 4) {
            float x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int ii = min(i + u, i1 - 1);
                x[u] = ii == 0 ? Plast[int64_t(c) * E + col] : Pfirst[int64_t(c + ii) * E + col];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (i + u < i1) acc[u] += x[u];
        }
        part_s[w * E + col] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    }
    __syncthreads();
    for (int col = threadIdx.x; col < E; col += blockDim.x)
        S[int64_t(head) * E + col] = ((part_s[col] + part_s[E + col]) + part_s[2 * E + col]) + part_s[3 * E + col];
}

// ---------------------------------------------------------------- dG_last
// One wave per (vs, chunk c): it walks the segment heads among sorted
// positions [c nv / chunks, (c + 1) nv / chunks) in order, keeps those whose
// id ends in digit vs, stages each head's prefix block A[vp] and row S in its
// own LDS region, and accumulates A[vp]^T S into registers (lane a holds
// dG_last[a, vs, :]).  Every (chunk, vs) slot of `part` is written by exactly
// one wave; the chunk partials are summed in chunk order afterwards.
__device__ __forceinline__ void wave_sync_lds() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ void wave_copy(float *dst, const float *__restrict__ src, int count) {
    const int lane = threadIdx.x & 63;
    if ((reinterpret_cast<uintptr_t>(src) & 15) == 0 && (count & 3) == 0) {
        const float4 *s4 = reinterpret_cast<const float4 *>(src);
        float4 *d4 = reinterpret_cast<float4 *>(dst);
        const int n4 = count / 4;
        for (int i0 = 0; i0 < n4; i0 += 64 * 8) {
            float4 r[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int i = i0 + u * 64 + lane;
                r[u] = s4[min(i, n4 - 1)];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int i = i0 + u * 64 + lane;
                if (i < n4) d4[i] = r[u];
            }
        }
    } else {
        for (int i = lane; i < count; i += 64) dst[i] = src[i];
    }
}

__global__ __launch_bounds__(256) void embed_dglast_kernel(const int *__restrict__ meta,
                                                           const uint32_t *__restrict__ keys,
                                                           const float *__restrict__ S,
                                                           const float *__restrict__ Apre, int Ep, int R, int Vs,
                                                           int Es, int chunks, float *__restrict__ part) {
    extern __shared__ float lds[];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int E = Ep * Es;
    float *sa = lds + w * (E + Ep * R);      // [Ep][R]
    float *ss = sa + Ep * R;                  // [Ep][Es]
    const int64_t wid = int64_t(blockIdx.x) * 4 + w;
    if (wid >= int64_t(Vs) * chunks) return;
    const int vs = int(wid % Vs), c = int(wid / Vs);
    const int nv = meta[0];
    const int q0 = int(int64_t(c) * nv / chunks), q1 = int(int64_t(c + 1) * nv / chunks);
    const int64_t tot = int64_t(R) * Vs * Es;
    const int la = min(lane, R - 1);
    for (int e0 = 0; e0 < Es; e0 += kMaxEs) {
        const int ne = min(kMaxEs, Es - e0);
        float acc[kMaxEs];
#pragma unroll
        for (int j = 0; j < kMaxEs; ++j) acc[j] = 0.f;
        for (int base = q0; base < q1; base += 64) {
            const int p = base + lane;
            bool take = false;
            if (p < q1) {
                const uint32_t kk = keys[p];
                take = (p == 0 || keys[p - 1] != kk) && int(kk % uint32_t(Vs)) == vs;
            }
            uint64_t m = __ballot(take);
            while (m) {
                const int h = __builtin_ctzll(m);
                m &= m - 1;
                const int hp = base + h;
                const int64_t vp = keys[hp] / uint32_t(Vs);
                wave_sync_lds();
                if (Apre) wave_copy(sa, Apre + vp * Ep * R, Ep * R);
                else if (lane == 0) sa[0] = 1.f;
                wave_copy(ss, S + int64_t(hp) * E, E);
                wave_sync_lds();
                for (int ep = 0; ep < Ep; ++ep) {
                    const float av = sa[ep * R + la];
                    const float *sr = ss + ep * Es + e0;
#pragma unroll
                    for (int j = 0; j < kMaxEs; ++j) acc[j] += av * sr[min(j, ne - 1)];
                }
            }
        }
        if (lane < R) {
            float *dst = part + int64_t(c) * tot + (int64_t(lane) * Vs + vs) * Es + e0;
#pragma unroll
            for (int j = 0; j < kMaxEs; ++j)
                if (j < ne) dst[j] = acc[j];
        }
    }
}

// ---------------------------------------------------------------- dA
// One wave per prefix vp: the ids of vp sit between two wave searches in the
// sorted keys; lane ep accumulates dA[vp, ep, :] (RMAX registers, RMAX >= r)
// over the segment heads in order, S[ep, :] by vector loads and
// G_last[:, vs, :] by scalar loads.  dA is written blocked for the
// projections onto the prefix cores.
template <int RMAX>
__global__ __launch_bounds__(256) void embed_dapre_kernel(const int *__restrict__ meta,
                                                          const uint32_t *__restrict__ keys,
                                                          const float *__restrict__ S, const float *__restrict__ Gs,
                                                          int64_t Vp, int Ep, int R, int Vs, int Es, int vq, int eq,
                                                          float *__restrict__ dA) {
    extern __shared__ float gs_s[];   // [R][Vs][Es]
    stage_to_lds(gs_s, Gs, R * Vs * Es);
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int64_t vp = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (vp >= Vp) return;
    const int nv = meta[0];
    const int pb = wave_lower_bound(keys, 0, nv, uint32_t(vp * Vs));
    const int pe = wave_lower_bound(keys, pb, nv, uint32_t((vp + 1) * Vs));
    const int E = Ep * Es;
    const int64_t NEq = Ep / eq;
    for (int ep0 = 0; ep0 < Ep; ep0 += 64) {
        const int ep = ep0 + lane;
        const int epc = min(ep, Ep - 1);
        float acc[RMAX];
#pragma unroll
        for (int a = 0; a < RMAX; ++a) acc[a] = 0.f;
        for (int base = pb; base < pe; base += 64) {
            const int p = base + lane;
            const bool head = p < pe && (p == 0 || keys[p - 1] != keys[p]);
            uint64_t m = __ballot(head);
            while (m) {
                const int h = __builtin_ctzll(m);
                m &= m - 1;
                const int hp = base + h;
                const int vs = int(keys[hp] % uint32_t(Vs));
                const float *sr = S + int64_t(hp) * E + int64_t(epc) * Es;
                for (int e0 = 0; e0 < Es; e0 += kMaxEs) {
                    const int ne = min(kMaxEs, Es - e0);
                    float sv[kMaxEs];
#pragma unroll
                    for (int j = 0; j < kMaxEs; ++j) sv[j] = j < ne ? sr[e0 + min(j, ne - 1)] : 0.f;
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int a = 0; a < RMAX; ++a) {
                        const float *g = gs_s + (min(a, R - 1) * Vs + vs) * Es + e0;
                        float v = 0.f;
#pragma unroll
                        for (int j = 0; j < kMaxEs; ++j) v += sv[j] * g[min(j, ne - 1)];
                        acc[a] += v;
                    }
                }
            }
        }
        if (ep < Ep) {
            const int64_t Vh = vp / vq, x = vp % vq, Eh = ep / eq, y = ep % eq;
            float *dst = dA + (((Vh * NEq + Eh) * vq + x) * eq + y) * R;
#pragma unroll
            for (int a = 0; a < RMAX; ++a)
                if (a < R) dst[a] = acc[a];
        }
    }
}

}  // namespace

bool embed_kernels_support(int Ep, int R, int Es, int64_t E) {
    const int64_t gs = int64_t(R) * 32 * Es;   // upper bound check done at launch with the real Vs
    (void)gs;
    return R <= 64 && E * 4 * int64_t(sizeof(float)) <= 64 * 1024 &&
           4 * (E + int64_t(Ep) * R) * int64_t(sizeof(float)) <= 64 * 1024;
}

bool embed_gs_fits(int R, int Vs, int Es) { return int64_t(R) * Vs * Es * int64_t(sizeof(float)) <= 64 * 1024; }

int launch_embed_rows(const int64_t *ids, int64_t n, int64_t V, const float *Apre, const float *Gs, float *Y, int Ep,
                      int R, int Vs, int Es, int *err_flag, void *stream) {
    if (n <= 0) return 0;
    const int64_t groups = (n + 3) / 4;
    const int grid = int(std::min<int64_t>(groups, 512));
    const size_t lds = sizeof(float) * size_t(R) * Vs * Es;
#define COMERA_ROWS(RM)                                                                                       \
    hipLaunchKernelGGL((embed_rows_kernel<RM>), dim3(grid), dim3(256), lds, hipStream_t(stream), ids, n, V, Apre, \
                       Gs, Y, Ep, R, Vs, Es, err_flag)
    if (R <= 8) COMERA_ROWS(8);
    else if (R <= 16) COMERA_ROWS(16);
    else if (R <= 32) COMERA_ROWS(32);
    else COMERA_ROWS(64);
#undef COMERA_ROWS
    return int(hipGetLastError());
}

const uint32_t *sorted_keys(const EmbedWs &w, int64_t V) {
    int bits = 0;
    while ((int64_t(1) << bits) <= V) ++bits;
    const int passes = (bits + 7) / 8;
    return (passes & 1) ? w.keysA : w.keysB;
}
const uint32_t *sorted_vals(const EmbedWs &w, int64_t V) {
    int bits = 0;
    while ((int64_t(1) << bits) <= V) ++bits;
    const int passes = (bits + 7) / 8;
    return (passes & 1) ? w.valsA : w.valsB;
}

int launch_embed_sort(const int64_t *ids, int n, int64_t V, const EmbedWs &w, int *err_flag, void *stream) {
    int bits = 0;
    while ((int64_t(1) << bits) <= V) ++bits;  // keys 0..V inclusive (V marks an out-of-range id)
    const int nblk = (n + kBlk - 1) / kBlk;
    const uint32_t *kin = nullptr, *vin = nullptr;
    uint32_t *kout = w.keysA, *vout = w.valsA;
    for (int shift = 0, pass = 0; shift < bits; shift += 8, ++pass) {
        hipLaunchKernelGGL(radix_hist_kernel, dim3(nblk), dim3(256), 0, hipStream_t(stream), ids, kin, n, V, shift,
                           nblk, w.hist, pass == 0 ? err_flag : nullptr);
        hipLaunchKernelGGL(radix_scan_kernel, dim3(1), dim3(1024), 0, hipStream_t(stream), w.hist, 256 * nblk);
        hipLaunchKernelGGL(radix_scatter_kernel, dim3(nblk), dim3(256), 0, hipStream_t(stream), ids, kin, vin, n, V,
                           shift, nblk, w.hist, kout, vout);
        if (int e = int(hipGetLastError())) return e;
        kin = kout;
        vin = vout;
        kout = (kout == w.keysA) ? w.keysB : w.keysA;
        vout = (vout == w.valsA) ? w.valsB : w.valsA;
    }
    hipLaunchKernelGGL(nvalid_kernel, dim3(1), dim3(64), 0, hipStream_t(stream), sorted_keys(w, V), n, V, w.meta);
    return int(hipGetLastError());
}

int launch_embed_segsum(const float *dY, int E, int n, int64_t V, const EmbedWs &w, void *stream) {
    const int chunks = (n + kEmbedItem - 1) / kEmbedItem;
    const uint32_t *keys = sorted_keys(w, V), *vals = sorted_vals(w, V);
    hipLaunchKernelGGL(embed_segsum_kernel, dim3(chunks), dim3(256), 0, hipStream_t(stream), dY, E, w.meta, keys, vals,
                       w.S, w.Pfirst, w.Plast);
    if (int e = int(hipGetLastError())) return e;
    hipLaunchKernelGGL(embed_segfix_kernel, dim3(chunks), dim3(256), sizeof(float) * 4 * size_t(E),
                       hipStream_t(stream), E, w.meta, keys, w.Pfirst, w.Plast, w.S);
    return int(hipGetLastError());
}

int launch_embed_dglast(const EmbedWs &w, int n, int64_t V, const float *Apre, int Ep, int R, int Vs, int Es,
                        void *stream) {
    (void)n;
    const int64_t waves = int64_t(Vs) * kEmbedChunks;
    const size_t lds = sizeof(float) * 4 * size_t(Ep * Es + Ep * R);
    hipLaunchKernelGGL(embed_dglast_kernel, dim3(unsigned((waves + 3) / 4)), dim3(256), lds, hipStream_t(stream), w.meta,
                       sorted_keys(w, V), w.S, Apre, Ep, R, Vs, Es, kEmbedChunks, w.dglast_part);
    return int(hipGetLastError());
}

int launch_embed_dapre(const EmbedWs &w, int n, int64_t V, const float *Gs, int64_t Vp, int Ep, int R, int Vs, int Es,
                       int vq, int eq, float *dA, void *stream) {
    (void)n;
    const dim3 grid(unsigned((Vp + 3) / 4));
    const uint32_t *keys = sorted_keys(w, V);
    const size_t lds = sizeof(float) * size_t(R) * Vs * Es;
    if (R <= 16)
        hipLaunchKernelGGL((embed_dapre_kernel<16>), grid, dim3(256), lds, hipStream_t(stream), w.meta, keys, w.S, Gs,
                           Vp, Ep, R, Vs, Es, vq, eq, dA);
    else if (R <= 32)
        hipLaunchKernelGGL((embed_dapre_kernel<32>), grid, dim3(256), lds, hipStream_t(stream), w.meta, keys, w.S, Gs,
                           Vp, Ep, R, Vs, Es, vq, eq, dA);
    else
        hipLaunchKernelGGL((embed_dapre_kernel<64>), grid, dim3(256), lds, hipStream_t(stream), w.meta, keys, w.S, Gs,
                           Vp, Ep, R, Vs, Es, vq, eq, dA);
    return int(hipGetLastError());
}

}  // namespace comera
