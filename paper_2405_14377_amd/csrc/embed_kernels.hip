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
// linearity): tokens are grouped by id with a stable radix sort, dY rows of
// equal ids are summed in token order (in chunks of at most kItem tokens so
// that hot ids spread over many workgroups), and the per-id sums S_u feed
//   dG_last[a, vs, es] = sum_u sum_ep A[vp_u, ep, a] S_u[ep, es]
//   dA[vp, ep, a]      = sum_{u in vp} sum_es S_u[ep, es] G_last[a, vs_u, es]
// after which dA is projected onto the prefix cores exactly like dW is for a
// linear layer.  Every sum has a fixed order, so results are bitwise
// reproducible.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "embed_internal.h"

namespace comera {
namespace {

inline int grid_for(int64_t n, int threads = 256, int64_t cap = 65536) {
    int64_t g = (n + threads - 1) / threads;
    return int(std::max<int64_t>(1, std::min<int64_t>(g, cap)));
}

// ---------------------------------------------------------------- forward rows
// One workgroup per group of tokens; the prefix row block A[vp] (Ep x r) and
// the suffix slice G_last[:, vs, :] (r x Es) are staged in LDS per token.
__global__ __launch_bounds__(256) void embed_rows_kernel(const int64_t *__restrict__ ids, int64_t n_tokens,
                                                         int64_t V, const float *__restrict__ Apre,
                                                         const float *__restrict__ Gs, float *__restrict__ Y, int Ep,
                                                         int R, int Vs, int Es, int *__restrict__ err_flag) {
    extern __shared__ float lds[];
    float *sa = lds;                 // [Ep][R]
    float *sg = lds + Ep * R;        // [R][Es]
    const int E = Ep * Es;
    for (int64_t t = blockIdx.x; t < n_tokens; t += gridDim.x) {
        const int64_t id = ids[t];
        const bool ok = id >= 0 && id < V;
        if (!ok) {
            if (threadIdx.x == 0 && err_flag) *err_flag = 1;
            for (int o = threadIdx.x; o < E; o += blockDim.x) Y[t * E + o] = 0.f;
            continue;
        }
        const int64_t vp = id / Vs;
        const int vs = int(id % Vs);
        __syncthreads();
        if (Apre) {
            const float *ap = Apre + vp * int64_t(Ep) * R;
            for (int i = threadIdx.x; i < Ep * R; i += blockDim.x) sa[i] = ap[i];
        } else {
            if (threadIdx.x == 0) sa[0] = 1.f;
        }
        for (int i = threadIdx.x; i < R * Es; i += blockDim.x) {
            int a = i / Es, es = i % Es;
            sg[i] = Gs[(int64_t(a) * Vs + vs) * Es + es];
        }
        __syncthreads();
        for (int o = threadIdx.x; o < E; o += blockDim.x) {
            const int ep = o / Es, es = o % Es;
            float acc = 0.f;
            for (int a = 0; a < R; ++a) acc += sa[ep * R + a] * sg[a * Es + es];
            Y[t * E + o] = acc;
        }
    }
}

// ---------------------------------------------------------------- sort + segments
// Single workgroup of 1024 threads.  LSD radix sort (8-bit digits) of the
// keys id (out-of-range ids get the key V and sort last), values = token
// index; each pass is stable, so equal ids keep token order.  Then the
// unique-id segments and the work items (runs of at most `item` tokens of one
// id) are listed.
constexpr int kSortThreads = 1024;
constexpr int kWaves = kSortThreads / 64;

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int lane = threadIdx.x & 63;
    return lane ? ((~0ull) >> (64 - lane)) : 0ull;
}

// exclusive block scan of one int per thread; returns the total
__device__ int block_exclusive_scan(int v, int *excl, int *wsum) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int x = v;
    for (int off = 1; off < 64; off <<= 1) {
        int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int i = 0; i < kWaves; ++i) {
            int c = wsum[i];
            wsum[i] = run;
            run += c;
        }
        wsum[kWaves] = run;
    }
    __syncthreads();
    *excl = wsum[w] + x - v;
    int total = wsum[kWaves];
    __syncthreads();
    return total;
}

__global__ __launch_bounds__(kSortThreads) void embed_sort_kernel(
    const int64_t *__restrict__ ids, int n, int64_t V, int bits, uint32_t *keysA, uint32_t *valsA, uint32_t *keysB,
    uint32_t *valsB, int *meta, int *uid, int *ustart, int *useg_item, int *item_u, int *item_beg, int *item_len,
    int *err_flag, int item) {
    __shared__ int hist[256];
    __shared__ int base[256];
    __shared__ int tile_total[256];
    __shared__ int wcount[kWaves][256];
    __shared__ int wsum[kWaves + 1];
    __shared__ int carry_s;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const uint32_t sentinel = uint32_t(V);

    uint32_t *kin = keysA, *vin = valsA, *kout = keysB, *vout = valsB;
    // pass 0 reads the ids directly
    int bad = 0;
    for (int shift = 0, pass = 0; shift < bits; shift += 8, ++pass) {
        for (int i = tid; i < 256; i += kSortThreads) hist[i] = 0;
        __syncthreads();
        for (int i = tid; i < n; i += kSortThreads) {
            uint32_t key;
            if (pass == 0) {
                int64_t id = ids[i];
                bool ok = id >= 0 && id < V;
                bad |= !ok;
                key = ok ? uint32_t(id) : sentinel;
            } else {
                key = kin[i];
            }
            atomicAdd(&hist[(key >> shift) & 255u], 1);
        }
        __syncthreads();
        if (tid == 0) {
            int run = 0;
            for (int dgt = 0; dgt < 256; ++dgt) {
                base[dgt] = run;
                run += hist[dgt];
            }
        }
        for (int i = tid; i < kWaves * 256; i += kSortThreads) (&wcount[0][0])[i] = 0;
        __syncthreads();
        for (int t0 = 0; t0 < n; t0 += kSortThreads) {
            const int i = t0 + tid;
            const bool valid = i < n;
            uint32_t key = 0, val = 0;
            if (valid) {
                if (pass == 0) {
                    int64_t id = ids[i];
                    key = (id >= 0 && id < V) ? uint32_t(id) : sentinel;
                    val = uint32_t(i);
                } else {
                    key = kin[i];
                    val = vin[i];
                }
            }
            const uint32_t dg = (key >> shift) & 255u;
            uint64_t peers = __ballot(valid);
            for (int bt = 0; bt < 8; ++bt) {
                const bool set = (dg >> bt) & 1u;
                const uint64_t bb = __ballot(valid && set);
                peers &= set ? bb : ~bb;
            }
            const int rank = __popcll(peers & lanemask_lt());
            if (valid && rank == 0) wcount[w][dg] = __popcll(peers);
            __syncthreads();
            if (tid < 256) {
                int run = 0;
                for (int ww = 0; ww < kWaves; ++ww) {
                    int c = wcount[ww][tid];
                    wcount[ww][tid] = run;
                    run += c;
                }
                tile_total[tid] = run;
            }
            __syncthreads();
            if (valid) {
                const int pos = base[dg] + wcount[w][dg] + rank;
                kout[pos] = key;
                vout[pos] = val;
            }
            __syncthreads();
            if (tid < 256) base[tid] += tile_total[tid];
            for (int i2 = tid; i2 < kWaves * 256; i2 += kSortThreads) (&wcount[0][0])[i2] = 0;
            __syncthreads();
        }
        // the next pass reads what this one wrote
        uint32_t *tk = kin, *tv = vin;
        kin = kout;
        vin = vout;
        kout = tk;
        vout = tv;
        __syncthreads();
    }
    // after the loop the sorted data is in (kin, vin)
    if (bad && err_flag) *err_flag = 1;
    // record which buffer holds the result: 0 = A, 1 = B
    if (tid == 0) meta[3] = (kin == keysA) ? 0 : 1;

    // unique-id segments
    if (tid == 0) carry_s = 0;
    __syncthreads();
    int nvalid_local = 0;
    for (int t0 = 0; t0 < n; t0 += kSortThreads) {
        const int i = t0 + tid;
        uint32_t key = i < n ? kin[i] : sentinel;
        const bool valid = i < n && key != sentinel;
        nvalid_local += valid;
        const bool head = valid && (i == 0 || kin[i - 1] != key);
        int excl;
        int total = block_exclusive_scan(head ? 1 : 0, &excl, wsum);
        const int carry = carry_s;
        if (head) {
            uid[carry + excl] = int(key);
            ustart[carry + excl] = i;
        }
        __syncthreads();
        if (tid == 0) carry_s = carry + total;
        __syncthreads();
    }
    int nv_excl;
    const int n_valid = block_exclusive_scan(nvalid_local, &nv_excl, wsum);
    const int U = carry_s;
    if (tid == 0) {
        ustart[U] = n_valid;
        meta[0] = U;
        meta[2] = n_valid;
        carry_s = 0;
    }
    __syncthreads();
    // work items per segment
    for (int u0 = 0; u0 < U; u0 += kSortThreads) {
        const int u = u0 + tid;
        int cnt = 0, beg = 0, len = 0;
        if (u < U) {
            beg = ustart[u];
            len = ustart[u + 1] - beg;
            cnt = (len + item - 1) / item;
        }
        int excl;
        int total = block_exclusive_scan(cnt, &excl, wsum);
        const int carry = carry_s;
        if (u < U) {
            useg_item[u] = carry + excl;
            for (int j = 0; j < cnt; ++j) {
                item_u[carry + excl + j] = u;
                item_beg[carry + excl + j] = beg + j * item;
                item_len[carry + excl + j] = min(item, len - j * item);
            }
        }
        __syncthreads();
        if (tid == 0) carry_s = carry + total;
        __syncthreads();
    }
    if (tid == 0) {
        useg_item[U] = carry_s;
        meta[1] = carry_s;
    }
}

// Sum the dY rows of each work item (token order).  A segment with a single
// item writes its sum straight to S[u]; otherwise to Spart[item].
__global__ __launch_bounds__(256) void embed_segsum_kernel(const float *__restrict__ dY, int E, const int *meta,
                                                           const uint32_t *keysA, const uint32_t *valsA,
                                                           const uint32_t *valsB, const int *useg_item,
                                                           const int *item_u, const int *item_beg,
                                                           const int *item_len, float *__restrict__ S,
                                                           float *__restrict__ Spart) {
    const int n_items = meta[1];
    const uint32_t *vals = meta[3] == 0 ? valsA : valsB;
    for (int it = blockIdx.x; it < n_items; it += gridDim.x) {
        const int u = item_u[it];
        const int beg = item_beg[it], len = item_len[it];
        const bool single = (useg_item[u + 1] - useg_item[u]) == 1;
        float *dst = single ? S + int64_t(u) * E : Spart + int64_t(it) * E;
        for (int c = threadIdx.x; c < E; c += blockDim.x) {
            float acc = 0.f;
            for (int j = 0; j < len; ++j) acc += dY[int64_t(vals[beg + j]) * E + c];
            dst[c] = acc;
        }
    }
}

// S[u] = sum of the item partials of u in order, for segments with > 1 item
__global__ __launch_bounds__(256) void embed_idsum_kernel(int E, const int *meta, const int *useg_item,
                                                          const float *__restrict__ Spart, float *__restrict__ S) {
    const int U = meta[0];
    for (int u = blockIdx.x; u < U; u += gridDim.x) {
        const int i0 = useg_item[u], i1 = useg_item[u + 1];
        if (i1 - i0 <= 1) continue;
        for (int c = threadIdx.x; c < E; c += blockDim.x) {
            float acc = 0.f;
            for (int it = i0; it < i1; ++it) acc += Spart[int64_t(it) * E + c];
            S[int64_t(u) * E + c] = acc;
        }
    }
}

// dG_last partials: workgroup c of `chunks` takes unique ids
// [c*U/chunks, (c+1)*U/chunks) and accumulates into LDS [R][Vs][Es].
__global__ __launch_bounds__(256) void embed_dglast_kernel(const int *meta, const int *uid,
                                                           const float *__restrict__ S,
                                                           const float *__restrict__ Apre, int Ep, int R, int Vs,
                                                           int Es, int chunks, float *__restrict__ part) {
    extern __shared__ float acc_s[];  // [R][Vs][Es]
    const int U = meta[0];
    const int c = blockIdx.x;
    const int u0 = int(int64_t(c) * U / chunks), u1 = int(int64_t(c + 1) * U / chunks);
    const int tot = R * Vs * Es;
    for (int i = threadIdx.x; i < tot; i += blockDim.x) acc_s[i] = 0.f;
    __syncthreads();
    const int E = Ep * Es;
    for (int u = u0; u < u1; ++u) {
        const int id = uid[u];
        const int64_t vp = id / Vs;
        const int vs = id % Vs;
        const float *srow = S + int64_t(u) * E;
        const float *ap = Apre ? Apre + vp * int64_t(Ep) * R : nullptr;
        for (int o = threadIdx.x; o < R * Es; o += blockDim.x) {
            const int a = o / Es, es = o % Es;
            float v = 0.f;
            for (int ep = 0; ep < Ep; ++ep) v += (ap ? ap[ep * R + a] : 1.f) * srow[ep * Es + es];
            acc_s[(a * Vs + vs) * Es + es] += v;
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < tot; i += blockDim.x) part[int64_t(c) * tot + i] = acc_s[i];
}

// dA[vp, ep, a] over the unique ids whose prefix is vp (binary search in the
// sorted unique list); prefixes with no id get zeros.
__global__ __launch_bounds__(256) void embed_dapre_kernel(const int *meta, const int *uid,
                                                          const float *__restrict__ S, const float *__restrict__ Gs,
                                                          int64_t Vp, int Ep, int R, int Vs, int Es,
                                                          float *__restrict__ dA) {
    const int U = meta[0];
    const int E = Ep * Es;
    for (int64_t vp = blockIdx.x; vp < Vp; vp += gridDim.x) {
        // first u with uid[u] >= vp * Vs, then first with uid[u] >= (vp + 1) * Vs
        auto lower = [&](int64_t key) {
            int lo = 0, hi = U;
            while (lo < hi) {
                int mid = (lo + hi) >> 1;
                if (int64_t(uid[mid]) < key) lo = mid + 1;
                else hi = mid;
            }
            return lo;
        };
        const int ub = lower(vp * Vs), ue = lower((vp + 1) * Vs);
        for (int o = threadIdx.x; o < Ep * R; o += blockDim.x) {
            const int ep = o / R, a = o % R;
            float acc = 0.f;
            for (int u = ub; u < ue; ++u) {
                const int vs = uid[u] % Vs;
                const float *srow = S + int64_t(u) * E + ep * Es;
                const float *g = Gs + (int64_t(a) * Vs + vs) * Es;
                for (int es = 0; es < Es; ++es) acc += srow[es] * g[es];
            }
            dA[vp * int64_t(Ep) * R + o] = acc;
        }
    }
}

}  // namespace

int launch_embed_rows(const int64_t *ids, int64_t n, int64_t V, const float *Apre, const float *Gs, float *Y, int Ep,
                      int R, int Vs, int Es, int *err_flag, void *stream) {
    if (n <= 0) return 0;
    size_t lds = sizeof(float) * (size_t(Ep) * R + size_t(R) * Es);
    int grid = int(std::min<int64_t>(n, 8192));
    hipLaunchKernelGGL(embed_rows_kernel, dim3(grid), dim3(256), lds, hipStream_t(stream), ids, n, V, Apre, Gs, Y,
                       Ep, R, Vs, Es, err_flag);
    return int(hipGetLastError());
}

int launch_embed_sort(const int64_t *ids, int n, int64_t V, const EmbedWs &w, int *err_flag, void *stream) {
    int bits = 0;
    while ((int64_t(1) << bits) <= V) ++bits;  // keys 0..V inclusive (V = sentinel)
    hipLaunchKernelGGL(embed_sort_kernel, dim3(1), dim3(kSortThreads), 0, hipStream_t(stream), ids, n, V, bits,
                       w.keysA, w.valsA, w.keysB, w.valsB, w.meta, w.uid, w.ustart, w.useg_item, w.item_u,
                       w.item_beg, w.item_len, err_flag, kEmbedItem);
    return int(hipGetLastError());
}

int launch_embed_segsum(const float *dY, int E, int n, const EmbedWs &w, void *stream) {
    int grid = std::max(1, std::min(n, 16384));
    hipLaunchKernelGGL(embed_segsum_kernel, dim3(grid), dim3(256), 0, hipStream_t(stream), dY, E, w.meta, w.keysA,
                       w.valsA, w.valsB, w.useg_item, w.item_u, w.item_beg, w.item_len, w.S, w.Spart);
    if (int e = int(hipGetLastError())) return e;
    hipLaunchKernelGGL(embed_idsum_kernel, dim3(grid), dim3(256), 0, hipStream_t(stream), E, w.meta, w.useg_item,
                       w.Spart, w.S);
    return int(hipGetLastError());
}

int launch_embed_dglast(const EmbedWs &w, const float *Apre, int Ep, int R, int Vs, int Es, void *stream) {
    size_t lds = sizeof(float) * size_t(R) * Vs * Es;
    hipLaunchKernelGGL(embed_dglast_kernel, dim3(kEmbedChunks), dim3(256), lds, hipStream_t(stream), w.meta, w.uid,
                       w.S, Apre, Ep, R, Vs, Es, kEmbedChunks, w.dglast_part);
    return int(hipGetLastError());
}

int launch_embed_dapre(const EmbedWs &w, const float *Gs, int64_t Vp, int Ep, int R, int Vs, int Es, float *dA,
                       void *stream) {
    int grid = int(std::max<int64_t>(1, std::min<int64_t>(Vp, 65536)));
    hipLaunchKernelGGL(embed_dapre_kernel, dim3(grid), dim3(256), 0, hipStream_t(stream), w.meta, w.uid, w.S, Gs, Vp,
                       Ep, R, Vs, Es, dA);
    return int(hipGetLastError());
}

}  // namespace comera
