// Fused batch-free build of a three-core layer (eq. TTM with the rank masks
// folded in as in eq. Wcompress), one launch:
//   folded cores  G~_k = G_k with its right bond scaled by D_k and both bonds
//                 compacted to their active entries (written out for the
//                 backward's projections),
//   left chain    P_2[(x0 x1)][(y0 y1)][c] = sum_a G~_0[x0 y0 a] G~_1[a x1 y1 c],
//   W             W[(x0 x1 x2)][(y0 y1 y2)] = sum_c P_2[(x0 x1)(y0 y1)][c] G~_2[c x2 y2]
// as W [N_in][N_out] and / or W^T [N_out][N_in], fp32 or bf16 (x_k runs over
// the input factor n_k, y_k over the output factor m_k).
//
// A workgroup of eight waves owns SX x SY slices (x1, y1) of the middle core
// and PX x PY pairs (x0, y0) of the first: R = SX SY PX PY <= 64 rows
// (slice, pair) of P_2.  Every global load of the workgroup is issued before
// any is used (the bond maps come as kernel arguments for uniform indices
// and from the active bits per lane, so no address waits on LDS): the last
// core, the pair rows of G~_0, and per thread one (slice, c) item, the
// slice's column c of G~_1 (rank A values straight from the raw core, the
// mask applied) that it contracts with the PP pair rows, so the middle core,
// the largest of the three, is read once per pair block and never staged.
// The R x C rows of P_2 then meet the last core (C x n2 m2, staged
// transposed) on v_mfma_f32_16x16x4f32, each 16-row block split over two
// waves by columns; the tile goes through LDS and out as runs of SY m2
// consecutive entries of W rows and SX n2 of W^T rows, four entries per
// store where the factors allow it.  Tiles divide the factors exactly.
//
// Replaces three launches (fold, chain step, W tile) of a d = 3 layer whose
// compacted ranks are at most 64 and whose last core has at most 256
// entries per rank pair.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "internal.h"

namespace comera {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kB3Threads = 512;     // eight waves: two per SIMD
constexpr int kB3Rows = 64;         // (slice, pair) rows of a workgroup: four 16-row MFMA blocks
constexpr int kB3MaxRank = 64;
constexpr int kB3MaxNC = 256;       // n_2 m_2
constexpr int kB3MaxPairs = 16;
constexpr size_t kB3Lds = 96 * 1024;

__host__ __device__ inline int b3_r16(int x) { return (x + 15) & ~15; }

// LDS floats for KK = the larger compacted rank rounded up to 16: the last
// core transposed [NC16][KK + 4], the P_2 rows [64][KK + 4], the pair rows of
// G~_0 [PP][KK] and the output tile [64][NC16 + 4]
__host__ __device__ inline size_t b3_lds_floats(int KK, int NC, int PP) {
    const int pk = KK + 4, NC16 = b3_r16(NC);
    return size_t(NC16) * pk + size_t(kB3Rows) * pk + size_t(PP) * KK + size_t(kB3Rows) * (NC16 + 4);
}
// (slice, rank) items of a workgroup: one per thread, loaded up front
__host__ __device__ inline int b3_max_items(int) { return kB3Threads; }

// two floats -> two bf16 (round to nearest even) in one dword, a low: one
// v_cvt_pk_bf16_f32
typedef __bf16 b3_bf16x2 __attribute__((ext_vector_type(2)));
typedef float b3_f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t b3_pack2(float a, float b) {
    const b3_f32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, b3_bf16x2));
}

// full index of the k-th active entry of a bond (k below the active count),
// per lane: the word by the running popcounts, then a binary search
__device__ __forceinline__ int b3_kth(const BondBits &b, int k) {
    const int c0 = __popcll(b.w[0]), c1 = c0 + __popcll(b.w[1]), c2 = c1 + __popcll(b.w[2]);
    const uint64_t w = k < c0 ? b.w[0] : k < c1 ? b.w[1] : k < c2 ? b.w[2] : b.w[3];
    int kk = k < c0 ? k : k < c1 ? k - c0 : k < c2 ? k - c1 : k - c2;
    int pos = 0;
#pragma unroll
    for (int h = 32; h >= 1; h >>= 1) {
        const int cnt = __popcll((w >> pos) & ((uint64_t(1) << h) - 1));
        const bool up = kk >= cnt;
        kk -= up ? cnt : 0;
        pos += up ? h : 0;
    }
    return (k < c0 ? 0 : k < c1 ? 64 : k < c2 ? 128 : 192) + pos;
}

// one output piece: V consecutive entries (V = 4: 16 bytes fp32 / 8 bf16)
template <int V, int BF>
__device__ __forceinline__ void b3_put(void *out, int off, float e0, float e1, float e2, float e3) {
    if (V == 4) {
        if (BF) {
            uint2 u;
            u.x = b3_pack2(e0, e1);
            u.y = b3_pack2(e2, e3);
            *reinterpret_cast<uint2 *>(reinterpret_cast<uint16_t *>(out) + off) = u;
        } else {
            *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(out) + off) = f32x4{e0, e1, e2, e3};
        }
    } else if (BF) {
        reinterpret_cast<uint16_t *>(out)[off] = uint16_t(b3_pack2(e0, 0.f) & 0xffffu);
    } else {
        reinterpret_cast<float *>(out)[off] = e0;
    }
}

// Geometry of a workgroup's tile for the write-out.
struct B3Tile {
    int n1, n2, m1, m2, SX, SY, PX, PY, PP, tp;
    int x0b, y0b, x1b, y1b, Nin, Nout;
};

// Write-out of one layout.  A run is the part of one output row the tile
// holds: for W, row (x0, x1, x2) and entries (y1, y2) of one y0; for W^T,
// row (y0, y1, y2) and entries (x1, x2) of one x0.  Runs are numbered by
// four digits (rad, least significant first); a run has QL pieces of V
// entries.  Where QL <= 64, every lane keeps one piece index for good and
// the runs advance by a constant step (digits added with carries); else the
// pieces are numbered flat over the workgroup.
template <int V, int BF, bool T>
__device__ __forceinline__ void b3_write(const B3Tile &g, const float *tile, void *out, int tid) {
    const int lane = tid & 63, wave = tid >> 6;
    constexpr int NW = kB3Threads / 64;
    // W: pieces over e = (sy, y2) in [0, SY m2); W^T: e = (sx, x2) in [0, SX n2)
    const int ext = T ? g.n2 : g.m2, ES = T ? g.SX : g.SY;
    const int QL = ES * ext / V;
    const int rad0 = T ? g.PX : g.PY, rad1 = T ? g.m2 : g.n2, rad2 = T ? g.SY : g.SX;
    const int nruns = rad0 * rad1 * rad2 * (T ? g.PY : g.PX);
    auto piece = [&](int d0, int d1, int d2, int d3, int e) {
        const int hi = e / ext, lo = e - hi * ext;
        if (!T) {
            const int py = d0, x2 = d1, sx = d2, px = d3, sy = hi, y2 = lo;
            const float *src = tile + ((sx * g.SY + sy) * g.PP + px * g.PY + py) * g.tp + x2 * g.m2 + y2;
            const int gi = ((g.x0b + px) * g.n1 + g.x1b + sx) * g.n2 + x2;
            const int off = gi * g.Nout + ((g.y0b + py) * g.m1 + g.y1b) * g.m2 + e;
            if (V == 4) {
                const f32x4 v = *reinterpret_cast<const f32x4 *>(src);
                b3_put<V, BF>(out, off, v[0], v[1], v[2], v[3]);
            } else {
                b3_put<V, BF>(out, off, *src, 0.f, 0.f, 0.f);
            }
        } else {
            const int px = d0, y2 = d1, sy = d2, py = d3, sx = hi, x2 = lo;
            const float *src = tile + ((sx * g.SY + sy) * g.PP + px * g.PY + py) * g.tp + x2 * g.m2 + y2;
            const int gj = ((g.y0b + py) * g.m1 + g.y1b + sy) * g.m2 + y2;
            const int off = gj * g.Nin + ((g.x0b + px) * g.n1 + g.x1b) * g.n2 + e;
            if (V == 4)
                b3_put<V, BF>(out, off, src[0], src[g.m2], src[2 * g.m2], src[3 * g.m2]);
            else
                b3_put<V, BF>(out, off, *src, 0.f, 0.f, 0.f);
        }
    };
    if (QL <= 64) {
        const int QLP = QL <= 1 ? 1 : 1 << (32 - __clz(QL - 1)), RPW = 64 / QLP;
        const int q = lane & (QLP - 1), sub = lane / QLP;
        if (q >= QL) return;
        const int e = V * q, step = NW * RPW;
        int r = wave * RPW + sub;
        int d0 = r % rad0, t = r / rad0, d1 = t % rad1;
        t /= rad1;
        int d2 = t % rad2, d3 = t / rad2;
        const int s0 = step % rad0, s1 = (step / rad0) % rad1, s2 = (step / (rad0 * rad1)) % rad2,
                  s3 = step / (rad0 * rad1 * rad2);
#pragma unroll 4
        for (; r < nruns; r += step) {
            piece(d0, d1, d2, d3, e);
            int c;
            d0 += s0;
            c = d0 >= rad0;
            d0 -= c ? rad0 : 0;
            d1 += s1 + c;
            c = d1 >= rad1;
            d1 -= c ? rad1 : 0;
            d2 += s2 + c;
            c = d2 >= rad2;
            d2 -= c ? rad2 : 0;
            d3 += s3 + c;
        }
    } else {
        const int total = nruns * QL;
        for (int f = tid; f < total; f += kB3Threads) {
            const int r = f / QL, q = f - r * QL;
            const int d0 = r % rad0, t = r / rad0, d1 = t % rad1, t2 = t / rad1, d2 = t2 % rad2, d3 = t2 / rad2;
            piece(d0, d1, d2, d3, V * q);
        }
    }
}

template <int KK, int BF>
__global__ __launch_bounds__(kB3Threads) void build3_kernel(Build3Args a) {
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int A = a.A, C = a.C;
    const int n0 = a.n[0], n1 = a.n[1], n2 = a.n[2], m0 = a.m[0], m1 = a.m[1], m2 = a.m[2];
    const int SX = a.SX, SY = a.SY, PX = a.PX, PY = a.PY;
    const int S = SX * SY, PP = PX * PY, R = S * PP;
    const int NC = n2 * m2, NC16 = b3_r16(NC), pk = KK + 4, tp = NC16 + 4;
    float *Gt = sm;                              // [NC16][pk]: G~_2[c][x2 y2] at (x2 m2 + y2, c)
    float *Ps = Gt + NC16 * pk;                  // [64][pk]: P_2 row (s PP + p), rank c
    float *P1s = Ps + kB3Rows * pk;              // [PP][KK]
    float *tile = P1s + PP * KK;                 // [64][tp]
    const bool cmp = a.compacted != 0;

    // tile of this workgroup: consecutive tiles (slice blocks fastest) on
    // one XCD, so the W rows they share meet in one L2
    const int gsy = m1 / SY, gsx = n1 / SX, gpx = n0 / PX;
    const int T = int(gridDim.x), b = int(blockIdx.x);
    const int L = (T % 8 == 0) ? (b % 8) * (T / 8) + b / 8 : b;
    const int syb = L % gsy, sxb = (L / gsy) % gsx, pxb = (L / (gsy * gsx)) % gpx, pyb = L / (gsy * gsx * gpx);
    const int x1b = sxb * SX, y1b = syb * SY, x0b = pxb * PX, y0b = pyb * PY;
    const bool wr0 = sxb == 0 && syb == 0;       // writes its pairs' rows of G~_0
    const bool wr1 = pxb == 0 && pyb == 0;       // writes its slices of G~_1
    const bool wr2 = wr0 && wr1;                 // writes G~_2

    // ---- every global load of the workgroup is issued before any is used
    // (one round trip): the bond maps come as kernel arguments (uniform
    // entries) or from the active-entry bits (per lane)
    // (1) raw column q = y2 n2 + x2 of the last core: ranks [0, KK/2) by
    // threads q, [KK/2, KK) by threads 256 + q
    constexpr int KH = KK / 2;
    const int gq = tid & 255, gh = tid >> 8;
    const bool gin = gq < NC;
    float gv[KH];
    if (gq < NC16) {    // whole waves past the last row skip the loads
        const float *G2 = a.G[2] + (gin ? gq : 0);
#pragma unroll
        for (int j = 0; j < KH; ++j) {
            const int c = gh * KH + j;
            gv[j] = G2[int(a.map2[c < C ? c : 0]) * NC];
        }
    }
    // (2) pair rows of G~_0: entry i = (p, al), two per thread at most
    float pv[2], pd[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int i = tid + u * kB3Threads;
        const int p = i / KK, al = i - p * KK;
        const bool ok = p < PP && al < A;
        const int fa = ok ? (cmp ? b3_kth(a.act1, al) : al) : 0;
        const int px = ok ? p / PY : 0, py = ok ? p - px * PY : 0;
        pv[u] = a.G[0][((y0b + py) * n0 + x0b + px) * a.r1 + fa];
        pd[u] = a.D[0] ? a.D[0][fa] : 1.f;
    }
    // (3) the middle core's column c of slice s for item it = tid; entries
    // past A up to the next multiple of four read an active entry (they
    // meet zeros in the pair rows), the rest are left at zero by leaving the
    // loop (uniform branches: per-entry tests were hoisted out of the loop
    // by the compiler and spilled)
    const int nit = S * C;
    float g0[KK], dc0 = 0.f;
#pragma unroll
    for (int al = 0; al < KK; ++al) g0[al] = 0.f;
    const int strA = m1 * n1 * a.r2;             // raw stride of the middle core's left bond
    if (tid < nit) {
        const int s = tid / C, c = tid - s * C;
        const int sx = s / SY, sy = s - sx * SY;
        const int fc = cmp ? b3_kth(a.act2, c) : c;
        const float *base = a.G[1] + ((y1b + sy) * n1 + x1b + sx) * a.r2 + fc;
        dc0 = a.D[1] ? a.D[1][fc] : 1.f;
#pragma unroll
        for (int q = 0; q < KK / 4; ++q) {
            if (4 * q >= A) break;
#pragma unroll
            for (int j = 0; j < 4; ++j) g0[4 * q + j] = base[int(a.map1[4 * q + j]) * strA];
        }
    }

    // ---- staging: the last core transposed (rows NC .. NC16 - 1 and ranks
    // C .. KK - 1 zero), the pair rows (entries past A zero)
    if (gq < NC16) {
        const int y2 = gin ? gq / n2 : 0, x2 = gin ? gq - y2 * n2 : 0;
        float *dst = Gt + (gin ? x2 * m2 + y2 : gq) * pk + gh * KH;
#pragma unroll
        for (int j = 0; j < KH; j += 4) {
            const int c = gh * KH + j;
            *reinterpret_cast<f32x4 *>(dst + j) =
                f32x4{(gin && c < C) ? gv[j] : 0.f, (gin && c + 1 < C) ? gv[j + 1] : 0.f,
                      (gin && c + 2 < C) ? gv[j + 2] : 0.f, (gin && c + 3 < C) ? gv[j + 3] : 0.f};
        }
        if (wr2 && gin) {
            const CoreStrides st = a.st[2];
            float *gc = a.Gc[2] + y2 * st.sm + x2 * st.sn + gh * KH * st.sa;
#pragma unroll
            for (int j = 0; j < KH; ++j) {
                if (gh * KH + j >= C) break;
                gc[j * st.sa] = gv[j];
            }
        }
    }
    {
        const CoreStrides st = a.st[0];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int i = tid + u * kB3Threads;
            const int p = i / KK, al = i - p * KK;
            if (p < PP) {
                const float v = al < A ? pv[u] * pd[u] : 0.f;
                P1s[i] = v;
                if (wr0 && al < A) {
                    const int px = p / PY, py = p - px * PY;
                    a.Gc[0][(y0b + py) * st.sm + (x0b + px) * st.sn + al * st.sc] = v;
                }
            }
        }
    }
    __syncthreads();

    // ---- P_2 rows: each item's column of G~_1 (mask applied) against every
    // pair row; written to LDS for the products, to P_2 and (once) to G~_1
    {
        const CoreStrides st = a.st[1];
        const int NJ = m0 * m1;
        auto item = [&](int it, const float *g, float dc) {
            const int s = it / C, c = it - s * C;
            const int sx = s / SY, sy = s - sx * SY;
            const int x1 = x1b + sx, y1 = y1b + sy;
            float gm[KK];
#pragma unroll
            for (int al = 0; al < KK; ++al) gm[al] = g[al] * dc;
            if (wr1) {
                float *dst = a.Gc[1] + x1 * st.sn + y1 * st.sm + c * st.sc;
#pragma unroll
                for (int al = 0; al < KK; ++al) {
                    if (al >= A) break;
                    dst[al * st.sa] = gm[al];
                }
            }
            for (int p = 0; p < PP; ++p) {
                const float *pr = P1s + p * KK;
                float acc = 0.f;
#pragma unroll
                for (int q = 0; q < KK / 4; ++q) {
                    const f32x4 x = *reinterpret_cast<const f32x4 *>(pr + 4 * q);
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc = fmaf(x[j], gm[4 * q + j], acc);
                }
                Ps[(s * PP + p) * pk + c] = acc;
                const int px = p / PY, py = p - px * PY;
                const int I = (x0b + px) * n1 + x1, J = (y0b + py) * m1 + y1;
                a.P2[(I * NJ + J) * C + c] = acc;
            }
        };
        if (tid < nit) item(tid, g0, dc0);
        // zero padding: ranks C .. KK - 1 of the rows in use, rows R .. 63
        const int padc = KK - C;
        for (int i = tid; i < R * padc; i += kB3Threads) {
            const int r = i / padc;
            Ps[r * pk + C + (i - r * padc)] = 0.f;
        }
        for (int i = tid; i < (kB3Rows - R) * KK; i += kB3Threads) Ps[(R + i / KK) * pk + i % KK] = 0.f;
    }
    __syncthreads();

    // ---- W tile = P_2 rows x G~_2 on 16x16x4 MFMA, one 16-column block at
    // a time (k = 16 g + 4 q + j: one 16-byte read per operand), straight
    // into the tile
    if ((wave & 3) * 16 < R) {
        const int li = lane & 15, lq = lane >> 4, rb = wave & 3;
        const float *pa = Ps + (rb * 16 + li) * pk + 4 * lq;
        float *to = tile + (rb * 16 + 4 * lq) * tp + li;
        const int NB = NC16 / 16;
#pragma unroll 2
        for (int t = wave >> 2; t < NB; t += kB3Threads / 256) {
            const float *pb = Gt + (t * 16 + li) * pk + 4 * lq;
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int g = 0; g < KK / 16; ++g) {
                const f32x4 x = *reinterpret_cast<const f32x4 *>(pa + 16 * g);
                const f32x4 y = *reinterpret_cast<const f32x4 *>(pb + 16 * g);
#pragma unroll
                for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(x[j], y[j], acc, 0, 0, 0);
            }
#pragma unroll
            for (int v = 0; v < 4; ++v) to[v * tp + t * 16] = acc[v];
        }
    }
    __syncthreads();

    // ---- write-out
    B3Tile g;
    g.n1 = n1;
    g.n2 = n2;
    g.m1 = m1;
    g.m2 = m2;
    g.SX = SX;
    g.SY = SY;
    g.PX = PX;
    g.PY = PY;
    g.PP = PP;
    g.tp = tp;
    g.x0b = x0b;
    g.y0b = y0b;
    g.x1b = x1b;
    g.y1b = y1b;
    g.Nin = n0 * n1 * n2;                        // Nin * Nout < 2^31 (host check)
    g.Nout = m0 * m1 * m2;
    if (a.w) {
        if (a.vec_w)
            b3_write<4, BF, false>(g, tile, a.w, tid);
        else
            b3_write<1, BF, false>(g, tile, a.w, tid);
    }
    if (a.wt) {
        if (a.vec_t)
            b3_write<4, BF, true>(g, tile, a.wt, tid);
        else
            b3_write<1, BF, true>(g, tile, a.wt, tid);
    }
}

template <int KK, int BF>
int launch_b3(const Build3Args &b, size_t lds, int64_t nwg, void *stream) {
    static int set = -1;     // the LDS limit, once per instantiation
    if (!launch_check_mode() && set != 0) {
        set = int(hipFuncSetAttribute(reinterpret_cast<const void *>(build3_kernel<KK, BF>),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, int(kB3Lds)));
        if (set) return set;
    }
    COMERA_LAUNCH_NAMED("build3_kernel", (build3_kernel<KK, BF>), dim3(unsigned(nwg)), dim3(kB3Threads), lds,
                        hipStream_t(stream), b);
    return launch_status();
}

}  // namespace

bool build3_tiles(const int *n, const int *m, int A, int C, int &SX, int &SY, int &PX, int &PY) {
    if (A < 1 || A > kB3MaxRank || C < 1 || C > kB3MaxRank) return false;
    for (int k = 0; k < 3; ++k)
        if (n[k] < 1 || m[k] < 1) return false;
    const int NC = n[2] * m[2];
    if (NC > kB3MaxNC) return false;
    const int KK = std::max(b3_r16(A), b3_r16(C));
    // every tile divides the factors; prefer (in order) at least 16 rows per
    // workgroup (one whole MFMA block), a grid of at least 256 workgroups,
    // more rows, output runs of at least 48 entries in both layouts, fewer
    // middle-core slices per workgroup
    auto divs = [](int x, int cap, int *out) {
        int c = 0;
        for (int v = 1; v <= std::min(x, cap); ++v)
            if (x % v == 0) out[c++] = v;
        return c;
    };
    int dsx[kB3Rows], dsy[kB3Rows], dpx[kB3Rows], dpy[kB3Rows];
    const int nsx = divs(n[1], kB3Rows, dsx), nsy = divs(m[1], kB3Rows, dsy);
    const int npx = divs(n[0], kB3MaxPairs, dpx), npy = divs(m[0], kB3MaxPairs, dpy);
    int64_t best = -1;
    for (int i = 0; i < nsx; ++i)
        for (int j = 0; j < nsy; ++j)
            for (int k = 0; k < npx; ++k)
                for (int l = 0; l < npy; ++l) {
                    const int sx = dsx[i], sy = dsy[j], px = dpx[k], py = dpy[l];
                    const int R = sx * sy * px * py;
                    if (R > kB3Rows || px * py > kB3MaxPairs || sx * sy * C > b3_max_items(KK)) continue;
                    if (b3_lds_floats(KK, NC, px * py) * sizeof(float) > kB3Lds) continue;
                    const int64_t nwg = int64_t(n[1] / sx) * (m[1] / sy) * (n[0] / px) * (m[0] / py);
                    const int runw = sy == m[1] ? py * m[1] * m[2] : sy * m[2];
                    const int runt = sx == n[1] ? px * n[1] * n[2] : sx * n[2];
                    const int64_t score = int64_t(std::min(R, 16)) * (int64_t(1) << 42) +
                                          std::min<int64_t>(nwg, 256) * (int64_t(1) << 32) +
                                          int64_t(R) * (int64_t(1) << 20) +
                                          int64_t(std::min(48, std::min(runw, runt))) * (int64_t(1) << 10) +
                                          (kB3Rows - sx * sy);
                    if (score > best) {
                        best = score;
                        SX = sx;
                        SY = sy;
                        PX = px;
                        PY = py;
                    }
                }
    return best >= 0;
}

int launch_build3(const Build3Args &a, void *stream) {
    if (!a.w && !a.wt) return int(hipErrorInvalidValue);
    const int A = a.A, C = a.C, NC = a.n[2] * a.m[2];
    if (A < 1 || A > kB3MaxRank || C < 1 || C > kB3MaxRank || NC < 1 || NC > kB3MaxNC) return int(hipErrorInvalidValue);
    if (a.SX < 1 || a.SY < 1 || a.PX < 1 || a.PY < 1 || a.n[1] % a.SX || a.m[1] % a.SY || a.n[0] % a.PX ||
        a.m[0] % a.PY)
        return int(hipErrorInvalidValue);
    const int PP = a.PX * a.PY, KK = std::max(b3_r16(A), b3_r16(C));
    if (a.SX * a.SY * PP > kB3Rows || PP > kB3MaxPairs || a.SX * a.SY * C > b3_max_items(KK))
        return int(hipErrorInvalidValue);
    // compacted bonds are at most 256 wide (their active bits); uncompacted
    // ranks are the compacted ones (at most 64)
    if (a.compacted ? (a.r1 > 256 || a.r2 > 256) : (a.r1 != A || a.r2 != C)) return int(hipErrorInvalidValue);
    if (!a.G[0] || !a.G[1] || !a.G[2] || !a.Gc[0] || !a.Gc[1] || !a.Gc[2] || !a.P2) return int(hipErrorInvalidValue);
    // raw middle-core, W and P_2 offsets are 32-bit
    const int64_t nw = int64_t(a.n[0]) * a.n[1] * a.n[2] * a.m[0] * a.m[1] * a.m[2];
    const int64_t np2 = int64_t(a.n[0]) * a.n[1] * a.m[0] * a.m[1] * C;
    if (int64_t(a.r1) * a.m[1] * a.n[1] * a.r2 >= (int64_t(1) << 31) || nw >= (int64_t(1) << 31) ||
        np2 >= (int64_t(1) << 31))
        return int(hipErrorInvalidValue);
    const size_t lds = b3_lds_floats(KK, NC, PP) * sizeof(float);
    if (lds > kB3Lds) return int(hipErrorInvalidValue);
    const int64_t nwg = int64_t(a.n[1] / a.SX) * (a.m[1] / a.SY) * (a.n[0] / a.PX) * (a.m[0] / a.PY);
    if (nwg < 1 || nwg >= (int64_t(1) << 31)) return int(hipErrorInvalidValue);
    Build3Args b = a;
    // bond maps (compacted entry -> full entry) from the active bits; the
    // entries past the rank repeat the first active one (they are read in
    // whole groups of four and meet zeros)
    auto fill = [&](const BondBits &bits, int r, int rc, uint8_t *map) -> bool {
        int k = 0;
        for (int e = 0; e < r && k < 64; ++e)
            if (!a.compacted || ((bits.w[e >> 6] >> (e & 63)) & 1)) map[k++] = uint8_t(e);
        if (k != rc) return false;
        for (; k < 64; ++k) map[k] = map[0];
        return true;
    };
    if (!fill(a.act1, a.r1, A, b.map1) || !fill(a.act2, a.r2, C, b.map2)) return int(hipErrorInvalidValue);
    // four entries per store where the runs and the addresses allow it
    const uintptr_t al = a.out_bf16 ? 7 : 15;
    b.vec_w = a.w && a.m[2] % 4 == 0 && (reinterpret_cast<uintptr_t>(a.w) & al) == 0;
    b.vec_t = a.wt && a.n[2] % 4 == 0 && (reinterpret_cast<uintptr_t>(a.wt) & al) == 0;
    const bool bf = a.out_bf16 != 0;
    switch (KK) {
        case 16: return bf ? launch_b3<16, 1>(b, lds, nwg, stream) : launch_b3<16, 0>(b, lds, nwg, stream);
        case 32: return bf ? launch_b3<32, 1>(b, lds, nwg, stream) : launch_b3<32, 0>(b, lds, nwg, stream);
        case 48: return bf ? launch_b3<48, 1>(b, lds, nwg, stream) : launch_b3<48, 0>(b, lds, nwg, stream);
        default: return bf ? launch_b3<64, 1>(b, lds, nwg, stream) : launch_b3<64, 0>(b, lds, nwg, stream);
    }
}

}  // namespace comera
