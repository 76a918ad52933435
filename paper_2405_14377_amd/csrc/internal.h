// Internal declarations shared by the planner, the entry points and the
// kernel launchers.  Nothing here is part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <memory>
#include <string>
#include <vector>

#include "comera.h"

namespace comera {

constexpr int kMaxCores = COMERA_MAX_CORES;

// Active entries of one bond, as a bit set (ranks up to 256 are compacted;
// larger ranks are used uncompacted).
struct BondBits {
    uint64_t w[4];
};

struct Order {
    int kind = COMERA_ORDER_DENSE;     // COMERA_ORDER_*
    uint32_t cuts = 0;                  // bit k set = a group boundary after core k
    double flops_fwd = 0, flops_bwd = 0, bytes = 0, t_pred = 0;
    bool executable = false;
    std::string desc;
};

// Placement of one compacted core copy: element (a, m, n, c) (left bond,
// output factor, input factor, right bond; bonds compacted) sits at
// a * sa + m * sm + n * sn + c * sc.
struct CoreStrides {
    int sa, sm, sn, sc;
};

// Byte offsets of every workspace region used by the dense order.
struct DenseLayout {
    size_t gc[kMaxCores];      // compacted, mask-folded cores (fp32)
    size_t p[kMaxCores + 1];   // left chains P_k, k = 1..d-1 (fp32); p[d] unused
    size_t w;                  // W [N_in, N_out] in the activation dtype
    size_t wt;                 // W^T [N_out, N_in] in the activation dtype
    size_t ones;               // a single 1.0f (left operand of the d = 1 build)
    size_t dw_part;            // split-K partials of dW (fp32)
    size_t dw;                 // dW (fp32)
    size_t e[kMaxCores + 1];   // right environments E_k, k = 1..d-1 (fp32)
    size_t gpart[kMaxCores];   // split partials of the compacted core gradients
    size_t total;
    int dw_splits;             // split-K count of dW = X^T dY
    int64_t dw_kchunk;         // tokens per split
    int meet_splits[kMaxCores];
    int dx_splits;             // split of dX = dY W^T over N_out (1: none)
    int64_t dx_kchunk;
    size_t dx_part;            // split partials of dX (fp32)
    int adj_splits[kMaxCores];  // split-K of the adjoint step producing E_k
    size_t adj_part;           // shared scratch for adjoint split partials
    size_t part;               // split partials of the forward / dX products at small batch
    int64_t part_elems;
    // fused projection route (all ranks within proj_supported): step k reads
    // E_{k+1} as e_slices[k+1] slices and writes E_k as e_slices[k] slices
    // (one per column chunk) and meet_splits[k] meet partials (one per row chunk)
    bool proj;
    int proj_rt[kMaxCores];
    int proj_ct[kMaxCores];
    int e_slices[kMaxCores + 1];
};

// FP8 mixed precision of the dense order: W is built in fp32 (region
// DenseLayout::w) and the three batch products read E4M3 codes.  K of every
// product is padded with zero codes to a multiple of 128 (N_in_p, N_out_p,
// b_p for the planned batch).
struct Fp8Layout {
    int64_t nin_p, nout_p, b_p;
    size_t w8;      // W codes [N_in][N_out_p]      (B of dX = dY W^T)
    size_t w8t;     // W^T codes [N_out][N_in_p]    (B of Y = X W)
    size_t x8;      // X codes [b][N_in_p]          (A of Y)
    size_t x8t;     // X^T codes [N_in][b_p]        (A of dW = X^T dY)
    size_t dy8;     // dY codes [b][N_out_p]        (A of dX)
    size_t dy8t;    // dY^T codes [N_out][b_p]      (B of dW)
    size_t pmax;    // partial maxima of the tensor being quantised
    size_t sc;      // scales: kScW, kScX, kScDY, then the GEMM output factors kScFwd, kScDX, kScDW
};
constexpr int kScW = 0, kScX = 1, kScDY = 2, kScFwd = 3, kScDX = 4, kScDW = 5;

// Sweep orders (groups of consecutive cores, activations swept through the
// groups in sequence).  Each group g (cores s[g] .. e[g]) is treated as a
// layer of its own whose outer bonds are folded into its outer factors:
//   right to left:  W'_g [(N_g, ae_g)][(as_g, M_g)]
//   left to right:  W'_g [(as_g, N_g)][(M_g, ae_g)]
// where N_g, M_g are the products of the group's input and output factors
// and as_g, ae_g its left and right (compacted) bond ranks.  The states of
// both sweeps are stored with the next contraction's index last:
//   right to left, activation state Z_g (input of step g-1):
//       [(b, N_<g-1, M_>=g)][(N_{g-1}, ae_{g-1})]
//   right to left, dY state H_g (input of step g): [(b, N_<g, M_>g)][(as_g, M_g)]
//   left to right, activation state Z_g (input of step g): [(b, M_<g, N_>g)][(as_g, N_g)]
//   left to right, dY state H_g (input of step g): [(b, M_<g, N_>g)][(M_g, ae_g)]
// so the gradient of W'_g is one product A^T B of the two states that meet
// at group g, with the token-like index (b and the outer factors) as K.
struct SweepLayout {
    int G = 0;
    int dir = 0;                       // COMERA_ORDER_SWEEP_RL or _LR
    int s[kMaxCores], e[kMaxCores];
    int64_t N[kMaxCores], M[kMaxCores], as[kMaxCores], ae[kMaxCores];
    size_t base[kMaxCores];            // workspace offset of each group's own layout
    size_t z[kMaxCores + 1];           // activation states Z_g, g = 1 .. G-1
    size_t h[kMaxCores + 1];           // dY states (RL: H_g, g = 1 .. G-1; LR: H_g, g = 0 .. G-2)
    size_t tin;                        // per-token transposed dY (RL) or X (LR)
    bool need_t = false;
    size_t part = 0;                   // split partials of the sweep products
    int64_t part_elems = 0;
    CoreStrides st[kMaxCores];         // placement of each folded core in its group
    size_t total = 0;
};

}  // namespace comera

namespace comera {
// Event pairs recorded around the batch-product launches when timing is on.
struct KernelTiming {
    bool on = false;
    std::vector<std::pair<void *, void *>> ev[3];
};
}  // namespace comera

namespace comera {
// Fused single-core sweep (chain.hip): the forward and the backward of a
// whole layer, one workgroup per TB tokens at a time, states in LDS.  Ranks
// are the compacted ones (rc), amap[k][x] is the full index of compacted
// entry x of bond k (k = 1 .. d-1); every offset below is in floats.
constexpr int kChainMaxRank = 64;
struct ChainArgs {
    const float *G[kMaxCores];
    const float *D[kMaxCores];
    uint8_t amap[kMaxCores + 1][kChainMaxRank];
    int d, TB, act_bf16;
    int r[kMaxCores + 1], rc[kMaxCores + 1], m[kMaxCores], n[kMaxCores];
    int Nl[kMaxCores], Mg[kMaxCores];   // prod of n before core k, prod of m after core k
    int ssz[kMaxCores + 1];             // floats of state k per token
    int cstart[kMaxCores + 1];          // first element of core k in one flat index over the cores
    int smap;                           // LDS copy of amap (ints)
    int cm[kMaxCores], km[kMaxCores];   // folded cores, c-major and k-major
    int cp[kMaxCores], kp[kMaxCores];   // their row pitches (floats)
    int compacted;                      // amap is not the identity
    int wave0[kMaxCores + 1];           // staging: first wave of core k's block
    int st0, st1;                       // ping-pong state buffers
    int sk[kMaxCores + 1];              // backward: forward states S_1 .. S_d
    int tab;                            // backward: row tables of the meets (ints)
    int want[kMaxCores];                // backward: core gradients asked for
    int64_t b;
    const void *X, *dY;
    void *Y, *dX;
    float *part;                        // backward: partials of the masked-core gradients, core k at
    int64_t poff[kMaxCores];            // part + poff[k] as [grid][rc_k m_k n_k rc_{k+1}]
    size_t lds_bytes;
};
}  // namespace comera

namespace comera {
// The fused single-core sweep of a plan: kernel arguments with the geometry
// filled in (forward and backward), grids, and the workspace region of the
// backward's core-gradient partials.
struct ChainLayout {
    ChainArgs fa, ba;
    int grid_f = 0, grid_b = 0;
    size_t part = 0;
    size_t total = 0;
};
}  // namespace comera

struct comera_ttm_plan_s {
    comera_ttm_shape s;
    int64_t batch = 0;
    int d = 0;
    int64_t N_in = 0, N_out = 0;
    int64_t rho[comera::kMaxCores + 1];          // effective (compacted) ranks
    bool compacted = false;                       // some rank is compacted below r
    comera::BondBits act[comera::kMaxCores + 1];  // act[k] for bond k = 1..d-1
    bool zero = false;                            // a bond has no active entry
    std::vector<comera::Order> orders;
    int chosen = 0;
    comera::DenseLayout dense;
    comera::SweepLayout sweep;                    // when the chosen order is a sweep
    bool chain = false;                           // the chosen order is the fused single-core sweep
    comera::ChainLayout ch;
    std::unique_ptr<comera_ttm_plan_s> sub[comera::kMaxCores];   // one layer per sweep group
    size_t ws_bytes = 0;
    bool reuse = false;                           // backward reuses the forward's build
    bool fp8 = false;                             // batch products on E4M3 codes (dense order)
    comera::Fp8Layout f8{};
    comera::KernelTiming timing;
};

namespace comera {

// Workspace layout of the dense order for a plan (fills p->dense).  Without
// with_dx no region for split partials of dX is reserved.
void layout_dense(comera_ttm_plan_s *p, bool with_dx = true);
// Workspace layout of a sweep order: fills L and one layer per group in sub;
// false when the order cannot run (workspace above the cap or a group
// outside the kernels' index limits).
bool layout_sweep(const comera_ttm_plan_s *p, int kind, uint32_t cuts, SweepLayout &L,
                  std::unique_ptr<comera_ttm_plan_s> *sub);

// Launchers (ttm_kernels.hip).  All return a hipError_t value as int.

// [a][m][n][c], or [a][n][m][c] when swap
CoreStrides core_strides(int A, int m, int n, int C, bool swap);

struct FoldArgs {
    const float *G[kMaxCores];
    const float *D[kMaxCores];   // D[k] for k < d-1, may be null (= ones)
    float *Gc[kMaxCores];
    BondBits act[kMaxCores + 1];
    int r[kMaxCores + 1];        // full ranks
    int rc[kMaxCores + 1];       // compacted ranks
    int m[kMaxCores];
    int n[kMaxCores];
    int d;
    int nfold;                   // cores folded (grid.y); d for a linear layer
    int compacted;
    CoreStrides st[kMaxCores];   // placement of each copy
};
int launch_fold(const FoldArgs &a, void *stream);

struct ExpandArgs {
    const float *part[kMaxCores];   // [splits][compacted core placed by st[k]]
    const float *D[kMaxCores];
    float *dG[kMaxCores];
    BondBits act[kMaxCores + 1];
    int r[kMaxCores + 1];
    int rc[kMaxCores + 1];
    int m[kMaxCores];
    int n[kMaxCores];
    int splits[kMaxCores];
    int d;
    int compacted;
    CoreStrides st[kMaxCores];      // placement of the compacted partials
    int groups[kMaxCores];          // set by launch_expand
    int blk0[kMaxCores];            // set by launch_expand
};
int launch_expand(const ExpandArgs &a, void *stream);

// dD_k (k = 0..d-2, r_{k+1} floats each, null = skip) from the compacted
// split partials of the masked-core gradients (as for expand) and the raw
// cores G_k
struct MaskGradArgs {
    const float *part[kMaxCores];
    int splits[kMaxCores];
    CoreStrides st[kMaxCores];
    const float *G[kMaxCores];
    float *dD[kMaxCores];
    BondBits act[kMaxCores + 1];
    int r[kMaxCores + 1];
    int rc[kMaxCores + 1];
    int m[kMaxCores];
    int n[kMaxCores];
    int d;
    int compacted;
    int blk0[kMaxCores];            // set by launch_mask_grad
};
int launch_mask_grad(const MaskGradArgs &a, void *stream);

// FP8 operands (fp8.hip): x [R][C] (fp32 or bf16 by dtype) -> per-tensor
// power-of-two scale s (written to s_out[0]), E4M3 codes q [R][ldq] (columns
// C .. ldq-1 zero) and / or qt [C][ldt] (x^T, columns R .. ldt-1 zero), and
// 1 / (s * *pa) -> *oa, 1 / (s * *pb) -> *ob for the GEMMs that consume the
// codes (any of q, qt, pa / oa, pb / ob may be null).  pmax:
// fp8_amax_blocks() floats of scratch.
int fp8_amax_blocks();
int launch_fp8_quant(const void *x, int dtype, int64_t R, int64_t C, float *pmax, uint8_t *q, int64_t ldq,
                     uint8_t *qt, int64_t ldt, float *s_out, const float *pa, float *oa, const float *pb, float *ob,
                     void *stream);

// Output index remap of a GEMM: write idx in mixed radix (digit 0 most
// significant and unbounded, digit t < nd has radix radix[t] for t >= 1) and
// return sum_t digit_t * stride[t].
struct Remap {
    int nd;
    int64_t radix[4];
    int64_t stride[4];
};
Remap remap_linear(int64_t stride);

// Fused projection step of the core gradients for one core k (dense order):
// with En = E_{k+1} (rows (I, J), columns (x, y, c)), the folded core
// Gc = G~_k [A][cols] and the left chain P = P_k [rows][A],
//   adjoint  E_k[row][a]   = sum_c En[row][c] Gc[a][c]       (per column chunk)
//   meet     part[a][c]    = sum_row P[row][a] En[row][c]     (per row chunk)
// En may come as `nin` slices that are summed in slice order on load.  The
// adjoint output of column chunk j goes to Eout + j * out_stride +
// rmap(row) + a; the meet partial of row chunk i to part + i * A * cols.
struct ProjArgs {
    const float *En;
    int nin;
    int64_t in_stride;
    const float *Gc;    // null: no adjoint
    const float *P;     // null: no meet
    float *Eout;
    int64_t out_stride;
    Remap rmap;
    float *part;
    int64_t rows, cols;
    int A;
    int RT, CT;
};
// tile choice (rows per chunk RT, columns per chunk CT) for a projection step
void proj_tiles(int64_t rows, int64_t cols, int A, int &RT, int &CT);
bool proj_supported(int A);
int launch_proj(const ProjArgs &a, void *stream);

// Last step of the W rebuild (proj.hip): W [N_in][N_out] to out and / or
// W^T [N_out][N_in] to out_t (either may be null) from P_{d-1} [NI][NJ][A]
// and the folded last core [A][nx][ny], in tiles of QI x QJ prefixes.
struct WBuildArgs {
    const float *P;
    const float *G;
    void *out;
    void *out_t;
    int64_t NI, NJ;
    int A, nx, ny;
    int out_bf16;
    int QI, QJ;
};
bool wbuild_tiles(int64_t NI, int64_t NJ, int A, int nx, int ny, int &QI, int &QJ);
int launch_wbuild(const WBuildArgs &a, void *stream);

// One inner step of the chain (proj.hip), fp32, ranks A up to 64: with the
// left chain P [NI][NJ][A] and the folded core G [A][nx][ny][C],
//   out[(I x)][(J y)][c] = sum_a P[I][J][a] G[a][x][y][c]
struct LChainArgs {
    const float *P;
    const float *G;
    float *out;
    int64_t NI, NJ;
    int A, nx, ny, C;
};
bool lchain_supported(int A);
int launch_lchain(const LChainArgs &a, void *stream);

// Whole batch-free build of a three-core layer in one launch (build3.hip):
// from the raw cores G_k [r_k][m_k][n_k][r_{k+1}] and the masks of bonds 1
// and 2 (D[k] scales core k's right bond; null = ones), the folded copies
// Gc[k] (placed by st[k]), the left chain P_2 [(x0 x1)][(y0 y1)][C] and W
// [N_in][N_out] (w) and / or W^T [N_out][N_in] (wt).  A, C: compacted ranks
// of bonds 1 and 2 (at most 64); r1, r2 full ranks; tiles of SX x SY middle
// slices and PX x PY pairs from build3_tiles.
struct Build3Args {
    const float *G[3];
    const float *D[2];
    float *Gc[3];
    CoreStrides st[3];
    float *P2;
    void *w, *wt;
    BondBits act1, act2;
    int r1, r2;
    int A, C;
    int n[3], m[3];
    int compacted;
    int out_bf16;
    int SX, SY, PX, PY;
    uint8_t map1[64], map2[64];   // compacted -> full entry of bonds 1 and 2 (set by launch_build3)
    int vec_w, vec_t;             // set by launch_build3
};
bool build3_tiles(const int *n, const int *m, int A, int C, int &SX, int &SY, int &PX, int &PY);
int launch_build3(const Build3Args &a, void *stream);


// operand type code of FP8 (OCP E4M3) GEMM operands, beside COMERA_F32 / COMERA_BF16
constexpr int kDtypeFp8 = 2;

struct GemmArgs {
    int dtype = COMERA_F32;          // operand type (COMERA_F32, COMERA_BF16 or kDtypeFp8)
    bool a_kc = true, b_kc = true;   // k contiguous in memory for A / B
    bool out_bf16 = false;
    const void *A = nullptr, *B = nullptr;
    void *C = nullptr;
    int64_t M = 0, N = 0, K = 0, lda = 0, ldb = 0;
    Remap rmap{}, cmap{};
    int splits = 1;
    int64_t kchunk = 0;              // k per split (0 = K)
    int64_t split_stride = 0;        // elements between split outputs
    int tile = -1;                   // general-kernel tile (-1 = automatic)
    int fast = -1;                   // fast-kernel tile (-1 = automatic, -2 = never)
    // automatic split over K for products whose output tiles alone leave
    // the chip idle: the remapped output must cover out_elems consecutive
    // elements; the fp32 partials go to scratch (at most scratch_elems) and
    // are summed in a fixed order into C
    float *scratch = nullptr;
    int64_t scratch_elems = 0;
    int64_t out_elems = 0;
    const float *oscale = nullptr;   // device scalar multiplying every result (fast path), or null
};
// C[rmap(m) + cmap(n)] = sum_k Aop(m, k) Bop(k, n); see gemm.hip.
int launch_gemm(const GemmArgs &g, void *stream);
// split count launch_gemm takes for an M x N x K product given scratch room
int gemm_auto_splits(int64_t M, int64_t N, int64_t K);

// Core contractions as GEMMs (gemm.hip).  A core copy Gc has layout
// [A][nx][ny][C]; x runs over the factors of the left index X, y over those
// of the right index Y.
//   chain:   out[(I x)][(J y)][c] = sum_a P[I][J][a] Gc[a][x][y][c]   (P == null: a single 1)
//   adjoint: E[(I, J)][a] = sum_{x y c} En[(I, J)][(x y c)] Gc[a][(x y c)], written
//            blocked for the next step: [(I', J')][(x', y')][a], I = I' nxp + x',
//            J = J' nyp + y'
//   meet:    part[s][a][(x y c)] = sum_{(I, J) in split s} P[(I, J)][a] En[(I, J)][(x y c)]
//   layout kChainT (last core, C == 1): out[(J y)][(I x)] instead
//   layout kChainRankMajor: out[(I x)][c][(J y)] instead
constexpr int kChainNormal = 0, kChainT = 1, kChainRankMajor = 2;
int chain_gemm(const float *P, const float *Gc, void *out, bool out_bf16, int64_t NI, int64_t NJ, int A, int nx,
               int ny, int C, void *stream, int layout = kChainNormal);

// Batched staging into LDS: count elements, element i = src(i), U loads in
// flight per thread before the stores (threads t0, t0 + nt, ...).
template <int U, class Src>
__device__ __forceinline__ void stage_lds(float *dst, int count, int t0, int nt, Src src) {
    for (int i0 = t0; i0 < count; i0 += nt * U) {
        float v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * nt;
            v[u] = i < count ? src(i) : 0.f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * nt;
            if (i < count) dst[i] = v[u];
        }
    }
}
// Two regions staged together (one memory round trip when countA + countB
// <= U * nt): element i < countA goes to dstA[i] = srcA(i), the rest to
// dstB[i - countA] = srcB(i - countA).
template <int U, class SrcA, class SrcB>
__device__ __forceinline__ void stage2_lds(float *dstA, int countA, SrcA srcA, float *dstB, int countB, SrcB srcB,
                                           int t0, int nt) {
    const int count = countA + countB;
    for (int i0 = t0; i0 < count; i0 += nt * U) {
        float v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * nt;
            v[u] = i < countA ? srcA(i) : (i < count ? srcB(i - countA) : 0.f);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * nt;
            if (i < countA)
                dstA[i] = v[u];
            else if (i < count)
                dstB[i - countA] = v[u];
        }
    }
}
// With splits > 1 the split partials go to `scratch` (splits * NI * NJ * A
// floats) and are summed into `out` in a fixed order.
int adjoint_gemm(const float *En, const float *Gc, float *out, int64_t NI, int64_t NJ, int A, int nx, int ny, int C,
                 int nxp, int nyp, int splits, float *scratch, void *stream);
// split count for a GEMM with few output tiles and a long K
int split_for(int64_t M, int64_t N, int64_t K);
int meet_gemm(const float *P, const float *En, float *part, int64_t NI, int64_t NJ, int A, int nx, int ny, int C,
              int splits, void *stream);

int launch_sum_splits(const float *part, float *out, int64_t n, int splits, void *stream);
// the same sum rounded once to bf16
int launch_sum_splits_bf16(const float *part, void *out, int64_t n, int splits, void *stream);
int launch_fill_zero(void *ptr, size_t bytes, void *stream);
int launch_fill_one(float *ptr, void *stream);

// Steps of one (virtual) layer, shared by the dense order and the groups of
// a sweep order (api_ttm.hip).
struct DenseBuild {
    float *gc[kMaxCores];      // folded cores [rho_k][n_k][m_k][rho_{k+1}]
    float *P[kMaxCores + 1];   // left chains P_k = [I_<k][J_<k][rho_k], k = 1..d-1
    void *w;                   // W [N_in][N_out] in the activation dtype
    void *wt;                  // W^T [N_out][N_in] in the activation dtype
};
// which layouts of W build_chain writes
constexpr int kWantW = 1, kWantWT = 2;
// folded-core pointers of a layer whose workspace starts at ws
void dense_ptrs(const comera_ttm_plan_s *sp, void *ws, DenseBuild &bd);
// fold the masks into compacted copies of every core of layer p (eq. Wcompress):
// core k goes to dst[k], placed by st[k]
int fold_cores(const comera_ttm_plan_s *p, const float *const *G, const float *const *D, float *const *dst,
               const CoreStrides *st, void *stream);
// left chains and W (want & kWantW) and / or W^T (want & kWantWT) of a
// layer from its folded cores
int build_chain(const comera_ttm_plan_s *sp, void *ws, DenseBuild &bd, int want, void *stream);
// pointers of the build that build_chain(want) left in the workspace of an
// earlier call (no device work)
void built_dense(const comera_ttm_plan_s *p, void *ws, DenseBuild &bd, int want);
// dW = A^T B (A [K][N_in] with leading dimension lda, B [K][N_out] with ldb),
// split over K, written blocked for the projections; *dwp, *splits describe
// the split partials.  With oscale (FP8 codes): A [N_in][lda] and B
// [N_out][ldb] hold the transposed operands, K a multiple of 128, and every
// result is multiplied by *oscale.
int dw_gemm(const comera_ttm_plan_s *sp, const void *A, int64_t lda, const void *B, int64_t ldb, int64_t K,
            void *ws, float **dwp, int *splits, void *stream, const float *oscale = nullptr);
// core gradients (compacted, as split partials part[k] x nsplit[k]) from the
// partials of dW; want[k] false skips core k
int project_cores(const comera_ttm_plan_s *sp, const DenseBuild &bd, const float *dwp, int splits,
                  const bool *want, void *ws, const float **part, int *nsplit, void *stream);
// sum the partials of every core of layer p, unfold and apply the masks
int expand_cores(const comera_ttm_plan_s *p, const float *const *part, const int *nsplit, const CoreStrides *st,
                 const float *const *D, float *const *dG, void *stream);
// mask gradients dD_k of layer p from the same partials (dD null: nothing)
int mask_grads(const comera_ttm_plan_s *p, const float *const *part, const int *nsplit, const CoreStrides *st,
               const float *const *G, float *const *dD, void *stream);
// out[t][j][i] = in[t][i][j] for t < b, i < M, j < T (elements of esz bytes)
int launch_permute_tokens(const void *in, void *out, int64_t b, int64_t M, int64_t T, int esz, void *stream);

// fills the size fields for TB tokens per workgroup; false when they do not
// fit the LDS of a CU
bool chain_fits(ChainArgs &a, int64_t b, bool backward, int TB);
int launch_chain(const ChainArgs &a, bool backward, int grid, void *stream);
// geometry, grids and workspace of the fused order of plan p; false when the
// layer is outside the fused kernels' limits
bool layout_chain(const comera_ttm_plan_s *p, ChainLayout &L);
comera_status chain_forward(const comera_ttm_plan_s *p, int64_t b, const void *X, const float *const *G,
                            const float *const *D, void *Y, void *ws, void *stream);
comera_status chain_backward(const comera_ttm_plan_s *p, int64_t b, const void *X, const void *dY,
                             const float *const *G, const float *const *D, void *dX, float *const *dG,
                             float *const *dD, void *ws, void *stream);

// sweep orders (sweep.hip)
comera_status sweep_forward(const comera_ttm_plan_s *p, int64_t b, const void *X, const float *const *G,
                            const float *const *D, void *Y, void *ws, void *stream);
comera_status sweep_backward(const comera_ttm_plan_s *p, int64_t b, const void *X, const void *dY,
                             const float *const *G, const float *const *D, void *dX, float *const *dG,
                             float *const *dD, void *ws, void *stream);

// Every kernel launch goes through COMERA_LAUNCH.  In launch check mode
// (comera_debug_launch_check) the configuration is validated and recorded
// instead of launched; launch_status() then returns the first failed check
// since the last call, otherwise hipGetLastError().
bool launch_check_mode();
void launch_check(const char *name, dim3 grid, dim3 block, size_t lds);
int launch_status();
#define COMERA_LAUNCH_NAMED(name, kern, grid, block, lds, stream, ...)                        \
    do {                                                                                      \
        if (::comera::launch_check_mode())                                                    \
            ::comera::launch_check(name, dim3(grid), dim3(block), size_t(lds));               \
        else                                                                                  \
            hipLaunchKernelGGL(kern, grid, block, lds, stream, __VA_ARGS__);                  \
    } while (0)
#define COMERA_LAUNCH(kern, grid, block, lds, stream, ...) \
    COMERA_LAUNCH_NAMED(#kern, kern, grid, block, lds, stream, __VA_ARGS__)

// record a failed launcher result (hipError_t value e != 0) with the step
// name for comera_last_hip_error; returns e (api_ttm.hip)
int note_hip(int e, const char *where);

// timing hooks (api_ttm.hip)
void timing_begin(comera_ttm_plan_s *p, int kernel, void *stream, void **ev0);
void timing_end(comera_ttm_plan_s *p, int kernel, void *stream, void *ev0);
void timing_clear(comera_ttm_plan_s *p);

}  // namespace comera
