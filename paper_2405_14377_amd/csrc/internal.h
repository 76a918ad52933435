// Internal declarations shared by the planner, the entry points and the
// kernel launchers.  Nothing here is part of the public ABI.
#pragma once

#include <cstddef>
#include <cstdint>
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

// Byte offsets of every workspace region used by the dense order.
struct DenseLayout {
    size_t gc[kMaxCores];      // compacted, mask-folded cores (fp32)
    size_t p[kMaxCores + 1];   // left chains P_k, k = 1..d-1 (fp32); p[d] unused
    size_t w;                  // W [N_in, N_out] in the activation dtype
    size_t dw_part;            // split-K partials of dW (fp32)
    size_t dw;                 // dW (fp32)
    size_t e[kMaxCores + 1];   // right environments E_k, k = 1..d-1 (fp32)
    size_t gpart[kMaxCores];   // split partials of the compacted core gradients
    size_t total;
    int dw_splits;             // split-K count of dW = X^T dY
    int64_t dw_kchunk;         // tokens per split
    int meet_splits[kMaxCores];
};

}  // namespace comera

namespace comera {
// Event pairs recorded around the batch-product launches when timing is on.
struct KernelTiming {
    bool on = false;
    std::vector<std::pair<void *, void *>> ev[3];
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
    size_t ws_bytes = 0;
    comera::KernelTiming timing;
};

namespace comera {

// Workspace layout of the dense order for a plan (fills p->dense).
void layout_dense(comera_ttm_plan_s *p);

// Launchers (ttm_kernels.hip).  All return a hipError_t value as int.
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
};
int launch_fold(const FoldArgs &a, void *stream);

struct ExpandArgs {
    const float *part[kMaxCores];   // [splits][rc_{k}, m, n, rc_{k+1}]
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
};
int launch_expand(const ExpandArgs &a, void *stream);

// out[(X x), (Y y), c] = sum_a P[X, Y, a] * G[a, .., .., c]; x is core axis
// `xaxis` (1 or 2), y the other one.  P == nullptr means a single 1.
// If out_bf16 is set (and c == 1), the result is written as bf16 instead.
int launch_chain(const float *P, const float *G, float *out, uint16_t *out_bf16, int64_t NX,
                 int64_t NY, int A, int m, int n, int C, int xaxis, void *stream);
// out[X, Y, a] = sum_{x, y, c} E[(X x), (Y y), c] * G[a, .., .., c]
int launch_adjoint(const float *E, const float *G, float *out, int64_t NX, int64_t NY, int A,
                   int m, int n, int C, int xaxis, void *stream);
// part[s][a, m, n, c] = sum_{(X, Y) in split s} P[X, Y, a] * E[(X x), (Y y), c]
int launch_meet(const float *P, const float *E, float *part, int64_t NX, int64_t NY, int A,
                int m, int n, int C, int xaxis, int splits, void *stream);

// C = op(A) op(B): see ttm_kernels.hip for the operand conventions.
int launch_gemm(int dtype, bool a_kcontig, bool b_kcontig, bool out_bf16, const void *A,
                const void *B, void *C, int64_t M, int64_t N, int64_t K, int64_t lda,
                int64_t ldb, int64_t ldc, int splits, int64_t kchunk, void *stream);
int launch_sum_splits(const float *part, float *out, int64_t n, int splits, void *stream);
int launch_fill_zero(void *ptr, size_t bytes, void *stream);

// timing hooks (api_ttm.hip)
void timing_begin(comera_ttm_plan_s *p, int kernel, void *stream, void **ev0);
void timing_end(comera_ttm_plan_s *p, int kernel, void *stream, void *ev0);
void timing_clear(comera_ttm_plan_s *p);

}  // namespace comera
