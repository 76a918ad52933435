// Internal declarations for the TTM embedding path.
#pragma once

#include <cstddef>
#include <cstdint>

#include "internal.h"

namespace comera {

constexpr int kEmbedItem = 16;     // sorted positions per chunk of the backward segment sums
constexpr int kEmbedChunks = 256;  // fixed split of the sorted positions for dG_last

struct EmbedDims {
    int d;
    int64_t V, E;           // rows, width
    int64_t Vp, Ep;         // prefix rows / width (cores 0..d-2)
    int Vs, Es, R;          // last core: v, e, left rank
};

struct EmbedLayout {
    size_t gc[kMaxCores];      // mask-folded prefix cores
    size_t p[kMaxCores];       // prefix chains P_k, k = 1..d-1 (P_{d-1} = prefix table)
    size_t keysA, valsA, keysB, valsB, hist, meta;
    size_t S, Pfirst, Plast, dA, dglast_part;
    size_t e[kMaxCores];       // environments E_k, k = 1..d-2
    size_t gpart[kMaxCores];   // meet partials for the prefix cores
    int meet_splits[kMaxCores];
    int adj_splits[kMaxCores];
    size_t adj_part;
    size_t total;
};

struct EmbedWs {
    uint32_t *keysA, *valsA, *keysB, *valsB;
    int *hist;
    int *meta;   // meta[0] = number of in-range ids
    float *S, *Pfirst, *Plast, *dglast_part;
};

int launch_embed_rows(const int64_t *ids, int64_t n, int64_t V, const float *Apre, const float *Gs, float *Y, int Ep,
                      int R, int Vs, int Es, int *err_flag, void *stream);
int launch_embed_sort(const int64_t *ids, int n, int64_t V, const EmbedWs &w, int *err_flag, void *stream);
int launch_embed_segsum(const float *dY, int E, int n, int64_t V, const EmbedWs &w, void *stream);
int launch_embed_dglast(const EmbedWs &w, int n, int64_t V, const float *Apre, int Ep, int R, int Vs, int Es,
                        void *stream);
// dA is written blocked for the prefix-core projections: [(V', E')][(vq, eq)][R]
// with vp = V' vq + x, ep = E' eq + y (vq, eq = factors of the last prefix core)
int launch_embed_dapre(const EmbedWs &w, int n, int64_t V, const float *Gs, int64_t Vp, int Ep, int R, int Vs, int Es,
                       int vq, int eq, float *dA, void *stream);
// shapes the embedding kernels handle (rank of the last bond <= 64, a dY row
// of the backward fix-up fits in LDS four times)
bool embed_kernels_support(int Ep, int R, int Es, int64_t E);
// the last core fits in LDS (staged whole by the row and dA kernels)
bool embed_gs_fits(int R, int Vs, int Es);

}  // namespace comera
