// Internal declarations for the TTM embedding path.
#pragma once

#include <cstddef>
#include <cstdint>

#include "internal.h"

namespace comera {

constexpr int kEmbedItem = 32;     // tokens per work item of the backward segment sums
constexpr int kEmbedChunks = 256;  // fixed split of the unique ids for dG_last

struct EmbedDims {
    int d;
    int64_t V, E;           // rows, width
    int64_t Vp, Ep;         // prefix rows / width (cores 0..d-2)
    int Vs, Es, R;          // last core: v, e, left rank
};

struct EmbedLayout {
    size_t gc[kMaxCores];      // mask-folded prefix cores
    size_t p[kMaxCores];       // prefix chains P_k, k = 1..d-1 (P_{d-1} = prefix table)
    size_t keysA, valsA, keysB, valsB, meta, uid, ustart, useg_item, item_u, item_beg, item_len;
    size_t S, Spart, dA, dglast_part;
    size_t e[kMaxCores];       // environments E_k, k = 1..d-2
    size_t gpart[kMaxCores];   // meet partials for the prefix cores
    int meet_splits[kMaxCores];
    size_t total;
};

struct EmbedWs {
    uint32_t *keysA, *valsA, *keysB, *valsB;
    int *meta, *uid, *ustart, *useg_item, *item_u, *item_beg, *item_len;
    float *S, *Spart, *dglast_part;
};

int launch_embed_rows(const int64_t *ids, int64_t n, int64_t V, const float *Apre, const float *Gs, float *Y, int Ep,
                      int R, int Vs, int Es, int *err_flag, void *stream);
int launch_embed_sort(const int64_t *ids, int n, int64_t V, const EmbedWs &w, int *err_flag, void *stream);
int launch_embed_segsum(const float *dY, int E, int n, const EmbedWs &w, void *stream);
int launch_embed_dglast(const EmbedWs &w, const float *Apre, int Ep, int R, int Vs, int Es, void *stream);
int launch_embed_dapre(const EmbedWs &w, const float *Gs, int64_t Vp, int Ep, int R, int Vs, int Es, float *dA,
                       void *stream);

}  // namespace comera
