// Internal declarations for the TTM embedding path.
#pragma once

#include <cstddef>
#include <cstdint>

#include "internal.h"

namespace comera {

constexpr int kEmbedItem = 16;     // sorted positions per chunk of the backward segment sums

struct EmbedDims {
    int d;
    int64_t V, E;           // rows, width
    int64_t Vp, Ep;         // prefix rows / width (cores 0..d-2)
    int Vs, Es, R;          // last core: v, e, left rank
};

struct EmbedLayout {
    size_t gc[kMaxCores];      // mask-folded prefix cores
    size_t p[kMaxCores];       // prefix chains P_k, k = 1..d-1 (P_{d-1} = prefix table)
    size_t keysA, valsA, keysB, valsB, hist, meta, headpos;
    size_t S, Pfirst, Plast, dA, dglast_part;
    int passes;                // radix passes
    int nvp;                   // dG_last partials (chunks of prefixes)
    // projections onto the prefix cores k = d-2 .. 1 (as for a linear layer)
    size_t e[kMaxCores];       // environment slices E_k
    size_t gpart[kMaxCores];   // meet partials of core k
    int e_slices[kMaxCores + 1];
    int meet_splits[kMaxCores];
    int proj_rt[kMaxCores], proj_ct[kMaxCores];
    size_t total;
};

struct EmbedWs {
    uint32_t *keysA, *valsA, *keysB, *valsB;
    int *hist;      // [256][nblk] digit counts of the current pass, then [nblk] out-of-range counts
    int *meta;      // meta[0] = number of in-range ids
    int *headpos;   // [V] sorted position of the first token of each id, -1 if absent
    float *S, *Pfirst, *Plast, *dA, *dglast_part;
};

// A = prefix table [Vp][Ep][R], or [Vp][R][Ep] when rank_major
int launch_embed_rows(const int64_t *ids, int64_t n, int64_t V, const float *Apre, bool rank_major, const float *Gs,
                      float *Y, int Ep, int R, int Vs, int Es, int *err_flag, void *stream);
// stable LSD radix sort of the ids (out-of-range ids get the key V and sort
// last) and n_valid into meta[0]; its first kernel also clears
// headpos[0 .. nclear) to -1 and zero[0 .. nzero) to 0
int launch_embed_sort(const int64_t *ids, int n, int64_t V, int passes, const EmbedWs &w, int *err_flag,
                      int64_t nclear, float *zero, int64_t nzero, void *stream);
const uint32_t *embed_sorted_keys(const EmbedWs &w, int passes);
// per-id sums of dY rows in token order: S[head] (and headpos[id] = head)
int launch_embed_segsum(const float *dY, int E, int n, int passes, const EmbedWs &w, void *stream);
// dA [Vp][Ep][R] per prefix (written blocked for the prefix projections:
// [(V', E')][(vq, eq)][R] with vp = V' vq + x, ep = E' eq + y)
int launch_embed_dapre(const EmbedWs &w, const float *Gs, int64_t Vp, int Ep, int R, int Vs, int Es, int vq, int eq,
                       void *stream);
// dG_last partials, one per chunk of prefixes: [chunk][R][Vs][Es]
int launch_embed_dglast(const EmbedWs &w, const float *Apre, bool rank_major, int64_t Vp, int Ep, int R, int Vs,
                        int Es, void *stream);
int embed_dglast_chunks(int64_t Vp);
// prefix table of a three-core table straight from the raw cores 0 and 1
// (masks folded on the fly), rank-major [v0 v1][r2][e0 e1]; also writes the
// folded cores gc0 [v0][e0][r1] and gc1 [r1][v1][e1][r2]
bool embed_table_supported(int r1, int e0);
int launch_embed_table(const float *G0, const float *D0, const float *G1, const float *D1, float *A, float *gc0,
                       float *gc1, int v0, int v1, int e0, int e1, int r1, int r2, void *stream);
// d = 1: dG_0[0, v, e, 0] = S[headpos[v]][e] (0 for absent ids)
int launch_embed_gather(const EmbedWs &w, int64_t V, int E, float *dG0, void *stream);
// shapes the embedding kernels handle (LDS staging limits)
bool embed_kernels_support(int64_t Ep, int R, int Vs, int Es, int d);

}  // namespace comera
