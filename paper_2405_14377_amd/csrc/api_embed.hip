// extern "C" entry points for the TTM embedding table (Sec. 4.1):
// comera_tt_embed_workspace_bytes, comera_tt_embed_forward and
// comera_tt_embed_backward.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "embed_internal.h"

using namespace comera;

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
inline char *at(void *ws, size_t off) { return reinterpret_cast<char *>(ws) + off; }

bool embed_dims(const comera_tt_embed_shape *s, EmbedDims &dm) {
    if (!s || s->d < 1 || s->d > kMaxCores) return false;
    if (s->r[0] != 1 || s->r[s->d] != 1) return false;
    double V = 1, E = 1;
    for (int k = 0; k < s->d; ++k) {
        if (s->v[k] < 1 || s->e[k] < 1 || s->r[k] < 1 || s->r[k + 1] < 1 || s->r[k] > 4096) return false;
        if (double(s->r[k]) * double(s->v[k]) * double(s->e[k]) * double(s->r[k + 1]) > 2147483647.0) return false;
        V *= double(s->v[k]);
        E *= double(s->e[k]);
    }
    if (V >= 2147483647.0 || E >= 2147483647.0) return false;
    dm.d = s->d;
    dm.V = 1;
    dm.E = 1;
    dm.Vp = 1;
    dm.Ep = 1;
    for (int k = 0; k < s->d; ++k) {
        dm.V *= s->v[k];
        dm.E *= s->e[k];
        if (k < s->d - 1) {
            dm.Vp *= s->v[k];
            dm.Ep *= s->e[k];
        }
    }
    dm.Vs = int(s->v[s->d - 1]);
    dm.Es = int(s->e[s->d - 1]);
    dm.R = int(s->r[s->d - 1]);
    return true;
}

// Limits of the kernels' LDS staging; larger tables are refused.
bool embed_supported(const EmbedDims &dm) {
    double table = double(dm.Vp) * double(dm.Ep) * double(dm.R) * 4.0;
    return embed_kernels_support(int(dm.Ep), dm.R, dm.Es, dm.E) && embed_gs_fits(dm.R, dm.Vs, dm.Es) && table <= 8.0e9;
}

void embed_layout(const comera_tt_embed_shape *s, const EmbedDims &dm, int64_t n, EmbedLayout &L) {
    std::memset(&L, 0, sizeof(L));
    const int d = dm.d;
    size_t off = 0;
    for (int k = 0; k < d - 1; ++k) {
        L.gc[k] = off;
        off = align_up(off + sizeof(float) * size_t(s->r[k] * s->v[k] * s->e[k] * s->r[k + 1]));
    }
    int64_t Vl = 1, El = 1;
    for (int k = 1; k < d; ++k) {
        Vl *= s->v[k - 1];
        El *= s->e[k - 1];
        L.p[k] = off;
        off = align_up(off + sizeof(float) * size_t(Vl * El * s->r[k]));
    }
    const size_t nn = size_t(std::max<int64_t>(n, 1));
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + bytes);
        return o;
    };
    L.keysA = take(4 * nn);
    L.valsA = take(4 * nn);
    L.keysB = take(4 * nn);
    L.valsB = take(4 * nn);
    const size_t nblk = (nn + 1023) / 1024, nchunk = (nn + kEmbedItem - 1) / kEmbedItem;
    L.hist = take(4 * 256 * nblk);
    L.meta = take(4 * 16);
    L.S = take(sizeof(float) * nn * size_t(dm.E));
    L.Pfirst = take(sizeof(float) * nchunk * size_t(dm.E));
    L.Plast = take(sizeof(float) * nchunk * size_t(dm.E));
    L.dA = take(sizeof(float) * size_t(dm.Vp * dm.Ep * dm.R));
    L.dglast_part = take(sizeof(float) * size_t(kEmbedChunks) * size_t(dm.R) * dm.Vs * dm.Es);
    Vl = 1;
    El = 1;
    for (int k = 1; k < d - 1; ++k) {
        Vl *= s->v[k - 1];
        El *= s->e[k - 1];
        L.e[k] = take(sizeof(float) * size_t(Vl * El * s->r[k]));
    }
    {
        size_t adj_max = 0;
        int64_t Va = dm.Vp, Ea = dm.Ep;
        for (int k = d - 2; k >= 1; --k) {
            Va /= s->v[k];
            Ea /= s->e[k];
            int64_t M = Va * Ea, N = s->r[k], K = s->v[k] * s->e[k] * s->r[k + 1];
            int sp = split_for(M, N, K);
            L.adj_splits[k] = sp;
            if (sp > 1) adj_max = std::max(adj_max, sizeof(float) * size_t(sp) * size_t(M * N));
        }
        L.adj_part = take(adj_max);
    }
    Vl = 1;
    El = 1;
    for (int k = 0; k < d - 1; ++k) {
        int64_t K = Vl * El;
        int64_t M = s->r[k], N = s->v[k] * s->e[k] * s->r[k + 1];
        int64_t sp = split_for(M, N, K);
        L.meet_splits[k] = int(sp);
        L.gpart[k] = take(sizeof(float) * size_t(sp * M * N));
        Vl *= s->v[k];
        El *= s->e[k];
    }
    L.total = off;
}

// fold the masks into the prefix cores and build the prefix table
// A = P_{d-1}[Vp, Ep, r_{d-1}] (eq. emb_A1 over cores 0..d-2)
int build_prefix(const comera_tt_embed_shape *s, const EmbedLayout &L, const float *const *G, const float *const *D,
                 void *ws, void *stream, float **gc, float **P) {
    const int d = s->d;
    if (d == 1) return 0;
    FoldArgs fa;
    std::memset(&fa, 0, sizeof(fa));
    fa.d = d;
    fa.nfold = d - 1;
    fa.compacted = 0;
    fa.swap = 0;
    for (int k = 0; k < d; ++k) {
        fa.G[k] = G[k];
        fa.D[k] = (D && k < d - 1) ? D[k] : nullptr;
        gc[k] = k < d - 1 ? reinterpret_cast<float *>(at(ws, L.gc[k])) : nullptr;
        fa.Gc[k] = gc[k];
        fa.m[k] = int(s->v[k]);
        fa.n[k] = int(s->e[k]);
    }
    for (int k = 0; k <= d; ++k) {
        fa.r[k] = int(s->r[k]);
        fa.rc[k] = int(s->r[k]);
    }
    int e = launch_fold(fa, stream);
    if (e) return e;
    P[1] = gc[0];  // r_0 = 1: [v_0][e_0][r_1] is the folded core itself
    int64_t Vl = s->v[0], El = s->e[0];
    for (int k = 1; k < d - 1; ++k) {
        float *out = reinterpret_cast<float *>(at(ws, L.p[k + 1]));
        e = chain_gemm(P[k], gc[k], out, false, Vl, El, int(s->r[k]), int(s->v[k]), int(s->e[k]), int(s->r[k + 1]),
                       stream);
        if (e) return e;
        P[k + 1] = out;
        Vl *= s->v[k];
        El *= s->e[k];
    }
    return 0;
}

EmbedWs embed_ws(const EmbedLayout &L, void *ws) {
    EmbedWs w;
    w.keysA = reinterpret_cast<uint32_t *>(at(ws, L.keysA));
    w.valsA = reinterpret_cast<uint32_t *>(at(ws, L.valsA));
    w.keysB = reinterpret_cast<uint32_t *>(at(ws, L.keysB));
    w.valsB = reinterpret_cast<uint32_t *>(at(ws, L.valsB));
    w.hist = reinterpret_cast<int *>(at(ws, L.hist));
    w.meta = reinterpret_cast<int *>(at(ws, L.meta));
    w.S = reinterpret_cast<float *>(at(ws, L.S));
    w.Pfirst = reinterpret_cast<float *>(at(ws, L.Pfirst));
    w.Plast = reinterpret_cast<float *>(at(ws, L.Plast));
    w.dglast_part = reinterpret_cast<float *>(at(ws, L.dglast_part));
    return w;
}

comera_status hip_status(int e) { return e ? COMERA_ERR_HIP : COMERA_OK; }

}  // namespace

extern "C" {

size_t comera_tt_embed_workspace_bytes(const comera_tt_embed_shape *s, int64_t n_tokens) {
    EmbedDims dm;
    if (!embed_dims(s, dm) || n_tokens < 0) return 0;
    EmbedLayout L;
    embed_layout(s, dm, n_tokens, L);
    return L.total;
}

comera_status comera_tt_embed_forward(const comera_tt_embed_shape *s, const int64_t *ids, int64_t n_tokens,
                                      const float *const *G, const float *const *D, float *Y, void *ws,
                                      size_t ws_bytes, int32_t *err_flag, void *stream) {
    EmbedDims dm;
    if (!embed_dims(s, dm) || n_tokens < 0 || n_tokens >= 2147483647) return COMERA_ERR_INVALID_ARG;
    if (!embed_supported(dm)) return COMERA_ERR_UNSUPPORTED;
    if (n_tokens == 0) return COMERA_OK;
    if (!ids || !Y || !G) return COMERA_ERR_INVALID_ARG;
    for (int k = 0; k < s->d; ++k)
        if (!G[k]) return COMERA_ERR_INVALID_ARG;
    EmbedLayout L;
    embed_layout(s, dm, n_tokens, L);
    if (!ws || ws_bytes < L.total) return COMERA_ERR_WORKSPACE;
    float *gc[kMaxCores] = {};
    float *P[kMaxCores + 1] = {};
    int e = build_prefix(s, L, G, D, ws, stream, gc, P);
    if (e) return COMERA_ERR_HIP;
    const float *Apre = s->d > 1 ? P[s->d - 1] : nullptr;
    return hip_status(launch_embed_rows(ids, n_tokens, dm.V, Apre, G[s->d - 1], Y, int(dm.Ep), dm.R, dm.Vs, dm.Es,
                                        err_flag, stream));
}

comera_status comera_tt_embed_backward(const comera_tt_embed_shape *s, const int64_t *ids, int64_t n_tokens,
                                       const float *dY, const float *const *G, const float *const *D,
                                       float *const *dG, int32_t deterministic, void *ws, size_t ws_bytes,
                                       int32_t *err_flag, void *stream) {
    (void)deterministic;
    EmbedDims dm;
    if (!embed_dims(s, dm) || n_tokens < 0 || n_tokens >= 2147483647) return COMERA_ERR_INVALID_ARG;
    if (!embed_supported(dm)) return COMERA_ERR_UNSUPPORTED;
    if (!dG || !G) return COMERA_ERR_INVALID_ARG;
    const int d = s->d;
    for (int k = 0; k < d; ++k)
        if (!dG[k] || !G[k]) return COMERA_ERR_INVALID_ARG;
    if (n_tokens == 0) {
        for (int k = 0; k < d; ++k) {
            int e = launch_fill_zero(dG[k], sizeof(float) * size_t(s->r[k] * s->v[k] * s->e[k] * s->r[k + 1]), stream);
            if (e) return COMERA_ERR_HIP;
        }
        return COMERA_OK;
    }
    if (!ids || !dY) return COMERA_ERR_INVALID_ARG;
    EmbedLayout L;
    embed_layout(s, dm, n_tokens, L);
    if (!ws || ws_bytes < L.total) return COMERA_ERR_WORKSPACE;
    float *gc[kMaxCores] = {};
    float *P[kMaxCores + 1] = {};
    int e = build_prefix(s, L, G, D, ws, stream, gc, P);
    if (e) return COMERA_ERR_HIP;
    const float *Apre = d > 1 ? P[d - 1] : nullptr;
    EmbedWs w = embed_ws(L, ws);
    e = launch_embed_sort(ids, int(n_tokens), dm.V, w, err_flag, stream);
    if (e) return COMERA_ERR_HIP;
    e = launch_embed_segsum(dY, int(dm.E), int(n_tokens), dm.V, w, stream);
    if (e) return COMERA_ERR_HIP;
    e = launch_embed_dglast(w, int(n_tokens), dm.V, Apre, int(dm.Ep), dm.R, dm.Vs, dm.Es, stream);
    if (e) return COMERA_ERR_HIP;
    ExpandArgs xa;
    std::memset(&xa, 0, sizeof(xa));
    xa.d = d;
    xa.compacted = 0;
    for (int k = 0; k <= d; ++k) {
        xa.r[k] = int(s->r[k]);
        xa.rc[k] = int(s->r[k]);
    }
    for (int k = 0; k < d; ++k) {
        xa.D[k] = (D && k < d - 1) ? D[k] : nullptr;
        xa.dG[k] = dG[k];
        xa.m[k] = int(s->v[k]);
        xa.n[k] = int(s->e[k]);
    }
    xa.part[d - 1] = w.dglast_part;
    xa.splits[d - 1] = kEmbedChunks;
    if (d > 1) {
        // E_{d-1} = dA over the prefix table (blocked), then right
        // environments and meets on the prefix cores as for a linear layer
        float *Ek[kMaxCores + 1] = {};
        Ek[d - 1] = reinterpret_cast<float *>(at(ws, L.dA));
        e = launch_embed_dapre(w, int(n_tokens), dm.V, G[d - 1], dm.Vp, int(dm.Ep), dm.R, dm.Vs, dm.Es, int(s->v[d - 2]),
                               int(s->e[d - 2]), Ek[d - 1], stream);
        if (e) return COMERA_ERR_HIP;
        int64_t Vl = dm.Vp, El = dm.Ep;
        for (int k = d - 2; k >= 1; --k) {
            Vl /= s->v[k];
            El /= s->e[k];
            Ek[k] = reinterpret_cast<float *>(at(ws, L.e[k]));
            e = adjoint_gemm(Ek[k + 1], gc[k], Ek[k], Vl, El, int(s->r[k]), int(s->v[k]), int(s->e[k]),
                             int(s->r[k + 1]), int(s->v[k - 1]), int(s->e[k - 1]), L.adj_splits[k],
                             reinterpret_cast<float *>(at(ws, L.adj_part)), stream);
            if (e) return COMERA_ERR_HIP;
        }
        Vl = 1;
        El = 1;
        for (int k = 0; k < d - 1; ++k) {
            if (k == 0) {
                xa.part[0] = Ek[1];
                xa.splits[0] = 1;
            } else {
                float *part = reinterpret_cast<float *>(at(ws, L.gpart[k]));
                e = meet_gemm(P[k], Ek[k + 1], part, Vl, El, int(s->r[k]), int(s->v[k]), int(s->e[k]),
                              int(s->r[k + 1]), L.meet_splits[k], stream);
                if (e) return COMERA_ERR_HIP;
                xa.part[k] = part;
                xa.splits[k] = L.meet_splits[k];
            }
            Vl *= s->v[k];
            El *= s->e[k];
        }
    }
    return hip_status(launch_expand(xa, stream));
}

}  // extern "C"
