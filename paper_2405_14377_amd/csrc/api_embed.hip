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
constexpr size_t kMaxLds = 64 * 1024;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
inline char *at(void *ws, size_t off) { return reinterpret_cast<char *>(ws) + off; }

bool embed_dims(const comera_tt_embed_shape *s, EmbedDims &dm) {
    if (!s || s->d < 1 || s->d > kMaxCores) return false;
    if (s->r[0] != 1 || s->r[s->d] != 1) return false;
    double V = 1, E = 1;
    for (int k = 0; k < s->d; ++k) {
        if (s->v[k] < 1 || s->e[k] < 1 || s->r[k] < 1 || s->r[k + 1] < 1 || s->r[k] > 4096) return false;
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
    size_t rows_lds = sizeof(float) * (size_t(dm.Ep) * dm.R + size_t(dm.R) * dm.Es);
    size_t dg_lds = sizeof(float) * size_t(dm.R) * dm.Vs * dm.Es;
    double table = double(dm.Vp) * double(dm.Ep) * double(dm.R) * 4.0;
    return rows_lds <= kMaxLds && dg_lds <= kMaxLds && table <= 8.0e9;
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
    L.meta = take(4 * 16);
    L.uid = take(4 * (nn + 1));
    L.ustart = take(4 * (nn + 1));
    L.useg_item = take(4 * (nn + 1));
    L.item_u = take(4 * (nn + 1));
    L.item_beg = take(4 * (nn + 1));
    L.item_len = take(4 * (nn + 1));
    L.S = take(sizeof(float) * nn * size_t(dm.E));
    L.Spart = take(sizeof(float) * nn * size_t(dm.E));
    L.dA = take(sizeof(float) * size_t(dm.Vp * dm.Ep * dm.R));
    L.dglast_part = take(sizeof(float) * size_t(kEmbedChunks) * size_t(dm.R) * dm.Vs * dm.Es);
    Vl = 1;
    El = 1;
    for (int k = 1; k < d - 1; ++k) {
        Vl *= s->v[k - 1];
        El *= s->e[k - 1];
        L.e[k] = take(sizeof(float) * size_t(Vl * El * s->r[k]));
    }
    Vl = 1;
    El = 1;
    for (int k = 0; k < d - 1; ++k) {
        int64_t XY = Vl * El;
        int64_t outs = s->r[k] * s->v[k] * s->e[k] * s->r[k + 1];
        int64_t sp = std::min<int64_t>((XY + 511) / 512, 4096);
        sp = std::max<int64_t>(1, std::min<int64_t>(sp, std::max<int64_t>(1, (1 << 20) / std::max<int64_t>(outs, 1))));
        L.meet_splits[k] = int(sp);
        L.gpart[k] = take(sizeof(float) * size_t(sp * outs));
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
    int64_t Vl = 1, El = 1;
    const float *prev = nullptr;
    for (int k = 0; k < d - 1; ++k) {
        float *out = reinterpret_cast<float *>(at(ws, L.p[k + 1]));
        e = launch_chain(prev, gc[k], out, nullptr, Vl, El, int(s->r[k]), int(s->v[k]), int(s->e[k]),
                         int(s->r[k + 1]), 1, stream);
        if (e) return e;
        P[k + 1] = out;
        prev = out;
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
    w.meta = reinterpret_cast<int *>(at(ws, L.meta));
    w.uid = reinterpret_cast<int *>(at(ws, L.uid));
    w.ustart = reinterpret_cast<int *>(at(ws, L.ustart));
    w.useg_item = reinterpret_cast<int *>(at(ws, L.useg_item));
    w.item_u = reinterpret_cast<int *>(at(ws, L.item_u));
    w.item_beg = reinterpret_cast<int *>(at(ws, L.item_beg));
    w.item_len = reinterpret_cast<int *>(at(ws, L.item_len));
    w.S = reinterpret_cast<float *>(at(ws, L.S));
    w.Spart = reinterpret_cast<float *>(at(ws, L.Spart));
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
    e = launch_embed_segsum(dY, int(dm.E), int(n_tokens), w, stream);
    if (e) return COMERA_ERR_HIP;
    e = launch_embed_dglast(w, Apre, int(dm.Ep), dm.R, dm.Vs, dm.Es, stream);
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
        // E_{d-1} = dA over the prefix table, then environments and meets on
        // the prefix cores as for a linear layer (row factor = core axis 1)
        float *Ek[kMaxCores + 1] = {};
        Ek[d - 1] = reinterpret_cast<float *>(at(ws, L.dA));
        e = launch_embed_dapre(w, G[d - 1], dm.Vp, int(dm.Ep), dm.R, dm.Vs, dm.Es, Ek[d - 1], stream);
        if (e) return COMERA_ERR_HIP;
        int64_t Vl = dm.Vp, El = dm.Ep;
        for (int k = d - 2; k >= 1; --k) {
            Vl /= s->v[k];
            El /= s->e[k];
            Ek[k] = reinterpret_cast<float *>(at(ws, L.e[k]));
            e = launch_adjoint(Ek[k + 1], gc[k], Ek[k], Vl, El, int(s->r[k]), int(s->v[k]), int(s->e[k]),
                               int(s->r[k + 1]), 1, stream);
            if (e) return COMERA_ERR_HIP;
        }
        Vl = 1;
        El = 1;
        for (int k = 0; k < d - 1; ++k) {
            float *part = reinterpret_cast<float *>(at(ws, L.gpart[k]));
            e = launch_meet(k == 0 ? nullptr : P[k], Ek[k + 1], part, Vl, El, int(s->r[k]), int(s->v[k]),
                            int(s->e[k]), int(s->r[k + 1]), 1, L.meet_splits[k], stream);
            if (e) return COMERA_ERR_HIP;
            xa.part[k] = part;
            xa.splits[k] = L.meet_splits[k];
            Vl *= s->v[k];
            El *= s->e[k];
        }
    }
    return hip_status(launch_expand(xa, stream));
}

}  // extern "C"
