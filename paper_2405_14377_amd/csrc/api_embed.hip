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
    const double table = double(dm.Vp) * double(dm.Ep) * double(dm.R) * 4.0;
    return embed_kernels_support(dm.Ep, dm.R, dm.Vs, dm.Es, dm.d) && table <= 8.0e9;
}

int radix_passes(int64_t V) {
    int bits = 0;
    while ((int64_t(1) << bits) <= V) ++bits;   // keys 0..V inclusive (V marks an out-of-range id)
    return (bits + 7) / 8;
}

void embed_layout(const comera_tt_embed_shape *s, const EmbedDims &dm, int64_t n, EmbedLayout &L) {
    std::memset(&L, 0, sizeof(L));
    const int d = dm.d;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + bytes);
        return o;
    };
    for (int k = 0; k < d - 1; ++k) L.gc[k] = take(sizeof(float) * size_t(s->r[k] * s->v[k] * s->e[k] * s->r[k + 1]));
    int64_t Vl = 1, El = 1;
    for (int k = 1; k < d; ++k) {
        Vl *= s->v[k - 1];
        El *= s->e[k - 1];
        L.p[k] = take(sizeof(float) * size_t(Vl * El * s->r[k]));
    }
    const size_t nn = size_t(std::max<int64_t>(n, 1));
    L.passes = radix_passes(dm.V);
    L.keysA = take(4 * nn);
    L.valsA = take(4 * nn);
    L.keysB = take(4 * nn);
    L.valsB = take(4 * nn);
    const size_t nblk = (nn + 1023) / 1024, nchunk = (nn + kEmbedItem - 1) / kEmbedItem;
    L.hist = take(4 * (256 * nblk + nblk));   // one pass's digit histograms, then out-of-range counts
    L.meta = take(4 * 16);
    L.headpos = take(4 * size_t(dm.V));
    L.S = take(sizeof(float) * nn * size_t(dm.E));
    L.Pfirst = take(sizeof(float) * nchunk * size_t(dm.E));
    L.Plast = take(sizeof(float) * nchunk * size_t(dm.E));
    L.nvp = embed_dglast_chunks(dm.Vp);
    if (d > 1) {
        L.dA = take(sizeof(float) * size_t(dm.Vp * dm.Ep * dm.R));
        L.dglast_part = take(sizeof(float) * size_t(L.nvp) * size_t(dm.R) * dm.Vs * dm.Es);
    }
    // projections of dA onto the prefix cores k = d-2 .. 1, as for a linear
    // layer: rows (V_<k, E_<k), columns (v_k, e_k, r_{k+1}), rank r_k
    L.e_slices[d - 1] = 1;
    int64_t Va = dm.Vp, Ea = dm.Ep;
    for (int k = d - 2; k >= 1; --k) {
        Va /= s->v[k];
        Ea /= s->e[k];
        const int64_t rows = Va * Ea, cols = s->v[k] * s->e[k] * s->r[k + 1];
        const int A = int(s->r[k]);
        int RT = 0, CT = 0;
        proj_tiles(rows, cols, A, RT, CT);
        L.proj_rt[k] = RT;
        L.proj_ct[k] = CT;
        L.e_slices[k] = int((cols + CT - 1) / CT);
        L.meet_splits[k] = int((rows + RT - 1) / RT);
        L.e[k] = take(sizeof(float) * size_t(L.e_slices[k]) * size_t(rows * A));
        L.gpart[k] = take(sizeof(float) * size_t(L.meet_splits[k]) * size_t(A * cols));
    }
    L.total = off;
}

// fold the masks into the prefix cores and build the prefix table
// A = P_{d-1} (eq. emb_A1 over cores 0..d-2), stored [Vp][r_{d-1}][Ep]
int build_prefix(const comera_tt_embed_shape *s, const EmbedLayout &L, const float *const *G, const float *const *D,
                 void *ws, void *stream, float **gc, float **P) {
    const int d = s->d;
    if (d == 1) return 0;
    if (d == 3 && embed_table_supported(int(s->r[1]), int(s->e[0]))) {
        // one kernel: the table straight from the raw cores 0 and 1, and their
        // folded copies for the backward's projections
        gc[0] = reinterpret_cast<float *>(at(ws, L.gc[0]));
        gc[1] = reinterpret_cast<float *>(at(ws, L.gc[1]));
        P[1] = gc[0];
        P[2] = reinterpret_cast<float *>(at(ws, L.p[2]));
        return launch_embed_table(G[0], D ? D[0] : nullptr, G[1], D ? D[1] : nullptr, P[2], gc[0], gc[1],
                                  int(s->v[0]), int(s->v[1]), int(s->e[0]), int(s->e[1]), int(s->r[1]),
                                  int(s->r[2]), stream);
    }
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
        fa.st[k] = core_strides(int(s->r[k]), fa.m[k], fa.n[k], int(s->r[k + 1]), false);
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
        // the prefix table itself (k = d-2) is written rank-major, [Vp][R][Ep],
        // so that a wave reads a row A[vp, :, a] with coalesced loads
        e = chain_gemm(P[k], gc[k], out, false, Vl, El, int(s->r[k]), int(s->v[k]), int(s->e[k]), int(s->r[k + 1]),
                       stream, k == d - 2 ? kChainRankMajor : kChainNormal);
        if (e) return e;
        P[k + 1] = out;
        Vl *= s->v[k];
        El *= s->e[k];
    }
    return 0;
}

// pointers of the folded prefix cores and chains that build_prefix wrote
int prefix_ptrs(const comera_tt_embed_shape *s, const EmbedLayout &L, void *ws, float **gc, float **P) {
    const int d = s->d;
    if (d == 1) return 0;
    for (int k = 0; k < d - 1; ++k) gc[k] = reinterpret_cast<float *>(at(ws, L.gc[k]));
    P[1] = gc[0];
    for (int k = 1; k < d - 1; ++k) P[k + 1] = reinterpret_cast<float *>(at(ws, L.p[k + 1]));
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
    w.headpos = reinterpret_cast<int *>(at(ws, L.headpos));
    w.S = reinterpret_cast<float *>(at(ws, L.S));
    w.Pfirst = reinterpret_cast<float *>(at(ws, L.Pfirst));
    w.Plast = reinterpret_cast<float *>(at(ws, L.Plast));
    w.dA = L.dA ? reinterpret_cast<float *>(at(ws, L.dA)) : nullptr;
    w.dglast_part = L.dglast_part ? reinterpret_cast<float *>(at(ws, L.dglast_part)) : nullptr;
    return w;
}

// the prefix-core projections take ranks up to the projection kernel's limit
bool embed_proj_ok(const comera_tt_embed_shape *s) {
    for (int k = 1; k < s->d - 1; ++k)
        if (!proj_supported(int(s->r[k]))) return false;
    return true;
}

comera_status hip_status(int e) { return note_hip(e, "embedding kernel") ? COMERA_ERR_HIP : COMERA_OK; }

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
    // the prefix table is rank-major when it comes from a chain (d >= 3)
    return hip_status(launch_embed_rows(ids, n_tokens, dm.V, Apre, s->d >= 3, G[s->d - 1], Y, int(dm.Ep), dm.R, dm.Vs,
                                        dm.Es, err_flag, stream));
}

comera_status comera_tt_embed_backward(const comera_tt_embed_shape *s, const int64_t *ids, int64_t n_tokens,
                                       const float *dY, const float *const *G, const float *const *D,
                                       float *const *dG, int32_t deterministic, void *ws, size_t ws_bytes,
                                       int32_t *err_flag, void *stream) {
    (void)deterministic;
    return comera_tt_embed_backward_ex(s, ids, n_tokens, dY, G, D, dG, 0, ws, ws_bytes, err_flag, stream);
}

comera_status comera_tt_embed_backward_ex(const comera_tt_embed_shape *s, const int64_t *ids, int64_t n_tokens,
                                          const float *dY, const float *const *G, const float *const *D,
                                          float *const *dG, int32_t flags, void *ws, size_t ws_bytes,
                                          int32_t *err_flag, void *stream) {
    if (flags & ~int32_t(COMERA_EMBED_REUSE_FORWARD)) return COMERA_ERR_INVALID_ARG;
    EmbedDims dm;
    if (!embed_dims(s, dm) || n_tokens < 0 || n_tokens >= 2147483647) return COMERA_ERR_INVALID_ARG;
    if (!embed_supported(dm) || !embed_proj_ok(s)) return COMERA_ERR_UNSUPPORTED;
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
    int e = (flags & COMERA_EMBED_REUSE_FORWARD) ? prefix_ptrs(s, L, ws, gc, P)
                                                 : build_prefix(s, L, G, D, ws, stream, gc, P);
    if (e) return COMERA_ERR_HIP;
    const float *Apre = d > 1 ? P[d - 1] : nullptr;
    EmbedWs w = embed_ws(L, ws);
    const int n = int(n_tokens);
    // group tokens by id (dA cleared on the way: prefixes without ids keep 0)
    e = launch_embed_sort(ids, n, dm.V, L.passes, w, err_flag, dm.V, w.dA, d > 1 ? dm.Vp * dm.Ep * dm.R : 0, stream);
    if (e) return COMERA_ERR_HIP;
    e = launch_embed_segsum(dY, int(dm.E), n, L.passes, w, stream);
    if (e) return COMERA_ERR_HIP;
    if (d == 1) return hip_status(launch_embed_gather(w, dm.V, int(dm.E), dG[0], stream));
    e = launch_embed_dapre(w, G[d - 1], dm.Vp, int(dm.Ep), dm.R, dm.Vs, dm.Es, int(s->v[d - 2]), int(s->e[d - 2]),
                           stream);
    if (e) return COMERA_ERR_HIP;
    e = launch_embed_dglast(w, Apre, d >= 3, dm.Vp, int(dm.Ep), dm.R, dm.Vs, dm.Es, stream);
    if (e) return COMERA_ERR_HIP;
    // dA is E_{d-1} for the prefix cores: project it right to left as for a
    // linear layer (folded cores gc[k], left chains P[k])
    ExpandArgs xa;
    std::memset(&xa, 0, sizeof(xa));
    const float *En = w.dA;
    int nin = 1;
    int64_t in_stride = 0;
    int64_t Vl = dm.Vp, El = dm.Ep;
    for (int k = d - 2; k >= 1; --k) {
        Vl /= s->v[k];
        El /= s->e[k];
        const int A = int(s->r[k]);
        const int64_t rows = Vl * El, cols = s->v[k] * s->e[k] * s->r[k + 1];
        ProjArgs pa;
        pa.En = En;
        pa.nin = nin;
        pa.in_stride = in_stride;
        pa.Gc = gc[k];
        pa.P = P[k];
        pa.Eout = reinterpret_cast<float *>(at(ws, L.e[k]));
        pa.out_stride = rows * A;
        const int64_t nxp = s->v[k - 1], nyp = s->e[k - 1], NJp = El / nyp;
        pa.rmap.nd = 4;
        pa.rmap.radix[1] = nxp;
        pa.rmap.radix[2] = NJp;
        pa.rmap.radix[3] = nyp;
        pa.rmap.stride[0] = NJp * nxp * nyp * A;
        pa.rmap.stride[1] = nyp * A;
        pa.rmap.stride[2] = nxp * nyp * A;
        pa.rmap.stride[3] = A;
        pa.part = reinterpret_cast<float *>(at(ws, L.gpart[k]));
        pa.rows = rows;
        pa.cols = cols;
        pa.A = A;
        pa.RT = L.proj_rt[k];
        pa.CT = L.proj_ct[k];
        e = launch_proj(pa, stream);
        if (e) return COMERA_ERR_HIP;
        xa.part[k] = pa.part;
        xa.splits[k] = L.meet_splits[k];
        En = pa.Eout;
        nin = L.e_slices[k];
        in_stride = pa.out_stride;
    }
    xa.part[0] = En;     // the gradient of core 0 is E_1 (or dA itself when d = 2)
    xa.splits[0] = nin;
    xa.part[d - 1] = w.dglast_part;
    xa.splits[d - 1] = L.nvp;
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
        xa.st[k] = core_strides(int(s->r[k]), xa.m[k], xa.n[k], int(s->r[k + 1]), false);
    }
    return hip_status(launch_expand(xa, stream));
}

}  // extern "C"
