// Host-side planner for TTM layers: shape validation, rank-mask compaction,
// enumeration of contraction orders, cost model and workspace layout.
//
// The order family is the one of Prop. 4.1 (Sec. 4.2): contract consecutive
// cores into groups first, then sweep the activations through the groups in
// sequence.  A single group is the dense order (rebuild W, then one GEMM per
// batch product), which the large-batch analysis of Sec. 4.2 favours when the
// ranks are not small next to the mode sizes.  Rank masks (eq. Wcompress)
// with zero entries shrink the bonds: inactive slices are removed before any
// contraction.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>

#include "internal.h"

namespace comera {
namespace {

constexpr double kPeakF32 = 157.3e12;    // MI355X dense fp32 (vector and MFMA)
constexpr double kPeakBF16 = 2.5e15;     // MI355X dense bf16 MFMA
constexpr double kHbm = 8.0e12;          // MI355X HBM3E bytes/s
constexpr double kLaunch = 2.0e-6;       // cost charged per kernel launch
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int popcount_bits(const BondBits &b) {
    int c = 0;
    for (int i = 0; i < 4; ++i) c += __builtin_popcountll(b.w[i]);
    return c;
}

struct GroupDims {
    double I, J, rs, re, build_flops;
};

// Dimensions and build cost of the group of cores [s, e] (inclusive).
GroupDims group_dims(const comera_ttm_plan_s *p, int s, int e) {
    GroupDims g{1, 1, double(p->rho[s]), double(p->rho[e + 1]), 0};
    for (int k = s; k <= e; ++k) {
        if (k > s) g.build_flops += 2.0 * g.rs * g.I * g.J * p->s.n[k] * p->s.m[k] * p->rho[k] * p->rho[k + 1];
        g.I *= double(p->s.n[k]);
        g.J *= double(p->s.m[k]);
    }
    return g;
}

void describe(Order &o, int d) {
    char buf[160];
    int pos = 0;
    const char *name = o.kind == COMERA_ORDER_DENSE ? "dense" : o.kind == COMERA_ORDER_SWEEP_RL ? "sweep-rl"
                       : o.kind == COMERA_ORDER_SWEEP_LR ? "sweep-lr" : "zero";
    pos += snprintf(buf + pos, sizeof(buf) - pos, "%s [", name);
    for (int k = 0; k < d; ++k) {
        pos += snprintf(buf + pos, sizeof(buf) - pos, "%d", k);
        if (k + 1 < d) pos += snprintf(buf + pos, sizeof(buf) - pos, (o.cuts >> k) & 1u ? "][" : ",");
    }
    snprintf(buf + pos, sizeof(buf) - pos, "]");
    o.desc = buf;
}

void cost_order(const comera_ttm_plan_s *p, Order &o) {
    const int d = p->d;
    const double b = double(p->batch);
    const double peak = p->s.act == COMERA_BF16 ? kPeakBF16 : kPeakF32;
    const double esz = p->s.act == COMERA_BF16 ? 2.0 : 4.0;
    const double Nin = double(p->N_in), Nout = double(p->N_out);
    if (o.kind == COMERA_ORDER_ZERO) {
        o.flops_fwd = o.flops_bwd = 0;
        o.bytes = b * (Nout + Nin) * esz;
        o.t_pred = o.bytes / kHbm + 2 * kLaunch;
        return;
    }
    // groups
    std::vector<std::pair<int, int>> groups;
    int s = 0;
    for (int k = 0; k < d; ++k) {
        if (k == d - 1 || ((o.cuts >> k) & 1u)) {
            groups.push_back({s, k});
            s = k + 1;
        }
    }
    double build = 0;
    std::vector<GroupDims> gd;
    for (auto &g : groups) {
        gd.push_back(group_dims(p, g.first, g.second));
        build += gd.back().build_flops;
    }
    if (o.kind == COMERA_ORDER_DENSE) {
        // projections of dW onto every core: one adjoint step and one meet
        // per core, each 2 * |E_{k+1}| * rho_k flops.
        double proj = 0, Il = Nin, Jl = Nout;
        for (int k = d - 1; k >= 0; --k) {
            double Esz = Il * Jl * double(p->rho[k + 1]);
            proj += (k > 0 ? 4.0 : 0.0) * Esz * double(p->rho[k]);
            Il /= double(p->s.n[k]);
            Jl /= double(p->s.m[k]);
        }
        o.flops_fwd = build + 2.0 * b * Nin * Nout;
        o.flops_bwd = build + 4.0 * b * Nin * Nout + proj;
        o.bytes = b * (Nin + Nout) * esz * 2 + b * (Nin + Nout) * esz * 2 + Nin * Nout * (esz * 3 + 12.0);
        double launches = double(d) + 1 + double(d) + 3 + 2.0 * d;
        o.t_pred = (o.flops_fwd + o.flops_bwd - 2 * build) / peak + 2 * build / kPeakF32 + o.bytes / kHbm +
                   launches * kLaunch;
        return;
    }
    // sweeps
    const int G = int(groups.size());
    double sweep = 0, inter_bytes = 0;
    for (int gi = 0; gi < G; ++gi) {
        double Ib = 1, Ja = 1, Jb = 1, Ia = 1;  // I before / J after (RL); J before / I after (LR)
        for (int h = 0; h < gi; ++h) { Ib *= gd[h].I; Jb *= gd[h].J; }
        for (int h = gi + 1; h < G; ++h) { Ja *= gd[h].J; Ia *= gd[h].I; }
        const GroupDims &g = gd[gi];
        double outer = o.kind == COMERA_ORDER_SWEEP_RL ? Ib * Ja : Jb * Ia;
        sweep += 2.0 * b * outer * g.I * g.re * g.rs * g.J;
        double state = o.kind == COMERA_ORDER_SWEEP_RL ? b * Ib * g.rs * g.J * Ja : b * Jb * g.J * g.re * Ia;
        if (gi != (o.kind == COMERA_ORDER_SWEEP_RL ? 0 : G - 1)) inter_bytes += state * 4.0 * 2;
    }
    o.flops_fwd = build + sweep;
    o.flops_bwd = build + 2.0 * sweep;
    o.bytes = b * (Nin + Nout) * esz * 4 + inter_bytes * 3;
    double launches = 3.0 * G + 2.0 * d;
    o.t_pred = (3.0 * sweep) / peak + 2 * build / kPeakF32 + o.bytes / kHbm + launches * kLaunch;
}

bool validate(const comera_ttm_shape *s, int64_t batch) {
    if (!s || s->d < 1 || s->d > kMaxCores || batch < 0) return false;
    if (s->act != COMERA_F32 && s->act != COMERA_BF16) return false;
    if (s->r[0] != 1 || s->r[s->d] != 1) return false;
    double nin = 1, nout = 1;
    for (int k = 0; k < s->d; ++k) {
        if (s->n[k] < 1 || s->m[k] < 1 || s->r[k] < 1 || s->r[k + 1] < 1) return false;
        if (s->r[k] > 4096) return false;
        // every core (and its gradient) is indexed with 32-bit offsets
        if (double(s->r[k]) * double(s->m[k]) * double(s->n[k]) * double(s->r[k + 1]) > 2147483647.0) return false;
        nin *= double(s->n[k]);
        nout *= double(s->m[k]);
    }
    if (nin > 2147483647.0 || nout > 2147483647.0) return false;
    return true;
}

}  // namespace

void layout_dense(comera_ttm_plan_s *p) {
    DenseLayout &L = p->dense;
    std::memset(&L, 0, sizeof(L));
    const int d = p->d;
    const size_t esz = p->s.act == COMERA_BF16 ? 2 : 4;
    size_t off = 0;
    for (int k = 0; k < d; ++k) {
        L.gc[k] = off;
        off = align_up(off + sizeof(float) * size_t(p->rho[k] * p->s.m[k] * p->s.n[k] * p->rho[k + 1]));
    }
    int64_t Il = 1, Jl = 1;
    for (int k = 1; k < d; ++k) {
        Il *= p->s.n[k - 1];
        Jl *= p->s.m[k - 1];
        L.p[k] = off;
        off = align_up(off + sizeof(float) * size_t(Il * Jl * p->rho[k]));
    }
    L.w = off;
    off = align_up(off + esz * size_t(p->N_in * p->N_out));
    L.ones = off;
    off = align_up(off + sizeof(float));
    // dW = X^T dY split over tokens so that the grid holds >= ~512 workgroups
    // (fp32: about three 128 x 128 tiles per CU, measured best on gfx950)
    int64_t tiles = ((p->N_in + 127) / 128) * ((p->N_out + 127) / 128);
    int64_t b = std::max<int64_t>(p->batch, 1);
    int64_t splits = std::max<int64_t>(1, (512 + tiles - 1) / tiles);
    if (p->s.act == COMERA_F32) splits = std::max<int64_t>(1, (768 + tiles / 2) / tiles);
    splits = std::min<int64_t>(splits, std::max<int64_t>(1, b / 256));
    splits = std::min<int64_t>(splits, 64);
    int64_t kchunk = (b + splits - 1) / splits;
    kchunk = (kchunk + 31) / 32 * 32;
    splits = (b + kchunk - 1) / kchunk;
    L.dw_splits = int(splits);
    L.dw_kchunk = kchunk;
    // fp32 dX = dY W^T split over N_out when the output alone gives too few
    // 128 x 128 tiles (the partials are summed in a fixed order)
    L.dx_splits = 1;
    L.dx_kchunk = p->N_out;
    if (p->s.act == COMERA_F32) {
        const int64_t xt = ((b + 127) / 128) * ((p->N_in + 127) / 128);
        int64_t sx = std::max<int64_t>(1, (768 + xt / 2) / xt);
        sx = std::min<int64_t>(std::min<int64_t>(sx, 8), std::max<int64_t>(1, p->N_out / 512));
        if (sx > 1) {
            int64_t kc = (p->N_out + sx - 1) / sx;
            kc = (kc + 31) / 32 * 32;
            L.dx_splits = int((p->N_out + kc - 1) / kc);
            L.dx_kchunk = kc;
            L.dx_part = off;
            off = align_up(off + sizeof(float) * size_t(L.dx_splits) * size_t(b) * size_t(p->N_in));
        }
    }
    L.proj = true;
    for (int k = 1; k < d; ++k) L.proj = L.proj && proj_supported(int(p->rho[k]));
    if (L.proj) {
        // fused projections: dW stays as its split partials, each step writes
        // its environment as column-chunk slices and its meet partials
        L.dw_part = off;
        off = align_up(off + sizeof(float) * size_t(splits) * size_t(p->N_in * p->N_out));
        L.dw = L.dw_part;
        L.e_slices[d] = int(splits);
        int64_t Ia = p->N_in, Ja = p->N_out;
        for (int k = d - 1; k >= 1; --k) {
            Ia /= p->s.n[k];
            Ja /= p->s.m[k];
            const int64_t rows = Ia * Ja, cols = p->s.n[k] * p->s.m[k] * p->rho[k + 1];
            const int A = int(p->rho[k]);
            int RT = 0, CT = 0;
            proj_tiles(rows, cols, A, RT, CT);
            L.proj_rt[k] = RT;
            L.proj_ct[k] = CT;
            L.e_slices[k] = int((cols + CT - 1) / CT);
            L.meet_splits[k] = int((rows + RT - 1) / RT);
            L.e[k] = off;
            off = align_up(off + sizeof(float) * size_t(L.e_slices[k]) * size_t(rows * A));
            L.gpart[k] = off;
            off = align_up(off + sizeof(float) * size_t(L.meet_splits[k]) * size_t(A * cols));
        }
        L.meet_splits[0] = L.e_slices[1];
        L.total = off;
        return;
    }
    L.dw_part = off;
    if (splits > 1) off = align_up(off + sizeof(float) * size_t(splits) * size_t(p->N_in * p->N_out));
    L.dw = off;
    off = align_up(off + sizeof(float) * size_t(p->N_in * p->N_out));
    Il = 1;
    Jl = 1;
    for (int k = 1; k < d; ++k) {
        Il *= p->s.n[k - 1];
        Jl *= p->s.m[k - 1];
        L.e[k] = off;
        off = align_up(off + sizeof(float) * size_t(Il * Jl * p->rho[k]));
    }
    // adjoint k (k = d-1..1): M = I_<k J_<k, N = rho_k, K = n_k m_k rho_{k+1}
    size_t adj_max = 0;
    {
        int64_t Ia = p->N_in, Ja = p->N_out;
        for (int k = d - 1; k >= 1; --k) {
            Ia /= p->s.n[k];
            Ja /= p->s.m[k];
            int64_t M = Ia * Ja, N = p->rho[k], K = p->s.n[k] * p->s.m[k] * p->rho[k + 1];
            int sp = split_for(M, N, K);
            L.adj_splits[k] = sp;
            if (sp > 1) adj_max = std::max(adj_max, sizeof(float) * size_t(sp) * size_t(M * N));
        }
    }
    L.adj_part = off;
    off = align_up(off + adj_max);
    // meet k: M = rho_k, N = n_k m_k rho_{k+1}, K = I_<k J_<k, split over K so
    // that the grid holds a few hundred workgroups and each split keeps >= 512 k
    Il = 1;
    Jl = 1;
    for (int k = 0; k < d; ++k) {
        int64_t K = Il * Jl;
        int64_t M = p->rho[k], N = p->s.n[k] * p->s.m[k] * p->rho[k + 1];
        int64_t sp = split_for(M, N, K);
        L.meet_splits[k] = int(sp);
        L.gpart[k] = off;
        off = align_up(off + sizeof(float) * size_t(sp * M * N));
        Il *= p->s.n[k];
        Jl *= p->s.m[k];
    }
    L.total = off;
}

}  // namespace comera

using namespace comera;

extern "C" {

comera_status comera_ttm_plan(const comera_ttm_shape *s, int64_t batch, const uint8_t *mask_active,
                              int32_t force_order, comera_ttm_plan_t *out) {
    if (!out) return COMERA_ERR_INVALID_ARG;
    *out = nullptr;
    if (!validate(s, batch)) return COMERA_ERR_INVALID_ARG;
    comera_ttm_plan_s *p = new (std::nothrow) comera_ttm_plan_s();
    if (!p) return COMERA_ERR_INTERNAL;
    p->s = *s;
    p->batch = batch;
    p->d = s->d;
    p->N_in = 1;
    p->N_out = 1;
    for (int k = 0; k < p->d; ++k) {
        p->N_in *= s->n[k];
        p->N_out *= s->m[k];
    }
    std::memset(p->act, 0, sizeof(p->act));
    for (int k = 0; k <= p->d; ++k) p->rho[k] = s->r[k];
    // rank-mask compaction (bond k sits between cores k-1 and k, 0-based)
    bool can_compact = true;
    for (int k = 1; k < p->d; ++k) can_compact = can_compact && s->r[k] <= 256;
    if (mask_active) {
        size_t off = 0;
        for (int k = 1; k < p->d; ++k) {
            int cnt = 0;
            for (int a = 0; a < s->r[k]; ++a) {
                bool on = mask_active[off + a] != 0;
                cnt += on;
                if (on && a < 256) p->act[k].w[a >> 6] |= 1ull << (a & 63);
            }
            off += size_t(s->r[k]);
            if (cnt == 0) p->zero = true;
            if (can_compact) {
                p->rho[k] = cnt;
                if (cnt != s->r[k]) p->compacted = true;
            }
        }
    }
    if (!p->compacted) {
        for (int k = 1; k < p->d; ++k) {
            std::memset(&p->act[k], 0, sizeof(BondBits));
            for (int a = 0; a < std::min<int64_t>(s->r[k], 256); ++a) p->act[k].w[a >> 6] |= 1ull << (a & 63);
            p->rho[k] = s->r[k];
        }
    }
    // enumerate: index 0 = dense; then per cut mask (increasing) RL, LR
    const int d = p->d;
    {
        Order o;
        o.kind = COMERA_ORDER_DENSE;
        o.cuts = 0;
        p->orders.push_back(o);
    }
    for (uint32_t cuts = 1; cuts < (1u << (d - 1)); ++cuts) {
        for (int dir = 0; dir < 2; ++dir) {
            Order o;
            o.kind = dir == 0 ? COMERA_ORDER_SWEEP_RL : COMERA_ORDER_SWEEP_LR;
            o.cuts = cuts;
            p->orders.push_back(o);
        }
    }
    for (auto &o : p->orders) {
        describe(o, d);
        if (p->zero) {
            Order z;
            z.kind = COMERA_ORDER_ZERO;
            cost_order(p, z);
            o.flops_fwd = z.flops_fwd;
            o.flops_bwd = z.flops_bwd;
            o.bytes = z.bytes;
            o.t_pred = z.t_pred;
            o.executable = true;
        } else {
            cost_order(p, o);
            o.executable = o.kind == COMERA_ORDER_DENSE;
        }
    }
    if (force_order >= 0) {
        if (force_order >= int32_t(p->orders.size())) {
            delete p;
            return COMERA_ERR_INVALID_ARG;
        }
        if (!p->orders[force_order].executable) {
            delete p;
            return COMERA_ERR_UNSUPPORTED;
        }
        p->chosen = force_order;
    } else {
        int best = -1;
        for (int i = 0; i < int(p->orders.size()); ++i) {
            if (!p->orders[i].executable) continue;
            if (best < 0 || p->orders[i].t_pred < p->orders[best].t_pred) best = i;
        }
        p->chosen = best < 0 ? 0 : best;
    }
    if (!p->zero) layout_dense(p);
    p->ws_bytes = p->zero ? 0 : p->dense.total;
    *out = p;
    return COMERA_OK;
}

int32_t comera_ttm_plan_num_orders(comera_ttm_plan_t p) { return p ? int32_t(p->orders.size()) : 0; }

int32_t comera_ttm_plan_chosen(comera_ttm_plan_t p) { return p ? p->chosen : -1; }

comera_status comera_ttm_plan_order_info(comera_ttm_plan_t p, int32_t i, char *desc, size_t len,
                                         int32_t *kind, double *flops_fwd, double *flops_bwd,
                                         double *bytes, int32_t *executable) {
    if (!p || i < 0 || i >= int32_t(p->orders.size())) return COMERA_ERR_INVALID_ARG;
    const Order &o = p->orders[i];
    if (desc && len > 0) {
        std::strncpy(desc, o.desc.c_str(), len - 1);
        desc[len - 1] = 0;
    }
    if (kind) *kind = p->zero ? COMERA_ORDER_ZERO : o.kind;
    if (flops_fwd) *flops_fwd = o.flops_fwd;
    if (flops_bwd) *flops_bwd = o.flops_bwd;
    if (bytes) *bytes = o.bytes;
    if (executable) *executable = o.executable ? 1 : 0;
    return COMERA_OK;
}

size_t comera_ttm_workspace_bytes(comera_ttm_plan_t p) { return p ? p->ws_bytes : 0; }

void comera_ttm_plan_destroy(comera_ttm_plan_t p) {
    if (!p) return;
    timing_clear(p);
    delete p;
}

const char *comera_status_string(comera_status s) {
    switch (s) {
        case COMERA_OK: return "ok";
        case COMERA_ERR_INVALID_ARG: return "invalid argument";
        case COMERA_ERR_UNSUPPORTED: return "unsupported request";
        case COMERA_ERR_WORKSPACE: return "workspace missing or too small";
        case COMERA_ERR_HIP: return "HIP runtime error";
        case COMERA_ERR_INTERNAL: return "internal error";
    }
    return "unknown status";
}

}  // extern "C"
