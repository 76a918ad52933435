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
constexpr double kLaunch = 6.0e-6;       // cost of one small kernel launch (measured 5-10 us back to back)
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
                       : o.kind == COMERA_ORDER_SWEEP_LR ? "sweep-lr" : o.kind == COMERA_ORDER_FUSED_RL ? "fused-rl"
                       : "zero";
    pos += snprintf(buf + pos, sizeof(buf) - pos, "%s [", name);
    for (int k = 0; k < d; ++k) {
        pos += snprintf(buf + pos, sizeof(buf) - pos, "%d", k);
        if (k + 1 < d) pos += snprintf(buf + pos, sizeof(buf) - pos, (o.cuts >> k) & 1u ? "][" : ",");
    }
    snprintf(buf + pos, sizeof(buf) - pos, "]");
    o.desc = buf;
}

// Time of one launch: its work at half the dense peak plus its bytes at the
// HBM rate, and never below the launch cost.
double launch_time(double flops, double bytes, double peak) {
    return std::max(kLaunch, flops / (0.5 * peak) + bytes / kHbm);
}

// Flops of the projections of a group's matrix gradient onto its cores (one
// environment step and one meet per core but the first; eq. back Gi).
double proj_flops(const comera_ttm_plan_s *p, int s, int e, double rs, double re) {
    double I = 1, J = 1;
    for (int k = s; k <= e; ++k) {
        I *= double(p->s.n[k]);
        J *= double(p->s.m[k]);
    }
    double f = 0;
    for (int k = e; k > s; --k) {
        I /= double(p->s.n[k]);
        J /= double(p->s.m[k]);
        const double right = k == e ? re : double(p->rho[k + 1]);
        f += 4.0 * rs * I * J * double(p->s.n[k]) * double(p->s.m[k]) * right * double(p->rho[k]);
    }
    return f;
}

// Predicted flops, bytes and time of one forward plus one backward call.
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
    const int G = int(groups.size());
    double build = 0, t_build = kLaunch;   // the fold
    std::vector<GroupDims> gd;
    for (auto &g : groups) {
        gd.push_back(group_dims(p, g.first, g.second));
        build += gd.back().build_flops;
        const int dg = g.second - g.first + 1;
        const double steps = dg > 1 ? dg - 1 : (p->s.act == COMERA_BF16 || o.kind == COMERA_ORDER_DENSE ? 1 : 0);
        t_build += steps * kLaunch + gd.back().build_flops / (0.5 * kPeakF32);
    }
    if (o.kind == COMERA_ORDER_FUSED_RL) {
        // per token, core k (0-based) is a product of (prod n before k) x
        // (prod m after k) rows, n_k rho_{k+1} contraction and rho_k m_k
        // columns; the backward recomputes the forward states (all but the
        // last step), sweeps dY and takes one meet per core of the same size
        double f_all = 0, f_first = 0;
        for (int k = 0; k < d; ++k) {
            double nl = 1, mg = 1;
            for (int h = 0; h < k; ++h) nl *= double(p->s.n[h]);
            for (int h = k + 1; h < d; ++h) mg *= double(p->s.m[h]);
            const double f = 2.0 * nl * mg * double(p->s.n[k]) * double(p->rho[k + 1]) * double(p->rho[k]) *
                             double(p->s.m[k]);
            f_all += f;
            if (k == 0) f_first = f;
        }
        o.flops_fwd = b * f_all;
        o.flops_bwd = b * (f_all - f_first + 2.0 * f_all);
        o.bytes = b * (2.0 * Nin + 2.0 * Nout) * esz;
        // one CU per workgroup (token) on fp32 MFMA fed from LDS at a quarter
        // of its rate; launches: forward, backward, expand of the partials
        const double cus = std::min(b, 256.0);
        o.t_pred = 3.0 * kLaunch + (o.flops_fwd + o.flops_bwd) / (0.25 * (kPeakF32 / 256.0) * cus) +
                   o.bytes / kHbm;
        return;
    }
    if (o.kind == COMERA_ORDER_DENSE) {
        const double proj = proj_flops(p, 0, d - 1, 1.0, 1.0);
        const double gemm = 2.0 * b * Nin * Nout;
        o.flops_fwd = build + gemm;
        o.flops_bwd = build + 2.0 * gemm + proj;
        const double act = b * (Nin + Nout) * esz, w = Nin * Nout * esz;
        o.bytes = 3.0 * act + 3.0 * w + Nin * Nout * 4.0;
        o.t_pred = 2.0 * t_build + 3.0 * launch_time(gemm, act + w, peak) + (d - 1) * kLaunch +
                   proj / (0.5 * kPeakF32) + kLaunch;
        return;
    }
    // sweeps: step g contracts rows x (K = in-side of the group) into C
    const bool rl = o.kind == COMERA_ORDER_SWEEP_RL;
    double sweep = 0, t_step = 0, out_step = 0, out_flops = 0, inter_bytes = 0, proj = 0, t_meet = 0;
    for (int gi = 0; gi < G; ++gi) {
        double Ib = 1, Ja = 1, Jb = 1, Ia = 1;  // I before / J after (RL); J before / I after (LR)
        for (int h = 0; h < gi; ++h) { Ib *= gd[h].I; Jb *= gd[h].J; }
        for (int h = gi + 1; h < G; ++h) { Ja *= gd[h].J; Ia *= gd[h].I; }
        const GroupDims &g = gd[gi];
        const double rows = b * (rl ? Ib * Ja : Jb * Ia);
        const double K = rl ? g.I * g.re : g.rs * g.I, C = rl ? g.rs * g.J : g.J * g.re;
        const double f = 2.0 * rows * K * C;
        sweep += f;
        const double by = rows * (K + C) * esz + K * C * esz;
        inter_bytes += rows * (K + C) * esz;
        t_step += launch_time(f, by, peak);
        if (gi == (rl ? 0 : G - 1)) {
            out_step = launch_time(f, by, peak);
            out_flops = f;
        }
        proj += proj_flops(p, groups[gi].first, groups[gi].second, g.rs, g.re);
        t_meet += launch_time(f, by, peak);
        t_meet += (groups[gi].second - groups[gi].first) * kLaunch;
    }
    // backward: the activation states are recomputed (every step but the one
    // writing Y), then the dY sweep and one meet per group
    o.flops_fwd = build + sweep;
    o.flops_bwd = build + 2.0 * sweep + (sweep - out_flops) + proj;
    o.bytes = inter_bytes * 4.0;
    const double t_perm = G > 1 ? 2.0 * kLaunch : 0.0;
    o.t_pred = 2.0 * t_build + t_step + (t_step - out_step) + t_step + t_meet + proj / (0.5 * kPeakF32) +
               kLaunch + t_perm;
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

namespace {

// regions of the FP8 codes, scales and partial maxima from offset off
size_t layout_fp8(comera_ttm_plan_s *p, size_t off) {
    Fp8Layout &F = p->f8;
    auto r128 = [](int64_t v) { return (std::max<int64_t>(v, 1) + 127) / 128 * 128; };
    F.nin_p = r128(p->N_in);
    F.nout_p = r128(p->N_out);
    F.b_p = r128(p->batch);
    const int64_t b = std::max<int64_t>(p->batch, 1);
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = align_up(off + bytes);
        return at;
    };
    F.w8 = take(size_t(p->N_in * F.nout_p));
    F.w8t = take(size_t(p->N_out * F.nin_p));
    F.x8 = take(size_t(b * F.nin_p));
    F.x8t = take(size_t(p->N_in * F.b_p));
    F.dy8 = take(size_t(b * F.nout_p));
    F.dy8t = take(size_t(p->N_out * F.b_p));
    F.pmax = take(sizeof(float) * size_t(fp8_amax_blocks()));
    F.sc = take(sizeof(float) * 8);
    return off;
}

}  // namespace

void layout_dense(comera_ttm_plan_s *p, bool with_dx) {
    DenseLayout &L = p->dense;
    std::memset(&L, 0, sizeof(L));
    const int d = p->d;
    // FP8: W is built in fp32 and W^T is never formed in the activation dtype
    const size_t esz = (p->s.act == COMERA_BF16 && !p->fp8) ? 2 : 4;
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
    L.wt = off;
    if (!p->fp8) off = align_up(off + esz * size_t(p->N_in * p->N_out));
    L.ones = off;
    off = align_up(off + sizeof(float));
    // dW = X^T dY split over tokens so that the grid holds >= ~512 workgroups
    // (fp32: about three 128 x 128 tiles per CU, measured best on gfx950)
    int64_t tiles = ((p->N_in + 127) / 128) * ((p->N_out + 127) / 128);
    int64_t b = std::max<int64_t>(p->batch, 1);
    int64_t splits = std::max<int64_t>(1, (512 + tiles - 1) / tiles);
    if (p->s.act == COMERA_F32) splits = std::max<int64_t>(1, (768 + tiles / 2) / tiles);
    // bf16 (256 x 256 tiles): the split count minimising a measured model,
    // waves of tiles x tokens per split x 40 ns plus writing and reading
    // back the split partials at 4 TB/s
    if ((p->s.act == COMERA_BF16 || p->fp8) && p->N_in >= 256 && p->N_out >= 256) {
        const int64_t t256 = ((p->N_in + 255) / 256) * ((p->N_out + 255) / 256);
        double best = -1.0;
        for (int64_t s = 1; s <= 64; ++s) {
            const int64_t kc = ((b + s - 1) / s + 63) / 64 * 64;
            const int64_t sp = (b + kc - 1) / kc;
            if (sp != s) continue;
            const double rounds = double((t256 * s + 255) / 256);
            const double t = rounds * double(kc) * 40e-9 + 2.0 * double(s) * double(p->N_in * p->N_out) * 4.0 / 4e12;
            if (best < 0 || t < best) {
                best = t;
                splits = s;
            }
        }
    }
    // a side of 64 or less (the meets of the paper's TT layout): the product
    // only streams the token rows, so about 1024 workgroups of the skinny
    // 32 x 128 tiles keep enough loads in flight
    if (std::min(p->N_in, p->N_out) <= 64 && !p->fp8) {
        const int64_t st = ((std::min(p->N_in, p->N_out) + 31) / 32) * ((std::max(p->N_in, p->N_out) + 127) / 128);
        splits = std::max<int64_t>(splits, (1024 + st - 1) / st);
    }
    splits = std::min<int64_t>(splits, std::max<int64_t>(1, b / 256));
    splits = std::min<int64_t>(splits, 64);
    int64_t kchunk = (b + splits - 1) / splits;
    kchunk = (kchunk + 31) / 32 * 32;
    if (p->fp8) kchunk = (kchunk + 127) / 128 * 128;   // whole 128-token K tiles of codes
    splits = (b + kchunk - 1) / kchunk;
    L.dw_splits = int(splits);
    L.dw_kchunk = kchunk;
    // fp32 dX = dY W^T split over N_out when the output alone gives too few
    // 128 x 128 tiles (the partials are summed in a fixed order)
    L.dx_splits = 1;
    L.dx_kchunk = p->N_out;
    if (with_dx && p->s.act == COMERA_F32 && !p->fp8) {
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
    if (p->fp8) off = layout_fp8(p, off);
    // forward and dX products with too few output tiles are split over K
    if (with_dx && !p->fp8) {
        const int sf = gemm_auto_splits(b, p->N_out, p->N_in);
        const int sx = L.dx_splits > 1 ? 1 : gemm_auto_splits(b, p->N_in, p->N_out);
        const int64_t pe = std::max<int64_t>(sf > 1 ? sf * b * p->N_out : 0, sx > 1 ? sx * b * p->N_in : 0);
        if (pe > 0) {
            L.part = off;
            L.part_elems = pe;
            off = align_up(off + sizeof(float) * size_t(pe));
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

namespace {
constexpr double kSweepCap = 64.0 * 1024 * 1024 * 1024;   // workspace cap of a sweep order (bytes)

// placement of core k (local index j of a group of dg cores, bonds A and C)
// in the group's layer: right to left the group's left bond joins the output
// factor of its first core and its right bond the input factor of its last
// core; left to right (left bond before the first input factor, right bond
// after the last output factor) the placement is the plain swapped one
CoreStrides sweep_strides(int dir, int j, int dg, int A, int m, int n, int C) {
    if (dir == COMERA_ORDER_SWEEP_LR || (j > 0 && j < dg - 1)) return core_strides(A, m, n, C, true);
    CoreStrides s;
    if (dg == 1) {           // [1][(n, c)][(a, m)][1]
        s.sn = C * A * m;
        s.sc = A * m;
        s.sa = m;
        s.sm = 1;
    } else if (j == 0) {     // [1][n][(a, m)][c]
        s.sn = A * m * C;
        s.sa = m * C;
        s.sm = C;
        s.sc = 1;
    } else {                 // [a][(n, c)][m][1]
        s.sa = n * C * m;
        s.sn = C * m;
        s.sc = m;
        s.sm = 1;
    }
    return s;
}
}  // namespace

bool layout_sweep(const comera_ttm_plan_s *p, int kind, uint32_t cuts, SweepLayout &L,
                  std::unique_ptr<comera_ttm_plan_s> *sub) {
    L = SweepLayout();
    const int d = p->d;
    const bool rl = kind == COMERA_ORDER_SWEEP_RL;
    L.dir = kind;
    int G = 0, s0 = 0;
    for (int k = 0; k < d; ++k) {
        if (k == d - 1 || ((cuts >> k) & 1u)) {
            L.s[G] = s0;
            L.e[G] = k;
            ++G;
            s0 = k + 1;
        }
    }
    L.G = G;
    for (int g = 0; g < G; ++g) {
        L.N[g] = 1;
        L.M[g] = 1;
        for (int k = L.s[g]; k <= L.e[g]; ++k) {
            L.N[g] *= p->s.n[k];
            L.M[g] *= p->s.m[k];
        }
        L.as[g] = p->rho[L.s[g]];
        L.ae[g] = p->rho[L.e[g] + 1];
    }
    auto prod = [&](const int64_t *v, int lo, int hi) {   // product of v[lo .. hi)
        double x = 1;
        for (int h = lo; h < hi; ++h) x *= double(v[h]);
        return x;
    };
    const double b = double(std::max<int64_t>(p->batch, 1));
    const size_t esz = p->s.act == COMERA_BF16 ? 2 : 4;
    double off = 0;
    // one layer per group
    for (int g = 0; g < G; ++g) {
        const int dg = L.e[g] - L.s[g] + 1;
        sub[g].reset(new (std::nothrow) comera_ttm_plan_s());
        comera_ttm_plan_s *sp = sub[g].get();
        if (!sp) return false;
        std::memset(&sp->s, 0, sizeof(sp->s));
        std::memset(sp->act, 0, sizeof(sp->act));
        sp->s.d = dg;
        sp->s.act = p->s.act;
        for (int j = 0; j < dg; ++j) {
            sp->s.n[j] = p->s.n[L.s[g] + j];
            sp->s.m[j] = p->s.m[L.s[g] + j];
            sp->s.r[j] = j == 0 ? 1 : p->rho[L.s[g] + j];
        }
        sp->s.r[dg] = 1;
        if (rl) {
            sp->s.m[0] *= L.as[g];
            sp->s.n[dg - 1] *= L.ae[g];
        } else {
            sp->s.n[0] *= L.as[g];
            sp->s.m[dg - 1] *= L.ae[g];
        }
        sp->d = dg;
        sp->N_in = 1;
        sp->N_out = 1;
        double nin = 1, nout = 1;
        for (int j = 0; j < dg; ++j) {
            nin *= double(sp->s.n[j]);
            nout *= double(sp->s.m[j]);
            if (double(sp->s.r[j]) * double(sp->s.m[j]) * double(sp->s.n[j]) * double(sp->s.r[j + 1]) >
                2147483647.0)
                return false;
            sp->N_in *= sp->s.n[j];
            sp->N_out *= sp->s.m[j];
        }
        if (nin > 2147483647.0 || nout > 2147483647.0 || nin * nout * 4.0 > kSweepCap) return false;
        for (int j = 0; j <= dg; ++j) sp->rho[j] = sp->s.r[j];
        sp->compacted = false;
        // K of the product that meets at this group: tokens times the outer factors
        const double kappa = rl ? b * prod(L.N, 0, g) * prod(L.M, g + 1, G) : b * prod(L.M, 0, g) * prod(L.N, g + 1, G);
        if (kappa > 4.0e18) return false;
        sp->batch = int64_t(kappa);
        layout_dense(sp, false);
        for (int j = 0; j < dg; ++j) {
            const int k = L.s[g] + j;
            L.st[k] = sweep_strides(kind, j, dg, int(p->rho[k]), int(p->s.m[k]), int(p->s.n[k]), int(p->rho[k + 1]));
        }
        L.base[g] = size_t(off);
        off += double(align_up(sp->dense.total));
    }
    // states: both sweeps store G-1 intermediate states of equal sizes
    for (int g = 1; g < G; ++g) {
        double zs, hs;
        if (rl) {
            zs = b * prod(L.N, 0, g) * double(L.ae[g - 1]) * prod(L.M, g, G);   // Z_g
            hs = zs;                                                                    // H_g
        } else {
            zs = b * prod(L.M, 0, g) * double(L.as[g]) * prod(L.N, g, G);       // Z_g
            hs = b * prod(L.M, 0, g) * double(L.ae[g - 1]) * prod(L.N, g, G);           // H_{g-1}
        }
        L.z[g] = size_t(off);
        off += double(align_up(size_t(zs * double(esz))));
        if (off > kSweepCap) return false;
        const int hi = rl ? g : g - 1;
        L.h[hi] = size_t(off);
        off += double(align_up(size_t(hs * double(esz))));
        if (off > kSweepCap) return false;
    }
    // per-token transpose of the input whose first-swept factor is not last
    const double trail = rl ? prod(L.M, 1, G) : prod(L.N, 1, G);
    L.need_t = G > 1 && trail > 1;
    if (L.need_t) {
        L.tin = size_t(off);
        off += double(align_up(size_t(b * double(rl ? p->N_out : p->N_in) * double(esz))));
    }
    // split partials of the sweep products whose output tiles are too few
    double pe = 0;
    for (int g = 0; g < G; ++g) {
        const double R = rl ? b * prod(L.N, 0, g) * prod(L.M, g + 1, G) : b * prod(L.M, 0, g) * prod(L.N, g + 1, G);
        const double Kx = rl ? double(L.N[g] * L.ae[g]) : double(L.as[g] * L.N[g]);
        const double Cx = rl ? double(L.as[g] * L.M[g]) : double(L.M[g] * L.ae[g]);
        const int s1 = gemm_auto_splits(int64_t(R), int64_t(Cx), int64_t(Kx));
        const int s2 = gemm_auto_splits(int64_t(R), int64_t(Kx), int64_t(Cx));
        if (s1 > 1) pe = std::max(pe, s1 * R * Cx);
        if (s2 > 1) pe = std::max(pe, s2 * R * Kx);
    }
    if (pe > 0) {
        L.part = size_t(off);
        L.part_elems = int64_t(pe);
        off += double(align_up(size_t(pe * 4.0)));
    }
    if (off > kSweepCap) return false;
    L.total = size_t(off);
    return true;
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
    {
        // every core its own group, swept right to left by the fused kernels
        Order o;
        o.kind = COMERA_ORDER_FUSED_RL;
        o.cuts = (1u << (d - 1)) - 1u;
        p->orders.push_back(o);
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
            if (o.kind == COMERA_ORDER_DENSE) {
                o.executable = true;
            } else if (o.kind == COMERA_ORDER_FUSED_RL) {
                ChainLayout cl;
                o.executable = layout_chain(p, cl);
            } else {
                SweepLayout sl;
                std::unique_ptr<comera_ttm_plan_s> tmp[kMaxCores];
                o.executable = layout_sweep(p, o.kind, o.cuts, sl, tmp);
            }
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
    p->ws_bytes = 0;
    if (!p->zero) {
        const Order &o = p->orders[p->chosen];
        if (o.kind == COMERA_ORDER_DENSE) {
            layout_dense(p);
            p->ws_bytes = p->dense.total;
        } else if (o.kind == COMERA_ORDER_FUSED_RL) {
            if (!layout_chain(p, p->ch)) {
                delete p;
                return COMERA_ERR_INTERNAL;
            }
            p->chain = true;
            p->ws_bytes = p->ch.total;
        } else {
            if (!layout_sweep(p, o.kind, o.cuts, p->sweep, p->sub)) {
                delete p;
                return COMERA_ERR_INTERNAL;
            }
            p->ws_bytes = p->sweep.total;
        }
    }
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

comera_status comera_ttm_plan_set_fp8(comera_ttm_plan_t p, int32_t enable) {
    if (!p) return COMERA_ERR_INVALID_ARG;
    const bool on = enable != 0;
    if (on == p->fp8) return COMERA_OK;
    if (p->zero) {
        // W == 0: nothing is multiplied, the workspace stays empty
        p->fp8 = on;
        return COMERA_OK;
    }
    if (p->orders[p->chosen].kind != COMERA_ORDER_DENSE) return COMERA_ERR_UNSUPPORTED;
    // every code buffer is addressed with 32-bit offsets by the GEMM
    const int64_t b = std::max<int64_t>(p->batch, 1);
    const int64_t nin_p = (p->N_in + 127) / 128 * 128, nout_p = (p->N_out + 127) / 128 * 128;
    const int64_t b_p = (b + 127) / 128 * 128;
    const int64_t lim = int64_t(1) << 32;
    if (b * nin_p >= lim || b * nout_p >= lim || p->N_in * b_p >= lim || p->N_out * b_p >= lim ||
        p->N_in * nout_p >= lim || p->N_out * nin_p >= lim)
        return COMERA_ERR_UNSUPPORTED;
    p->fp8 = on;
    layout_dense(p);
    p->ws_bytes = p->dense.total;
    return COMERA_OK;
}

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
