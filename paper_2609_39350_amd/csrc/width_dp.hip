// Per-stage data-parallel widths (stage_types = 3): the non-uniform PP/DP
// partitioning of the paper's contributions -- stage-wise parallelism knobs
// chosen jointly with the layer assignment (Section 1, the ablation of the
// evaluation) -- on the block device layout.  The devices are listed type by
// type in the candidate's ordering; stage i takes the next w_i half-groups of
// g/2 devices (g = G/PP), w_i in {1, 2, 3}, sum w_i = 2 PP, and runs DP_i =
// w_i DP / 2 replicas.  Every stage processes the same global micro-batch, so a
// replica holds r = 2 / w_i of the nominal tokens: the Section 3.2 terms are
// evaluated at that token count, the ZeRO-1 optimizer state over DP_i, the
// activations and MoE buffers at r; the boundary transfer is the sender's
// per-rank activation; the pruning-1 window follows the stage's share w_i P_i
// (g/2) / sum_h m_h P_h of the cluster's compute; pruning 3 and T_dp-sync +
// T_opt keep their nominal values.
//
// Kernel W1 (k_width_tables, one workgroup per configuration) writes layer
// prefix sums of the stage time without / with recomputation and of its
// communication for every device-type set at each width, and of the memory
// terms at each width.  Kernel W2 (k_width_dp, persistent workgroups over the
// candidates) runs, per candidate, the threshold DP over (stage, end layer,
// half-groups used): F_t[i][b][u] = min over (a, w) of F_t[i-1][a][u-w] +
// c_{i-1}(u-w, w; a, b) over stage costs <= t, ties to the smallest a, then the
// smallest w, and sweeps the thresholds downwards over the (max, sum) Pareto
// points (a pass at t gives a partition whose largest stage m keeps F constant
// on [m, t]; the next threshold is min(m - 1, the largest that can still beat
// the incumbent)).  The incumbent is replaced by a lower sum + (B-1) max, or an
// equal one with a lower max, so the result is the least objective, the least
// threshold reaching it and the back-trace there.  Plain int64 min-plus work on
// the VALU; F of two levels, the memory prefix sums and the stage layouts of the
// half-group ranges live in LDS, the back-trace pointers in the workgroup's
// slice of the workspace.
#include "internal.h"

namespace hapmoe {
namespace {

constexpr int kThreads = 256;
constexpr int kLayerSlots = 128;   // >= kMaxLayers + 1
constexpr int kMaxUnits = 2 * kMaxStages;
constexpr int64_t kNone = INT64_MAX;

__device__ inline int lg2i(int v) { return 31 - __clz(v); }

__device__ inline int64_t qterm(double x, unsigned *flag)
{
    if (!(x < (double)kTermLimit)) {
        atomicOr(flag, 1u);
        return kTermLimit;
    }
    return (int64_t)ceil(x);
}

// slowest link inside a device-type set (largest latency, smallest bandwidth)
__device__ inline void set_link(const ImageHeader &H, int mask, double &alpha, double &bw)
{
    bool first = true;
    alpha = 0.0;
    bw = 0.0;
    for (int h = 0; h < H.n_types; ++h) {
        if (!((mask >> h) & 1)) continue;
        for (int g = 0; g < H.n_types; ++g) {
            if (!((mask >> g) & 1)) continue;
            const double a = H.alpha[h * kMaxTypes + g], b = H.bw[h * kMaxTypes + g];
            if (first || a > alpha) alpha = a;
            if (first || b < bw) bw = b;
            first = false;
        }
    }
}

__device__ inline double ring_ar(double bytes, int w, double alpha, double bw)
{
    if (w == 1) return 0.0;
    const double steps = (double)(2 * (w - 1));
    return steps * alpha + ((steps * bytes) / (double)w) / bw;
}

// token share of one replica of a width-w stage
__device__ inline double ratio(int w) { return 2.0 / (double)w; }

// ---- kernel W1: width tables, one 256-thread workgroup per configuration ----
__global__ __launch_bounds__(kThreads) void k_width_tables(const unsigned char *__restrict__ img,
                                                           const hapmoe_candidate *__restrict__ cand,
                                                           int64_t per_config, int64_t cfg_lo, TablesLayout L,
                                                           unsigned char *__restrict__ tab)
{
    const ImageHeader &H = *reinterpret_cast<const ImageHeader *>(img);
    const uint8_t *is_moe = img + H.off_is_moe;
    const int64_t *pdense = reinterpret_cast<const int64_t *>(img + H.off_pdense);
    const int64_t *pexp = reinterpret_cast<const int64_t *>(img + H.off_pexp);
    const int64_t *act = reinterpret_cast<const int64_t *>(img + H.off_act);
    const int64_t *tdense = reinterpret_cast<const int64_t *>(img + H.off_tdense);
    const int64_t *tffn = reinterpret_cast<const int64_t *>(img + H.off_tffn);
    const double *skew = reinterpret_cast<const double *>(tab + L.off_layer);

    const int64_t cfg = cfg_lo + blockIdx.x;
    const int tid = threadIdx.x;
    const hapmoe_candidate c = cand[cfg * per_config];
    const int N = H.n_layers, T = H.n_types;
    const int64_t np = L.np;
    const int nm = (int)L.n_masks;

    __shared__ int64_t s_qce[3][kMaxTypes][kLayerSlots];   // q(comp) + q(expert) per width, type, layer
    __shared__ int64_t s_val[3][3][kLayerSlots];            // per width: w, a0, a1 of each layer
    __shared__ unsigned s_flag;
    if (tid == 0) s_flag = 0;
    __syncthreads();

    const double tok0 = (double)((int64_t)H.seq_len * H.mbs / c.cp);
    // per-layer terms at each width
    for (int i = tid; i < 3 * N; i += kThreads) {
        const int wi = i / N, l = i - wi * N, w = wi + 1;
        const double r = ratio(w);
        const double tok = tok0 * r;
        const bool moe = is_moe[l] != 0;
        for (int h = 0; h < T; ++h) {
            const int64_t off = (((int64_t)h * 4 + lg2i(c.tp)) * 4 + lg2i(c.cp)) * N + l;
            const double td = (double)tdense[off], tf = (double)tffn[off];
            double comp, expert;
            if (!moe) {
                comp = td * r;
                expert = 0.0;
            } else {
                const double route = H.route_coef[h] * (tok * (double)H.hidden);
                comp = (td - tf) * r + route;
                const double xexp = (H.moe_ffn_mult * (tf * r)) / ((H.eff[h] * (double)c.ep) * (double)c.tpe);
                expert = skew[l] * xexp;
            }
            s_qce[wi][h][l] = qterm(comp, &s_flag) + qterm(expert, &s_flag);
        }
        const int dp_i = c.dp * w / 2;
        const double beta_opt = 6.0 + 12.0 / (double)dp_i;
        const double wt = ((double)pdense[l] / (double)c.tp + (double)pexp[l] / (double)(c.ep * c.tpe)) * beta_opt;
        const double a0 = ((double)act[l] * r) / (double)(c.tp * c.cp);
        const int64_t qa0 = qterm(a0, &s_flag);
        s_val[wi][0][l] = qterm(wt, &s_flag);
        s_val[wi][1][l] = qa0;
        s_val[wi][2][l] = qterm(H.rc_act * (double)qa0, &s_flag);
    }
    __syncthreads();

    // memory prefix sums: one thread a (width, field) row
    int64_t *wmem = reinterpret_cast<int64_t *>(tab + L.off_wmem) + cfg * 3 * 4 * np;
    if (tid < 12) {
        const int wi = tid / 4, f = tid % 4;
        int64_t *row = wmem + (wi * 4 + f) * np;
        int64_t acc = 0;
        row[0] = 0;
        for (int l = 0; l < N; ++l) {
            acc += f < 3 ? s_val[wi][f][l] : (int64_t)(is_moe[l] != 0);
            row[l + 1] = acc;
        }
    }
    // stage times of every device-type set at every width: one thread a (set, width)
    // row, the per-layer terms evaluated in order
    int64_t *wtime = reinterpret_cast<int64_t *>(tab + L.off_wtime) + cfg * nm * 3 * 3 * np;
    for (int i = tid; i < nm * 3; i += kThreads) {
        const int m = i / 3 + 1, wi = i % 3;
        const double r = ratio(wi + 1);
        double alpha, bw;
        set_link(H, m, alpha, bw);
        const double D = ((tok0 * r) * (double)H.hidden) * (double)H.elem_bytes;
        int64_t *P0 = wtime + ((int64_t)(m - 1) * 3 + wi) * 3 * np;
        int64_t *P1 = P0 + np, *P2 = P1 + np;
        int64_t a0 = 0, a1 = 0, a2 = 0;
        P0[0] = P1[0] = P2[0] = 0;
        for (int l = 0; l < N; ++l) {
            double a2a, tp;
            if (!is_moe[l]) {
                a2a = 0.0;
                tp = 4.0 * ring_ar(D, c.tp, alpha, bw);
            } else {
                const double sk = skew[l];
                const double dm = (D * (double)H.top_k) * (1.0 - 1.0 / (double)c.ep);
                const double f_a2a = (double)(c.ep - 1) * alpha + dm / bw;
                const double f_ag = (double)(c.ep - 1) * alpha + (D * (double)(c.ep - 1)) / bw;
                a2a = sk * (4.0 * (f_ag < f_a2a ? f_ag : f_a2a));
                tp = 2.0 * ring_ar(D, c.tp, alpha, bw) + 2.0 * ring_ar(D, c.tpe, alpha, bw);
            }
            const double cpt =
                c.cp == 1 ? 0.0 : 3.0 * ((double)(c.cp - 1) * (alpha + ((2.0 * D) / (double)c.tp) / bw));
            const int64_t comm = qterm(a2a, &s_flag) + qterm(tp, &s_flag) + qterm(cpt, &s_flag);
            int64_t ce = -1;
            for (int h = 0; h < T; ++h)
                if ((m >> h) & 1) ce = s_qce[wi][h][l] > ce ? s_qce[wi][h][l] : ce;
            const int64_t t0 = ce + comm;
            a0 += t0;
            a1 += qterm(H.rc_time * (double)t0, &s_flag);
            a2 += comm;
            P0[l + 1] = a0;
            P1[l + 1] = a1;
            P2[l + 1] = a2;
        }
    }
    if (tid >= 64 && tid < 67) {   // MoE buffers of each width
        const int wi = tid - 64;
        const double r = ratio(wi + 1);
        const double tok = tok0 * r;
        const double D = (tok * (double)H.hidden) * (double)H.elem_bytes;
        const double dm = (D * (double)H.top_k) * (1.0 - 1.0 / (double)c.ep);
        reinterpret_cast<int64_t *>(tab + L.off_wx)[cfg * 4 + wi] =
            qterm(((8.0 * tok) * (double)H.top_k) + 2.0 * dm, &s_flag);
    }
    __syncthreads();
    if (tid == 0 && s_flag) reinterpret_cast<PiInfo *>(tab + L.off_pi)[cfg].status = HAPMOE_STATUS_OVERFLOW;
}

// ---- kernel W2: the DP, one candidate per workgroup pass of the queue ----
struct WStage {     // stage on half-groups [u, u + w)
    int64_t cap, p2p;
    uint8_t mask, lo, hi, flags;   // flags: 1 mixed, 2 next stage starts on another type
};

struct WCtl {
    uint32_t qi;
    int32_t pad;
    int64_t t;
};

// floor(x / d) for d > 0 where only its sign matters below zero (-1)
__device__ inline int64_t floor_div(int64_t x, int64_t d) { return x < 0 ? -1 : x / d; }

template <bool STATS>
__global__ __launch_bounds__(kThreads) void k_width_dp(const unsigned char *__restrict__ img,
                                                       const hapmoe_candidate *__restrict__ cand, TablesLayout L,
                                                       const unsigned char *__restrict__ tab, int64_t first,
                                                       int64_t count, unsigned char *__restrict__ slots,
                                                       int64_t slot_bytes, hapmoe_dp_result *__restrict__ res,
                                                       uint8_t *__restrict__ types_out,
                                                       uint8_t *__restrict__ widths_out, int32_t *__restrict__ stats,
                                                       uint32_t *__restrict__ queue)
{
    const ImageHeader &H = *reinterpret_cast<const ImageHeader *>(img);
    const int tid = threadIdx.x;
    const int N = H.n_layers, W = N + 1, T = H.n_types;
    const int64_t np = L.np;

    __shared__ int64_t s_mw[3][kLayerSlots], s_ma0[3][kLayerSlots], s_ma1[3][kLayerSlots];
    __shared__ int32_t s_moe[kLayerSlots];
    __shared__ WStage s_st[kMaxUnits + 1][3];
    __shared__ int64_t s_x[3];
    __shared__ WCtl ctl;
    __shared__ int64_t s_pF, s_pM;   // last pass: stage sum and largest stage
    __shared__ uint32_t s_prm;
    __shared__ uint8_t s_plen[kMaxStages], s_pw[kMaxStages], s_pmask[kMaxStages];
    __shared__ uint32_t s_relax;
    // the candidates of the key's current group (equal min(B, PP)): their B index
    // j and their incumbents, and the next threshold each still needs
    __shared__ int32_t s_mj[HAPMOE_MAX_MICRO];
    __shared__ int64_t s_best[HAPMOE_MAX_MICRO], s_bestM[HAPMOE_MAX_MICRO], s_bestF[HAPMOE_MAX_MICRO];
    __shared__ int64_t s_next[HAPMOE_MAX_MICRO];
    __shared__ uint32_t s_brm[HAPMOE_MAX_MICRO];
    __shared__ uint8_t s_blen[HAPMOE_MAX_MICRO][kMaxStages], s_bw[HAPMOE_MAX_MICRO][kMaxStages],
        s_bmask[HAPMOE_MAX_MICRO][kMaxStages];
    __shared__ int s_nmem, s_vj;

    // F of two levels in LDS; the back-trace pointers in the workgroup's slice
    extern __shared__ __align__(16) unsigned char w_dyn[];
    int64_t *F = reinterpret_cast<int64_t *>(w_dyn);
    int16_t *const ARG = reinterpret_cast<int16_t *>(slots + (int64_t)blockIdx.x * slot_bytes);
    // the (configuration, ordering) keys holding candidates [first, first + count)
    const int64_t key_lo = first / H.n_micro, n_keys = (first + count - 1) / H.n_micro - key_lo + 1;
    for (;;) {
        if (tid == 0) ctl.qi = atomicAdd(queue, 1u);
        __syncthreads();
        const int64_t k = ctl.qi;
        __syncthreads();
        if (k >= n_keys) break;   // every workgroup exits once the queue is drained
        const int64_t key = key_lo + k;
        const int nB = H.n_micro;
        const hapmoe_candidate c = cand[key * nB];
        const int64_t cfg = key / H.n_orders;
        const int o = (int)(key - cfg * H.n_orders);
        const int PP = c.pp, U = 2 * PP, UP = U + 1;
        const PiInfo *pi = reinterpret_cast<const PiInfo *>(tab + L.off_pi) + cfg;
        const KeyInfo *ki = reinterpret_cast<const KeyInfo *>(tab + L.off_key) + key;
        // candidate j of the key, when it lies in [first, first + count)
        auto in_range = [&](int j) {
            const int64_t idx = key * nB + j;
            return idx >= first && idx < first + count;
        };
        if (pi->status != HAPMOE_STATUS_OK) {
            for (int j = 0; j < nB; ++j) {
                if (!in_range(j)) continue;
                const int64_t r = key * nB + j - first;
                hapmoe_dp_result *out = res + r;
                if (tid == 0) {
                    out->objective = out->stage_sum = out->t_max = kInf;
                    out->status = HAPMOE_STATUS_OVERFLOW;
                    out->recompute_mask = 0;
                    if (STATS) stats[4 * r] = stats[4 * r + 1] = stats[4 * r + 2] = stats[4 * r + 3] = 0;
                }
                if (tid < kMaxStages) out->layers[tid] = types_out[r * kMaxStages + tid] = widths_out[r * kMaxStages + tid] = 0;
            }
            __syncthreads();
            continue;
        }
        // memory prefix sums of the three widths
        const int64_t *wmem = reinterpret_cast<const int64_t *>(tab + L.off_wmem) + cfg * 3 * 4 * np;
        for (int i = tid; i < 3 * W; i += kThreads) {
            const int wi = i / W, b = i - wi * W;
            s_mw[wi][b] = wmem[(wi * 4 + 0) * np + b];
            s_ma0[wi][b] = wmem[(wi * 4 + 1) * np + b];
            s_ma1[wi][b] = wmem[(wi * 4 + 2) * np + b];
            if (wi == 0) s_moe[b] = (int32_t)wmem[3 * np + b];
        }
        if (tid < 3) s_x[tid] = reinterpret_cast<const int64_t *>(tab + L.off_wx)[cfg * 4 + tid];
        // the stage on half-groups [u, u + w) of this ordering
        {
            const int G = H.total_devices, half = G / PP / 2;
            int pos_type[kMaxTypes], pos_end[kMaxTypes];
            int acc = 0;
            int64_t total_speed = 0;
            for (int j = 0; j < T; ++j) {
                pos_type[j] = H.perm[o][j];
                acc += H.count[pos_type[j]];
                pos_end[j] = acc;
                total_speed += (int64_t)H.count[j] * H.speed[j];
            }
            auto type_of = [&](int d) {
                int t = pos_type[T - 1];
                for (int j = T - 1; j >= 0; --j)
                    if (d < pos_end[j]) t = pos_type[j];
                return t;
            };
            for (int i = tid; i < UP * 3; i += kThreads) {
                const int u = i / 3, w = i % 3 + 1;
                WStage x = {0, 0, 0, 0, 0, 0};
                if (u + w <= U) {
                    const int d0 = u * half, d1 = (u + w) * half;
                    int mask = 0;
                    for (int j = 0; j < T; ++j)
                        if (pos_end[j] - H.count[pos_type[j]] < d1 && pos_end[j] > d0) mask |= 1 << pos_type[j];
                    int64_t cap = -1;
                    int sp = 0;
                    for (int h = 0; h < T; ++h) {
                        if (!((mask >> h) & 1)) continue;
                        if (cap < 0 || H.mem_bytes[h] < cap) cap = H.mem_bytes[h];
                        if (sp == 0 || H.speed[h] < sp) sp = H.speed[h];
                    }
                    const int last = type_of(d1 - 1);
                    int flags = __popc(mask) > 1 ? 1 : 0;
                    int64_t p2p = 0;
                    if (u + w < U) {
                        const int nt = type_of(d1);
                        if (nt != last) flags |= 2;
                        const double a = H.alpha[last * kMaxTypes + nt], b = H.bw[last * kMaxTypes + nt];
                        const double r = ratio(w);
                        const double D = (((double)((int64_t)H.seq_len * H.mbs / c.cp) * r) * (double)H.hidden) *
                                         (double)H.elem_bytes;
                        p2p = (int64_t)ceil(2.0 * (a + (D / (double)c.tp) / b));
                    }
                    int64_t lo = 1, hi = N;
                    if (H.prune_window == 1) {
                        const int64_t dn = H.delta_num, dd = H.delta_den;
                        const int64_t num = (int64_t)w * sp * half * N, den = dd * total_speed;
                        lo = ((dd - dn) * num) / den;
                        hi = ((dd + dn) * num + den - 1) / den;
                        lo = lo < 1 ? 1 : lo;
                        hi = hi > N ? N : hi;
                    } else if (H.prune_window == 2) {
                        lo = N / PP;
                        hi = (N + PP - 1) / PP;
                    }
                    x.cap = cap;
                    x.p2p = p2p;
                    x.mask = (uint8_t)mask;
                    x.lo = (uint8_t)lo;
                    x.hi = (uint8_t)hi;
                    x.flags = (uint8_t)flags;
                }
                s_st[u][w - 1] = x;
            }
        }
        if (tid == 0) s_relax = 0;
        __syncthreads();

        const int64_t *wtime = reinterpret_cast<const int64_t *>(tab + L.off_wtime) + cfg * L.n_masks * 3 * 3 * np;
        const int64_t eta_tbar = (int64_t)H.eta_prune * pi->tbar;
        const bool prune_het = H.prune_hetero != 0, recomp = H.allow_recompute != 0;
        int64_t B = 1;   // the current group's min(B, PP): every stage's stored micro-batches

        // cost of stage s on half-groups [u0, u0 + w) and layers [a, b), kNone if
        // pruned; *rf = 1 if it needs recomputation
        auto stage_cost = [&](int s, int u0, int w, int a, int b, int *rf) -> int64_t {
            const WStage &x = s_st[u0][w - 1];
            const int n = b - a;
            if (n < x.lo || n > x.hi) return kNone;
            const int wi = w - 1;
            const int64_t ms = (int64_t)(PP - s) < B ? (int64_t)(PP - s) : B;   // B: the group's min(B, PP)
            const int64_t ex = (s_moe[b] - s_moe[a]) > 0 ? s_x[wi] : 0;
            const int64_t dw = s_mw[wi][b] - s_mw[wi][a];
            const int64_t *P = wtime + ((int64_t)(x.mask - 1) * 3 + wi) * 3 * np;
            int64_t t;
            if (dw + ms * (s_ma0[wi][b] - s_ma0[wi][a]) + ex <= x.cap) {
                t = P[b] - P[a];
                *rf = 0;
            } else if (recomp && dw + ms * (s_ma1[wi][b] - s_ma1[wi][a]) + ex <= x.cap) {
                t = P[np + b] - P[np + a];
                *rf = 1;
            } else {
                return kNone;
            }
            if (prune_het) {
                const int64_t hc = ((x.flags & 1) ? P[2 * np + b] - P[2 * np + a] : 0) + ((x.flags & 2) ? x.p2p : 0);
                if (hc > eta_tbar) return kNone;
            }
            return t + x.p2p;
        };

        // one pass at threshold t: F over the levels, then the back-trace by thread 0
        auto pass = [&](int64_t t) {
            int64_t *F0 = F, *F1 = F + (int64_t)W * UP;
            for (int i = tid; i < W * UP; i += kThreads) F0[i] = i == 0 ? 0 : kNone;   // level 0: (b, u) = (0, 0)
            __syncthreads();
            uint32_t relax = 0;
            for (int i = 1; i <= PP; ++i) {
                const int64_t *Fp = (i & 1) ? F0 : F1;
                int64_t *Fc = (i & 1) ? F1 : F0;
                int16_t *Ai = ARG + (int64_t)i * W * UP;
                // states of level i: b in [i, N - (PP - i)], u in [max(i, U - 3 (PP - i)), min(3 i, U - (PP - i))]
                const int blo = i, bhi = N - (PP - i);
                const int ulo = i > U - 3 * (PP - i) ? i : U - 3 * (PP - i);
                const int uhi = 3 * i < U - (PP - i) ? 3 * i : U - (PP - i);
                const int nb = bhi - blo + 1, nu = uhi - ulo + 1;
                for (int e = tid; e < W * UP; e += kThreads) Fc[e] = kNone;
                __syncthreads();
                for (int e = tid; nb > 0 && nu > 0 && e < nb * nu; e += kThreads) {
                    const int b = blo + e / nu, u = ulo + e % nu;
                    int64_t best = kNone;
                    int ba = -1, bwid = 0;
                    for (int w = 1; w <= 3; ++w) {
                        const int u0 = u - w;
                        if (u0 < i - 1 || u0 > 3 * (i - 1)) continue;
                        const WStage &x = s_st[u0][w - 1];
                        if (x.mask == 0) continue;
                        int alo = b - x.hi, ahi = b - x.lo;   // the window: n = b - a in [lo, hi]
                        alo = alo < i - 1 ? i - 1 : alo;
                        // stage_cost with its end-layer terms read once per (b, w)
                        const int wi = w - 1;
                        const int64_t ms = (int64_t)(PP - (i - 1)) < B ? (int64_t)(PP - (i - 1)) : B;
                        const int64_t *P = wtime + ((int64_t)(x.mask - 1) * 3 + wi) * 3 * np;
                        const int64_t p0b = P[b], p1b = P[np + b], p2b = (x.flags & 1) ? P[2 * np + b] : 0;
                        const int64_t mwb = s_mw[wi][b], ma0b = s_ma0[wi][b], ma1b = s_ma1[wi][b];
                        const int moeb = s_moe[b];
                        const int64_t xw = s_x[wi], hc_b = (x.flags & 2) ? x.p2p : 0;
                        for (int a = alo; a <= ahi; ++a) {
                            const int64_t prev = Fp[(int64_t)a * UP + u0];
                            if (prev == kNone) continue;
                            const int64_t ex = (moeb - s_moe[a]) > 0 ? xw : 0;
                            const int64_t dw = mwb - s_mw[wi][a];
                            int64_t cst;
                            if (dw + ms * (ma0b - s_ma0[wi][a]) + ex <= x.cap)
                                cst = p0b - P[a];
                            else if (recomp && dw + ms * (ma1b - s_ma1[wi][a]) + ex <= x.cap)
                                cst = p1b - P[np + a];
                            else
                                continue;
                            if (prune_het && ((x.flags & 1) ? p2b - P[2 * np + a] : 0) + hc_b > eta_tbar) continue;
                            cst += x.p2p;
                            if (cst > t) continue;
                            if (STATS) ++relax;
                            const int64_t v = prev + cst;
                            if (v < best || (v == best && (a < ba || (a == ba && w < bwid)))) {
                                best = v;
                                ba = a;
                                bwid = w;
                            }
                        }
                    }
                    Fc[(int64_t)b * UP + u] = best;
                    Ai[(int64_t)b * UP + u] = (int16_t)(best == kNone ? -1 : ba * 4 + bwid);
                }
                __syncthreads();
            }
            if (STATS && relax) atomicAdd(&s_relax, relax);
            if (tid == 0) {
                const int64_t *Fl = (PP & 1) ? F1 : F0;
                const int64_t f = Fl[(int64_t)N * UP + U];
                s_pF = f;
                s_pM = 0;
                s_prm = 0;
                if (f != kNone) {
                    int b = N, u = U;
                    int64_t m = 0;
                    uint32_t rm = 0;
                    for (int i = PP; i >= 1; --i) {
                        const int x = ARG[((int64_t)i * W + b) * UP + u];
                        const int a = x >> 2, w = x & 3, u0 = u - w;
                        int rf = 0;
                        const int64_t cst = stage_cost(i - 1, u0, w, a, b, &rf);
                        m = cst > m ? cst : m;
                        if (rf) rm |= 1u << (i - 1);
                        s_plen[i - 1] = (uint8_t)(b - a);
                        s_pw[i - 1] = (uint8_t)w;
                        s_pmask[i - 1] = s_st[u0][w - 1].mask;
                        b = a;
                        u = u0;
                    }
                    s_pM = m;
                    s_prm = rm;
                }
            }
            __syncthreads();
        };

        // ---- the descending Pareto sweep, one per group of the key's candidates
        // with equal min(B, PP) (their stored micro-batch counts, hence every DP
        // pass, are the same); one incumbent per candidate, replaced by a lower
        // sum + (B-1) max or an equal one with a lower max.  The next threshold is
        // the largest any member still needs: a member skips only points that
        // cannot beat its own incumbent, so each gets the result of its own sweep.
        for (int g = 0; g < nB; ++g) {
            // group g: the candidates whose min(B, PP) equals that of the g-th B,
            // taken at its first occurrence
            if (tid == 0) {
                const int vg = H.micro[g] < PP ? H.micro[g] : PP;
                bool firstv = true;
                for (int j = 0; j < g; ++j) firstv = firstv && (H.micro[j] < PP ? H.micro[j] : PP) != vg;
                int nm = 0;
                if (firstv)
                    for (int j = g; j < nB; ++j)
                        if ((H.micro[j] < PP ? H.micro[j] : PP) == vg && in_range(j)) s_mj[nm++] = j;
                s_nmem = nm;
                s_vj = vg;
                s_relax = 0;
            }
            __syncthreads();
            const int nmem = s_nmem;
            B = s_vj;
            __syncthreads();   // every thread has read them before thread 0 moves on
            if (nmem == 0) continue;   // uniform
            for (int m = tid; m < nmem; m += kThreads) {
                s_best[m] = s_bestM[m] = s_bestF[m] = kInf;
                s_brm[m] = 0;
            }
            int passes = 0;
            int64_t t = kInf;
            for (;;) {
                pass(t);
                ++passes;
                const int64_t f = s_pF, mx = s_pM;
                if (f == kNone) break;
                for (int m = tid; m < nmem; m += kThreads) {
                    const int64_t Bm = H.micro[s_mj[m]];
                    const int64_t obj = f + (Bm - 1) * mx;
                    if (obj < s_best[m] || (obj == s_best[m] && mx < s_bestM[m])) {
                        s_best[m] = obj;
                        s_bestM[m] = mx;
                        s_bestF[m] = f;
                        s_brm[m] = s_prm;
                        for (int q = 0; q < PP; ++q) {
                            s_blen[m][q] = s_plen[q];
                            s_bw[m][q] = s_pw[q];
                            s_bmask[m][q] = s_pmask[q];
                        }
                    }
                    // a lower threshold t' gives a sum >= f: it can win only if
                    // f + (B-1) t' <= best (equal objectives go to the lower max)
                    int64_t next = mx - 1;
                    if (Bm > 1) {
                        const int64_t lim = floor_div(s_best[m] - f, Bm - 1);
                        next = lim < next ? lim : next;
                    } else if (f > s_best[m]) {
                        next = -1;
                    }
                    s_next[m] = next;
                }
                __syncthreads();
                int64_t next = -1;
                for (int m = 0; m < nmem; ++m) next = s_next[m] > next ? s_next[m] : next;
                __syncthreads();
                if (next < 0) break;
                t = next;
            }
            __syncthreads();
            for (int m = 0; m < nmem; ++m) {
                const int64_t r = key * nB + s_mj[m] - first;
                hapmoe_dp_result *out = res + r;
                uint8_t *tout = types_out + r * kMaxStages, *wout = widths_out + r * kMaxStages;
                const int64_t best = s_best[m];
                if (tid == 0) {
                    if (best == kInf) {
                        out->objective = out->stage_sum = out->t_max = kInf;
                        out->status = HAPMOE_STATUS_INFEASIBLE;
                        out->recompute_mask = 0;
                    } else {
                        out->objective = best + ki->dp_const;
                        out->stage_sum = s_bestF[m];
                        out->t_max = s_bestM[m];
                        out->status = HAPMOE_STATUS_OK;
                        out->recompute_mask = s_brm[m];
                    }
                    if (STATS) {   // the shared sweep's relaxations on its first candidate
                        stats[4 * r] = passes;
                        stats[4 * r + 1] = m == 0 ? (int32_t)s_relax : 0;
                        stats[4 * r + 2] = 0;
                        stats[4 * r + 3] = 0;
                    }
                }
                if (tid < kMaxStages) {
                    const bool on = best != kInf && tid < PP;
                    out->layers[tid] = on ? s_blen[m][tid] : 0;
                    tout[tid] = on ? s_bmask[m][tid] : 0;
                    wout[tid] = on ? s_bw[m][tid] : 0;
                }
            }
            __syncthreads();
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_width_tables(const void *d_image, const hapmoe_candidate *d_cand, int64_t per_config,
                               const TablesLayout &L, int64_t cfg_lo, int64_t n_cfg, void *d_tables, hipStream_t s)
{
    if (n_cfg <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_width_tables, dim3((unsigned)n_cfg), dim3(kThreads), 0, s,
                       static_cast<const unsigned char *>(d_image), d_cand, per_config, cfg_lo, L,
                       static_cast<unsigned char *>(d_tables));
    return hipGetLastError();
}

// one workgroup's slice: the back-trace pointers of every level (int16),
// [levels][end layer][half-groups used]
int64_t width_dp_slot_bytes(int n_layers, int ppmax)
{
    const int64_t W = n_layers + 1, UP = 2 * ppmax + 1;
    return align256((ppmax + 1) * W * UP * 2);
}

// LDS of one workgroup beyond its static arrays: F of two levels (int64),
// [end layer][half-groups used]; at most 2 x 128 x 65 x 8 = 133,120 bytes
int width_dp_lds_bytes(int n_layers, int ppmax)
{
    return 2 * (n_layers + 1) * (2 * ppmax + 1) * 8;
}

int64_t width_dp_ws_bytes(int n_layers, int ppmax, int64_t n_cand)
{
    const int64_t slots = n_cand < kWidthDpMaxSlots ? (n_cand > 0 ? n_cand : 1) : kWidthDpMaxSlots;
    return 256 + slots * width_dp_slot_bytes(n_layers, ppmax);
}

__global__ void k_width_reset(uint32_t *q) { q[0] = 0; }

hipError_t launch_width_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_layers, int ppmax,
                           const TablesLayout &L, const void *d_tables, int64_t first, int64_t count,
                           hapmoe_dp_result *d_res, uint8_t *d_types, uint8_t *d_widths, int32_t *d_stats, void *d_ws,
                           hipStream_t s)
{
    if (count == 0) return hipSuccess;
    const int64_t slot = width_dp_slot_bytes(n_layers, ppmax);
    const int64_t grid = count < kWidthDpMaxSlots ? count : kWidthDpMaxSlots;
    auto *queue = static_cast<uint32_t *>(d_ws);
    auto *slots = static_cast<unsigned char *>(d_ws) + 256;
    hipLaunchKernelGGL(k_width_reset, dim3(1), dim3(1), 0, s, queue);
    const auto *img = static_cast<const unsigned char *>(d_image);
    const auto *tab = static_cast<const unsigned char *>(d_tables);
    const int lds = width_dp_lds_bytes(n_layers, ppmax);
    auto go = [&](auto kern) -> hipError_t {
        if (lds > 65536) {
            const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, lds);
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, s, img, d_cand, L, tab, first, count,
                           slots, slot, d_res, d_types, d_widths, d_stats, queue);
        return hipGetLastError();
    };
    return d_stats ? go(k_width_dp<true>) : go(k_width_dp<false>);
}

}  // namespace hapmoe
