// Cost-table kernel: the MoE-aware per-layer cost model of the paper
// (Section 3.2: Eq. 2 compute, Eq. 3 dispatch/combine volume with the best of
// the all-to-all and all-gather primitives, the load-imbalance factor, the
// stage memory model; Section 3.3: compute and primitive tables) evaluated
// for every configuration pi, quantised to int64 ns / bytes and stored as
// prefix sums over layers for the stage DP.  It also lays out the stages of
// every (pi, device-type ordering): device-type set, pruning-1 window,
// boundary link, and the partition-independent T_dp-sync + T_opt of Eq. 4.
//
// One workgroup (4 wave64) per configuration.  Arithmetic is fp64 with IEEE
// + - * / and ceil only, in a fixed order, compiled with -ffp-contract=off so
// every rounded value is reproducible bit for bit.
#include "internal.h"

namespace hapmoe {
namespace {

constexpr int kThreads = 256;
constexpr int kLayerSlots = 128;   // >= kMaxLayers + 1

__device__ inline int lg2i(int v) { return 31 - __clz(v); }

// Rounded-up term; values at or above the int64 budget of the DP set the
// overflow flag instead (and are clamped so the conversion stays defined).
__device__ inline int64_t qterm(double x, unsigned *flag)
{
    if (!(x < (double)kTermLimit)) {
        atomicOr(flag, 1u);
        return kTermLimit;
    }
    return (int64_t)ceil(x);
}

// Slowest link inside a device-type set: largest latency, smallest bandwidth
// over all (h, h') pairs of the set.
__device__ inline void set_link(const ImageHeader &H, int mask, double &alpha, double &bw)
{
    // (unrolled over all kMaxTypes x kMaxTypes pairs so that every load is issued at
    // once; pairs outside the set take no part)
    bool first = true;
    alpha = 0.0;
    bw = 0.0;
#pragma unroll
    for (int h = 0; h < kMaxTypes; ++h) {
#pragma unroll
        for (int g = 0; g < kMaxTypes; ++g) {
            const double a = H.alpha[h * kMaxTypes + g], b = H.bw[h * kMaxTypes + g];
            if (h < H.n_types && g < H.n_types && ((mask >> h) & 1) && ((mask >> g) & 1)) {
                if (first || a > alpha) alpha = a;
                if (first || b < bw) bw = b;
                first = false;
            }
        }
    }
}

// Ring all-reduce over w ranks: 2(w-1) latency steps, 2(w-1)/w of the bytes.
__device__ inline double ring_ar(double bytes, int w, double alpha, double bw)
{
    if (w == 1) return 0.0;
    const double steps = (double)(2 * (w - 1));
    return steps * alpha + ((steps * bytes) / (double)w) / bw;
}

// K exclusive wave scans side by side (their shuffles overlap): x[f] becomes the
// sum of x[f] over the lower lanes
template <int K>
__device__ inline void wave_excl_scan_k(int64_t (&x)[K], int lane)
{
    int64_t inc[K];
#pragma unroll
    for (int f = 0; f < K; ++f) inc[f] = x[f];
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int64_t y[K];
#pragma unroll
        for (int f = 0; f < K; ++f) y[f] = __shfl_up(inc[f], d, 64);
#pragma unroll
        for (int f = 0; f < K; ++f)
            if (lane >= d) inc[f] += y[f];
    }
#pragma unroll
    for (int f = 0; f < K; ++f) x[f] = inc[f] - x[f];
}

__device__ inline int64_t wave_sum(int64_t x)
{
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d, 64);
    return x;
}

__device__ inline int64_t wave_max(int64_t x)
{
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const int64_t y = __shfl_xor(x, d, 64);
        x = y > x ? y : x;
    }
    return x;
}

// Load-imbalance factor of every layer (Section 3.2, router skew): one block a
// layer, rho = max / mean token count over its experts.  It depends on the
// model only, so it is computed once per launch, not once per configuration.
__global__ __launch_bounds__(kThreads) void k_layer_skew(const unsigned char *__restrict__ img, TablesLayout L,
                                                         unsigned char *__restrict__ tab)
{
    const ImageHeader &H = *reinterpret_cast<const ImageHeader *>(img);
    const uint8_t *is_moe = img + H.off_is_moe;
    const int64_t *tokens = reinterpret_cast<const int64_t *>(img + H.off_tokens);
    const int l = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int E = H.n_experts;
    __shared__ int64_t s_sum[kThreads / 64], s_max[kThreads / 64];
    double sk = 1.0;
    if (is_moe[l]) {   // block-uniform
        int64_t sum = 0, mx = 0;
        for (int e = tid; e < E; e += kThreads) {
            const int64_t v = tokens[(int64_t)l * E + e];
            sum += v;
            mx = v > mx ? v : mx;
        }
        sum = wave_sum(sum);
        mx = wave_max(mx);
        if (lane == 0) {
            s_sum[wave] = sum;
            s_max[wave] = mx;
        }
        __syncthreads();
        if (tid == 0) {
            for (int w = 1; w < kThreads / 64; ++w) {
                sum += s_sum[w];
                mx = s_max[w] > mx ? s_max[w] : mx;
            }
            const double rho = sum > 0 ? (double)(mx * E) / (double)sum : 1.0;
            sk = 1.0 + H.gamma * (rho - 1.0);
        }
    }
    if (tid == 0) reinterpret_cast<double *>(tab + L.off_layer)[l] = sk;
}

// Eight workgroups a CU (64 VGPRs): each workgroup is a short latency-bound
// sequence of phases, and 2,510 of them on 256 CUs finish sooner with twice the
// workgroups resident, even though a few small per-thread arrays then live in
// scratch (0.105 -> 0.087 ms on the 96-layer MoE workload).
__global__ __launch_bounds__(kThreads, 8) void k_cost_tables(const unsigned char *__restrict__ img,
                                                          const hapmoe_candidate *__restrict__ cand,
                                                          int64_t per_config, int64_t cfg_lo, TablesLayout L,
                                                          unsigned char *__restrict__ tab,
                                                          double *__restrict__ dbg, DebugLayout D)
{
    const ImageHeader &H = *reinterpret_cast<const ImageHeader *>(img);
    const uint8_t *is_moe = img + H.off_is_moe;
    const int64_t *pdense = reinterpret_cast<const int64_t *>(img + H.off_pdense);
    const int64_t *pexp = reinterpret_cast<const int64_t *>(img + H.off_pexp);
    const int64_t *act = reinterpret_cast<const int64_t *>(img + H.off_act);
    const int64_t *tdense = reinterpret_cast<const int64_t *>(img + H.off_tdense);
    const int64_t *tffn = reinterpret_cast<const int64_t *>(img + H.off_tffn);

    const int64_t cfg = cfg_lo + blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const hapmoe_candidate c = cand[cfg * per_config];
    const int N = H.n_layers, T = H.n_types;
    // MoE flags of layers 2 lane and 2 lane + 1, the layers this lane takes in the
    // prefix sums and for every device-type set
    const bool moe2[2] = {2 * lane < N && is_moe[2 * lane] != 0, 2 * lane + 1 < N && is_moe[2 * lane + 1] != 0};
    double *dcfg = dbg ? dbg + cfg * D.per_cfg : nullptr;

    __shared__ int64_t s_qce[kMaxTypes][kLayerSlots];   // q(comp) + q(expert) per type, layer
    __shared__ int64_t s_maxce[kLayerSlots];
    __shared__ double s_skew[kLayerSlots];
    __shared__ double s_link_a[1 << kMaxTypes], s_link_b[1 << kMaxTypes];   // per device-type set
    __shared__ int64_t s_w[kLayerSlots], s_a0[kLayerSlots], s_a1[kLayerSlots];
    __shared__ double s_pavg;
    __shared__ unsigned s_used, s_flag;
    __shared__ int64_t s_tbar;
    __shared__ int32_t s_ospd[kMaxOrders][kMaxStages];   // block orderings: speed of each stage
    __shared__ int32_t s_perm[kMaxOrders][kMaxTypes], s_count[kMaxTypes], s_speed[kMaxTypes];   // orderings, devices
    __shared__ uint8_t s_omask[kMaxOrders][kMaxStages];  //   and its device-type set
    __shared__ int64_t s_osum[kMaxOrders];               //   summed stage speeds

    // tokens of one micro-batch per rank, activation tensor bytes, D_moe (Eq. 3)
    const double tok = (double)((int64_t)H.seq_len * H.mbs / c.cp);
    const double Dact = (tok * (double)H.hidden) * (double)H.elem_bytes;
    const double dmoe = (Dact * (double)H.top_k) * (1.0 - 1.0 / (double)c.ep);

    if (tid == 0) {
        s_used = 0;
        s_flag = 0;
    }
    if (wave == 0) {   // parameters per device, averaged over the stages (exact int64 sums)
        int64_t pd = 0, pe = 0;
#pragma unroll
        for (int r = 0; r < kLayerSlots / 64; ++r) {   // N < kLayerSlots: every load at once
            const int l = lane + 64 * r;
            pd += l < N ? pdense[l] : 0;
            pe += l < N ? pexp[l] : 0;
        }
        pd = wave_sum(pd);
        pe = wave_sum(pe);
        if (lane == 0) s_pavg = ((double)pd / (double)c.tp + (double)pe / (double)(c.ep * c.tpe)) / (double)c.pp;
    }
    // load-imbalance factors (k_layer_skew) and the slowest link of every
    // device-type set
    for (int l = tid; l < N; l += kThreads) s_skew[l] = reinterpret_cast<const double *>(tab + L.off_layer)[l];
    if (tid >= 1 && tid < (1 << T)) set_link(H, tid, s_link_a[tid], s_link_b[tid]);
    // the orderings, device counts and speeds, read by the stage layouts below
    if (tid < kMaxOrders * kMaxTypes) s_perm[tid / kMaxTypes][tid % kMaxTypes] = H.perm[tid / kMaxTypes][tid % kMaxTypes];
    if (tid < kMaxTypes) {
        s_count[tid] = H.count[tid];
        s_speed[tid] = H.speed[tid];
    }
    __syncthreads();

    // ---- stage layout of the block orderings: (ordering, stage) pairs over the threads ----
    // (stage_types 3, per-stage widths, keeps this uniform layout for its constants)
    if (H.stage_types == 0 || H.stage_types == 3) {
        const int nord = H.n_orders, PP = c.pp, g = H.total_devices / PP, npair = nord * PP;
        for (int i = tid; i < npair; i += kThreads) {
            const int o = i / PP, s = i - o * PP;
            // (loops over all kMaxTypes positions, unrolled, so that the arrays stay in
            // registers; positions j >= T take no part)
            int pos_type[kMaxTypes], pos_cnt[kMaxTypes], pos_end[kMaxTypes];
            int acc = 0;
#pragma unroll
            for (int j = 0; j < kMaxTypes; ++j) {
                pos_type[j] = j < T ? s_perm[o][j] : 0;
                pos_cnt[j] = j < T ? s_count[pos_type[j]] : 0;
                acc += pos_cnt[j];
                pos_end[j] = acc;
            }
            // the type of device d: that of the first block ending past d, else the last block's
            auto type_of = [&](int d) {
                int t = 0;
#pragma unroll
                for (int j = kMaxTypes - 1; j >= 0; --j)
                    if (j == T - 1 || (j < T && d < pos_end[j])) t = pos_type[j];
                return t;
            };
            const int d0 = s * g, d1 = d0 + g;
            int mask = 0;
#pragma unroll
            for (int j = 0; j < kMaxTypes; ++j)
                if (j < T && pos_end[j] - pos_cnt[j] < d1 && pos_end[j] > d0) mask |= 1 << pos_type[j];
            const int bpair = s < PP - 1 ? (type_of(d1 - 1) << 2) | type_of(d1) : 0;
            int sp = 0;
#pragma unroll
            for (int h = 0; h < kMaxTypes; ++h)
                if (h < T && ((mask >> h) & 1)) sp = (sp == 0 || s_speed[h] < sp) ? s_speed[h] : sp;
            KeyInfo *K = reinterpret_cast<KeyInfo *>(tab + L.off_key) + (cfg * L.n_orders + o);
            K->mask[s] = (uint8_t)mask;
            K->bpair[s] = (uint8_t)bpair;
            atomicOr(&s_used, 1u << (mask - 1));
            s_ospd[o][s] = sp;
            s_omask[o][s] = (uint8_t)mask;
        }
        __syncthreads();
        // per ordering: summed speed, slowest link over the stages, T_dp-sync + T_opt
        for (int o = tid; o < nord; o += kThreads) {
            int64_t sum_speed = 0;
            double al_k = 0.0, bw_k = 0.0;
            for (int s = 0; s < PP; ++s) {
                sum_speed += s_ospd[o][s];
                const int m = s_omask[o][s];
                const double a = s_link_a[m], b = s_link_b[m];
                if (s == 0 || a > al_k) al_k = a;
                if (s == 0 || b < bw_k) bw_k = b;
            }
            s_osum[o] = sum_speed;
            KeyInfo *K = reinterpret_cast<KeyInfo *>(tab + L.off_key) + (cfg * L.n_orders + o);
            const double pavg = s_pavg;
            K->dp_const = qterm(ring_ar(4.0 * pavg, c.dp, al_k, bw_k) + (H.opt_coef * pavg) / (double)c.dp, &s_flag);
        }
        __syncthreads();
        // pruning-1 window: n_s in [(1-delta) w_s N, (1+delta) w_s N], w_s = P_s / sum P
        const int64_t dn = H.delta_num, dd = H.delta_den;
        for (int i = tid; i < npair; i += kThreads) {
            const int o = i / PP, s = i - o * PP;
            int64_t lo = 1, hi = N;
            if (H.prune_window == 2) {   // uniform: floor(N / PP) .. ceil(N / PP) layers per stage
                lo = N / PP;
                hi = (N + PP - 1) / PP;
            } else if (H.prune_window) {
                const int64_t den = dd * s_osum[o];
                lo = ((dd - dn) * s_ospd[o][s] * (int64_t)N) / den;
                hi = ((dd + dn) * s_ospd[o][s] * (int64_t)N + den - 1) / den;
                lo = lo < 1 ? 1 : lo;
                hi = hi > N ? N : hi;
            }
            KeyInfo *K = reinterpret_cast<KeyInfo *>(tab + L.off_key) + (cfg * L.n_orders + o);
            K->lo[s] = (uint8_t)lo;
            K->hi[s] = (uint8_t)hi;
        }
    }

    // ---- free stage types: the layout of every stage-type sequence (one thread each) ----
    for (int o = tid; (H.stage_types == 1 || H.stage_types == 2) && o < H.n_orders; o += kThreads) {
        const int g = H.total_devices / c.pp;
        KeyInfo *K = reinterpret_cast<KeyInfo *>(tab + L.off_key) + (cfg * L.n_orders + o);
        int seq[kMaxStages];   // free stage types: the type of each stage
        if (H.stage_types) {
            // the o-th distinct arrangement of k_h = m_h / g stages of type h, in
            // lexicographic order: at each position take the smallest type whose
            // block of arrangements (the multinomial of what remains) holds o
            int k[kMaxTypes];
            int64_t M = 1;   // multinomial of the counts so far; it never falls, and stays <= 2^20
            int r = 0;
            for (int h = 0; h < kMaxTypes; ++h) {
                k[h] = h < T ? s_count[h] / g : 0;
                for (int i = 1; i <= k[h]; ++i) M = M * ++r / i;
            }
            if (o >= M) {   // past this pipeline's sequences: no partition is feasible
                K->dp_const = 0;
                for (int s = 0; s < kMaxStages; ++s) {
                    K->mask[s] = 1;
                    K->lo[s] = K->hi[s] = K->bpair[s] = 0;
                }
                continue;
            }
            int64_t rest = o;
            for (int s = 0; s < c.pp; ++s) {
                const int left = c.pp - s;
                for (int h = 0; h < T; ++h) {
                    if (k[h] == 0) continue;
                    const int64_t block = M * k[h] / left;   // arrangements that put h here
                    if (rest < block) {
                        seq[s] = h;
                        M = block;
                        --k[h];
                        break;
                    }
                    rest -= block;
                }
            }
        }
        int pos_type[kMaxTypes], pos_start[kMaxTypes], pos_end[kMaxTypes];
        int acc = 0;
        for (int j = 0; j < T; ++j) {
            pos_type[j] = H.stage_types ? j : s_perm[o][j];   // perm holds |H|! <= 24 rows
            pos_start[j] = acc;
            acc += s_count[pos_type[j]];
            pos_end[j] = acc;
        }
        auto type_of = [&](int d) {
            int t = pos_type[T - 1];
            for (int j = T - 1; j >= 0; --j)
                if (d < pos_end[j]) t = pos_type[j];
            return t;
        };
        int spd[kMaxStages];
        int64_t sum_speed = 0;
        double al_k = 0.0, bw_k = 0.0;
        for (int s = 0; s < c.pp; ++s) {
            const int d0 = s * g, d1 = d0 + g;
            int mask = 0, bpair = 0;
            if (H.stage_types) {
                mask = 1 << seq[s];
                if (s < c.pp - 1) bpair = (seq[s] << 2) | seq[s + 1];
            } else {
                for (int j = 0; j < T; ++j)
                    if (pos_start[j] < d1 && pos_end[j] > d0) mask |= 1 << pos_type[j];
                if (s < c.pp - 1) bpair = (type_of(d1 - 1) << 2) | type_of(d1);
            }
            int sp = 0;
            for (int h = 0; h < T; ++h)
                if ((mask >> h) & 1) sp = (sp == 0 || s_speed[h] < sp) ? s_speed[h] : sp;
            spd[s] = sp;
            sum_speed += sp;
            double a, b;
            set_link(H, mask, a, b);
            if (s == 0 || a > al_k) al_k = a;
            if (s == 0 || b < bw_k) bw_k = b;
            atomicOr(&s_used, 1u << (mask - 1));
            K->mask[s] = (uint8_t)mask;
            K->bpair[s] = (uint8_t)bpair;
        }
        // pruning-1 window: n_s in [(1-delta) w_s N, (1+delta) w_s N], w_s = P_s / sum P
        const int64_t dn = H.delta_num, dd = H.delta_den;
        const int64_t den = dd * sum_speed;
        for (int s = 0; s < c.pp; ++s) {
            int64_t lo = 1, hi = N;
            if (H.prune_window == 2) {   // uniform: floor(N / PP) .. ceil(N / PP) layers per stage
                lo = N / c.pp;
                hi = (N + c.pp - 1) / c.pp;
            } else if (H.prune_window) {
                lo = ((dd - dn) * spd[s] * (int64_t)N) / den;
                hi = ((dd + dn) * spd[s] * (int64_t)N + den - 1) / den;
                lo = lo < 1 ? 1 : lo;
                hi = hi > N ? N : hi;
            }
            K->lo[s] = (uint8_t)lo;
            K->hi[s] = (uint8_t)hi;
        }
        const double pavg = s_pavg;
        K->dp_const = qterm(ring_ar(4.0 * pavg, c.dp, al_k, bw_k) + (H.opt_coef * pavg) / (double)c.dp, &s_flag);
    }

    // ---- per-layer terms: Eq. 2 per device type, load imbalance, memory ----
    for (int l = tid; l < N; l += kThreads) {
        const bool moe = is_moe[l] != 0;
        const double sk = s_skew[l];
        int64_t mce = 0;
        for (int h = 0; h < T; ++h) {
            const int64_t off = (((int64_t)h * 4 + lg2i(c.tp)) * 4 + lg2i(c.cp)) * N + l;
            const double td = (double)tdense[off], tf = (double)tffn[off];
            double comp, expert;
            if (!moe) {
                comp = td;
                expert = 0.0;
            } else {
                const double route = H.route_coef[h] * (tok * (double)H.hidden);
                comp = (td - tf) + route;
                const double xexp = (H.moe_ffn_mult * tf) / ((H.eff[h] * (double)c.ep) * (double)c.tpe);
                expert = sk * xexp;
            }
            const int64_t q = qterm(comp, &s_flag) + qterm(expert, &s_flag);
            s_qce[h][l] = q;
            mce = q > mce ? q : mce;
            if (dcfg) {
                dcfg[D.off_type + ((int64_t)l * T + h) * 2 + 0] = comp;
                dcfg[D.off_type + ((int64_t)l * T + h) * 2 + 1] = expert;
            }
        }
        s_maxce[l] = mce;
        const double beta_opt = 6.0 + 12.0 / (double)c.dp;
        const double w = ((double)pdense[l] / (double)c.tp + (double)pexp[l] / (double)(c.ep * c.tpe)) * beta_opt;
        const double a0 = (double)act[l] / (double)(c.tp * c.cp);
        const int64_t qa0 = qterm(a0, &s_flag);
        s_w[l] = qterm(w, &s_flag);
        s_a0[l] = qa0;
        s_a1[l] = qterm(H.rc_act * (double)qa0, &s_flag);
        if (dcfg) {
            dcfg[D.off_mem + (int64_t)l * 2 + 0] = w;
            dcfg[D.off_mem + (int64_t)l * 2 + 1] = a0;
        }
    }
    __syncthreads();

    const int64_t np = L.np;
    // ---- memory prefix sums and the pruning-3 compute bound (wave 0) ----
    if (wave == 0) {
        int64_t *mem = reinterpret_cast<int64_t *>(tab + L.off_mem) + cfg * 4 * np;
        const int l0 = 2 * lane, l1 = 2 * lane + 1;
        int64_t v[4][2];
        for (int k = 0; k < 2; ++k) {
            const int l = k ? l1 : l0;
            const bool ok = l < N;
            v[0][k] = ok ? s_w[l] : 0;
            v[1][k] = ok ? s_a0[l] : 0;
            v[2][k] = ok ? s_a1[l] : 0;
            v[3][k] = ok ? (int64_t)moe2[k] : 0;
        }
        int64_t exs[4];
#pragma unroll
        for (int f = 0; f < 4; ++f) exs[f] = v[f][0] + v[f][1];
        wave_excl_scan_k(exs, lane);
#pragma unroll
        for (int f = 0; f < 4; ++f) {
            const int64_t ex = exs[f];
            if (lane == 0) mem[f * np] = 0;
            if (l0 < N) mem[f * np + l0 + 1] = ex + v[f][0];
            if (l1 < N) mem[f * np + l1 + 1] = ex + v[f][0] + v[f][1];
        }
        const int64_t tot = wave_sum((l0 < N ? s_maxce[l0] : 0) + (l1 < N ? s_maxce[l1] : 0));
        if (lane == 0) s_tbar = (tot + c.pp - 1) / c.pp;
    }

    // ---- per device-type set: communication and stage times (all waves) ----
    const unsigned used = s_used;
    int k = 0;
    for (int m = 1; m <= (int)L.n_masks; ++m) {
        if (!((used >> (m - 1)) & 1)) continue;
        if ((k++ & 3) != wave) continue;
        const double alpha = s_link_a[m], bw = s_link_b[m];
        int64_t *P = reinterpret_cast<int64_t *>(tab + L.off_time) + (cfg * L.n_masks + (m - 1)) * 3 * np;
        int64_t v[3][2];
        for (int kk = 0; kk < 2; ++kk) {
            const int l = 2 * lane + kk;
            v[0][kk] = v[1][kk] = v[2][kk] = 0;
            if (l >= N) continue;
            double a2a, tp;
            if (!moe2[kk]) {
                a2a = 0.0;
                tp = 4.0 * ring_ar(Dact, c.tp, alpha, bw);
            } else {
                const double sk = s_skew[l];
                const double f_a2a = (double)(c.ep - 1) * alpha + dmoe / bw;
                const double f_ag = (double)(c.ep - 1) * alpha + (Dact * (double)(c.ep - 1)) / bw;
                const double sel = f_ag < f_a2a ? f_ag : f_a2a;
                a2a = sk * (4.0 * sel);
                tp = 2.0 * ring_ar(Dact, c.tp, alpha, bw) + 2.0 * ring_ar(Dact, c.tpe, alpha, bw);
            }
            const double cpt = c.cp == 1 ? 0.0
                                         : 3.0 * ((double)(c.cp - 1) * (alpha + ((2.0 * Dact) / (double)c.tp) / bw));
            const int64_t comm = qterm(a2a, &s_flag) + qterm(tp, &s_flag) + qterm(cpt, &s_flag);
            int64_t ce = 0;
#pragma unroll
            for (int h = 0; h < kMaxTypes; ++h)
                if (h < T && ((m >> h) & 1)) ce = s_qce[h][l] > ce ? s_qce[h][l] : ce;
            const int64_t t0 = ce + comm;
            v[0][kk] = t0;
            v[1][kk] = qterm(H.rc_time * (double)t0, &s_flag);
            v[2][kk] = comm;
            if (dcfg) {
                double *dm = dcfg + D.off_mask + ((int64_t)(m - 1) * N + l) * 3;
                dm[0] = a2a;
                dm[1] = tp;
                dm[2] = cpt;
            }
        }
        const int l0 = 2 * lane, l1 = 2 * lane + 1;
        int64_t exs[3];
#pragma unroll
        for (int f = 0; f < 3; ++f) exs[f] = v[f][0] + v[f][1];
        wave_excl_scan_k(exs, lane);
#pragma unroll
        for (int f = 0; f < 3; ++f) {
            const int64_t ex = exs[f];
            if (lane == 0) P[f * np] = 0;
            if (l0 < N) P[f * np + l0 + 1] = ex + v[f][0];
            if (l1 < N) P[f * np + l1 + 1] = ex + v[f][0] + v[f][1];
        }
    }

    // ---- per-configuration record ----
    PiInfo *pi = reinterpret_cast<PiInfo *>(tab + L.off_pi) + cfg;
    if (tid < kMaxTypes * kMaxTypes) {
        // boundary transfer: activation forward + gradient back, tokens*H*beta/TP each
        // way; one (h, g) link a thread
        const int h = tid / kMaxTypes, g = tid % kMaxTypes;
        int64_t v = 0;
        if (h < T && g < T) {
            const double a = H.alpha[h * kMaxTypes + g], b = H.bw[h * kMaxTypes + g];
            v = qterm(2.0 * (a + (Dact / (double)c.tp) / b), &s_flag);
        }
        pi->p2p[tid] = v;
    } else if (tid == kMaxTypes * kMaxTypes) {
        // routing metadata (8 bytes per token and choice) + dispatch and combine buffers
        pi->x_bytes = qterm(((8.0 * tok) * (double)H.top_k) + 2.0 * dmoe, &s_flag);
    }
    __syncthreads();   // every overflow flag is in
    if (tid == 0) {
        pi->tbar = s_tbar;
        pi->used_masks = s_used;
        pi->status = s_flag ? HAPMOE_STATUS_OVERFLOW : HAPMOE_STATUS_OK;
    }
}

}  // namespace
}  // namespace hapmoe

namespace hapmoe {

hipError_t launch_cost_tables(const void *d_image, const hapmoe_candidate *d_cand, int64_t per_config,
                              int n_layers, const TablesLayout &L, int64_t cfg_lo, int64_t n_cfg, void *d_tables,
                              double *d_debug, const DebugLayout &D, hipStream_t s)
{
    if (n_cfg <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_layer_skew, dim3((unsigned)n_layers), dim3(kThreads), 0, s,
                       static_cast<const unsigned char *>(d_image), L, static_cast<unsigned char *>(d_tables));
    hipLaunchKernelGGL(k_cost_tables, dim3((unsigned)n_cfg), dim3(kThreads), 0, s,
                       static_cast<const unsigned char *>(d_image), d_cand, per_config, cfg_lo, L,
                       static_cast<unsigned char *>(d_tables), d_debug, D);
    return hipGetLastError();
}

}  // namespace hapmoe
