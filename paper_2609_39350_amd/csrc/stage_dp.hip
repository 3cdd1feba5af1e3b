// Stage-DP kernel: for every candidate (pi, device-type ordering, B) the
// pipeline partition of Section 3.4 -- the DP transition over split points
// with the three prunings of Algorithm 1 and the back-trace of the optimum --
// under the 1F1B objective in threshold form:
//     minimise  sum_i c_i + (B-1) max_i c_i,
// i.e. min over t of F_t + (B-1) t where F_t is the least stage-time sum with
// every stage <= t.  The thresholds are swept downwards from t = inf: each
// pass yields a partition whose largest stage m bounds the next threshold to
// m - 1 (F is constant on [m, t]), the min-max partition value t_bot (one
// min-max DP pass) is the floor, and thresholds that can no longer beat the
// incumbent are skipped.  This visits exactly the (max, sum) Pareto points in
// range and returns the same (objective, t*, partition) as an ascending sweep
// over every distinct stage cost.
//
// Mapping: one wave64 per candidate (workgroup = one wave), lanes over the end
// layer b of a stage (BPL = 1 or 2 values of b per lane), layer prefix sums
// staged in LDS, the per-(stage, b) feasible split interval computed once
// (memory with / without recomputation, pruning 1 and 3 are monotone in the
// segment length), then int64 min-plus passes.  No MFMA: this is min-plus
// scan work.
#include "internal.h"

namespace hapmoe {
namespace {

struct DpLds {
    int npad, kmax, ppmax;
    int off_amin, off_a0, off_arg, off_fr, off_mr, off_w, off_a0m, off_a1m, off_moe, total;
};

inline int align16(int x) { return (x + 15) & ~15; }

DpLds dp_lds(int bpl, int kmax, int ppmax)
{
    DpLds S;
    S.npad = 64 * bpl;
    S.kmax = kmax;
    S.ppmax = ppmax;
    const int np = S.npad;
    S.off_amin = kmax * 2 * np * 8;
    S.off_a0 = S.off_amin + ppmax * np;
    const int u = align16(S.off_a0 + ppmax * np);   // union: DP rows  |  memory prefixes
    S.off_arg = u;
    S.off_fr = align16(u + ppmax * np);
    S.off_mr = S.off_fr + np * 8;
    const int dp_end = S.off_mr + np * 8;
    S.off_w = u;
    S.off_a0m = u + np * 8;
    S.off_a1m = u + 2 * np * 8;
    S.off_moe = u + 3 * np * 8;
    const int mem_end = S.off_moe + np * 4;
    S.total = align16(dp_end > mem_end ? dp_end : mem_end);
    return S;
}

__device__ inline int rl32(int v, int src) { return __builtin_amdgcn_readlane(v, src); }

__device__ inline int64_t rl64(int64_t v, int src)
{
    const int lo = __builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)v, src);
    const int hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), src);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ inline unsigned wave_or(unsigned x)
{
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) x |= __shfl_xor(x, d, 64);
    return x;
}

__device__ inline int wave_sum32(int x)
{
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) x += __shfl_xor(x, d, 64);
    return x;
}

__device__ inline void write_result(hapmoe_dp_result *out, int status, int64_t obj, int64_t sum, int64_t tmax,
                                    uint32_t rmask, const uint8_t *layers, int pp)
{
    out->objective = obj;
    out->stage_sum = sum;
    out->t_max = tmax;
    out->status = status;
    out->recompute_mask = rmask;
    uint32_t w[kMaxStages / 4];
    for (int i = 0; i < kMaxStages / 4; ++i) w[i] = 0;
    for (int i = 0; i < pp; ++i) w[i >> 2] |= (uint32_t)layers[i] << (8 * (i & 3));
    uint32_t *dst = reinterpret_cast<uint32_t *>(out->layers);
    for (int i = 0; i < kMaxStages / 4; ++i) dst[i] = w[i];
}

template <int BPL, bool STATS>
__global__ __launch_bounds__(64) void k_stage_dp(const unsigned char *__restrict__ img,
                                                 const hapmoe_candidate *__restrict__ cand, TablesLayout L,
                                                 const unsigned char *__restrict__ tab, int64_t first,
                                                 int64_t count, DpLds S, hapmoe_dp_result *__restrict__ res,
                                                 int32_t *__restrict__ stats)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const ImageHeader &H = *reinterpret_cast<const ImageHeader *>(img);
    const int lane = threadIdx.x;
    const int NP = S.npad;

    // XCD-aware order: block b runs on XCD b % 8; give every XCD a contiguous
    // run of candidates so the candidates of one (pi, ordering) share an L2.
    const int64_t nb = gridDim.x, bid = blockIdx.x;
    const int64_t per = nb >> 3, rem = nb & 7, x = bid & 7, y = bid >> 3;
    const int64_t local = x * per + (x < rem ? x : rem) + y;
    const int64_t idx = first + local;
    hapmoe_dp_result *out = res + local;

    const hapmoe_candidate c = cand[idx];
    const int N = H.n_layers, PP = c.pp;
    const int64_t B = c.n_micro, Bm = B - 1;
    const int64_t key = idx / H.n_micro, cfg = key / H.n_orders;
    const PiInfo *pi = reinterpret_cast<const PiInfo *>(tab + L.off_pi) + cfg;
    const KeyInfo *ki = reinterpret_cast<const KeyInfo *>(tab + L.off_key) + key;

    uint8_t zero[kMaxStages];
    for (int i = 0; i < kMaxStages; ++i) zero[i] = 0;
    if (pi->status != HAPMOE_STATUS_OK) {
        if (lane == 0) write_result(out, HAPMOE_STATUS_OVERFLOW, kInf, kInf, kInf, 0, zero, 0);
        if (STATS && lane == 0) stats[2 * local] = stats[2 * local + 1] = 0;
        return;
    }

    // ---- stage s lives in lane s ----
    int mask = 0, lo = 1, hi = 0, bp = 0;
    if (lane < PP) {
        mask = ki->mask[lane];
        lo = ki->lo[lane];
        hi = ki->hi[lane];
        bp = ki->bpair[lane];
    }
    const unsigned used = wave_or(lane < PP ? (1u << mask) : 0u);   // device-type sets present
    const int nslot = __popc(used);
    const int slot = __popc(used & ((1u << mask) - 1u));
    int64_t cap = kInf;
    for (int h = 0; h < H.n_types; ++h)
        if ((mask >> h) & 1) cap = H.mem_bytes[h] < cap ? H.mem_bytes[h] : cap;
    const int64_t ms = (int64_t)(PP - lane) < B ? (int64_t)(PP - lane) : B;   // 1F1B stored micro-batches
    const bool inner = lane < PP - 1;
    const int64_t p2p = inner ? pi->p2p[(bp >> 2) * kMaxTypes + (bp & 3)] : 0;
    const int bdiff = inner && ((bp >> 2) != (bp & 3));
    const int mixed = __popc(mask) > 1;
    const int64_t X = pi->x_bytes, eta_tbar = (int64_t)H.eta_prune * pi->tbar;

    if (nslot > S.kmax || PP > S.ppmax) {   // host bound violated: refuse rather than overrun LDS
        if (lane == 0) write_result(out, HAPMOE_STATUS_OVERFLOW, kInf, kInf, kInf, 0, zero, 0);
        return;
    }

    int64_t *TM = reinterpret_cast<int64_t *>(smem);
    uint8_t *AMIN = smem + S.off_amin;
    uint8_t *A0B = smem + S.off_a0;
    uint8_t *ARG = smem + S.off_arg;
    int64_t *FR = reinterpret_cast<int64_t *>(smem + S.off_fr);
    int64_t *MR = reinterpret_cast<int64_t *>(smem + S.off_mr);
    int64_t *MW = reinterpret_cast<int64_t *>(smem + S.off_w);
    int64_t *MA0 = reinterpret_cast<int64_t *>(smem + S.off_a0m);
    int64_t *MA1 = reinterpret_cast<int64_t *>(smem + S.off_a1m);
    int32_t *MOE = reinterpret_cast<int32_t *>(smem + S.off_moe);

    // ---- stage the prefix sums of this candidate in LDS ----
    const int64_t np = L.np;
    const int64_t *time = reinterpret_cast<const int64_t *>(tab + L.off_time) + cfg * L.n_masks * 3 * np;
    const int64_t *mem = reinterpret_cast<const int64_t *>(tab + L.off_mem) + cfg * 4 * np;
    {
        unsigned rest = used;
        int k = 0;
        while (rest) {
            const int m = __ffs(rest) - 1;
            rest &= rest - 1;
            const int64_t *src = time + (int64_t)(m - 1) * 3 * np;
#pragma unroll
            for (int j = 0; j < BPL; ++j) {
                const int b = lane + 64 * j;
                if (b <= N) {
                    TM[(k * 2 + 0) * NP + b] = src[b];
                    TM[(k * 2 + 1) * NP + b] = src[np + b];
                }
            }
            ++k;
        }
#pragma unroll
        for (int j = 0; j < BPL; ++j) {
            const int b = lane + 64 * j;
            if (b <= N) {
                MW[b] = mem[b];
                MA0[b] = mem[np + b];
                MA1[b] = mem[2 * np + b];
                MOE[b] = (int32_t)mem[3 * np + b];
            }
        }
    }
    __syncthreads();

    // ---- feasible split interval of every (stage, b) ----
    // a in [AMIN, A0B) needs recomputation (r = 1), a in [A0B, b - lo] fits without.
    for (int s = 0; s < PP; ++s) {
        const int lo_s = rl32(lo, s), hi_s = rl32(hi, s), mask_s = rl32(mask, s);
        const int mixed_s = rl32(mixed, s), bdiff_s = rl32(bdiff, s);
        const int64_t cap_s = rl64(cap, s), ms_s = rl64(ms, s), p2p_s = rl64(p2p, s);
        const int64_t *CM = mixed_s ? time + ((int64_t)(mask_s - 1) * 3 + 2) * np : nullptr;
        const int64_t hc_b = bdiff_s ? p2p_s : 0;
#pragma unroll
        for (int j = 0; j < BPL; ++j) {
            const int b = lane + 64 * j;
            int amin = 255, a0 = 255;
            if (b <= N) {
                const int ahi = b - lo_s;
                const int alo = (b - hi_s) > s ? (b - hi_s) : s;
                const bool valid = b >= s + 1 && b <= N - (PP - 1 - s) && ahi >= alo;
                if (valid) {
                    amin = a0 = ahi + 1;
                    const int64_t wb = MW[b], a0b = MA0[b], a1b = MA1[b];
                    const int mb = MOE[b];
                    const int64_t cmb = CM ? CM[b] : 0;
                    bool phase0 = true;
                    for (int a = ahi; a >= alo; --a) {
                        if (H.prune_hetero) {
                            const int64_t hc = (CM ? cmb - CM[a] : 0) + hc_b;   // pruning 3
                            if (hc > eta_tbar) break;
                        }
                        const int64_t xb = (mb - MOE[a]) > 0 ? X : 0;
                        const int64_t dw = wb - MW[a];
                        if (phase0) {
                            if (dw + ms_s * (a0b - MA0[a]) + xb <= cap_s) {
                                a0 = a;
                                amin = a;
                                continue;
                            }
                            phase0 = false;
                        }
                        if (!H.allow_recompute) break;
                        if (dw + ms_s * (a1b - MA1[a]) + xb <= cap_s) {
                            amin = a;
                            continue;
                        }
                        break;   // pruning 2: no recomputation choice fits
                    }
                }
            }
            AMIN[s * NP + b] = (uint8_t)amin;
            A0B[s * NP + b] = (uint8_t)a0;
        }
    }
    __syncthreads();   // the memory prefixes are dead from here on (their LDS is reused)

    int passes = 0, relax = 0;

    // One DP pass at threshold t.  minimax: F = min over partitions of the
    // largest stage (the bottleneck); otherwise F = least sum with all stages
    // <= t and Mx = the largest stage along the back-trace path.
    auto pass = [&](int64_t t, bool minimax, int64_t &F_out, int64_t &M_out) {
        ++passes;
#pragma unroll
        for (int j = 0; j < BPL; ++j) {
            const int b = lane + 64 * j;
            FR[b] = b == 0 ? 0 : kInf;
            MR[b] = 0;
        }
        __syncthreads();
        for (int s = 0; s < PP; ++s) {
            const int slot_s = rl32(slot, s), lo_s = rl32(lo, s);
            const int64_t p2p_s = rl64(p2p, s);
            const int64_t *T0 = TM + slot_s * 2 * NP;
            const int64_t *T1 = T0 + NP;
            int64_t fn[BPL], mn[BPL];
            int an[BPL];
#pragma unroll
            for (int j = 0; j < BPL; ++j) {
                const int b = lane + 64 * j;
                int64_t best = kInf, bm = 0;
                int ba = 255;
                if (b <= N) {
                    const int amin = AMIN[s * NP + b], a0 = A0B[s * NP + b], ahi = b - lo_s;
                    const int e1 = (a0 - 1) < ahi ? (a0 - 1) : ahi;
                    const int64_t k1 = T1[b] + p2p_s;
                    for (int a = amin; a <= e1; ++a) {
                        const int64_t cst = k1 - T1[a];
                        const int64_t f = FR[a];
                        if (cst <= t && f != kInf) {
                            const int64_t v = minimax ? (f > cst ? f : cst) : f + cst;
                            if (v < best) {
                                best = v;
                                ba = a;
                                const int64_t mr = MR[a];
                                bm = mr > cst ? mr : cst;
                            }
                        }
                    }
                    const int64_t k0 = T0[b] + p2p_s;
                    const int s0 = a0 > amin ? a0 : amin;
                    for (int a = s0; a <= ahi; ++a) {
                        const int64_t cst = k0 - T0[a];
                        const int64_t f = FR[a];
                        if (cst <= t && f != kInf) {
                            const int64_t v = minimax ? (f > cst ? f : cst) : f + cst;
                            if (v < best) {
                                best = v;
                                ba = a;
                                const int64_t mr = MR[a];
                                bm = mr > cst ? mr : cst;
                            }
                        }
                    }
                    if (STATS) relax += (e1 >= amin ? e1 - amin + 1 : 0) + (ahi >= s0 ? ahi - s0 + 1 : 0);
                }
                fn[j] = best;
                mn[j] = bm;
                an[j] = ba;
            }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < BPL; ++j) {
                const int b = lane + 64 * j;
                FR[b] = fn[j];
                MR[b] = mn[j];
                ARG[s * NP + b] = (uint8_t)an[j];
            }
            __syncthreads();
        }
        F_out = FR[N];
        M_out = MR[N];
    };

    int64_t tbot, unused, F1, M1;
    pass(kInf, true, tbot, unused);
    int status = HAPMOE_STATUS_INFEASIBLE;
    int64_t best_s = kInf, best_m = kInf, best_t = kInf;
    if (tbot != kInf) {
        status = HAPMOE_STATUS_OK;
        pass(kInf, false, F1, M1);
        int64_t cur_t = kInf;
        best_s = F1 + Bm * M1;
        best_m = M1;
        best_t = kInf;
        if (tbot < M1) {
            int64_t Fb, Mb;
            pass(tbot, false, Fb, Mb);
            cur_t = tbot;
            if (Fb + Bm * Mb <= best_s) {
                best_s = Fb + Bm * Mb;
                best_m = Mb;
                best_t = tbot;
            }
            const int64_t lb = F1 + Bm * tbot;   // no score is below this
            if (!(best_m == tbot && best_s == lb)) {
                int64_t F = F1, t = M1 - 1;
                if (Bm > 0) {
                    const int64_t lim = (best_s - F) / Bm;
                    t = lim < t ? lim : t;
                }
                while (t > tbot && F + Bm * tbot <= best_s) {
                    int64_t Fc, Mc;
                    pass(t, false, Fc, Mc);
                    cur_t = t;
                    if (Fc + Bm * Mc <= best_s) {
                        best_s = Fc + Bm * Mc;
                        best_m = Mc;
                        best_t = t;
                    }
                    F = Fc;
                    t = Mc - 1;
                    if (Bm > 0) {
                        if (best_s < F) break;
                        const int64_t lim = (best_s - F) / Bm;
                        t = lim < t ? lim : t;
                    }
                }
            }
        }
        if (cur_t != best_t) {
            int64_t Fr, Mr;
            pass(best_t, false, Fr, Mr);
        }
    }

    if (STATS) {
        const int rsum = wave_sum32(relax);
        if (lane == 0) {
            stats[2 * local] = passes;
            stats[2 * local + 1] = rsum;
        }
    }
    if (lane == 0) {
        uint8_t layers[kMaxStages];
        uint32_t rmask = 0;
        if (status == HAPMOE_STATUS_OK) {
            int b = N;
            bool path_ok = true;
            for (int s = PP - 1; s >= 0; --s) {
                const int a = ARG[s * NP + b];
                if (a >= b) {   // no predecessor recorded: cannot happen for a feasible pass
                    path_ok = false;
                    break;
                }
                layers[s] = (uint8_t)(b - a);
                if (a < A0B[s * NP + b]) rmask |= 1u << s;
                b = a;
            }
            if (path_ok && b == 0)
                write_result(out, status, best_s + ki->dp_const, best_s - Bm * best_m, best_m, rmask, layers, PP);
            else
                write_result(out, HAPMOE_STATUS_OVERFLOW, kInf, kInf, kInf, 0, zero, 0);
        } else {
            write_result(out, status, kInf, kInf, kInf, 0, zero, 0);
        }
    }
}

}  // namespace

hipError_t launch_stage_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_layers, int n_micro,
                           int n_orders, const TablesLayout &L, const void *d_tables, int64_t first,
                           int64_t count, int kmax, int ppmax, hapmoe_dp_result *d_res, int32_t *d_stats,
                           hipStream_t s)
{
    (void)n_micro;
    (void)n_orders;
    if (count == 0) return hipSuccess;
    const int bpl = (n_layers + 1 <= 64) ? 1 : 2;
    const DpLds S = dp_lds(bpl, kmax, ppmax);
    const dim3 grid((unsigned)count), block(64);
    const auto *img = static_cast<const unsigned char *>(d_image);
    const auto *tab = static_cast<const unsigned char *>(d_tables);
    if (bpl == 1) {
        if (d_stats)
            hipLaunchKernelGGL((k_stage_dp<1, true>), grid, block, S.total, s, img, d_cand, L, tab, first, count,
                               S, d_res, d_stats);
        else
            hipLaunchKernelGGL((k_stage_dp<1, false>), grid, block, S.total, s, img, d_cand, L, tab, first, count,
                               S, d_res, d_stats);
    } else {
        if (d_stats)
            hipLaunchKernelGGL((k_stage_dp<2, true>), grid, block, S.total, s, img, d_cand, L, tab, first, count,
                               S, d_res, d_stats);
        else
            hipLaunchKernelGGL((k_stage_dp<2, false>), grid, block, S.total, s, img, d_cand, L, tab, first, count,
                               S, d_res, d_stats);
    }
    return hipGetLastError();
}

}  // namespace hapmoe
