// Stage-DP kernel: for every candidate (pi, device-type ordering, B) the
// pipeline partition of Section 3.4 -- the DP transition over split points
// with the three prunings of Algorithm 1 and the back-trace of the optimum --
// under the 1F1B objective in threshold form:
//     minimise  sum_i c_i + (B-1) max_i c_i,
// i.e. min over t of F_t + (B-1) t where F_t is the least stage-time sum with
// every stage <= t.  Thresholds are swept downwards from t = inf: a pass at t
// yields a partition whose largest stage m makes F constant on [m, t], so the
// next useful threshold is m - 1; the min-max partition value t_bot (one
// min-max pass) is the floor, and thresholds that can no longer beat an
// incumbent are skipped.  This visits exactly the (max, sum) Pareto points in
// range and returns the same (objective, t*, partition) as an ascending sweep
// over every distinct stage cost.
//
// Work sharing across B: B enters a candidate only through the 1F1B count of
// stored micro-batches min(PP - i, B) (memory) and through the (B-1) weight of
// the objective.  All candidates of one (pi, ordering) whose B gives the same
// min(B, PP) therefore share the feasible segments and every DP pass; one
// sweep serves all of them, with one incumbent per B held in its own lane.
//
// Mapping: persistent wave64 workgroups pull work items (pi, ordering,
// B-group) from an atomic queue, largest PP first.  Lanes run over the end
// layer b of a stage, restricted to the band of b reachable under the
// pruning-1 windows; split points a run over the previous stage's band.
// Layer prefix sums sit in LDS; the feasible split interval of every
// (stage, b) is computed once per work item (memory with / without
// recomputation and prunings 1 and 3 are monotone in the segment length).
// No MFMA: this is int64 min-plus scan work.
#include "internal.h"

namespace hapmoe {
namespace {

constexpr int64_t kBig = int64_t(1) << 62;   // "no partition" inside the DP (sums stay far from overflow)
constexpr int kMaxRuns = 32;

struct ItemRun {
    int64_t item_start;
    int32_t key_start, key_count, n_groups, pp;
};

// Work items: runs of consecutive (pi, ordering) keys with the same PP; each
// key of a run contributes n_groups items (one per distinct min(B, PP)).
struct ItemMap {
    int32_t n_runs, pad;
    int64_t total;
    ItemRun run[kMaxRuns];
};

struct DpLds {
    int np, kmax, ppmax;
    int off_amin, off_a0, off_u, off_arg, off_fm, off_w, off_a0m, off_a1m, off_moe, off_bt, total;
};

inline int align16(int x) { return (x + 15) & ~15; }

// LDS of one wave: TM [kmax][np] {T0, T1} | AMIN, A0B [ppmax][np] bytes |
// union( ARG [ppmax][np] bytes + FM [np] {F, M} ,  memory prefixes ) | back-trace scratch
DpLds dp_lds(int n_layers, int kmax, int ppmax)
{
    DpLds S;
    S.np = (n_layers + 1 + 15) & ~15;
    S.kmax = kmax;
    S.ppmax = ppmax;
    const int np = S.np;
    S.off_amin = kmax * np * 16;
    S.off_a0 = S.off_amin + ppmax * np;
    S.off_u = align16(S.off_a0 + ppmax * np);
    S.off_arg = S.off_u;
    S.off_fm = align16(S.off_arg + ppmax * np);
    const int dp_end = S.off_fm + np * 16;
    S.off_w = S.off_u;
    S.off_a0m = S.off_w + np * 8;
    S.off_a1m = S.off_a0m + np * 8;
    S.off_moe = S.off_a1m + np * 8;
    const int mem_end = S.off_moe + np * 4;
    S.off_bt = align16(dp_end > mem_end ? dp_end : mem_end);
    S.total = S.off_bt + 48;
    return S;
}

__device__ inline int rl32(int v, int src) { return __builtin_amdgcn_readlane(v, src); }

__device__ inline int64_t rl64(int64_t v, int src)
{
    const int lo = __builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)v, src);
    const int hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), src);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ inline uint64_t wave_or64(uint64_t x)
{
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) x |= __shfl_xor(x, d, 64);
    return x;
}

__device__ inline int64_t wave_max64(int64_t x)
{
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_xor(x, d, 64);
        x = y > x ? y : x;
    }
    return x;
}

__device__ inline int64_t wave_min64(int64_t x)
{
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_xor(x, d, 64);
        x = y < x ? y : x;
    }
    return x;
}

__device__ inline int wave_incl_scan(int x, int lane)
{
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    return x;
}

__device__ inline int wave_sum32(int x)
{
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) x += __shfl_xor(x, d, 64);
    return x;
}

// The workgroup is a single wave: LDS traffic of one wave is processed in
// order, so a wave-level fence (wait for outstanding LDS ops + no compiler
// motion) separates the reads of a row from its in-place update.
__device__ inline void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct I64x2 {
    int64_t x, y;
};

__device__ inline void write_result(hapmoe_dp_result *out, int status, int64_t obj, int64_t sum, int64_t tmax,
                                    uint32_t rmask, const uint32_t *layer_words)
{
    uint4 *dst = reinterpret_cast<uint4 *>(out);
    uint4 w0, w1, w2, w3;
    w0.x = (uint32_t)(uint64_t)obj;
    w0.y = (uint32_t)((uint64_t)obj >> 32);
    w0.z = (uint32_t)(uint64_t)sum;
    w0.w = (uint32_t)((uint64_t)sum >> 32);
    w1.x = (uint32_t)(uint64_t)tmax;
    w1.y = (uint32_t)((uint64_t)tmax >> 32);
    w1.z = (uint32_t)status;
    w1.w = rmask;
    w2.x = layer_words[0];
    w2.y = layer_words[1];
    w2.z = layer_words[2];
    w2.w = layer_words[3];
    w3.x = layer_words[4];
    w3.y = layer_words[5];
    w3.z = layer_words[6];
    w3.w = layer_words[7];
    dst[0] = w0;
    dst[1] = w1;
    dst[2] = w2;
    dst[3] = w3;
}

__global__ void k_reset_queue(uint32_t *q) { q[0] = 0; }

template <int R, bool STATS>
__global__ __launch_bounds__(64) void k_stage_dp(const unsigned char *__restrict__ img,
                                                 const hapmoe_candidate *__restrict__ cand, TablesLayout L,
                                                 const unsigned char *__restrict__ tab, int64_t first,
                                                 int64_t count, ItemMap M, DpLds S,
                                                 hapmoe_dp_result *__restrict__ res, int32_t *__restrict__ stats,
                                                 uint32_t *__restrict__ queue)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const ImageHeader &H = *reinterpret_cast<const ImageHeader *>(img);
    const int lane = threadIdx.x;
    const int NP = S.np;
    const int N = H.n_layers;
    const int nB = H.n_micro;
    const int64_t np = L.np;
    const uint32_t zero_words[8] = {0, 0, 0, 0, 0, 0, 0, 0};

    I64x2 *TM = reinterpret_cast<I64x2 *>(smem);
    uint8_t *AMIN = smem + S.off_amin;
    uint8_t *A0B = smem + S.off_a0;
    uint8_t *ARG = smem + S.off_arg;
    I64x2 *FM = reinterpret_cast<I64x2 *>(smem + S.off_fm);
    int64_t *MW = reinterpret_cast<int64_t *>(smem + S.off_w);
    int64_t *MA0 = reinterpret_cast<int64_t *>(smem + S.off_a0m);
    int64_t *MA1 = reinterpret_cast<int64_t *>(smem + S.off_a1m);
    int32_t *MOE = reinterpret_cast<int32_t *>(smem + S.off_moe);
    uint32_t *BT = reinterpret_cast<uint32_t *>(smem + S.off_bt);   // back-trace: 8 words of n_i + r mask

    for (;;) {
        uint32_t qi = 0;
        if (lane == 0) qi = atomicAdd(queue, 1u);
        qi = __shfl(qi, 0, 64);
        if ((int64_t)qi >= M.total) break;   // every wave exits once the queue is drained
        const int64_t item = M.total - 1 - (int64_t)qi;   // runs are PP-ascending: biggest work first
        int r = 0;
        while (r + 1 < M.n_runs && item >= M.run[r + 1].item_start) ++r;
        const int64_t rel = item - M.run[r].item_start;
        const int ng = M.run[r].n_groups;
        const int64_t key = M.run[r].key_start + rel / ng;
        const int g = (int)(rel % ng);
        const int64_t cfg = key / H.n_orders;
        const int64_t idx0 = key * nB;
        const int PP = cand[idx0].pp;

        // ---- the candidates of this item: lanes j < nB with min(B_j, PP) equal to the g-th value ----
        int Bj = 1, vj = 0;
        if (lane < nB) {
            Bj = H.micro[lane];
            vj = Bj < PP ? Bj : PP;
        }
        const uint64_t present = wave_or64(lane < nB ? (uint64_t(1) << vj) : 0);
        uint64_t rest = present;
        for (int k = 0; k < g; ++k) rest &= rest - 1;
        const int vg = __ffsll((unsigned long long)rest) - 1;
        const int64_t inst = idx0 + lane;
        const bool member = lane < nB && vj == vg && inst >= first && inst < first + count;
        if (!__any(member)) continue;
        hapmoe_dp_result *out = res + (inst - first);

        const PiInfo *pi = reinterpret_cast<const PiInfo *>(tab + L.off_pi) + cfg;
        const KeyInfo *ki = reinterpret_cast<const KeyInfo *>(tab + L.off_key) + key;
        if (pi->status != HAPMOE_STATUS_OK) {
            if (member) {
                write_result(out, HAPMOE_STATUS_OVERFLOW, kInf, kInf, kInf, 0, zero_words);
                if (STATS) stats[2 * (inst - first)] = stats[2 * (inst - first) + 1] = 0;
            }
            continue;
        }

        // ---- stage s lives in lane s ----
        int mask = 0, lo = 0, hi = 0, bp = 0;
        if (lane < PP) {
            mask = ki->mask[lane];
            lo = ki->lo[lane];
            hi = ki->hi[lane];
            bp = ki->bpair[lane];
        }
        const uint64_t used = wave_or64(lane < PP ? (uint64_t(1) << mask) : 0);
        const int nslot = __popcll(used);
        const int slot = __popcll(used & ((uint64_t(1) << mask) - 1));
        int64_t cap = kInf;
        for (int h = 0; h < H.n_types; ++h)
            if ((mask >> h) & 1) cap = H.mem_bytes[h] < cap ? H.mem_bytes[h] : cap;
        const int64_t ms = (int64_t)((PP - lane) < vg ? (PP - lane) : vg);   // 1F1B stored micro-batches
        const bool inner = lane < PP - 1;
        const int64_t p2p = inner ? pi->p2p[(bp >> 2) * kMaxTypes + (bp & 3)] : 0;
        const int bdiff = inner && ((bp >> 2) != (bp & 3));
        const int mixed = __popc(mask) > 1;
        const int64_t X = pi->x_bytes, eta_tbar = (int64_t)H.eta_prune * pi->tbar;
        // band of end layers reachable by stage s under the windows
        const int cumlo = wave_incl_scan(lane < PP ? lo : 0, lane);
        const int cumhi = wave_incl_scan(lane < PP ? hi : 0, lane);
        const int totlo = rl32(cumlo, 63), tothi = rl32(cumhi, 63);
        int blo = N - (tothi - cumhi), bhi = N - (totlo - cumlo);
        blo = blo > cumlo ? blo : cumlo;
        bhi = bhi < cumhi ? bhi : cumhi;
        const bool band_ok = !(lane < PP) || blo <= bhi;
        const bool feasible_shape = totlo <= N && tothi >= N && __all(band_ok);
        if (nslot > S.kmax || PP > S.ppmax || !feasible_shape) {
            if (member) {
                const int st = feasible_shape ? HAPMOE_STATUS_OVERFLOW : HAPMOE_STATUS_INFEASIBLE;
                write_result(out, st, kInf, kInf, kInf, 0, zero_words);
                if (STATS) stats[2 * (inst - first)] = stats[2 * (inst - first) + 1] = 0;
            }
            continue;
        }

        // ---- stage the prefix sums of this candidate in LDS ----
        const int64_t *time = reinterpret_cast<const int64_t *>(tab + L.off_time) + cfg * L.n_masks * 3 * np;
        const int64_t *mem = reinterpret_cast<const int64_t *>(tab + L.off_mem) + cfg * 4 * np;
        {
            uint64_t rs = used;
            int k = 0;
            while (rs) {
                const int m = __ffsll((unsigned long long)rs) - 1;
                rs &= rs - 1;
                const int64_t *src = time + (int64_t)(m - 1) * 3 * np;
#pragma unroll
                for (int q = 0; q < R; ++q) {
                    const int b = lane + 64 * q;
                    if (b <= N) TM[k * NP + b] = I64x2{src[b], src[np + b]};
                }
                ++k;
            }
#pragma unroll
            for (int q = 0; q < R; ++q) {
                const int b = lane + 64 * q;
                if (b <= N) {
                    MW[b] = mem[b];
                    MA0[b] = mem[np + b];
                    MA1[b] = mem[2 * np + b];
                    MOE[b] = (int32_t)mem[3 * np + b];
                }
            }
        }
        wave_sync();

        // ---- feasible split interval of every (stage, b in band) ----
        // a in [AMIN, A0B) fits only with recomputation (r = 1), a in [A0B, b - lo] without.
        for (int s = 0; s < PP; ++s) {
            const int lo_s = rl32(lo, s), hi_s = rl32(hi, s), mask_s = rl32(mask, s);
            const int blo_s = rl32(blo, s), bhi_s = rl32(bhi, s);
            const int plo = s ? rl32(blo, s - 1) : 0, phi = s ? rl32(bhi, s - 1) : 0;
            const int mixed_s = rl32(mixed, s), bdiff_s = rl32(bdiff, s);
            const int64_t cap_s = rl64(cap, s), ms_s = rl64(ms, s), p2p_s = rl64(p2p, s);
            const int64_t *CM = mixed_s ? time + ((int64_t)(mask_s - 1) * 3 + 2) * np : nullptr;
            const int64_t hc_b = bdiff_s ? p2p_s : 0;
            for (int q = 0; q * 64 <= bhi_s - blo_s; ++q) {
                const int k = lane + 64 * q;
                const int b = blo_s + k;
                if (b > bhi_s) continue;
                int amin = 255, a0 = 255;
                const int ahi = (b - lo_s) < phi ? (b - lo_s) : phi;
                const int alo = (b - hi_s) > plo ? (b - hi_s) : plo;
                if (ahi >= alo) {
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
                AMIN[s * NP + k] = (uint8_t)amin;
                A0B[s * NP + k] = (uint8_t)a0;
            }
        }
        wave_sync();   // the memory prefixes are dead from here on (their LDS holds ARG / FM)

        int passes = 0, relax = 0;

        // One DP pass at threshold t.  minimax: F = least possible largest stage;
        // otherwise F = least stage sum with all stages <= t and M = the largest
        // stage on the back-trace path (ties: smallest split point a).
        auto pass = [&](int64_t t, bool minimax, int64_t &F_out, int64_t &M_out) {
            ++passes;
            if (lane == 0) FM[0] = I64x2{0, 0};
            wave_sync();
            for (int s = 0; s < PP; ++s) {
                const int slot_s = rl32(slot, s), lo_s = rl32(lo, s);
                const int blo_s = rl32(blo, s), bhi_s = rl32(bhi, s);
                const int phi = s ? rl32(bhi, s - 1) : 0;
                const int64_t p2p_s = rl64(p2p, s);
                const I64x2 *T = TM + slot_s * NP;
                int64_t fbest[R], fm[R];
                int fa[R];
#pragma unroll
                for (int q = 0; q < R; ++q) {
                    const int k = lane + 64 * q;
                    const int b = blo_s + k;
                    int64_t best = kBig, bm = 0;
                    int ba = 255;
                    if (b <= bhi_s) {
                        const int amin = AMIN[s * NP + k], a0 = A0B[s * NP + k];
                        const int ahi = (b - lo_s) < phi ? (b - lo_s) : phi;
                        const I64x2 tb = T[b];
                        const int64_t k0 = tb.x + p2p_s, k1 = tb.y + p2p_s;
                        for (int a = amin; a <= ahi; ++a) {
                            const I64x2 ta = T[a];
                            const bool r1 = a < a0;
                            const int64_t cst = r1 ? k1 - ta.y : k0 - ta.x;
                            const I64x2 f = FM[a];
                            int64_t v = minimax ? (f.x > cst ? f.x : cst) : f.x + cst;
                            v = cst <= t ? v : kBig;
                            if (v < best) {
                                best = v;
                                ba = a;
                                bm = f.y > cst ? f.y : cst;
                            }
                        }
                        if (STATS) relax += ahi >= amin ? ahi - amin + 1 : 0;
                    }
                    fbest[q] = best;
                    fm[q] = bm;
                    fa[q] = ba;
                }
                wave_sync();
#pragma unroll
                for (int q = 0; q < R; ++q) {
                    const int k = lane + 64 * q;
                    const int b = blo_s + k;
                    if (b <= bhi_s) {
                        FM[b] = I64x2{fbest[q], fm[q]};
                        ARG[s * NP + k] = (uint8_t)fa[q];
                    }
                }
                wave_sync();
            }
            const I64x2 fin = FM[N];
            F_out = fin.x;
            M_out = fin.y;
        };

        // back-trace of the last pass into BT (lane 0), then shared by the writers
        auto backtrace = [&]() {
            if (lane == 0) {
                uint32_t words[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                uint32_t rmask = 0;
                int b = N;
                bool ok = true;
                for (int s = PP - 1; s >= 0; --s) {
                    const int k = b - rl32(blo, s);
                    const int a = ARG[s * NP + k];
                    if (a >= b) {
                        ok = false;
                        break;
                    }
                    words[s >> 2] |= (uint32_t)(b - a) << (8 * (s & 3));
                    if (a < A0B[s * NP + k]) rmask |= 1u << s;
                    b = a;
                }
                ok = ok && b == 0;
                for (int w = 0; w < 8; ++w) BT[w] = words[w];
                BT[8] = rmask;
                BT[9] = ok ? 1u : 0u;
            }
            wave_sync();
        };

        int64_t tbot, unused, F1, M1;
        pass(kInf, true, tbot, unused);
        if (tbot >= kBig) {
            if (member) {
                write_result(out, HAPMOE_STATUS_INFEASIBLE, kInf, kInf, kInf, 0, zero_words);
                if (STATS) {
                    stats[2 * (inst - first)] = passes;
                    stats[2 * (inst - first) + 1] = 0;
                }
            }
            if (STATS) {
                const int rs = wave_sum32(relax);
                const int leader = __ffsll((unsigned long long)__ballot(member)) - 1;
                if (lane == leader) stats[2 * (inst - first) + 1] = rs;
            }
            continue;
        }
        pass(kInf, false, F1, M1);
        int64_t last_t = kInf;
        const int64_t Bm = (int64_t)Bj - 1;
        int64_t bs = F1 + Bm * M1, bmx = M1, bt = kInf;   // this lane's incumbent
        if (tbot < M1) {
            int64_t Fb, Mb;
            pass(tbot, false, Fb, Mb);
            last_t = tbot;
            if (Fb + Bm * Mb <= bs) {
                bs = Fb + Bm * Mb;
                bmx = Mb;
                bt = tbot;
            }
            int64_t F = F1, t = M1 - 1;
            for (;;) {
                const bool done = bmx == tbot && bs == F1 + Bm * tbot;   // reached the lower bound
                const bool act = member && !done && F + Bm * tbot <= bs;
                const int64_t lim = act ? (Bm > 0 ? (bs - F) / Bm : kBig) : -1;
                const int64_t mx = wave_max64(lim);
                const int64_t tn = mx < t ? mx : t;
                if (tn <= tbot) break;
                int64_t Fc, Mc;
                pass(tn, false, Fc, Mc);
                last_t = tn;
                if (Fc + Bm * Mc <= bs) {
                    bs = Fc + Bm * Mc;
                    bmx = Mc;
                    bt = tn;
                }
                F = Fc;
                t = Mc - 1;
            }
        }

        // ---- results: one back-trace per distinct winning threshold ----
        bool pending = member;
        const int64_t dpc = ki->dp_const;
        while (__any(pending)) {
            const int64_t tr = wave_min64(pending ? bt : kInf);
            if (tr != last_t) {
                int64_t Fr, Mr;
                pass(tr, false, Fr, Mr);
                last_t = tr;
            }
            backtrace();
            if (pending && bt == tr) {
                uint32_t words[8];
                for (int w = 0; w < 8; ++w) words[w] = BT[w];
                if (BT[9])
                    write_result(out, HAPMOE_STATUS_OK, bs + dpc, bs - Bm * bmx, bmx, BT[8], words);
                else
                    write_result(out, HAPMOE_STATUS_OVERFLOW, kInf, kInf, kInf, 0, zero_words);
                pending = false;
            }
            wave_sync();
        }
        if (STATS) {
            const int rs = wave_sum32(relax);
            const int leader = __ffsll((unsigned long long)__ballot(member)) - 1;
            if (member) {
                stats[2 * (inst - first)] = passes;
                stats[2 * (inst - first) + 1] = lane == leader ? rs : 0;
            }
        }
    }
}

}  // namespace

int64_t stage_dp_ws_bytes() { return 256; }

hipError_t launch_stage_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_layers, int n_micro,
                           const std::vector<int32_t> &config_pp, int n_orders, const TablesLayout &L,
                           const void *d_tables, int64_t first, int64_t count, int kmax, int ppmax,
                           hapmoe_dp_result *d_res, int32_t *d_stats, void *d_ws, const int32_t *micro,
                           hipStream_t s)
{
    if (count == 0) return hipSuccess;
    // work items over the keys that hold candidates of [first, first + count)
    const int64_t key_lo = first / n_micro, key_hi = (first + count - 1) / n_micro;   // inclusive
    ItemMap M;
    M.n_runs = 0;
    M.pad = 0;
    M.total = 0;
    const int64_t ncfg = (int64_t)config_pp.size();
    for (int64_t c = 0; c < ncfg;) {
        int64_t e = c;
        while (e < ncfg && config_pp[e] == config_pp[c]) ++e;
        const int pp = config_pp[c];
        int64_t ks = c * n_orders, ke = e * n_orders - 1;
        ks = ks > key_lo ? ks : key_lo;
        ke = ke < key_hi ? ke : key_hi;
        if (ks <= ke) {
            uint64_t present = 0;
            for (int i = 0; i < n_micro; ++i) present |= uint64_t(1) << (micro[i] < pp ? micro[i] : pp);
            if (M.n_runs >= kMaxRuns) return hipErrorInvalidValue;
            ItemRun &r = M.run[M.n_runs++];
            r.item_start = M.total;
            r.key_start = (int32_t)ks;
            r.key_count = (int32_t)(ke - ks + 1);
            r.n_groups = __builtin_popcountll(present);
            r.pp = pp;
            M.total += (int64_t)r.key_count * r.n_groups;
        }
        c = e;
    }
    if (M.total == 0) return hipSuccess;
    const int R = (n_layers + 1 + 63) / 64;
    const DpLds S = dp_lds(n_layers, kmax, ppmax);
    const auto *img = static_cast<const unsigned char *>(d_image);
    const auto *tab = static_cast<const unsigned char *>(d_tables);
    uint32_t *queue = static_cast<uint32_t *>(d_ws);
    hipLaunchKernelGGL(k_reset_queue, dim3(1), dim3(1), 0, s, queue);
    int dev = 0, ncu = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return hipErrorUnknown;
    auto go = [&](auto kern) -> hipError_t {
        hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, 64, S.total);
        if (e != hipSuccess) return e;
        int64_t grid = (int64_t)ncu * (per_cu > 0 ? per_cu : 1);
        if (grid > M.total) grid = M.total;
        hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64), S.total, s, img, d_cand, L, tab, first, count, M,
                           S, d_res, d_stats, queue);
        return hipGetLastError();
    };
    if (R == 1)
        return d_stats ? go(k_stage_dp<1, true>) : go(k_stage_dp<1, false>);
    return d_stats ? go(k_stage_dp<2, true>) : go(k_stage_dp<2, false>);
}

}  // namespace hapmoe
