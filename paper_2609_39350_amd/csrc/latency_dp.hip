// Least 1F1B iteration latency over every partition (Appendix B, Eq. 5, with
// the steady-state term of Eq. 4): for each candidate the partition, with the
// Section 3.4 prunings and per-stage recomputation, that minimises
//     T = sum_i c_i + sum_{i <= s} ceil(c_i / 3) + max(0, B - s - 1) * t,
// t = max_i c_i and s the first (1-based) stage whose cost is t (a stage's
// forward part is ceil(c / 3), its backward part the rest).
//
// For a threshold t the least T among partitions whose largest stage is
// exactly t is a DP over (stage, end layer, z), z = 1 once the bottleneck
// stage is placed: before it a stage needs c < t and weighs c + ceil(c / 3);
// the bottleneck stage s has c = t and weighs t + ceil(t / 3) +
// max(0, B - s - 1) t; after it a stage needs c <= t and weighs c.  The
// thresholds are the distinct finite stage costs, taken in ascending order
// from t_bot, the least possible largest stage (one min-max pass: below it no
// partition exists, so those passes would change nothing); the sweep stops at the first t where F_inf + ceil(t / 3) +
// max(0, B - PP - 1) t (a lower bound of T for this and every larger t,
// F_inf the least stage sum) reaches the best T found.  Ties: the least T,
// then the lower largest stage (the first threshold reaching it), then the
// lexicographically smallest (b_{PP-1}, ..., b_1): the back-trace keeps the
// set of (end layer, z) states on optimal paths and at every stage takes the
// smallest split point through which one continues optimally.
//
// Thresholds are taken up to kLatSlots at a time and run side by side in one
// pass (a slot of DP states each), then examined in ascending order with the
// stop test; a pass past the stop is discarded.
//
// Mapping: one wave64 workgroup per (configuration, ordering) key, deepest first,
// lane j holding the key's j-th candidate and its incumbent; the candidates
// with B >= PP + 1 share one sweep, the others run one each.  A first launch
// with 24 KB of LDS a workgroup, then 40, 80 and 160 KB for the keys whose tables
// did not fit the previous one (more LDS also holds more threshold slots).  The candidate's
// stage costs -- every (stage, end layer b in the stage's band, split point a
// in the window) with the memory test of its stored micro-batch count,
// recomputation and prunings 1 and 3, exactly as the threshold DP prices them
// -- are evaluated once into LDS; a pass spreads the (end layer, z) states of
// a stage over the lanes, each lane taking the minimum over its window.  The
// next threshold is a wave-wide minimum over the cost table.  Integer min-plus
// work: no MFMA.
#include "internal.h"

namespace hapmoe {
namespace {

constexpr int64_t kLBig = int64_t(1) << 62;   // "no path" inside the DP, far from overflow
// Launches in tiers of LDS a workgroup: every key with 24 KB (six workgroups fit
// a CU), then the keys whose table did not fit with 40 KB (four), 80 KB (two)
// and 160 KB (one).
constexpr int kLatTiers = 4;
constexpr int kLatLdsTiers[kLatTiers] = {24 * 1024, 40 * 1024, 80 * 1024, 160 * 1024};
constexpr int64_t kLatMaxGrid = int64_t(1) << 30;   // workgroups a launch (keys beyond: grid-stride)
constexpr int kLatSlots = 8;                  // thresholds a latency pass may run side by side
constexpr int32_t kStatusRetry = 3;           // between the two launches only: table too big for the first

struct LatStage {
    int blo, wd;     // band of end layers [blo, blo + wd)
    int lo, win;     // window: n = b - a in [lo, lo + win)
    int plo, phi;    // band of the previous stage's end layers (split points)
    int coff, voff;  // offsets into the cost table and the DP states
};

struct LatHead {
    LatStage st[kMaxStages];
    int64_t red[64];         // wave reductions through LDS
    int32_t len[kMaxStages]; // best partition: layers per stage
    int32_t pad[kMaxStages];  // keeps the header at the documented 1,792 bytes
};

// the stage-cost table may use 160 KB less the header: 162,048 bytes (documented)
static_assert(sizeof(LatHead) == 1792, "LDS header size is part of the documented table limit");

__device__ inline int64_t ceil3(int64_t c) { return (c + 2) / 3; }

// The cost table holds each stage cost c as w = c + ceil(c / 3), the weight of a
// stage before the bottleneck (kLBig: no such stage).  w is strictly increasing
// in c, so comparisons with a threshold t can be made as w against t +
// ceil(t / 3), and c comes back without a division: c = 3m, 3m + 1, 3m + 2 give
// w = 4m, 4m + 2, 4m + 3, so c = 3 (w >> 2) + ((w & 3) + 1) / 2.  (Stage costs
// stay below 2^60, so w stays below kLBig.)
__device__ inline int64_t cost_weight(int64_t c) { return c >= kLBig ? kLBig : c + ceil3(c); }
__device__ inline int64_t weight_cost(int64_t w) { return 3 * (w >> 2) + (((w & 3) + 1) >> 1); }

__device__ inline int64_t shfl_xor64(int64_t v, int d)
{
    const int lo = __shfl_xor((int)(uint32_t)(uint64_t)v, d, 64);
    const int hi = __shfl_xor((int)(uint32_t)((uint64_t)v >> 32), d, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Wave-wide minimum and sum of an int64 (every lane gets the result; call with
// every lane of the wave active).
__device__ inline int64_t lat_min(int64_t v)
{
    // each 16-lane row by DPP row rotations (no LDS round trip), then the four
    // rows' results from lanes 0, 16, 32 and 48
#define LAT_ROT_MIN(CTRL)                                                                              \
    do {                                                                                               \
        const int lo_ = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(uint64_t)v, CTRL, 0xf, 0xf, false); \
        const int hi_ = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)((uint64_t)v >> 32), CTRL, 0xf, 0xf, false); \
        const int64_t o_ = (int64_t)(((uint64_t)(uint32_t)hi_ << 32) | (uint32_t)lo_);                \
        v = o_ < v ? o_ : v;                                                                           \
    } while (0)
    LAT_ROT_MIN(0x128);   // row_ror 8
    LAT_ROT_MIN(0x124);   // row_ror 4
    LAT_ROT_MIN(0x122);   // row_ror 2
    LAT_ROT_MIN(0x121);   // row_ror 1
#undef LAT_ROT_MIN
    int64_t m = kLBig + kLBig / 2;   // above every value
#pragma unroll
    for (int r = 0; r < 64; r += 16) {
        const int lo = __builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)v, r);
        const int hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), r);
        const int64_t o = (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
        m = o < m ? o : m;
    }
    return m;
}

__device__ inline int64_t lat_sum(int64_t v)
{
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += shfl_xor64(v, d);
    return v;
}

__device__ inline void lat_write(hapmoe_dp_result *out, int status, int64_t obj, int64_t sum, int64_t tmax,
                                 uint32_t rmask, const int32_t *len, int pp)
{
    out->objective = obj;
    out->stage_sum = sum;
    out->t_max = tmax;
    out->status = status;
    out->recompute_mask = rmask;
    for (int s = 0; s < kMaxStages; ++s) out->layers[s] = (uint8_t)(len && s < pp ? len[s] : 0);
}

// lds_bytes: the workgroup's LDS; retry: process only the keys whose candidates
// the first launch marked kStatusRetry (last: no larger launch follows, so a
// table that does not fit is HAPMOE_STATUS_OVERFLOW)
template <bool STATS>
__global__ __launch_bounds__(64) void k_latency_dp(const unsigned char *img, const hapmoe_candidate *cand,
                                                   const unsigned char *tab, TablesLayout L, int64_t first,
                                                   int64_t count, hapmoe_dp_result *res, int32_t *stats,
                                                   int lds_bytes, int retry, int last)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const ImageHeader &H = *reinterpret_cast<const ImageHeader *>(img);
    LatHead &D = *reinterpret_cast<LatHead *>(smem);
    unsigned char *dyn = smem + ((sizeof(LatHead) + 15) & ~size_t(15));
    const int dyn_bytes = lds_bytes - (int)((sizeof(LatHead) + 15) & ~size_t(15));
    const int lane = threadIdx.x;
    const int N = H.n_layers, nB = H.n_micro;
    const int64_t np = L.np;
    // the (configuration, ordering) keys holding candidates [first, first + count)
    const int64_t key_lo = first / nB, n_keys = (first + count - 1) / nB - key_lo + 1;

    for (int64_t kq = blockIdx.x; kq < n_keys; kq += gridDim.x) {
        // keys are PP-ascending: the deepest pipelines (the most work) go first
        const int64_t key = key_lo + n_keys - 1 - kq, cfg = key / H.n_orders;
        const int PP = cand[key * nB].pp;
        // lane j holds the key's j-th candidate (B = micro[j])
        const int64_t inst = key * nB + lane;
        const bool inr = lane < nB && inst >= first && inst < first + count;
        const int64_t Bj = lane < nB ? H.micro[lane] : 1;
        hapmoe_dp_result *out = res + (inst - first);   // dereferenced only where inr
        int32_t *st_out = STATS ? stats + 4 * (inst - first) : nullptr;
        if (retry && __ballot(inr && out->status == kStatusRetry) == 0) continue;   // wave-uniform
        const PiInfo *pi = reinterpret_cast<const PiInfo *>(tab + L.off_pi) + cfg;
        const KeyInfo *ki = reinterpret_cast<const KeyInfo *>(tab + L.off_key) + key;
        const int64_t *mem = reinterpret_cast<const int64_t *>(tab + L.off_mem) + cfg * 4 * np;
        const int64_t *time = reinterpret_cast<const int64_t *>(tab + L.off_time) + cfg * L.n_masks * 3 * np;
        auto finish_if = [&](bool mine, int status) {   // a result without a partition
            if (mine) {
                lat_write(out, status, kInf, kInf, kInf, 0, nullptr, PP);
                if (STATS) st_out[0] = st_out[1] = st_out[2] = st_out[3] = 0;
            }
        };
        if (pi->status != HAPMOE_STATUS_OK) {
            finish_if(inr, HAPMOE_STATUS_OVERFLOW);
            continue;
        }

        // ---- stage layout: bands of end layers under the pruning-1 windows ----
        int totlo = 0, tothi = 0, cumlo = 0, cumhi = 0;
        for (int s = 0; s < PP; ++s) {
            totlo += ki->lo[s];
            tothi += ki->hi[s];
            if (s <= lane) {
                cumlo += ki->lo[s];
                cumhi += ki->hi[s];
            }
        }
        int wd = 0;
        if (lane < PP) {
            int blo = N - (tothi - cumhi), bhi = N - (totlo - cumlo);
            blo = blo > cumlo ? blo : cumlo;
            bhi = bhi < cumhi ? bhi : cumhi;
            wd = bhi >= blo ? bhi - blo + 1 : 0;
            D.st[lane].blo = blo;
            D.st[lane].wd = wd;
            D.st[lane].lo = ki->lo[lane];
            D.st[lane].win = ki->hi[lane] - ki->lo[lane] + 1;
        }
        const bool shape = totlo <= N && tothi >= N && !__any(lane < PP && wd == 0);
        __syncthreads();
        if (!shape) {
            finish_if(inr, HAPMOE_STATUS_INFEASIBLE);
            __syncthreads();
            continue;
        }
        if (lane == 0) {
            int coff = 0, voff = 0;
            for (int s = 0; s < PP; ++s) {
                LatStage &S = D.st[s];
                S.plo = s ? D.st[s - 1].blo : 0;
                S.phi = s ? D.st[s - 1].blo + D.st[s - 1].wd - 1 : 0;
                S.coff = coff;
                S.voff = voff;
                coff += S.wd * S.win;
                voff += S.wd;
            }
            D.red[0] = coff;
            D.red[1] = voff;
        }
        __syncthreads();
        const int ncost = (int)D.red[0], nv = (int)D.red[1];
        __syncthreads();
        // LDS: cost table [ncost] int64 | recomputation flags [ncost] u8 | DP states
        // [nslot][nv][2] int64, one slot per threshold of a pass (at least one)
        const int fixed = ncost * 8 + ((ncost + 15) & ~15);
        const int need = fixed + nv * 16;
        if (need > dyn_bytes) {   // the table does not depend on B: the whole key
            finish_if(inr, last ? HAPMOE_STATUS_OVERFLOW : kStatusRetry);
            continue;
        }
        // thresholds a latency pass runs side by side, as many as the LDS allows (at
        // most kLatSlots): a stage's (slot, end layer) entries are spread over the
        // lanes together, so narrow bands fill the wave instead of a few lanes
        int nslot = (dyn_bytes - fixed) / (nv * 16);
        nslot = nslot < kLatSlots ? nslot : kLatSlots;
        nslot = nslot > 1 ? nslot : 1;
        int64_t *Cst = reinterpret_cast<int64_t *>(dyn);
        uint8_t *R = reinterpret_cast<uint8_t *>(Cst + ncost);
        int64_t *V = reinterpret_cast<int64_t *>(dyn + fixed);
        const int64_t X = pi->x_bytes, eta_tbar = (int64_t)H.eta_prune * pi->tbar;
        const bool prune_het = H.prune_hetero != 0, recomp = H.allow_recompute != 0;
        const LatStage SL = D.st[PP - 1];
        int64_t B = 1;   // the current group's reference B (see below)

        // One pass over the stages, every end layer of a stage (both its states z =
        // 0 / 1) on its own lane.  mode 0: the least stage sum (state z = 0 only); 1: the least
        // latency weight with the largest stage exactly t (states z = 0 / 1), for
        // nt thresholds D.red[8 + k] side by side, slot k's states at V + 2 nv k;
        // 2: the least possible largest stage (z = 0 only).  Returns the latency
        // relaxations this lane made.
        auto pass = [&](int mode, int nt) -> int64_t {
            const bool lat = mode == 1;
            int64_t nrel = 0;
            for (int s = 0; s < PP; ++s) {
                const LatStage S = D.st[s];
                const LatStage P = D.st[s ? s - 1 : 0];
                const int64_t steady = B - s - 2 > 0 ? B - s - 2 : 0;   // stage s + 1 (1-based) as bottleneck
                const int per = S.wd;
                for (int e = lane; e < nt * per; e += 64) {
                    // one lane an (end layer, threshold slot): both states z = 0 / 1 of
                    // the end layer from the same loads
                    const int ks = e / per, k = e - ks * per;
                    const int b = S.blo + k;
                    const int64_t t = lat ? D.red[8 + ks] : 0;
                    int64_t *Vk = V + 2 * (int64_t)nv * ks;
                    // a stage of cost t weighs wt before the bottleneck and wb as it
                    const int64_t wt = lat ? t + ceil3(t) : 0, wb = wt + steady * t;
                    const int64_t *Wp = Cst + S.coff + k * S.win;
                    int64_t best0 = kLBig, best1 = kLBig;
                    // the previous stage's states at split point a (stage 0: layer 0 at
                    // cost 0); a split point outside its band has no cost (w = kLBig),
                    // and the clamped index keeps the read inside the band
                    auto states = [&](int a, int64_t &v0, int64_t &v1) {
                        v0 = a == 0 ? 0 : kLBig;
                        v1 = kLBig;
                        if (s) {   // wave-uniform
                            int q = a - P.blo;
                            q = q < 0 ? 0 : (q >= P.wd ? P.wd - 1 : q);
                            const int64_t *vp = Vk + 2 * (P.voff + q);
                            v0 = vp[0];
                            v1 = vp[1];
                        }
                    };
                    auto relax = [&](int64_t w, int64_t v0, int64_t v1) {
                        const bool live = w < kLBig && v0 < kLBig;
                        if (mode == 0) {
                            const int64_t x = v0 + weight_cost(w);
                            best0 = live && x < best0 ? x : best0;
                        } else if (mode == 2) {
                            const int64_t c = weight_cost(w), m = v0 > c ? v0 : c;
                            best0 = live && m < best0 ? m : best0;
                        } else {
                            if (STATS) nrel += w < kLBig ? 2 : 0;   // both states
                            // (unsigned sums: a state or cost of kLBig gives a value that
                            // is not used, without a signed overflow)
                            const int64_t x0 = (int64_t)((uint64_t)v0 + (uint64_t)w);
                            const int64_t x1 = (int64_t)((uint64_t)v0 + (uint64_t)wb);
                            const int64_t y = (int64_t)((uint64_t)v1 + (uint64_t)weight_cost(w));
                            best0 = live && w < wt && x0 < best0 ? x0 : best0;
                            best1 = live && w == wt && x1 < best1 ? x1 : best1;
                            best1 = v1 < kLBig && w <= wt && y < best1 ? y : best1;
                        }
                    };
                    // two split points a trip, every load issued before either is used
                    const int a0 = b - S.lo;
                    int j = 0;
                    for (; j + 1 < S.win; j += 2) {
                        const int64_t w1 = Wp[j], w2 = Wp[j + 1];
                        int64_t p0, p1, q0, q1;
                        states(a0 - j, p0, p1);
                        states(a0 - j - 1, q0, q1);
                        relax(w1, p0, p1);
                        relax(w2, q0, q1);
                    }
                    if (j < S.win) {
                        int64_t v0, v1;
                        states(a0 - j, v0, v1);
                        relax(Wp[j], v0, v1);
                    }
                    Vk[2 * (S.voff + k)] = best0;
                    Vk[2 * (S.voff + k) + 1] = best1;
                }
                __syncthreads();
            }
            return nrel;
        };

        // Back-trace of the latency pass at threshold t with states Vt: the
        // smallest split point through which a live state continues optimally,
        // stage by stage from the last (lengths into D.len; sum and recomputation
        // mask returned).
        auto trace = [&](const int64_t *Vt, int64_t t, int64_t &sum, uint32_t &rmask) {
            int b = N;
            bool live0 = false, live1 = true;
            sum = 0;
            rmask = 0;
            for (int s = PP - 1; s >= 0; --s) {
                const LatStage S = D.st[s];
                const LatStage P = D.st[s ? s - 1 : 0];
                const int64_t steady = B - s - 2 > 0 ? B - s - 2 : 0;
                const int k = b - S.blo;
                const int64_t tg0 = Vt[2 * (S.voff + k)], tg1 = Vt[2 * (S.voff + k) + 1];
                int64_t amin = kLBig;
                bool m0 = false, m1 = false;
                int aj = -1;
                for (int j = lane; j < S.win; j += 64) {
                    const int64_t w = Cst[S.coff + k * S.win + j];
                    if (w >= kLBig) continue;
                    const int64_t c = weight_cost(w);
                    const int a = b - S.lo - j;
                    const int64_t v0 = s ? Vt[2 * (P.voff + a - P.blo)] : (a == 0 ? 0 : kLBig);
                    const int64_t v1 = s ? Vt[2 * (P.voff + a - P.blo) + 1] : kLBig;
                    const bool f0 = v0 < kLBig && ((live0 && c < t && v0 + c + ceil3(c) == tg0) ||
                                                   (live1 && c == t && v0 + c + ceil3(c) + steady * c == tg1));
                    const bool f1 = v1 < kLBig && live1 && c <= t && v1 + c == tg1;
                    if ((f0 || f1) && a < amin) {   // one lane may hold two split points (j, j + 64)
                        amin = a;
                        m0 = f0;
                        m1 = f1;
                        aj = j;
                    }
                }
                const int64_t na = lat_min(amin);
                const bool mine = amin == na && na < kLBig;
                const uint64_t b0 = __ballot(mine && m0), b1 = __ballot(mine && m1);
                const uint64_t who = __ballot(mine);
                const int src = who ? __ffsll((unsigned long long)who) - 1 : 0;
                const int jj = __shfl(aj, src, 64);
                if (na >= kLBig || jj < 0) break;   // cannot happen on an optimal path
                const int e = S.coff + k * S.win + jj;
                sum += weight_cost(Cst[e]);
                if (R[e]) rmask |= 1u << s;
                if (lane == 0) D.len[s] = b - (int)na;
                b = (int)na;
                live0 = b0 != 0;
                live1 = b1 != 0;
            }
        };

        // Groups of the key's candidates that share one sweep: all those with
        // B >= PP + 1, then each one with B <= PP alone.  With B >= PP + 1 no
        // stage's steady-state count max(0, B - s - 1) is clamped and every stage
        // stores PP - s + 1 micro-batches, so the DP at a threshold t differs
        // between two such B only by (B - B') t on the states past the bottleneck:
        // the same least-latency paths, latencies shifted by a constant.  One
        // sweep with the group's smallest B serves them all, each member keeping
        // its own incumbent and stopping bound; a member's bound says that no
        // larger threshold can beat its incumbent, so the extra thresholds the
        // others need change nothing for it.
        const uint64_t shared = __ballot(inr && Bj >= PP + 1);
        uint64_t pending = __ballot(inr);
        while (pending) {
            const uint64_t grp = (pending & shared) ? (pending & shared)
                                                    : (uint64_t(1) << (__ffsll((unsigned long long)pending) - 1));
            pending &= ~grp;
            const bool member = (grp >> lane) & 1;
            const int lead = __ffsll((unsigned long long)grp) - 1;
            B = lat_min(member ? Bj : kLBig);
            const int64_t dB = Bj - B;

            // ---- every stage cost of the group (stored micro-batches min(PP - s, B)) ----
            for (int e = lane; e < ncost; e += 64) {
                int s = 0;
                while (s + 1 < PP && D.st[s + 1].coff <= e) ++s;
                const LatStage S = D.st[s];
                const int k = (e - S.coff) / S.win, j = (e - S.coff) - k * S.win;
                const int b = S.blo + k, a = b - S.lo - j;
                int64_t c = kLBig;
                uint8_t r = 0;
                if (a >= S.plo && a <= S.phi && a >= 0) {
                    const int mask = ki->mask[s];
                    int64_t cap = kInf;
                    for (int h = 0; h < H.n_types; ++h)
                        if ((mask >> h) & 1) cap = H.mem_bytes[h] < cap ? H.mem_bytes[h] : cap;
                    const bool inner = s < PP - 1;
                    const int bp = ki->bpair[s];
                    const int64_t p2p = inner ? pi->p2p[(bp >> 2) * kMaxTypes + (bp & 3)] : 0;
                    const bool bdiff = inner && ((bp >> 2) != (bp & 3));
                    const bool mixed = __popc(mask) > 1;
                    const int64_t *tm = time + (int64_t)(mask - 1) * 3 * np;
                    const int64_t ms = (PP - s) < B ? (PP - s) : B;   // stored micro-batches
                    const int64_t base = mem[b] - mem[a] + ((mem[3 * np + b] - mem[3 * np + a]) > 0 ? X : 0);
                    const int64_t hc = (mixed ? tm[2 * np + b] - tm[2 * np + a] : 0) + (bdiff ? p2p : 0);
                    if (!prune_het || hc <= eta_tbar) {
                        if (base + ms * (mem[np + b] - mem[np + a]) <= cap) {
                            c = tm[b] - tm[a] + p2p;
                        } else if (recomp && base + ms * (mem[2 * np + b] - mem[2 * np + a]) <= cap) {
                            c = tm[np + b] - tm[np + a] + p2p;
                            r = 1;
                        }
                    }
                }
                Cst[e] = cost_weight(c);
                R[e] = r;
            }
            __syncthreads();

            pass(0, 1);
            const int64_t finf = V[2 * (SL.voff + (N - SL.blo))];
            __syncthreads();
            if (finf >= kLBig) {
                finish_if(member, HAPMOE_STATUS_INFEASIBLE);
                __syncthreads();
                continue;
            }
            // no partition has a largest stage below t_bot: the sweep starts there
            // (the passes below it find no path and change nothing)
            pass(2, 1);
            const int64_t tbot = V[2 * (SL.voff + (N - SL.blo))];
            __syncthreads();
            const int64_t steady_min = Bj - PP - 1 > 0 ? Bj - PP - 1 : 0;
            // this lane's incumbent (members only): latency, largest stage, sum,
            // recomputation mask and the stage lengths, four to a word
            int64_t best = kLBig, tbest = 0, bsum = 0;
            uint32_t brm = 0, lw[kMaxStages / 4] = {};
            int64_t tprev = tbot - 1, relax = 0;
            int swept = 0;
            for (bool more = true; more;) {
                // the next nslot distinct stage costs above tprev (stage costs are
                // positive), run side by side; then taken in ascending order, each
                // with the stop test against the incumbents as they stand there (a
                // pass past the stop is discarded)
                int nt = 0;
                for (int64_t lo_t = tprev; nt < nslot; ++nt) {
                    // in weights: the least w above lo_t's is the least cost above lo_t
                    const int64_t wlo = lo_t + ceil3(lo_t);
                    int64_t wn = kLBig;
                    for (int e = lane; e < ncost; e += 64) {
                        const int64_t w = Cst[e];
                        if (w > wlo && w < wn) wn = w;
                    }
                    const int64_t wmin = lat_min(wn);
                    if (wmin >= kLBig) break;
                    const int64_t t = weight_cost(wmin);
                    if (lane == 0) D.red[8 + nt] = t;
                    lo_t = t;
                }
                __syncthreads();
                if (nt == 0) break;
                if (__ballot(member && finf + ceil3(D.red[8]) + steady_min * D.red[8] < best) == 0) break;
                relax += pass(1, nt);
                for (int ks = 0; ks < nt; ++ks) {
                    const int64_t t = D.red[8 + ks];
                    if (ks > 0 && __ballot(member && finf + ceil3(t) + steady_min * t < best) == 0) {
                        more = false;
                        break;
                    }
                    ++swept;
                    tprev = t;
                    const int64_t *Vt = V + 2 * (int64_t)nv * ks;
                    const int64_t v = Vt[2 * (SL.voff + (N - SL.blo)) + 1];
                    const bool gain = member && v < kLBig && v + dB * t < best;
                    if (__ballot(gain) == 0) continue;
                    int64_t sum = 0;
                    uint32_t rmask = 0;
                    trace(Vt, t, sum, rmask);
                    __syncthreads();
                    if (gain) {
                        best = v + dB * t;
                        tbest = t;
                        bsum = sum;
                        brm = rmask;
#pragma unroll
                        for (int w = 0; w < kMaxStages / 4; ++w) {
                            uint32_t x = 0;
                            for (int q = 0; q < 4; ++q)
                                if (4 * w + q < PP) x |= (uint32_t)(uint8_t)D.len[4 * w + q] << (8 * q);
                            lw[w] = x;
                        }
                    }
                    __syncthreads();
                }
                __syncthreads();   // the thresholds of the next chunk overwrite D.red
            }
            const int64_t nrel = STATS ? lat_sum(relax) : 0;
            if (member) {
                if (best >= kLBig) {
                    lat_write(out, HAPMOE_STATUS_INFEASIBLE, kInf, kInf, kInf, 0, nullptr, PP);
                } else {
                    int32_t len[kMaxStages];
                    for (int q = 0; q < kMaxStages; ++q) len[q] = (lw[q / 4] >> (8 * (q % 4))) & 0xff;
                    lat_write(out, HAPMOE_STATUS_OK, best + ki->dp_const, bsum, tbest, brm, len, PP);
                }
                if (STATS) {   // the group's thresholds; its relaxations on its first candidate
                    st_out[0] = best >= kLBig ? 0 : swept;
                    st_out[1] = best >= kLBig || lane != lead ? 0 : (int32_t)(nrel < INT32_MAX ? nrel : INT32_MAX);
                    st_out[2] = st_out[3] = 0;
                }
            }
            __syncthreads();
        }
    }
}

}  // namespace

hipError_t launch_latency_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_micro,
                             const TablesLayout &L, const void *d_tables, int64_t first, int64_t count,
                             hapmoe_dp_result *d_res, int32_t *d_stats, hipStream_t stream)
{
    if (count == 0) return hipSuccess;
    const int64_t n_keys = (first + count - 1) / n_micro - first / n_micro + 1;
    const auto *img = static_cast<const unsigned char *>(d_image);
    const auto *tab = static_cast<const unsigned char *>(d_tables);
    auto go = [&](auto kern) -> hipError_t {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, kLatLdsTiers[kLatTiers - 1]);
        if (e != hipSuccess) return e;
        for (int tier = 0; tier < kLatTiers; ++tier) {
            // one workgroup a key: the dispatcher hands the next key to whichever
            // CU slot frees first, which balances keys of very different work
            const int64_t grid = n_keys < kLatMaxGrid ? n_keys : kLatMaxGrid;
            hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64), kLatLdsTiers[tier], stream, img, d_cand, tab, L,
                               first, count, d_res, d_stats, kLatLdsTiers[tier], tier > 0 ? 1 : 0,
                               tier == kLatTiers - 1 ? 1 : 0);
        }
        return hipGetLastError();
    };
    return d_stats ? go(k_latency_dp<true>) : go(k_latency_dp<false>);
}

}  // namespace hapmoe
