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
// over every distinct stage cost: the back-trace of the pass at the winning
// threshold is the lexicographically smallest sum-optimal partition there,
// which is also the smallest one at its own largest stage.
//
// Passes per sweep: one fused pass at t = inf that also carries the min-max
// row (t_bot = least possible largest stage), one pass at t_bot, then the
// descending sweep.  An incumbent is replaced by a lower objective, or by an
// equal one with a lower largest stage, so the result does not depend on the
// order of the passes.  A pass at any threshold t returns a genuine Pareto
// point (the one whose constant range holds t), so the descending sweep of a
// class can run as two chains side by side in two slots, each covering part of
// the threshold range: the upper chain starts at the top, the lower one at the
// middle of what remains, and an idle chain takes over the lower half of the
// other's range.  The passes of a sweep then run about a third fewer rounds.
//
// Work sharing across B: B enters a candidate only through the 1F1B count of
// stored micro-batches min(PP - i, B) (memory) and the (B-1) weight of the
// objective.  Candidates of one (pi, ordering) whose B values lead to identical
// feasible split intervals at every (stage, end layer) share every DP pass:
// one sweep serves them, one incumbent per B.  The groups of equal min(B, PP)
// are merged further into classes: the intervals of a (stage, end layer) change
// with the stored count m only at the m where some split point's memory stops
// fitting (m = floor(room / activation), computed exactly), so neighbouring
// group values fall into one class unless such a step lies between them.
//
// Mapping: persistent wave64 workgroups pull (pi, ordering) keys from an atomic
// queue, largest PP first.  The stage layout of a key is wave-uniform (one
// stage per lane, read with readlane).  Up to four classes of the key run at
// once as segments; the (segment, end layer b) entries of a stage -- b over the
// band a stage can reach under the pruning-1 windows -- are spread over the 64
// lanes in rounds, and each lane loops over the split points a of the previous
// stage's band (two per trip, wave-uniform trip count).  Layer prefix sums live
// in LDS once per key; feasible split intervals (memory with / without
// recomputation, prunings 1 and 3 -- all monotone in the segment length), DP
// rows (double-buffered) and back-trace pointers live in LDS per segment,
// packed by band.  Lane j also holds the incumbent of the key's j-th
// microbatch count.  Wave-wide reductions use DPP row rotations.  No MFMA:
// this is int64 min-plus scan work.
#include "internal.h"

namespace hapmoe {
namespace {

constexpr int64_t kBig = int64_t(1) << 62;   // "no partition" inside the DP (sums stay far from overflow)
constexpr int64_t kNegInf = INT64_MIN;        // a threshold no stage cost meets
constexpr int kRelaxUnroll = 2;   // split points per relaxation-loop trip
constexpr int kMaxSeg = 4;
constexpr int kParallelTrace = 4;    // pipelines at least this deep back-trace in two phases
constexpr int kEarlySlots = 4;       // slots whose time prefix sums are loaded ahead of the layout work
// Sweeps and 1F1B walks give every class up to kMaxChains slots (chains) while the
// batch has room for them and the slots' entries of the widest stage band take at
// most kChainEntries lanes.  A third chain saves passes but costs more per pass
// (a second round of entries and of back-trace work on deep pipelines).
constexpr int kMaxChains = 2;
constexpr int kChainEntries = 128;

// Optional section clocks (built with -DHAPMOE_SECTION_CLOCKS into a separate
// library): every wave accumulates the shader-clock cycles it spends in each
// part of the kernel and adds them to a device-wide table when it exits.
// Sections: key set-up and classification, feasibility scan, the relaxation
// rounds of the passes, the back-traces, and the sweep control in between.
#ifdef HAPMOE_SECTION_CLOCKS
__device__ unsigned long long g_section_clocks[kSectionClocks];
#define HAPMOE_CLOCK_VARS                                                           \
    unsigned long long clk_acc[kSectionClocks] = {};                                \
    const unsigned long long clk_start = clock64();                                 \
    unsigned long long clk_last = clk_start;                                        \
    const unsigned long long wall_start = wall_clock64();                           \
    unsigned long long key_start = 0;                                               \
    int key_pp = 0
#define HAPMOE_CLOCK(sec)                                                           \
    do {                                                                            \
        const unsigned long long clk_now = clock64();                               \
        clk_acc[sec] += clk_now - clk_last;                                         \
        clk_last = clk_now;                                                         \
    } while (0)
#define HAPMOE_CLOCK_RESTART() (clk_last = clock64())
// at the top of the key loop: the previous key of this wave has ended
#define HAPMOE_KEY_MARK(lane)                                                       \
    do {                                                                            \
        const unsigned long long now_ = wall_clock64();                             \
        if (key_start && (lane) == 0)                                               \
            atomicMax(&g_section_clocks[kKeyMax], ((now_ - key_start) << 6) | (unsigned long long)key_pp); \
        key_start = now_;                                                           \
    } while (0)
#define HAPMOE_KEY_PP(pp) (key_pp = (pp))
#define HAPMOE_COUNT(sec) (++clk_acc[sec])
#define HAPMOE_CLOCK_FLUSH(lane)                                                    \
    do {                                                                            \
        clk_acc[kClockTotal] = clock64() - clk_start;                               \
        if ((lane) == 0)                                                            \
            for (int i_ = 0; i_ < kCountPasses + 1; ++i_) atomicAdd(&g_section_clocks[i_], clk_acc[i_]); \
        const unsigned long long wend_ = wall_clock64();                            \
        if ((lane) == 0) {                                                          \
            atomicMax(&g_section_clocks[kWaveStartMinC], ~wall_start);              \
            atomicMax(&g_section_clocks[kWaveEndMinC], ~wend_);                     \
            atomicMax(&g_section_clocks[kWaveEndMax], wend_);                       \
        }                                                                           \
    } while (0)
#else
#define HAPMOE_CLOCK_VARS
#define HAPMOE_CLOCK(sec)
#define HAPMOE_CLOCK_RESTART()
#define HAPMOE_KEY_MARK(lane)
#define HAPMOE_KEY_PP(pp)
#define HAPMOE_COUNT(sec)
#define HAPMOE_CLOCK_FLUSH(lane)
#endif

// LDS of one wave: TM [kmax][np] {T0, T1} | memory prefixes | per-segment
// region | control.  The per-segment region holds, for each active segment:
// AMIN, A0B, ARG [sum of band widths] bytes and two DP rows [max band width].
struct DpLds {
    int np, kmax, ppmax, region;
    int off_region, off_ctl, total;
};

__host__ __device__ inline int align16(int x) { return (x + 15) & ~15; }

// Per-segment control block in LDS.
struct SegCtl {
    int64_t t;        // threshold of the next pass
    int64_t F, M;     // result of the last pass at b = N: stage sum, largest stage
    int64_t G;        // min-max value of the fused pass
    int32_t on;       // the segment takes part in the next pass
    int32_t pad;
    uint32_t bt[8];   // back-trace: n_i bytes
    uint32_t sb[8];   // back-trace of deep pipelines: first layer of each stage
    uint32_t rmask, ok;
    // 1F1B re-scoring: the traced partition's first largest stage s0 (0-based)
    // and the forward time sum_{i <= s0} ceil(c_i / 3); the pending frontier
    // candidate (the last point, confirmed once a lower threshold raises the sum)
    int64_t fwd;
    int32_t s0, pend;
    int64_t pF, pM, pfwd;
    int32_t ps0, prmask, pok, pad2;
    uint32_t pbt[8];
    // threshold sweep: the chain of passes this slot runs -- the sum of its last
    // pass (a lower bound for every lower threshold), the next threshold it
    // needs, and the threshold it stops above (the next chain covers the rest)
    int64_t cF, ct, cs;
};


// Bytes of the memory prefix sums (W, A0, A1 as int64, MoE count as int32).
__host__ __device__ inline int mem_bytes(int n_layers)
{
    const int w = n_layers + 1;
    return 3 * align16(w * 8) + align16(w * 4);
}

DpLds dp_lds(int n_layers, int kmax, int ppmax)
{
    DpLds S;
    S.np = n_layers + 1;
    S.kmax = kmax;
    S.ppmax = ppmax;
    S.off_region = kmax * S.np * 16;
    // one segment of any key always fits: every stage holds at least one
    // layer, so each of the PP stage bands of end layers is at most N - PP + 1
    // wide; the memory prefix sums share the space of the DP rows (they are
    // only read before the first DP pass of a batch)
    const int mb = mem_bytes(n_layers);
    int need = 0;
    for (int pp = 1; pp <= ppmax && pp <= n_layers; ++pp) {
        const int wmax = n_layers - pp + 1, rows = 2 * align16(wmax * 16);
        const int n = align16(3 * pp * wmax) + (rows > mb ? rows : mb);
        need = n > need ? n : need;
    }
    S.region = need + 64;
    S.off_ctl = S.off_region + S.region;
    S.total = S.off_ctl + kMaxSeg * (int)sizeof(SegCtl);
    return S;
}

__device__ inline int rl32(int v, int src) { return __builtin_amdgcn_readlane(v, src); }

__device__ inline int64_t rl64(int64_t v, int src)
{
    const int lo = __builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)v, src);
    const int hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), src);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Wave-wide reductions for a full wave (all 64 lanes active).  Each 16-lane
// row is all-reduced with DPP row rotations (register-to-register, no LDS round
// trip), then the four row results are combined from lanes 0/16/32/48 in scalar
// registers, so the result is wave-uniform.
template <int CTRL>
__device__ inline int dpp32(int x)
{
    return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xf, 0xf, false);
}

template <int CTRL>
__device__ inline int64_t dpp64(int64_t x)
{
    const int lo = dpp32<CTRL>((int)(uint32_t)(uint64_t)x);
    const int hi = dpp32<CTRL>((int)(uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

constexpr int kRowRor8 = 0x128, kRowRor4 = 0x124, kRowRor2 = 0x122, kRowRor1 = 0x121;

__device__ inline int64_t rows_max64(int64_t x)
{
    int64_t y = dpp64<kRowRor8>(x);
    x = y > x ? y : x;
    y = dpp64<kRowRor4>(x);
    x = y > x ? y : x;
    y = dpp64<kRowRor2>(x);
    x = y > x ? y : x;
    y = dpp64<kRowRor1>(x);
    return y > x ? y : x;
}

__device__ inline int64_t wave_max64(int64_t x)
{
    x = rows_max64(x);
    const int64_t r0 = rl64(x, 0), r1 = rl64(x, 16), r2 = rl64(x, 32), r3 = rl64(x, 48);
    const int64_t a = r0 > r1 ? r0 : r1, b = r2 > r3 ? r2 : r3;
    return a > b ? a : b;
}

__device__ inline int wave_max32(int x)
{
    int y = dpp32<kRowRor8>(x);
    x = y > x ? y : x;
    y = dpp32<kRowRor4>(x);
    x = y > x ? y : x;
    y = dpp32<kRowRor2>(x);
    x = y > x ? y : x;
    y = dpp32<kRowRor1>(x);
    x = y > x ? y : x;
    const int r0 = rl32(x, 0), r1 = rl32(x, 16), r2 = rl32(x, 32), r3 = rl32(x, 48);
    const int a = r0 > r1 ? r0 : r1, b = r2 > r3 ? r2 : r3;
    return a > b ? a : b;
}

__device__ inline int wave_sum32(int x)
{
    x += dpp32<kRowRor8>(x);
    x += dpp32<kRowRor4>(x);
    x += dpp32<kRowRor2>(x);
    x += dpp32<kRowRor1>(x);
    return rl32(x, 0) + rl32(x, 16) + rl32(x, 32) + rl32(x, 48);
}

__device__ inline uint64_t wave_or64(uint64_t x)
{
    int lo = (int)(uint32_t)x, hi = (int)(uint32_t)(x >> 32);
    lo |= dpp32<kRowRor8>(lo);
    hi |= dpp32<kRowRor8>(hi);
    lo |= dpp32<kRowRor4>(lo);
    hi |= dpp32<kRowRor4>(hi);
    lo |= dpp32<kRowRor2>(lo);
    hi |= dpp32<kRowRor2>(hi);
    lo |= dpp32<kRowRor1>(lo);
    hi |= dpp32<kRowRor1>(hi);
    const uint32_t l = (uint32_t)(rl32(lo, 0) | rl32(lo, 16) | rl32(lo, 32) | rl32(lo, 48));
    const uint32_t h = (uint32_t)(rl32(hi, 0) | rl32(hi, 16) | rl32(hi, 32) | rl32(hi, 48));
    return ((uint64_t)h << 32) | l;
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

// The largest count m of stored micro-batches whose activations (act each) still
// fit into room: floor(room / act), -1 if room < 0, 64 for "64 or more" (also
// act = 0).  Exact: an fp32 estimate is corrected by one integer step either way
// (its error is far below 1 for counts < 64).
__device__ inline int cap_count(int64_t room, int64_t act)
{
    if (room < 0) return -1;
    if (act <= 0 || room >= act * 64) return 64;
    if (room < act) return 0;
    // act <= room < 64 act, so the quotient lies in [1, 63].  Both are shifted
    // right until room fits 32 bits (act then keeps at least 25), and the fp32
    // product with act's approximate reciprocal is within one of the floor.
    const uint32_t rh = (uint32_t)((uint64_t)room >> 32);
    const int sh = rh ? 32 - __clz(rh) : 0;
    const float q = (float)(uint32_t)((uint64_t)room >> sh) *
                    __builtin_amdgcn_rcpf((float)(uint32_t)((uint64_t)act >> sh));
    int m = (int)q;
    m = m > 63 ? 63 : (m < 1 ? 1 : m);
    if ((int64_t)m * act > room)
        --m;
    else if ((int64_t)(m + 1) * act <= room)
        ++m;
    return m;
}

__device__ inline uint64_t step_bit(int m, int mtop)
{
    return (m >= 1 && m <= mtop) ? (uint64_t(1) << m) : 0;
}

// Entry e of a stage's (segment, end layer) list: segment q = e / wd and
// k = e % wd, as q = (e * ceil(2^16 / wd)) >> 16.  For 1 <= wd <= 128 this is
// the exact floor for every e < 4 wd + 64 (checked exhaustively), which covers
// the entries of up to four segments plus the lanes past the last one.  The
// multiplier of each stage is computed once a key, in the stage's lane.
__device__ inline uint32_t split_mul(int wd)
{
    return wd > 0 ? (65536u + (uint32_t)wd - 1u) / (uint32_t)wd : 0u;
}

__device__ inline void split_entry(int e, int wd, uint32_t mul, int &q, int &k)
{
    q = (int)(__umul24((uint32_t)e, mul) >> 16);
    k = e - q * wd;
}

// floor(x / d) for x >= 0 and d >= 1, with rd = 1 / d rounded to double: below
// 2^52 through the double product x * rd, whose truncation is within one of the
// floor (d = 1: exact; d >= 2: the two roundings leave an error below x / d *
// 2^-52 < 1/2), corrected by one integer step either way
__device__ inline int64_t div_recip(int64_t x, int64_t d, double rd)
{
    if (x < (int64_t(1) << 52)) {
        const int64_t q = (int64_t)((double)x * rd);
        const int64_t r = x - q * d;
        return r < 0 ? q - 1 : (r >= d ? q + 1 : q);
    }
    return x / d;
}

// Per-segment values held in registers, selected / updated without dynamic
// register indexing.
__device__ inline int sel4(const int (&v)[4], int q)
{
    return q == 0 ? v[0] : q == 1 ? v[1] : q == 2 ? v[2] : v[3];
}

__device__ inline void add4(int (&v)[4], int q, int x)
{
    v[0] += q == 0 ? x : 0;
    v[1] += q == 1 ? x : 0;
    v[2] += q == 2 ? x : 0;
    v[3] += q == 3 ? x : 0;
}

// The workgroup is a single wave whose LDS operations are processed in order;
// this fence keeps the compiler from moving LDS accesses across it and waits
// for the wave's outstanding LDS operations.
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

template <bool STATS, bool EXACT>
__global__ __launch_bounds__(64) void k_stage_dp(const unsigned char *__restrict__ img,
                                                 const hapmoe_candidate *__restrict__ cand, TablesLayout L,
                                                 const unsigned char *__restrict__ tab, int64_t first,
                                                 int64_t count, int64_t key_lo, int64_t n_keys, DpLds S,
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
    unsigned char *REG = smem + S.off_region;
    SegCtl *CTL = reinterpret_cast<SegCtl *>(smem + S.off_ctl);

    HAPMOE_CLOCK_VARS;
    // Keys come off the queue largest first, one at a time: fetching the next
    // key's index early (to hide the atomic's latency) binds a wave to it too
    // soon and costs more in balance than it saves, at every depth measured.
    for (;;) {
        HAPMOE_CLOCK_RESTART();
        HAPMOE_KEY_MARK(lane);
        uint32_t qi = 0;
        if (lane == 0) qi = atomicAdd(queue, 1u);
        // wave-uniform from here on: everything indexed by the key stays scalar
        qi = (uint32_t)__builtin_amdgcn_readlane((int)qi, 0);
        if ((int64_t)qi >= n_keys) break;   // every wave exits once the queue is drained
        const int64_t key = key_lo + n_keys - 1 - (int64_t)qi;   // keys are PP-ascending: biggest work first
        const int64_t cfg = key / H.n_orders;
        const int64_t idx0 = key * nB;
        const int PP = __builtin_amdgcn_readfirstlane(cand[idx0].pp);
        HAPMOE_KEY_PP(PP);
        const PiInfo *pi = reinterpret_cast<const PiInfo *>(tab + L.off_pi) + cfg;
        const KeyInfo *ki = reinterpret_cast<const KeyInfo *>(tab + L.off_key) + key;
        // stage s's layout fields in lane s, loaded with PP (the arrays hold
        // kMaxStages entries; lanes from PP on are cleared below)
        int mask = 0, lo = 0, hi = 0, bp = 0;
        if (lane < kMaxStages) {
            mask = ki->mask[lane];
            lo = ki->lo[lane];
            hi = ki->hi[lane];
            bp = ki->bpair[lane];
        }
        // The configuration's memory prefix sums (stored to LDS for the class
        // split) and, below, the slots' time prefix sums are loaded as soon as
        // their addresses are known, so that their latency overlaps the stage
        // layout work; lane l holds end layers l and l + 64 (N <= 127).
        const int64_t *time = reinterpret_cast<const int64_t *>(tab + L.off_time) + cfg * L.n_masks * 3 * np;
        const int64_t *mem = reinterpret_cast<const int64_t *>(tab + L.off_mem) + cfg * 4 * np;
        int64_t mv[2][3] = {{0, 0, 0}, {0, 0, 0}};
        int32_t mo[2] = {0, 0};
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int b = lane + 64 * c;
            if (b <= N) {
                mv[c][0] = mem[b];
                mv[c][1] = mem[np + b];
                mv[c][2] = mem[2 * np + b];
                mo[c] = (int32_t)mem[3 * np + b];
            }
        }

        // ---- lane j holds the key's j-th microbatch count ----
        const int64_t inst = idx0 + lane;
        const bool inr = lane < nB && inst >= first && inst < first + count;
        int Bj = 1, vj = 0;
        if (lane < nB) {
            Bj = H.micro[lane];
            vj = Bj < PP ? Bj : PP;
        }
        const uint64_t present = wave_or64(lane < nB ? (uint64_t(1) << vj) : 0);   // group values
        if (!__any(inr)) continue;
        hapmoe_dp_result *out = res + (inst - first);
        int32_t *st_out = STATS ? stats + 4 * (inst - first) : nullptr;
        if (pi->status != HAPMOE_STATUS_OK) {
            if (inr) {
                write_result(out, HAPMOE_STATUS_OVERFLOW, kInf, kInf, kInf, 0, zero_words);
                if (STATS) st_out[0] = st_out[1] = st_out[2] = st_out[3] = 0;
            }
            continue;
        }

        // ---- stage s lives in lane s ----
        if (lane >= PP) mask = lo = hi = bp = 0;
        const uint64_t used = wave_or64(lane < PP ? (uint64_t(1) << mask) : 0);
        const int nslot = __popcll(used);
        const int slot = __popcll(used & ((uint64_t(1) << mask) - 1));
        // time prefix sums (r = 0, 1) of the first kEarlySlots slots, in flight
        // during the layout work below
        int64_t tv[kEarlySlots][2][2];
        {
            uint64_t rs = used;
#pragma unroll
            for (int k = 0; k < kEarlySlots; ++k) {
                const int m = rs ? __ffsll((unsigned long long)rs) - 1 : 0;   // bit m: set m (>= 1)
                rs = rs ? rs & (rs - 1) : 0;
                const int64_t *src = time + (int64_t)(m > 0 ? m - 1 : 0) * 3 * np;
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    const int b = lane + 64 * c;
                    tv[k][c][0] = tv[k][c][1] = 0;
                    if (m > 0 && b <= N) {
                        tv[k][c][0] = src[b];
                        tv[k][c][1] = src[np + b];
                    }
                }
            }
        }
        int64_t cap = kInf;
        for (int h = 0; h < H.n_types; ++h)
            if ((mask >> h) & 1) cap = H.mem_bytes[h] < cap ? H.mem_bytes[h] : cap;
        const bool inner = lane < PP - 1;
        const int64_t p2p = inner ? pi->p2p[(bp >> 2) * kMaxTypes + (bp & 3)] : 0;
        const int bdiff = inner && ((bp >> 2) != (bp & 3));
        const int mixed = __popc(mask) > 1;
        const int64_t X = pi->x_bytes, eta_tbar = (int64_t)H.eta_prune * pi->tbar;
        const bool prune_het = H.prune_hetero != 0, recomp = H.allow_recompute != 0;
        // band [blo, bhi] of end layers stage s can reach under the windows
        const int cumlo = wave_incl_scan(lane < PP ? lo : 0, lane);
        const int cumhi = wave_incl_scan(lane < PP ? hi : 0, lane);
        const int totlo = rl32(cumlo, 63), tothi = rl32(cumhi, 63);
        int blo = N - (tothi - cumhi), bhi = N - (totlo - cumlo);
        blo = blo > cumlo ? blo : cumlo;
        bhi = bhi < cumhi ? bhi : cumhi;
        const int wd = lane < PP ? (bhi >= blo ? bhi - blo + 1 : 0) : 0;
        const int woff = wave_incl_scan(wd, lane) - wd;   // packed offset of stage s
        // stage s's band fields packed in lane s (one readlane each in the hot
        // loops): blo | bhi << 8 | lo << 16 | slot << 24 (all < 256), and
        // woff | wd << 16 (woff <= 32 * 128, wd <= 128)
        const int pk1 = (blo & 0xff) | ((bhi & 0xff) << 8) | ((lo & 0xff) << 16) | (slot << 24);
        const int pk2 = woff | (wd << 16);
        const int pkm = (int)split_mul(wd);   // the entry split's multiplier
        // and hi | mask << 8 | mixed << 16 | bdiff << 17, for the stage-flattened scans
        const int pk3 = (hi & 0xff) | (mask << 8) | (mixed << 16) | (bdiff << 17);
        // The classification and feasibility scans spread the (stage, end layer)
        // entries of all stages over the lanes at once (the stages are independent
        // there); each lane finds its stage by a binary search over the packed
        // offsets and reads the stage's fields from that lane.
        // (both read other lanes: call them with every lane of the wave active)
        auto stage_of = [&](int e) {   // the stage whose packed band holds entry e
            int st = 0;
#pragma unroll
            for (int step = 16; step >= 1; step >>= 1) {
                const int c = st + step;
                const int wc = __shfl(woff, c < 64 ? c : 63, 64);
                if (c < PP && wc <= e) st = c;
            }
            return st;
        };
        struct StageP {
            int lo, hi, blo, off, wd, mask, mixed, bdiff, plo, phi;
            int64_t cap, p2p;
        };
        auto stage_p = [&](int st) {   // stage st's fields (st may differ across lanes)
            StageP P;
            const int q1 = __shfl(pk1, st, 64), q2 = __shfl(pk2, st, 64), q3 = __shfl(pk3, st, 64);
            const int r1 = __shfl(pk1, st > 0 ? st - 1 : 0, 64);
            P.blo = q1 & 0xff;
            P.lo = (q1 >> 16) & 0xff;
            P.off = q2 & 0xffff;
            P.wd = q2 >> 16;
            P.hi = q3 & 0xff;
            P.mask = (q3 >> 8) & 0xff;
            P.mixed = (q3 >> 16) & 1;
            P.bdiff = (q3 >> 17) & 1;
            P.plo = st ? (r1 & 0xff) : 0;
            P.phi = st ? ((r1 >> 8) & 0xff) : 0;
            const int c0 = __shfl((int)(uint32_t)(uint64_t)cap, st, 64);
            const int c1 = __shfl((int)(uint32_t)((uint64_t)cap >> 32), st, 64);
            const int p0 = __shfl((int)(uint32_t)(uint64_t)p2p, st, 64);
            const int p1 = __shfl((int)(uint32_t)((uint64_t)p2p >> 32), st, 64);
            P.cap = (int64_t)(((uint64_t)(uint32_t)c1 << 32) | (uint32_t)c0);
            P.p2p = (int64_t)(((uint64_t)(uint32_t)p1 << 32) | (uint32_t)p0);
            return P;
        };
        const int sumwd = rl32(woff, 63) + rl32(wd, 63);
        const int maxw = wave_max32(wd);

        const bool feasible_shape = totlo <= N && tothi >= N && !__any(lane < PP && wd == 0);
        // region: [per-segment AMIN | A0B | ARG] [per-segment DP rows  or  memory prefixes]
        const int arr_bytes = align16(3 * sumwd), row_bytes = 2 * align16(maxw * 16);
        const int mbytes = mem_bytes(N);
        int smax = 0;
        for (int q = 1; q <= kMaxSeg; ++q) {
            const int need = q * arr_bytes + (q * row_bytes > mbytes ? q * row_bytes : mbytes);
            if (need <= S.region) smax = q;
        }
        if (nslot > S.kmax || PP > S.ppmax || !feasible_shape || smax == 0) {
            if (inr) {
                const int st = feasible_shape ? HAPMOE_STATUS_OVERFLOW : HAPMOE_STATUS_INFEASIBLE;
                write_result(out, st, kInf, kInf, kInf, 0, zero_words);
                if (STATS) st_out[0] = st_out[1] = st_out[2] = st_out[3] = 0;
            }
            continue;
        }

        // ---- the key's prefix sums in LDS ----
        {
            // negated, so that a stage cost T[b] - T[a] is one 64-bit add
#pragma unroll
            for (int k = 0; k < kEarlySlots; ++k) {
                if (k >= nslot) continue;
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    const int b = lane + 64 * c;
                    if (b <= N) TM[k * NP + b] = I64x2{-tv[k][c][0], -tv[k][c][1]};
                }
            }
            // further slots (device-type sets across the boundaries of an ordering)
            uint64_t rs = used;
            for (int k = 0; k < kEarlySlots && rs; ++k) rs &= rs - 1;
            int k = kEarlySlots;
            while (rs) {
                const int m = __ffsll((unsigned long long)rs) - 1;
                rs &= rs - 1;
                const int64_t *src = time + (int64_t)(m - 1) * 3 * np;
                // negated, so that a stage cost T[b] - T[a] is one 64-bit add
                for (int b = lane; b <= N; b += 64) TM[k * NP + b] = I64x2{-src[b], -src[np + b]};
                ++k;
            }
        }
        wave_sync();

        const int off_rows = smax * arr_bytes;   // start of the DP rows / memory prefixes
        int64_t *MW = reinterpret_cast<int64_t *>(REG + off_rows);
        int64_t *MA0 = MW + align16((N + 1) * 8) / 8;
        int64_t *MA1 = MA0 + align16((N + 1) * 8) / 8;
        int32_t *MOE = reinterpret_cast<int32_t *>(MA1 + align16((N + 1) * 8) / 8);

        // ---- classes of groups with identical feasible windows ----
        // Stage s of group v stores ms = min(PP - s, v) micro-batches.  For a fixed
        // (s, b) and split point a, the largest ms that still fits is cap(a) =
        // floor(room / activation), with and without recomputation, and it does
        // not fall as a grows; so the window bounds of (s, b), as functions of ms,
        // step exactly at the cap values of the window's split points.  Groups v <
        // v' see identical windows everywhere -- hence identical DP results at any
        // threshold -- unless some stage steps at an m in [v, min(PP - s, v') - 1]:
        // collect every step m <= PP - s - 1 into brk, then a present group value
        // opens a new class iff brk has a bit between the previous value and it.
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int b = lane + 64 * c;
            if (b <= N) {
                MW[b] = mv[c][0];
                MA0[b] = mv[c][1];
                MA1[b] = mv[c][2];
                MOE[b] = mo[c];
            }
        }
        wave_sync();
        uint64_t brk = 0;
        int cls_evals = 0;
        // one (stage, b) entry's window: every step m <= mtop of its fitting counts
        auto classify = [&](int b, int lo_s, int hi_s, int plo, int phi, int mtop, int64_t cap_s,
                            const int64_t *CM, int64_t hc_b) {
            const int ahi = (b - lo_s) < phi ? (b - lo_s) : phi;
            const int alo = (b - hi_s) > plo ? (b - hi_s) : plo;
            const int64_t wb = MW[b], a0b = MA0[b], a1b = MA1[b];
            const int mb = MOE[b];
            const int64_t cmb = CM ? CM[b] : 0;
            // the counts do not fall as a grows: once both exceed mtop, so do
            // all the later ones
            for (int a = alo; a <= ahi; ++a) {
                if (STATS) ++cls_evals;
                const int64_t xb = (mb - MOE[a]) > 0 ? X : 0;
                const int64_t room = cap_s - (wb - MW[a] + xb);
                const bool ok3 = !prune_het || (CM ? cmb - CM[a] : 0) + hc_b <= eta_tbar;
                if (!ok3) continue;
                const int m0 = cap_count(room, a0b - MA0[a]);
                const int m1 = recomp ? cap_count(room, a1b - MA1[a]) : 64;
                brk |= step_bit(m0, mtop) | (recomp ? step_bit(m1, mtop) : 0);
                if (m0 > mtop && m1 > mtop) break;
            }
        };
        const int nent = rl32(woff, PP - 1);   // the entries of stages 0 .. PP - 2
        for (int e0 = 0; e0 < nent; e0 += 64) {   // wave-uniform
            // every lane takes part in the cross-lane reads of stage_of and
            // stage_p (a read from an inactive lane is undefined); only the
            // lanes holding an entry classify it
            const int e = e0 + lane;
            const bool act = e < nent;
            const int st = stage_of(act ? e : 0);
            const StageP P = stage_p(st);
            const int64_t *CM = P.mixed ? time + ((int64_t)(P.mask - 1) * 3 + 2) * np : nullptr;
            if (act)
                classify(P.blo + (e - P.off), P.lo, P.hi, P.plo, P.phi, PP - st - 1, P.cap, CM,
                         P.bdiff ? P.p2p : 0);
        }
        brk = wave_or64(brk);
        const int cls_sum = STATS ? wave_sum32(cls_evals) : 0;
        uint64_t bnd;   // first group value of every class
        {
            const uint64_t below = present & ((uint64_t(1) << lane) - 1);
            bool first = true;
            if (below) {
                const int vprev = 63 - __clzll((long long)below);
                const uint64_t range = ((uint64_t(1) << lane) - 1) & ~((uint64_t(1) << vprev) - 1);
                first = (brk & range) != 0;
            }
            bnd = __builtin_amdgcn_ballot_w64(((present >> lane) & 1) && first);
        }
        const int ng = __popcll(bnd);   // classes
        const int gj = __popcll(bnd & ((uint64_t(2) << vj) - 1)) - 1;   // this lane's class

        HAPMOE_CLOCK(kClockSetup);
        HAPMOE_COUNT(kCountKeys);
        for (int g0 = 0; g0 < ng; g0 += smax) {
            HAPMOE_COUNT(kCountBatches);
            const int nact = (ng - g0) < smax ? (ng - g0) : smax;
            // with room for it, class q also runs in the slots q + nact, ..., each
            // covering a part of the class's threshold range (the chains of the
            // descending sweep and of the 1F1B frontier walk, below)
            int nchain = 1;
            while (nchain < kMaxChains && (nchain + 1) * nact <= smax && (nchain + 1) * nact <= kMaxSeg &&
                   (nchain + 1) * nact * maxw <= kChainEntries)
                ++nchain;
            const int nslot = nchain * nact;
            // class of every slot, 2 bits a slot
            int cmap = 0;
#pragma unroll
            for (int q = 0; q < kMaxSeg; ++q) cmap |= (q % (nact > 0 ? nact : 1)) << (2 * q);
            const int nseg = nslot <= 1 ? 1 : (nslot <= 2 ? 2 : 4);
            const int W = 64 / nseg;
            const int sg = lane / W, ll = lane % W;   // DP view: segment and lane in segment
            // class value (its smallest group value) of every segment of the batch
            int vq[kMaxSeg] = {1, 1, 1, 1};
            {
                uint64_t rest = bnd;
                for (int k = 0; k < g0 && rest; ++k) rest &= rest - 1;
#pragma unroll
                for (int q = 0; q < kMaxSeg; ++q) {
                    if (q < nact && rest) {
                        vq[q] = __ffsll((unsigned long long)rest) - 1;
                        rest &= rest - 1;
                    }
                }
            }
            const bool seg_live = sg < nslot;
            const int segi = seg_live ? sg : 0;
            // a slot reads the feasible intervals of its class and keeps its own
            // back-trace pointers and DP rows
            uint8_t *AMIN = REG + ((cmap >> (2 * segi)) & 3) * arr_bytes;
            uint8_t *A0B = AMIN + sumwd;
            uint8_t *ARG = REG + segi * arr_bytes + 2 * sumwd;
            unsigned char *RW = REG + off_rows + segi * row_bytes;
            int64_t *const FM0 = reinterpret_cast<int64_t *>(RW);
            int64_t *const FM1 = reinterpret_cast<int64_t *>(RW + row_bytes / 2);
            I64x2 *const FG0 = reinterpret_cast<I64x2 *>(RW);   // fused pass: {sum, min-max}
            I64x2 *const FG1 = reinterpret_cast<I64x2 *>(RW + row_bytes / 2);
            // memory prefix sums for the feasibility scan (they share the DP-row space;
            // the first batch finds them there from the class split)
            if (g0 > 0) {
                for (int b = lane; b <= N; b += 64) {
                    MW[b] = mem[b];
                    MA0[b] = mem[np + b];
                    MA1[b] = mem[2 * np + b];
                    MOE[b] = (int32_t)mem[3 * np + b];
                }
                wave_sync();
            }
            // candidate view: lane j's segment in this batch (-1: not in this batch)
            const int sj = (gj >= g0 && gj < g0 + nact) ? gj - g0 : -1;
            bool member = inr && sj >= 0;
            // groups whose candidates are all outside [first, first + count) still run;
            // their results are simply not written.

            // split-point evaluations per segment (stats); the classification counts once
            int evq[kMaxSeg] = {(STATS && g0 == 0 && lane == 0) ? cls_sum : 0, 0, 0, 0};
            // ---- feasible split interval of every (stage, b in band), per segment ----
            // a in [AMIN, A0B) fits only with recomputation (r = 1), a in [A0B, b - lo] without.
            // One (segment, stage, b) entry a lane, the entries of all segments and stages
            // spread over the lanes at once.
            auto scan_entry = [&](bool act, int q, int s, int k, int lo_s, int hi_s, int blo_s, int off_s, int plo,
                                  int phi, int64_t cap_s, const int64_t *CM, int64_t hc_b) {
                const int vs = sel4(vq, q);
                const int64_t ms = (int64_t)((PP - s) < vs ? (PP - s) : vs);   // 1F1B stored micro-batches
                uint8_t *const AMq = REG + q * arr_bytes;
                const int b = blo_s + k;
                const int ahi = (b - lo_s) < phi ? (b - lo_s) : phi;
                const int alo = (b - hi_s) > plo ? (b - hi_s) : plo;
                const bool has = act && ahi >= alo;
                // the feasible split points form a suffix [amin, ahi] of the window
                // (memory and pruning 3 only grow with the segment), and so do those
                // feasible without recomputation, [a0, ahi]: scanning a upwards, the
                // first hit of each is its bound, and a lane is done at its first
                // split point that fits without recomputation
                int amin = has ? ahi + 1 : 255, a0 = amin;
                const int64_t wb = MW[b], a0b = MA0[b], a1b = MA1[b];
                const int mb = MOE[b];
                const int64_t cmb = CM ? CM[b] : 0;
                const int aend = has ? ahi : plo;
                bool open = has;
                // one split point's test, gated by the lane still being open
                auto test = [&](int a, int64_t mwa, int64_t ma0, int64_t ma1, int moea, int64_t cma) {
                    const int64_t xb = (mb - moea) > 0 ? X : 0;
                    const int64_t base = wb - mwa + xb;
                    const bool ok3 = !prune_het | (cmb - cma + hc_b <= eta_tbar);
                    const bool f0 = open & ok3 & (base + ms * (a0b - ma0) <= cap_s);
                    const bool f1 = open & ok3 & recomp & (base + ms * (a1b - ma1) <= cap_s);
                    if (STATS) add4(evq, q, open ? 1 : 0);
                    amin = ((f0 | f1) & (a < amin)) ? a : amin;
                    a0 = f0 ? a : a0;
                    open = open & !f0 & (a < aend);
                };
                // two split points per trip, all loads issued before either test
                int a = has ? alo : plo;
                for (;;) {   // a lane closes at aend at the latest
                    const int a2 = a < aend ? a + 1 : a;
                    const int64_t w1 = MW[a], w2 = MW[a2], p1 = MA0[a], p2 = MA0[a2];
                    const int64_t q1 = MA1[a], q2 = MA1[a2];
                    const int m1 = MOE[a], m2 = MOE[a2];
                    const int64_t c1 = CM ? CM[a] : 0, c2 = CM ? CM[a2] : 0;
                    test(a, w1, p1, q1, m1, c1);
                    test(a2, w2, p2, q2, m2, c2);
                    if (__builtin_amdgcn_ballot_w64(open) == 0) break;
                    a = a2 < aend ? a2 + 1 : a2;   // stays inside the window
                }
                if (act) {
                    AMq[off_s + k] = (uint8_t)amin;
                    AMq[sumwd + off_s + k] = (uint8_t)a0;
                }
            };
            const int total = nact * sumwd;
            for (int e0 = 0; e0 < total; e0 += 64) {   // wave-uniform
                const int e = e0 + lane;
                const bool act = e < total;
                const int ee = act ? e : 0;
                const int q = ee / sumwd, ke = ee - q * sumwd;
                const int st = stage_of(ke);
                const StageP P = stage_p(st);
                const int64_t *CM = P.mixed ? time + ((int64_t)(P.mask - 1) * 3 + 2) * np : nullptr;
                scan_entry(act, q, st, ke - P.off, P.lo, P.hi, P.blo, P.off, P.plo, P.phi, P.cap, CM,
                           P.bdiff ? P.p2p : 0);
            }
            wave_sync();

            HAPMOE_CLOCK(kClockScan);
            int passes = 0;
            int relq[kMaxSeg] = {0, 0, 0, 0}, slq[kMaxSeg] = {0, 0, 0, 0};   // per segment (stats)

            // One DP pass of every segment with CTL.on set, at its CTL.t: F = least
            // stage sum with all stages <= t (ties: smallest split point a); lane
            // 0 of the segment then back-traces the partition and its largest
            // stage M into the segment's control block.  The fused pass (t = inf)
            // also carries the min-max row: G = least possible largest stage.
            auto pass = [&](bool fused) {
                HAPMOE_CLOCK(kClockControl);
                HAPMOE_COUNT(kCountPasses);
                const bool on = seg_live && CTL[sg].on != 0;
                if (STATS && sj >= 0) {
                    bool ran = false;
                    for (int k = 0; k < nchain; ++k) ran |= CTL[sj + k * nact].on != 0;
                    if (ran) ++passes;
                }
                if (on && ll == 0) {   // stage -1: layer 0 reached at cost 0
                    if (fused)
                        FG1[0] = I64x2{0, 0};
                    else
                        FM1[0] = 0;
                }
                // the running segments, in order (wave-uniform)
                // (all four flags are read at once -- one LDS round trip -- and masked)
                int nq = 0, qmap = 0, onq[kMaxSeg];
#pragma unroll
                for (int q = 0; q < kMaxSeg; ++q) onq[q] = CTL[q].on;
#pragma unroll
                for (int q = 0; q < kMaxSeg; ++q) {
                    const int o = __builtin_amdgcn_readfirstlane(onq[q]) & -(int)(q < nseg);
                    if (o) {
                        qmap |= q << (2 * nq);
                        ++nq;
                    }
                }
                wave_sync();
                for (int s = 0; s < PP; ++s) {
                    const int p1 = rl32(pk1, s), p2 = rl32(pk2, s), q1 = s ? rl32(pk1, s - 1) : 0;
                    const int blo_s = p1 & 0xff, lo_s = (p1 >> 16) & 0xff, slot_s = (p1 >> 24) & 0xff;
                    const int off_s = p2 & 0xffff, wd_s = p2 >> 16;
                    const int plo = q1 & 0xff, phi = (q1 >> 8) & 0xff;
                    const int64_t p2p_s = rl64(p2p, s);
                    const I64x2 *T = TM + slot_s * NP;
                    const int poff = (s & 1) ? 0 : row_bytes / 2, coff = row_bytes / 2 - poff;
                    // wave-uniform rounds over the (running segment, b) entries of the
                    // stage, and a wave-uniform split-point loop: a lane with less to
                    // do runs masked (clamped, in-range loads; predicated stores only)
                    const int total = nq * wd_s;
                    const uint32_t mul_wd = (uint32_t)rl32(pkm, s);
                    for (int e0 = 0; e0 < total; e0 += 64) {
                        const int e = e0 + lane;
                        const bool act = e < total;
                        int qi = 0, k = act ? e : 0;
                        if (nq > 1) split_entry(k, wd_s, mul_wd, qi, k);   // wave-uniform branch
                        const int q = (qmap >> (2 * qi)) & 3;
                        const int64_t t = CTL[q].t;
                        // (24-bit products: full-rate multiplies; every region offset is far below 2^24)
                        const uint8_t *const AMq = REG + __umul24((cmap >> (2 * q)) & 3, arr_bytes);   // class
                        uint8_t *const ARq = REG + __umul24(q, arr_bytes) + 2 * sumwd;                   // slot
                        unsigned char *const RWq = REG + off_rows + __umul24(q, row_bytes);
                        const int64_t *Fp = reinterpret_cast<const int64_t *>(RWq + poff);
                        int64_t *Fc = reinterpret_cast<int64_t *>(RWq + coff);
                        const I64x2 *Gp = reinterpret_cast<const I64x2 *>(RWq + poff);
                        I64x2 *Gc = reinterpret_cast<I64x2 *>(RWq + coff);
                        const int b = blo_s + k;
                        const int amin0 = AMq[off_s + k], a0 = AMq[sumwd + off_s + k];
                        const int ahi0 = (b - lo_s) < phi ? (b - lo_s) : phi;
                        const bool has = act && amin0 <= ahi0;
                        int left = has ? ahi0 - amin0 + 1 : 0;   // split points not yet relaxed
                        // a lane without a window reads split point plo under a
                        // threshold no stage cost meets
                        const int amin = has ? amin0 : plo;
                        const int64_t tl = has ? t : kNegInf;
                        const I64x2 tb = T[b];   // negated prefix sums
                        const int64_t k0 = p2p_s - tb.x, k1 = p2p_s - tb.y;
                        int64_t best = kBig, gbest = kBig;
                        int ba = 255;
                        // a runs downwards from b - lo and then stays at amin: repeating
                        // the last split point changes nothing ("<=" keeps the smallest
                        // split point among equal values, which is the current one)
                        // kRelaxUnroll split points per trip (more only add work: the
                        // threshold leaves most windows one or two points long): every
                        // load is issued before the first use, one exit test per trip;
                        // the trip count is bounded by the longest window, as a lane only
                        // goes on while a > amin
                        int a = has ? ahi0 : plo;
                        for (;;) {
                            int au[kRelaxUnroll];
                            I64x2 tu[kRelaxUnroll], fu[kRelaxUnroll];
#pragma unroll
                            for (int u = 0; u < kRelaxUnroll; ++u) {
                                au[u] = u == 0 ? a : (au[u - 1] > amin ? au[u - 1] - 1 : au[u - 1]);
                                tu[u] = T[au[u]];
                                fu[u] = fused ? Gp[au[u] - plo] : I64x2{Fp[au[u] - plo], 0};
                            }
                            bool ok = false;
                            int al = a;
#pragma unroll
                            for (int u = 0; u < kRelaxUnroll; ++u) {
                                al = au[u];
                                const int64_t cst = au[u] < a0 ? k1 + tu[u].y : k0 + tu[u].x;
                                ok = cst <= tl;
                                const int64_t v = fu[u].x + cst;
                                const bool le = ok && v <= best;
                                best = le ? v : best;
                                ba = le ? au[u] : ba;
                                if (fused) {
                                    const int64_t g = fu[u].y > cst ? fu[u].y : cst;
                                    gbest = ok && g < gbest ? g : gbest;
                                }
                                if (STATS) {
                                    add4(relq, q, ok && left > 0 ? 1 : 0);
                                    add4(slq, q, 1);
                                    --left;
                                }
                            }
                            // the stage cost only grows as a falls: the wave is done once
                            // no lane is both under its threshold and short of amin
                            if (__builtin_amdgcn_ballot_w64(ok && al > amin) == 0) break;
                            a = al > amin ? al - 1 : al;
                        }
                        if (act) {
                            if (fused)
                                Gc[k] = I64x2{best, gbest};
                            else
                                Fc[k] = best;
                            ARq[off_s + k] = (uint8_t)ba;
                        }
                    }
                    wave_sync();
                }
                HAPMOE_CLOCK(kClockRelax);
                const bool odd = ((PP - 1) & 1) != 0;
                const int64_t fin = fused ? (odd ? FG1[0].x : FG0[0].x) : (odd ? FM1[0] : FM0[0]);
                const bool tracer = on && ll == 0;
                if (tracer) {
                    CTL[sg].F = fin;
                    if (fused) CTL[sg].G = odd ? FG1[0].y : FG0[0].y;
#pragma unroll
                    for (int w = 0; w < 8; ++w) CTL[sg].bt[w] = 0;
                }
                if (PP >= kParallelTrace) {
                    // Deep pipelines: the lanes of each segment only follow the chain of
                    // split points (one byte load a stage) into CTL.sb; then every
                    // (segment, stage) entry recomputes its stage cost on its own lane
                    // and the segment's largest stage, recomputation mask and layer
                    // counts are combined with LDS atomics.  Same results as the
                    // stage-by-stage trace below.
                    {
                        // Every lane of a segment follows the segment's chain (with the
                        // same values), so the loop holds no branch and no store: lane ll
                        // keeps stage ll's split point and stage ll + W's (PP <= 2 W),
                        // stored once the chain is done -- one LDS round trip a stage.
                        uint8_t *const sbb = reinterpret_cast<uint8_t *>(CTL[segi].sb);
                        bool ok = on && fin < kBig;
                        int b = N, sv0 = 0, sv1 = 0;
                        for (int s = PP - 1; s >= 0; --s) {   // wave-uniform; clamped, in-range indices
                            const int q1 = rl32(pk1, s), q2 = rl32(pk2, s);
                            const int wdn = q2 >> 16;
                            int k = b - (q1 & 0xff);
                            k = k < 0 ? 0 : (k >= wdn ? wdn - 1 : k);
                            const int a = ARG[(q2 & 0xffff) + k];
                            ok = ok && a < b;
                            sv0 = s == ll ? a : sv0;
                            sv1 = s == ll + W ? a : sv1;
                            b = ok ? a : b;
                        }
                        ok = ok && b == 0;
                        if (on) {
                            if (ll < PP) sbb[ll] = (uint8_t)sv0;
                            if (ll + W < PP) sbb[ll + W] = (uint8_t)sv1;
                        }
                        if (tracer) {
                            CTL[sg].ok = ok ? 1u : 0u;
                            CTL[sg].M = 0;
                            CTL[sg].rmask = 0;
                            if (EXACT) {
                                CTL[sg].s0 = ok ? PP : 0;
                                CTL[sg].fwd = 0;
                            }
                        }
                    }
                    wave_sync();
                    const int nent = nslot * PP;   // <= 4 * 32: two rounds at most
                    int64_t ce[2] = {0, 0};
                    int qe[2] = {0, 0}, se[2] = {0, 0};
                    bool ve[2] = {false, false};
#pragma unroll
                    for (int r = 0; r < 2; ++r) {
                        if (r * 64 >= nent) break;   // wave-uniform
                        const int e = r * 64 + lane;
                        const bool act = e < nent;
                        const int q = act ? e / PP : 0, s = act ? e % PP : 0;
                        // only segments that ran this pass (the others keep their last trace)
                        const bool valid = act && q < nslot && CTL[q].on != 0 && CTL[q].ok != 0;
                        const int p1 = __shfl(pk1, s, 64), p2 = __shfl(pk2, s, 64);
                        const int plo = __shfl((int)(uint32_t)(uint64_t)p2p, s, 64);
                        const int phi = __shfl((int)(uint32_t)((uint64_t)p2p >> 32), s, 64);
                        const int64_t pc = (int64_t)(((uint64_t)(uint32_t)phi << 32) | (uint32_t)plo);
                        const uint8_t *sbq = reinterpret_cast<const uint8_t *>(CTL[q].sb);
                        const int a = valid ? sbq[s] : 0;
                        const int b = valid ? (s + 1 < PP ? sbq[s + 1] : N) : 0;
                        const int wdn = p2 >> 16;
                        int k = b - (p1 & 0xff);
                        k = k < 0 ? 0 : (k >= wdn ? wdn - 1 : k);
                        const int a0 = (REG + ((cmap >> (2 * q)) & 3) * arr_bytes + sumwd)[(p2 & 0xffff) + k];
                        const I64x2 *T = TM + ((p1 >> 24) & 0xff) * NP;
                        const I64x2 ta = T[a], tb = T[b];   // negated prefix sums
                        const bool r1 = a < a0;
                        const int64_t c = (r1 ? ta.y - tb.y : ta.x - tb.x) + pc;
                        if (valid) {
                            atomicMax(reinterpret_cast<unsigned long long *>(&CTL[q].M), (unsigned long long)c);
                            if (r1) atomicOr(&CTL[q].rmask, 1u << s);
                            reinterpret_cast<uint8_t *>(CTL[q].bt)[s] = (uint8_t)(b - a);
                        }
                        ce[r] = c;
                        qe[r] = q;
                        se[r] = s;
                        ve[r] = valid;
                    }
                    if (EXACT) {   // the first stage of largest cost, then the forward time up to it
                        wave_sync();
#pragma unroll
                        for (int r = 0; r < 2; ++r)
                            if (ve[r] && ce[r] == CTL[qe[r]].M) atomicMin(&CTL[qe[r]].s0, se[r]);
                        wave_sync();
#pragma unroll
                        for (int r = 0; r < 2; ++r)
                            if (ve[r] && se[r] <= CTL[qe[r]].s0)
                                atomicAdd(reinterpret_cast<unsigned long long *>(&CTL[qe[r]].fwd),
                                          (unsigned long long)((ce[r] + 2) / 3));
                    }
                } else {
                    // Back-trace of every running segment by its lane 0.  The loop over
                    // the stages is wave-uniform; the other lanes follow on clamped,
                    // in-range indices and drop what they compute.  The next stage's
                    // pointer and recomputation bound go out with this stage's prefix
                    // sums: one LDS round trip a stage.
                    {
                        uint8_t *const btb = reinterpret_cast<uint8_t *>(CTL[segi].bt);
                        uint32_t rmask = 0;
                        int64_t m = 0, tf = 0, tf_after = 0;   // forward times (1F1B re-scoring)
                        int s0 = 0;
                        int b = N;
                        bool ok = tracer && fin < kBig;
                        const int pl = rl32(pk2, PP - 1) & 0xffff, kl = N - (rl32(pk1, PP - 1) & 0xff);
                        int a = ARG[pl + kl], a0 = A0B[pl + kl];
                        for (int s = PP - 1; s >= 0; --s) {
                            ok = ok && a < b;
                            int an = 0, a0n = 0;
                            if (s > 0) {   // wave-uniform
                                const int q1 = rl32(pk1, s - 1), q2 = rl32(pk2, s - 1);
                                const int wdn = q2 >> 16;
                                int kn = (ok ? a : 0) - (q1 & 0xff);
                                kn = kn < 0 ? 0 : (kn >= wdn ? wdn - 1 : kn);
                                an = ARG[(q2 & 0xffff) + kn];
                                a0n = A0B[(q2 & 0xffff) + kn];
                            }
                            const int ai = ok ? a : 0;
                            const I64x2 *T = TM + ((rl32(pk1, s) >> 24) & 0xff) * NP;
                            const I64x2 ta = T[ai], tb = T[b];   // negated prefix sums
                            const bool r1 = ai < a0;
                            const int64_t c = (r1 ? ta.y - tb.y : ta.x - tb.x) + rl64(p2p, s);
                            if (ok) {
                                if (EXACT) {   // walking down, ">=" keeps the first stage of largest cost
                                    if (c >= m) {
                                        s0 = s;
                                        tf_after = tf;
                                    }
                                    tf += (c + 2) / 3;
                                }
                                m = c > m ? c : m;
                                btb[s] = (uint8_t)(b - a);
                                if (r1) rmask |= 1u << s;
                                b = a;
                            }
                            a = an;
                            a0 = a0n;
                        }
                        if (tracer) {
                            ok = ok && b == 0;
                            CTL[sg].M = m;
                            if (EXACT) {
                                CTL[sg].s0 = s0;
                                CTL[sg].fwd = tf - tf_after;
                            }
                            CTL[sg].rmask = rmask;
                            CTL[sg].ok = ok ? 1u : 0u;
                        }
                    }
                }
                wave_sync();
                HAPMOE_CLOCK(kClockTrace);
            };

            // per-segment control, written by lane 0 from wave-uniform values
            auto set_ctl = [&](int seg, bool on, int64_t t) {
                if (lane == 0) {
                    CTL[seg].on = on ? 1 : 0;
                    CTL[seg].t = t;
                }
            };

            // this lane's incumbent and its partition
            int64_t bs = 0, bmx = 0, bsum = 0;
            uint32_t pw[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            uint32_t prm = 0, pok = 0;
            const int64_t Bm = (int64_t)Bj - 1;
            const double rBm = Bm > 0 ? 1.0 / (double)Bm : 0.0;   // for the sweep bound below
            // offer the segment's last pass: a lower objective wins, and on equal
            // objectives the lower largest stage (the least threshold reaching the
            // optimum), whatever order the passes ran in; equal (objective, M)
            // points share the partition of threshold M
            auto take = [&](int slot) {
                const int64_t Fx = CTL[slot].F, Mx = CTL[slot].M;
                const int64_t sc = Fx + Bm * Mx;
                if (sc < bs || (sc == bs && Mx < bmx)) {
                    bs = sc;
                    bmx = Mx;
                    for (int w = 0; w < 8; ++w) pw[w] = CTL[slot].bt[w];
                    prm = CTL[slot].rmask;
                    pok = CTL[slot].ok;
                }
            };

            // ---- 1) least sum without a threshold, fused with the min-max pass ----
#pragma unroll
            for (int q = 0; q < kMaxSeg; ++q)
                if (q < nseg) set_ctl(q, q < nact, kInf);
            wave_sync();
            pass(true);
            const int64_t tbot = member ? CTL[sj].G : kBig;
            if (member && tbot >= kBig) {
                write_result(out, HAPMOE_STATUS_INFEASIBLE, kInf, kInf, kInf, 0, zero_words);
                member = false;
            }
            int64_t segF[kMaxSeg] = {kBig, kBig, kBig, kBig};   // t_bot of each segment
            bool segok[kMaxSeg] = {false, false, false, false};
#pragma unroll
            for (int q = 0; q < kMaxSeg; ++q) {
                if (q >= nact) continue;
                segF[q] = CTL[q].G;
                segok[q] = segF[q] < kBig;
            }
            const int sjc = sj >= 0 ? sj : 0;   // a candidate's segment, clamped for lanes outside the batch
            if (EXACT) {
                // ---- 1F1B re-scoring: walk the whole (max, sum) frontier ----
                // The last point of a segment is pending until a pass at its max - 1
                // shows a higher sum (then it is a frontier point and is scored) or
                // the same sum (then a lower max reaches it and it is dropped); a
                // point at t_bot is the segment's last frontier point.
                // With a second slot per class the walk runs as two chains: the upper
                // one (slot q) walks down to a middle threshold mid, where its last
                // pass only confirms its pending point; the lower one (slot q + nact)
                // starts with a pass at mid (pend = 2: nothing to confirm yet) and
                // walks on down.  A point both find is scored twice, which changes
                // nothing.  (Splitting again whenever one chain falls idle, as the
                // descending sweep does, measured slower here: every split adds a
                // confirming pass.)
                auto keep_pending = [&]() {   // lane 0 of a segment: the last pass's point
                    CTL[sg].pend = CTL[sg].F < kBig ? 1 : 0;
                    CTL[sg].pF = CTL[sg].F;
                    CTL[sg].pM = CTL[sg].M;
                    CTL[sg].pfwd = CTL[sg].fwd;
                    CTL[sg].ps0 = CTL[sg].s0;
                    CTL[sg].prmask = (int32_t)CTL[sg].rmask;
                    CTL[sg].pok = (int32_t)CTL[sg].ok;
                    for (int w = 0; w < 8; ++w) CTL[sg].pbt[w] = CTL[sg].bt[w];
                };
                auto latency = [&](const SegCtl &P) {
                    int64_t steady = (int64_t)Bj - P.ps0 - 2;   // B - s - 1 with s = s0 + 1
                    steady = steady > 0 ? steady : 0;
                    return P.pF + P.pfwd + steady * P.pM;
                };
                auto score = [&](int slot) {   // a candidate lane offers a slot's pending point
                    const SegCtl &P = CTL[slot];
                    const int64_t lat = latency(P);
                    if (lat < bs || (lat == bs && P.pM < bmx)) {
                        bs = lat;
                        bmx = P.pM;
                        bsum = P.pF;
                        for (int w = 0; w < 8; ++w) pw[w] = P.pbt[w];
                        prm = (uint32_t)P.prmask;
                        pok = (uint32_t)P.pok;
                    }
                };
                // A candidate needs no more of a chain once its incumbent is strictly
                // below the pending point's latency and below a bound for every point
                // further down: sum >= the pending sum, forward part >= ceil(t_bot/3)
                // (the largest stage's own), steady part >= max(0, B - PP - 1) t_bot.
                // Strict, so that a tie, which the lower max would win, still runs.
                auto needs_more = [&](int slot) {
                    const SegCtl &P = CTL[slot];
                    if (!member || P.pend != 1) return false;
                    const int64_t lat = latency(P);
                    int64_t slb = (int64_t)Bj - PP - 1;
                    slb = slb > 0 ? slb : 0;
                    const int64_t lb = P.pF + (P.G + 2) / 3 + slb * P.G;
                    return !(bs < lat && bs < lb);
                };
                if (seg_live && ll == 0) {
                    if (CTL[sg].on)
                        keep_pending();
                    else
                        CTL[sg].pend = 0;
                }
                if (member) bs = kInf;
                wave_sync();
                // the upper chains' stops and the lower chains' starts
                if (lane == 0) {
                    for (int q = 0; q < nact; ++q) {
                        CTL[q].cs = -1;   // no stop: walks to t_bot
                        if (nchain < 2) continue;
                        const int y = q + nact;
                        CTL[y].cs = -1;
                        CTL[y].G = CTL[q].G;
                        CTL[y].pend = 0;
                        const int64_t top = CTL[q].M - 1, g = CTL[q].G;
                        if (CTL[q].pend == 1 && top - g >= 2) {
                            const int64_t mid = g + (top - g) / 2;
                            CTL[q].cs = mid;
                            CTL[y].pend = 2;
                            CTL[y].pM = mid + 1;   // its first pass runs at mid
                        }
                    }
                }
                wave_sync();
                for (;;) {
                    bool any = false;
                    const uint64_t need0 = __builtin_amdgcn_ballot_w64(sj >= 0 && needs_more(sjc));
                    const uint64_t need1 =
                        nchain > 1 ? __builtin_amdgcn_ballot_w64(sj >= 0 && needs_more(sjc + nact)) : 0;
#pragma unroll
                    for (int q = 0; q < kMaxSeg; ++q) {
                        if (q >= nseg) continue;
                        const int c = q < nact ? q : q - nact;
                        const int pend = q < nslot ? CTL[q].pend : 0;
                        // a lower chain starts where its class still needs the upper one
                        const uint64_t need = (q < nact || pend == 2) ? need0 : need1;
                        const bool run = pend != 0 && CTL[q].pM > CTL[q].G &&
                                         (need & __builtin_amdgcn_ballot_w64(sj == c)) != 0;
                        set_ctl(q, run, pend ? CTL[q].pM - 1 : 0);
                        any |= run;
                    }
                    // a pending point at t_bot is the last frontier point
                    if (member)
                        for (int k = 0; k < nchain; ++k) {
                            const int slot = sjc + k * nact;
                            if (CTL[slot].pend == 1 && CTL[slot].pM <= CTL[slot].G) score(slot);
                        }
                    wave_sync();
                    if (seg_live && ll == 0 && CTL[sg].pend == 1 && CTL[sg].pM <= CTL[sg].G) CTL[sg].pend = 0;
                    wave_sync();
                    if (!any) break;
                    pass(false);
                    if (member)
                        for (int k = 0; k < nchain; ++k) {
                            const int slot = sjc + k * nact;
                            if (CTL[slot].on && CTL[slot].pend == 1 && CTL[slot].F > CTL[slot].pF) score(slot);   // confirmed
                        }
                    wave_sync();
                    if (seg_live && ll == 0 && CTL[sg].on) {
                        if (CTL[sg].t <= CTL[sg].cs)
                            CTL[sg].pend = 0;   // an upper chain's last pass only confirmed its point
                        else
                            keep_pending();
                    }
                    wave_sync();
                }
            }
            int64_t F1 = 0, M1 = 0;
            if (!EXACT && member) {
                F1 = CTL[sj].F;
                M1 = CTL[sj].M;
                bs = kInf;
                take(sj);
            }
            // lanes of segments where t_bot >= M1 are already final
            const bool sweeping = !EXACT && member && tbot < M1;
            // Chains of the descending sweep.  A chain runs passes at the largest
            // threshold some candidate of its class still needs, min(lim, ct): below
            // ct = (last largest stage) - 1 the sum is at least cF, so thresholds above
            // lim = (incumbent - cF) / (B - 1) cannot win.  It covers the thresholds
            // above its stop cs; together the chains of a class cover (t_bot, M1 - 1].
            // Chain k of class q runs in slot q + k nact.  The last chain starts at
            // the top (alongside the pass at t_bot, in slot q); whenever a chain is
            // idle and another one runs, the idle one takes the lower half of the
            // widest running range.  Each chain visits every Pareto point of its range
            // that can still win, and the incumbent rule does not depend on the order,
            // so the result is that of a single chain.
            if (!EXACT) {
                if (lane == 0) {
                    for (int q = 0; q < nslot; ++q) {
                        const int c = (cmap >> (2 * q)) & 3;
                        CTL[q].cF = CTL[c].F;
                        CTL[q].ct = q >= nslot - nact ? CTL[c].M - 1 : -1;   // -1: idle
                        CTL[q].cs = CTL[c].G;
                    }
                }
            }
            wave_sync();
            // this lane's threshold for the chain in a slot of its class (-1: none)
            auto need = [&](int slot) -> int64_t {
                const bool done = bmx == tbot && bs == F1 + Bm * tbot;   // reached the lower bound
                const int64_t cF = CTL[slot].cF, ct = CTL[slot].ct;
                if (!sweeping || done || cF + Bm * tbot > bs) return -1;
                if (Bm == 0 || cF + Bm * ct <= bs) return ct;   // ct binds: no division
                const int64_t lim = div_recip(bs - cF, Bm, rBm);
                return lim < ct ? lim : ct;
            };
            // the chains' passes: offer them, and move the chains on
            auto advance = [&](int from) {
                if (sweeping)
                    for (int k = from; k < nchain; ++k)
                        if (CTL[sj + k * nact].on) take(sj + k * nact);
                wave_sync();
                if (lane == 0) {
                    for (int q = from * nact; q < nslot; ++q) {
                        if (!CTL[q].on) continue;
                        CTL[q].cF = CTL[q].F;
                        CTL[q].ct = CTL[q].M - 1;
                    }
                }
                wave_sync();
            };

            // ---- 3) the bottleneck threshold itself (and the top chain's first pass) ----
            if (!EXACT) {
                bool any = false;
#pragma unroll
                for (int q = 0; q < kMaxSeg; ++q) {
                    if (q >= nact) continue;
                    const bool run = segok[q] && segF[q] < CTL[q].M;   // t_bot < M1
                    set_ctl(q, run, segF[q]);
                    any |= run;
                    if (nchain > 1) {
                        const int top = q + (nchain - 1) * nact;
                        const int64_t t1 = wave_max64(sj == q ? need(top) : -1);
                        const int64_t tb = wave_max64(sj == q && sweeping ? tbot : -1);
                        const bool run1 = t1 > tb;
                        set_ctl(top, run1, t1);
                        any |= run1;
                    }
                }
                wave_sync();
                if (any) {
                    pass(false);
                    if (member && CTL[sj].on) take(sj);   // the t_bot pass is no chain's
                    if (nchain > 1) advance(1);
                }
                wave_sync();
            }

            // ---- 4) descending Pareto sweep ----
            // each class's t_bot as seen by its sweeping candidates (-1: none), fixed
            // for the whole sweep
            int64_t tbq[kMaxSeg] = {-1, -1, -1, -1};
#pragma unroll
            for (int q = 0; q < kMaxSeg; ++q)
                if (!EXACT && q < nact) tbq[q] = wave_max64(sj == q && sweeping ? tbot : -1);
            while (!EXACT) {
                bool any = false;
                // this lane's thresholds for the chains of its class
                int64_t nk[kMaxChains];
#pragma unroll
                for (int k = 0; k < kMaxChains; ++k) nk[k] = (sweeping && k < nchain) ? need(sj + k * nact) : -1;
#pragma unroll
                for (int q = 0; q < kMaxSeg; ++q) {
                    if (q >= nact) continue;
                    const int64_t tb = tbq[q];
                    // every chain's threshold and the bound it runs above (wave-uniform)
                    int64_t tk[kMaxSeg], lk[kMaxSeg];
#pragma unroll
                    for (int k = 0; k < kMaxSeg; ++k) {
                        tk[k] = -1;
                        lk[k] = 0;
                        if (k >= nchain || k >= kMaxChains) continue;
                        const int slot = q + k * nact;
                        tk[k] = wave_max64(sj == q ? nk[k] : -1);
                        lk[k] = CTL[slot].cs > tb ? CTL[slot].cs : tb;
                    }
                    // idle chains take the lower half of the widest running range
                    for (int it = 1; it < nchain; ++it) {
                        int x = -1, y = -1;
                        int64_t wx = 1;
#pragma unroll
                        for (int k = 0; k < kMaxSeg; ++k) {
                            if (k >= nchain) continue;
                            if (tk[k] > lk[k]) {
                                if (tk[k] - lk[k] > wx) {
                                    wx = tk[k] - lk[k];
                                    x = k;
                                }
                            } else if (y < 0) {
                                y = k;
                            }
                        }
                        if (x < 0 || y < 0) break;   // wave-uniform
                        int64_t tx = 0, lx = 0;
#pragma unroll
                        for (int k = 0; k < kMaxSeg; ++k)
                            if (k == x) {
                                tx = tk[k];
                                lx = lk[k];
                            }
                        // the new chain starts at mid with x's sum: its lanes' thresholds
                        // are min(theirs for x, mid), whose largest is mid
                        const int64_t mid = lx + (tx - lx) / 2;
                        const int sx = q + x * nact, sy = q + y * nact;
                        const int64_t xF = CTL[sx].cF, xs = CTL[sx].cs;
                        wave_sync();
                        if (lane == 0) {
                            CTL[sy].cF = xF;
                            CTL[sy].ct = mid;
                            CTL[sy].cs = xs;
                            CTL[sx].cs = mid;
                        }
#pragma unroll
                        for (int k = 0; k < kMaxSeg; ++k) {
                            if (k == y) {
                                tk[k] = mid;
                                lk[k] = lx;
                            }
                            if (k == x) lk[k] = mid;
                        }
                    }
#pragma unroll
                    for (int k = 0; k < kMaxSeg; ++k) {
                        if (k >= nchain) continue;
                        const bool r = tk[k] > lk[k];
                        set_ctl(q + k * nact, r, tk[k]);
                        any |= r;
                    }
                }
                wave_sync();
                if (!any) break;
                pass(false);
                advance(0);
            }

            // ---- 5) results ----
            if (member) {
                if (pok)
                    write_result(out, HAPMOE_STATUS_OK, bs + ki->dp_const, EXACT ? bsum : bs - Bm * bmx, bmx, prm, pw);
                else
                    write_result(out, HAPMOE_STATUS_OVERFLOW, kInf, kInf, kInf, 0, zero_words);
            }

            if (STATS) {
                // per class: the passes its candidates took part in (rounds, counted
                // once when both of its slots ran), and the relaxations, split-point
                // evaluations and lane slots of the relaxation loops of its slots; the
                // shared work is counted once, on the class's first candidate in range
                int rq[kMaxSeg] = {0, 0, 0, 0}, eq[kMaxSeg] = {0, 0, 0, 0};
                int sq[kMaxSeg] = {0, 0, 0, 0};
                int lead[kMaxSeg] = {-1, -1, -1, -1};
    #pragma unroll
                for (int q = 0; q < kMaxSeg; ++q) {
                    if (q >= nseg) continue;
                    rq[q] = wave_sum32(relq[q]);
                    eq[q] = wave_sum32(evq[q]);
                    sq[q] = wave_sum32(slq[q]);
                    lead[q] = __ffsll((unsigned long long)__ballot(inr && sj == q)) - 1;
                }
    #pragma unroll
                for (int q = 0; q < kMaxSeg; ++q) {
                    if (q >= nact) continue;
                    for (int k = 1; k < nchain; ++k) {
                        rq[q] += sel4(rq, q + k * nact);
                        sq[q] += sel4(sq, q + k * nact);
                    }
                }
                if (inr && sj >= 0) {
                    const int p = passes;
                    const int r = sj == 0 ? rq[0] : sj == 1 ? rq[1] : sj == 2 ? rq[2] : rq[3];
                    const int e = sj == 0 ? eq[0] : sj == 1 ? eq[1] : sj == 2 ? eq[2] : eq[3];
                    const int l = sj == 0 ? lead[0] : sj == 1 ? lead[1] : sj == 2 ? lead[2] : lead[3];
                    const int z = sj == 0 ? sq[0] : sj == 1 ? sq[1] : sj == 2 ? sq[2] : sq[3];
                    st_out[0] = p;
                    st_out[1] = lane == l ? r : 0;
                    st_out[2] = lane == l ? e : 0;
                    st_out[3] = lane == l ? z : 0;
                }
            }
            wave_sync();
        }
    }
    HAPMOE_CLOCK(kClockControl);
    HAPMOE_CLOCK_FLUSH(lane);
}

}  // namespace

int32_t stage_dp_section_clocks(uint64_t *out, bool clear)
{
#ifdef HAPMOE_SECTION_CLOCKS
    if (hipMemcpyFromSymbol(out, HIP_SYMBOL(g_section_clocks), sizeof(uint64_t) * kSectionClocks) != hipSuccess)
        return HAPMOE_E_HIP;
    int dev = 0, khz = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
        return HAPMOE_E_HIP;
    out[kWallClockKHz] = (uint64_t)khz;
    if (clear) {
        const uint64_t z[kSectionClocks] = {};
        if (hipMemcpyToSymbol(HIP_SYMBOL(g_section_clocks), z, sizeof(z)) != hipSuccess) return HAPMOE_E_HIP;
    }
    return HAPMOE_OK;
#else
    (void)out;
    (void)clear;
    return HAPMOE_E_INVAL;   // built without the section clocks
#endif
}

int64_t stage_dp_ws_bytes() { return 256; }

hipError_t launch_stage_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_layers, int n_micro,
                           const std::vector<int32_t> &config_pp, int n_orders, const TablesLayout &L,
                           const void *d_tables, int64_t first, int64_t count, int kmax, int ppmax,
                           hapmoe_dp_result *d_res, int32_t *d_stats, void *d_ws, const int32_t *micro,
                           bool exact, hipStream_t s)
{
    (void)config_pp;
    (void)micro;
    (void)n_orders;
    if (count == 0) return hipSuccess;
    // keys holding candidates of [first, first + count)
    const int64_t key_lo = first / n_micro, key_hi = (first + count - 1) / n_micro;
    const int64_t n_keys = key_hi - key_lo + 1;
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
        if (grid > n_keys) grid = n_keys;
        hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64), S.total, s, img, d_cand, L, tab, first, count,
                           key_lo, n_keys, S, d_res, d_stats, queue);
        return hipGetLastError();
    };
    if (exact) return d_stats ? go(k_stage_dp<true, true>) : go(k_stage_dp<false, true>);
    return d_stats ? go(k_stage_dp<true, false>) : go(k_stage_dp<false, false>);
}

}  // namespace hapmoe
