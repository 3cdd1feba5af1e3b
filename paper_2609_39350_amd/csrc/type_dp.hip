// Device-count stage DP: free per-stage device types (Section 3.4 -- the DP
// state carries the devices left of each type, and every transition places
// one more stage, choosing its device type and its layers; Algorithm 1 with
// the three prunings).
//
// A pipeline of PP stages with g = G / PP devices a stage holds k_h = m_h / g
// stages of type h.  State (u, b, h'): u_h stages of type h placed (s = sum u
// of them), layers [0, b) covered, the next stage of type h'.  In threshold
// form
//     F_t(u, b, h') = min over (a, h) of F_t(u - e_h, a, h) + c_{s-1,h,h'}(a, b)
// over stage costs <= t, where c is the pure type-h stage's time on [a, b)
// (memory with min(PP - s + 1, B) stored micro-batches, recomputation only if
// needed) plus the transfer to the type-h' stage; the last stage has none
// (h' = T).  Ties keep the smallest a, then the smallest h, so the back-trace
// from (k, N, T) is the lexicographically smallest (b_{PP-1}, h_{PP-1}, ...,
// b_1, h_1, h_0) among the sum-optimal paths.
//
// Thresholds: a pass at t yields the canonical path, whose largest stage m
// gives the same path for every threshold in [m, t]; so the sweep goes down
// from t = inf to m - 1 each time, skipping thresholds that can no longer beat
// any incumbent (F_t >= F_inf).  An incumbent per B is replaced by a lower
// objective or an equal one with a lower largest stage: the result is the
// least sum + (B-1) max, the smallest threshold reaching it, and the
// back-trace there.  B enters through min(B, PP) (memory) and the objective
// weight: the B values with one min(B, PP) share every pass, and so do
// neighbouring values of min(B, PP) whose feasible split intervals agree at
// every (stage, type, end layer) -- one sweep per such class, one incumbent
// per B.
//
// Mapping: one 1024-thread workgroup per configuration, pulled from an atomic
// queue (largest PP first).  States of one level (equal sum u) are
// independent: their (u, b, h') entries are spread over the threads, and the
// levels follow one another with a barrier.  Only end layers b inside the
// band the pruning-1 windows leave for u are visited (the rest cannot lie on
// a feasible path).  F and the back-trace pointers live in the workgroup's
// slice of the workspace; the layer prefix sums, the level lists and the
// incumbents in LDS.  Plain int64 min-plus work: no MFMA.
#include "internal.h"

namespace hapmoe {
namespace {

constexpr int kThreads = 1024;
constexpr int64_t kNone = INT64_MAX;   // no path
constexpr int kTypeWin = 4;            // split points a predecessor type loads at once

struct TypePath {   // result of one pass, filled by thread 0
    int64_t F, M;
    int64_t fwd;        // forward time (ceil(c/3)) of the stages up to the first largest one
    int32_t s1;         // that stage, 1-based
    uint32_t rmask;
    uint8_t layers[kMaxStages];
    uint8_t types[kMaxStages];
};

struct TypeInc {   // incumbent of one microbatch count
    int64_t obj, M, F;
    uint32_t rmask;
    int32_t passes;
    uint8_t layers[kMaxStages];
    uint8_t types[kMaxStages];
};

struct TypeCtl {   // workgroup-uniform scalars set by thread 0
    uint32_t qi;
    int32_t go;
    int64_t t, finf, lastF;
    int32_t cnt[kMaxStages + 2];   // states per level
    int32_t start[kMaxStages + 2];
    int32_t wmax[kMaxStages + 2];  // widest end-layer band of a level
    uint32_t relax;
    int32_t diff;   // a later group's feasible intervals differ from the class's
};

// one state vector u of a level: u | 6-bit digits u_h | band start | band width
__device__ inline uint64_t pack_u(int u, const int *d, int blo, int wd)
{
    uint64_t x = (uint64_t)u | ((uint64_t)blo << 37) | ((uint64_t)wd << 45);
#pragma unroll
    for (int h = 0; h < kMaxTypes; ++h) x |= (uint64_t)d[h] << (13 + 6 * h);
    return x;
}

// exact q = floor(i / d), r = i - q d for 0 <= i < 2^24, d >= 1, inv = 1/d in fp32
__device__ inline void div_small(int i, int d, float inv, int &q, int &r)
{
    q = (int)((float)i * inv);
    r = i - q * d;
    if (r < 0) {
        --q;
        r += d;
    } else if (r >= d) {
        ++q;
        r -= d;
    }
}

// Layer prefix sums of one configuration in LDS: stage times of each pure type
// set without / with recomputation, weights, activations, MoE-layer count.
struct StageData {
    const int64_t *T0, *T1;        // [T][W]
    const int64_t *MW, *MA0, *MA1;
    const int32_t *MOE;
    int W;
};

// Cost of a pure type-h stage on layers [a, b) holding ms micro-batches of
// activations in capacity cap, plus its outgoing transfer pc: kNone if it does
// not fit even with recomputation, else the cost, *r = 1 if recomputation was
// needed.
__device__ inline int64_t stage_cost(const StageData &D, int h, int a, int b, int64_t ms, int64_t cap, int64_t X,
                                     bool recomp, int64_t pc, int *r)
{
    const int64_t dw = D.MW[b] - D.MW[a];
    const int64_t ex = (D.MOE[b] - D.MOE[a]) > 0 ? X : 0;
    if (dw + ms * (D.MA0[b] - D.MA0[a]) + ex <= cap) {
        *r = 0;
        return D.T0[h * D.W + b] - D.T0[h * D.W + a] + pc;
    }
    if (recomp && dw + ms * (D.MA1[b] - D.MA1[a]) + ex <= cap) {
        *r = 1;
        return D.T1[h * D.W + b] - D.T1[h * D.W + a] + pc;
    }
    return kNone;
}

template <bool STATS, bool EXACT>
__global__ __launch_bounds__(kThreads) void k_type_dp(const unsigned char *__restrict__ img,
                                                      const hapmoe_candidate *__restrict__ cand, TablesLayout L,
                                                      const unsigned char *__restrict__ tab, int64_t first,
                                                      int64_t count, int64_t key_lo, int64_t n_keys, TypeLds S,
                                                      unsigned char *__restrict__ slots, int64_t slot_bytes,
                                                      hapmoe_dp_result *__restrict__ res,
                                                      uint8_t *__restrict__ types_out, int32_t *__restrict__ stats,
                                                      uint32_t *__restrict__ queue)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const ImageHeader &H = *reinterpret_cast<const ImageHeader *>(img);
    const int tid = threadIdx.x;
    const int N = H.n_layers, W = N + 1, T = H.n_types, T1 = T + 1;
    const int nB = H.n_micro;
    const int64_t np = L.np;

    int64_t *sT0 = reinterpret_cast<int64_t *>(smem + S.off_t0);
    int64_t *sT1 = reinterpret_cast<int64_t *>(smem + S.off_t1);
    int64_t *sMW = reinterpret_cast<int64_t *>(smem + S.off_mw);
    int64_t *sMA0 = sMW + W, *sMA1 = sMA0 + W;
    int32_t *sMOE = reinterpret_cast<int32_t *>(smem + S.off_moe);
    uint64_t *ulist = reinterpret_cast<uint64_t *>(smem + S.off_ulist);
    // per (stage, type, end layer b) of the current B group: the least split
    // point that fits at all (low byte) and the least that fits without
    // recomputation (high byte); b itself means none
    uint16_t *bounds = reinterpret_cast<uint16_t *>(smem + S.off_bounds);
    TypeInc *inc = reinterpret_cast<TypeInc *>(smem + S.off_inc);
    TypePath &P = *reinterpret_cast<TypePath *>(smem + S.off_path);
    TypePath &Q = *(reinterpret_cast<TypePath *>(smem + S.off_path) + 1);   // 1F1B: the pending frontier point
    TypeCtl &C = *reinterpret_cast<TypeCtl *>(smem + S.off_ctl);
    const StageData D{sT0, sT1, sMW, sMA0, sMA1, sMOE, W};

    int64_t *F = reinterpret_cast<int64_t *>(slots + (int64_t)blockIdx.x * slot_bytes);
    int16_t *ARG = reinterpret_cast<int16_t *>(F + (int64_t)S.umax * W * T1);

    for (;;) {
        if (tid == 0) C.qi = atomicAdd(queue, 1u);
        __syncthreads();
        // wave-uniform: everything indexed by the key stays scalar
        const uint32_t qi = (uint32_t)__builtin_amdgcn_readfirstlane((int)C.qi);
        __syncthreads();
        if ((int64_t)qi >= n_keys) break;   // every workgroup exits once the queue is drained
        const int64_t key = key_lo + n_keys - 1 - (int64_t)qi;   // one key per configuration, PP-ascending
        const int64_t idx0 = key * nB;
        if (idx0 + nB <= first || idx0 >= first + count) continue;
        const int PP = __builtin_amdgcn_readfirstlane(cand[idx0].pp);
        const PiInfo *pi = reinterpret_cast<const PiInfo *>(tab + L.off_pi) + key;
        const KeyInfo *ki = reinterpret_cast<const KeyInfo *>(tab + L.off_key) + key;

        // ---- stage counts per type, radix of u, per-type windows ----
        const int g = H.total_devices / PP;
        int k[kMaxTypes], rad[kMaxTypes], lo[kMaxTypes], hi[kMaxTypes];
        int U = 1, sum_lo = 0, sum_hi = 0;
#pragma unroll
        for (int h = 0; h < kMaxTypes; ++h) {
            k[h] = h < T ? H.count[h] / g : 0;
            rad[h] = U;
            U *= k[h] + 1;
            lo[h] = hi[h] = 0;
            for (int s = 0; s < PP; ++s)   // the first sequence's layout holds every type's window
                if (ki->mask[s] == (1 << h)) {
                    lo[h] = ki->lo[s];
                    hi[h] = ki->hi[s];
                }
            sum_lo += k[h] * lo[h];
            sum_hi += k[h] * hi[h];
        }
        const bool shape_ok = pi->status == HAPMOE_STATUS_OK && sum_lo <= N && sum_hi >= N && U <= S.umax;

        // ---- levels: the u of each sum, then prefix sums to LDS ----
        if (tid < kMaxStages + 2) {
            C.cnt[tid] = 0;
            C.wmax[tid] = 0;
        }
        __syncthreads();
        auto level_of = [&](int u) {
            int l = 0;
#pragma unroll
            for (int h = 0; h < kMaxTypes; ++h) l += (u / rad[h]) % (k[h] + 1);
            return l;
        };
        if (shape_ok)
            for (int u = tid; u < U; u += kThreads) atomicAdd(&C.cnt[level_of(u)], 1);
        __syncthreads();
        if (tid == 0) {
            int acc = 0;
            for (int l = 0; l <= PP; ++l) {
                C.start[l] = acc;
                acc += C.cnt[l];
                C.cnt[l] = C.start[l];
            }
            C.start[PP + 1] = acc;
        }
        __syncthreads();
        if (shape_ok)
            for (int u = tid; u < U; u += kThreads) {   // digits and the band of end layers the windows leave
                int d[kMaxTypes], l = 0, ulo = 0, uhi = 0, rlo = 0, rhi = 0;
#pragma unroll
                for (int h = 0; h < kMaxTypes; ++h) {
                    d[h] = (u / rad[h]) % (k[h] + 1);
                    l += d[h];
                    ulo += d[h] * lo[h];
                    uhi += d[h] * hi[h];
                    rlo += (k[h] - d[h]) * lo[h];
                    rhi += (k[h] - d[h]) * hi[h];
                }
                const int blo = ulo > N - rhi ? ulo : N - rhi, bhi = uhi < N - rlo ? uhi : N - rlo;
                const int wd = bhi >= blo ? bhi - blo + 1 : 0;
                ulist[atomicAdd(&C.cnt[l], 1)] = pack_u(u, d, wd ? blo : 0, wd);
                atomicMax(&C.wmax[l], wd);
            }
        const int64_t *mem = reinterpret_cast<const int64_t *>(tab + L.off_mem) + key * 4 * np;
        const int64_t *time = reinterpret_cast<const int64_t *>(tab + L.off_time) + key * L.n_masks * 3 * np;
        for (int b = tid; b < W; b += kThreads) {
            sMW[b] = mem[b];
            sMA0[b] = mem[np + b];
            sMA1[b] = mem[2 * np + b];
            sMOE[b] = (int32_t)mem[3 * np + b];
            for (int h = 0; h < T; ++h) {
                const bool on = k[h] > 0;   // only the sets some stage uses are written
                sT0[h * W + b] = on ? time[((int64_t)((1 << h) - 1) * 3) * np + b] : 0;
                sT1[h * W + b] = on ? time[((int64_t)((1 << h) - 1) * 3 + 1) * np + b] : 0;
            }
        }
        __syncthreads();

        const int64_t X = pi->x_bytes, eta_tbar = (int64_t)H.eta_prune * pi->tbar;
        const bool recomp = H.allow_recompute != 0, prune_het = H.prune_hetero != 0;
        // ---- one pass at threshold t, groups of equal min(B, PP) = v ----
        auto pass = [&](int64_t t, int v) {
            uint32_t relax = 0;
            for (int i = tid; i < W * T1; i += kThreads) {   // u = 0: only b = 0
                const int b = i / T1, hn = i % T1;
                F[i] = (b == 0 && hn < T && k[hn] > 0) ? 0 : kNone;
            }
            __syncthreads();
            for (int l = 1; l <= PP; ++l) {
                const int s = l - 1;   // the stage that ends at b
                // one (u, b) state vector a thread: its predecessors are loaded once and
                // relaxed into every valid next type h' (the transfer and pruning 3
                // depend on h', the rest does not)
                const int wm = C.wmax[l];
                const int n_items = (C.start[l + 1] - C.start[l]) * wm;
                const float inv_wm = wm ? 1.0f / (float)wm : 0.0f;
                for (int i = tid; i < n_items; i += kThreads) {
                    int pos, j;
                    div_small(i, wm, inv_wm, pos, j);
                    const uint64_t x = ulist[C.start[l] + pos];
                    const int wd = (int)(x >> 45) & 0x1ff;
                    if (j >= wd) continue;
                    const int u = (int)(x & 0x1fff), b = ((int)(x >> 37) & 0xff) + j;
                    int d[kMaxTypes], ulo = 0, uhi = 0, rlo = 0, rhi = 0, hnmask = 0;
#pragma unroll
                    for (int h = 0; h < kMaxTypes; ++h) {
                        d[h] = (int)(x >> (13 + 6 * h)) & 63;
                        ulo += d[h] * lo[h];
                        uhi += d[h] * hi[h];
                        rlo += (k[h] - d[h]) * lo[h];
                        rhi += (k[h] - d[h]) * hi[h];
                        if (h < T && d[h] < k[h]) hnmask |= 1 << h;   // a stage of type h can follow
                    }
                    if (l == PP) hnmask = 1 << T;   // the last stage: no successor
                    int64_t best[kMaxTypes + 1];
                    int bk[kMaxTypes + 1];
#pragma unroll
                    for (int e = 0; e <= kMaxTypes; ++e) {
                        best[e] = kNone;
                        bk[e] = 0x7fff;
                    }
                    // the first kTypeWin split points of every predecessor type are
                    // loaded together (up to 16 loads in flight), then relaxed; longer
                    // windows (no pruning-1 windows) finish in a second loop
                    int wa0[kMaxTypes], wa1[kMaxTypes];
                    int64_t pv[kMaxTypes][kTypeWin];
#pragma unroll
                    for (int h = 0; h < kMaxTypes; ++h) {
                        wa0[h] = 1;
                        wa1[h] = 0;   // empty
                        if (h < T && d[h] > 0) {
                            // the predecessor's band: one stage of type h fewer
                            const int plo = (ulo - lo[h]) > N - (rhi + hi[h]) ? (ulo - lo[h]) : N - (rhi + hi[h]);
                            const int phi = (uhi - hi[h]) < N - (rlo + lo[h]) ? (uhi - hi[h]) : N - (rlo + lo[h]);
                            wa0[h] = (b - hi[h]) > plo ? (b - hi[h]) : plo;
                            wa1[h] = (b - lo[h]) < phi ? (b - lo[h]) : phi;
                        }
                        const int64_t *Fp = F + (int64_t)(u - rad[h]) * W * T1 + h;
#pragma unroll
                        for (int jj = 0; jj < kTypeWin; ++jj) {
                            const int a = wa0[h] + jj;
                            pv[h][jj] = a <= wa1[h] ? Fp[(int64_t)a * T1] : kNone;
                        }
                    }
#pragma unroll
                    for (int h = 0; h < kMaxTypes; ++h) {
                        if (wa0[h] > wa1[h]) continue;
                        // transfer to each next type, and pruning 3 on it
                        int64_t pc[kMaxTypes + 1];
                        int ok = 0;
#pragma unroll
                        for (int e = 0; e <= kMaxTypes; ++e) {
                            pc[e] = e < T ? pi->p2p[h * kMaxTypes + e] : 0;
                            const bool p3 = prune_het && e < T && e != h && pc[e] > eta_tbar;
                            if (((hnmask >> e) & 1) && !p3) ok |= 1 << e;
                        }
                        if (!ok) continue;
                        if (STATS) relax += (uint32_t)((wa1[h] - wa0[h] + 1) * __popc(ok));
                        const int bd = bounds[(s * T + h) * W + b];
                        const int amin = bd & 0xff, a0 = bd >> 8;
                        const int64_t tb0 = sT0[h * W + b], tb1 = sT1[h * W + b];
                        const int64_t *Fp = F + (int64_t)(u - rad[h]) * W * T1 + h;
                        for (int a = wa0[h]; a <= wa1[h]; ++a) {
                            const int jj = a - wa0[h];
                            int64_t prev = kNone;
#pragma unroll
                            for (int q = 0; q < kTypeWin; ++q) prev = jj == q ? pv[h][q] : prev;
                            if (jj >= kTypeWin) prev = Fp[(int64_t)a * T1];
                            if (prev == kNone || a < amin) continue;
                            const int64_t st = a < a0 ? tb1 - sT1[h * W + a] : tb0 - sT0[h * W + a];
                            const int key2 = a * 8 + h;
#pragma unroll
                            for (int e = 0; e <= kMaxTypes; ++e) {
                                if (!((ok >> e) & 1)) continue;
                                const int64_t c = st + pc[e];
                                if (c > t) continue;
                                const int64_t val = prev + c;
                                if (val < best[e] || (val == best[e] && key2 < bk[e])) {
                                    best[e] = val;
                                    bk[e] = key2;
                                }
                            }
                        }
                    }
                    const int64_t at = ((int64_t)u * W + b) * T1;
#pragma unroll
                    for (int e = 0; e <= kMaxTypes; ++e) {
                        if (!((hnmask >> e) & 1)) continue;
                        F[at + e] = best[e];
                        ARG[at + e] = (int16_t)(best[e] == kNone ? -1 : bk[e]);
                    }
                }
                __syncthreads();
            }
            if (STATS && relax) atomicAdd(&C.relax, relax);
            if (tid == 0) {   // back-trace the canonical path
                const int64_t fe = F[((int64_t)(U - 1) * W + N) * T1 + T];
                P.F = fe;
                P.M = 0;
                P.rmask = 0;
                P.fwd = 0;
                P.s1 = 0;
                if (fe != kNone) {
                    int u = U - 1, b = N, hn = T;
                    int64_t fsum = 0, fafter = 0;   // forward times: all stages, those after the first largest
                    for (int i = PP - 1; i >= 0; --i) {
                        const int x = ARG[((int64_t)u * W + b) * T1 + hn];
                        const int a = x >> 3, h = x & 7;
                        const int64_t msi = (PP - i) < v ? (PP - i) : v;
                        const int64_t pc = hn < T ? pi->p2p[h * kMaxTypes + hn] : 0;
                        int r = 0;
                        const int64_t c = stage_cost(D, h, a, b, msi, H.mem_bytes[h], X, recomp, pc, &r);
                        if (c >= P.M) {   // ">=": going down, the smaller stage index wins ties
                            P.M = c;
                            P.s1 = i + 1;
                            fafter = fsum;
                        }
                        fsum += (c + 2) / 3;
                        P.layers[i] = (uint8_t)(b - a);
                        P.types[i] = (uint8_t)h;
                        P.rmask |= (uint32_t)r << i;
                        u -= rad[h];
                        b = a;
                        hn = h;
                    }
                    P.fwd = fsum - fafter;
                }
            }
            __syncthreads();
        };

        auto take = [&](int j) {   // thread j: the pass's path for microbatch count j
            const int64_t B = H.micro[j];
            const int64_t obj = P.F + (B - 1) * P.M;
            TypeInc &I = inc[j];
            if (obj < I.obj || (obj == I.obj && P.M < I.M)) {
                I.obj = obj;
                I.M = P.M;
                I.F = P.F;
                I.rmask = P.rmask;
                for (int i = 0; i < kMaxStages; ++i) {
                    I.layers[i] = i < PP ? P.layers[i] : 0;
                    I.types[i] = i < PP ? P.types[i] : 0;
                }
            }
        };

        // 1F1B: thread j scores a frontier point for microbatch count j (least
        // latency, ties to the lower largest stage)
        auto take_exact = [&](int j, const TypePath &R) {
            const int64_t B = H.micro[j];
            const int64_t steady = B - R.s1 - 1 > 0 ? B - R.s1 - 1 : 0;
            const int64_t obj = R.F + R.fwd + steady * R.M;
            TypeInc &I = inc[j];
            if (obj < I.obj || (obj == I.obj && R.M < I.M)) {
                I.obj = obj;
                I.M = R.M;
                I.F = R.F;
                I.rmask = R.rmask;
                for (int i = 0; i < kMaxStages; ++i) {
                    I.layers[i] = i < PP ? R.layers[i] : 0;
                    I.types[i] = i < PP ? R.types[i] : 0;
                }
            }
        };

        int v_prev = 0;
        for (;;) {
            int v = 1 << 30;
            for (int j = 0; j < nB; ++j) {
                const int vj = H.micro[j] < PP ? H.micro[j] : PP;
                if (vj > v_prev && vj < v) v = vj;
            }
            if (v == 1 << 30) break;
            // feasible split points of every (stage, type, end layer) for this group:
            // memory only falls as the split point a rises, so they form a suffix of
            // the pruning-1 window; scan it downwards
            if (shape_ok)
                for (int i = tid; i < PP * T * W; i += kThreads) {
                    const int b = i % W, sh = i / W, h = sh % T, st = sh / T;
                    const int64_t ms = (PP - st) < v ? (PP - st) : v;
                    const int64_t cap = H.mem_bytes[h];
                    int amin = b, a0 = b;
                    const int top = b - (h == 0 ? lo[0] : h == 1 ? lo[1] : h == 2 ? lo[2] : lo[3]);
                    const int bot = b - (h == 0 ? hi[0] : h == 1 ? hi[1] : h == 2 ? hi[2] : hi[3]);
                    for (int a = top; a >= 0 && a >= bot; --a) {
                        const int64_t dw = sMW[b] - sMW[a];
                        const int64_t ex = (sMOE[b] - sMOE[a]) > 0 ? X : 0;
                        const bool fit0 = dw + ms * (sMA0[b] - sMA0[a]) + ex <= cap;
                        const bool fit1 = recomp && dw + ms * (sMA1[b] - sMA1[a]) + ex <= cap;
                        if (!(fit0 || fit1)) break;
                        amin = a;
                        if (fit0) a0 = a;
                    }
                    bounds[i] = (uint16_t)(amin | (a0 << 8));
                }
            __syncthreads();
            // The next group values join this class while their feasible split
            // intervals are the same at every (stage, type, end layer): then every
            // DP pass and back-trace is the same too (memory enters nothing else),
            // so one sweep serves them all, one incumbent per B.
            int vmax = v;
            for (;;) {
                int v2 = 1 << 30;
                for (int j = 0; j < nB; ++j) {
                    const int vj = H.micro[j] < PP ? H.micro[j] : PP;
                    if (vj > vmax && vj < v2) v2 = vj;
                }
                if (v2 == 1 << 30 || !shape_ok) break;   // uniform
                if (tid == 0) C.diff = 0;
                __syncthreads();
                for (int i = tid; i < PP * T * W; i += kThreads) {
                    const int b = i % W, sh = i / W, h = sh % T, st = sh / T;
                    const int64_t ms = (PP - st) < v2 ? (PP - st) : v2;
                    const int64_t cap = H.mem_bytes[h];
                    int amin = b, a0 = b;
                    const int top = b - (h == 0 ? lo[0] : h == 1 ? lo[1] : h == 2 ? lo[2] : lo[3]);
                    const int bot = b - (h == 0 ? hi[0] : h == 1 ? hi[1] : h == 2 ? hi[2] : hi[3]);
                    for (int a = top; a >= 0 && a >= bot; --a) {
                        const int64_t dw = sMW[b] - sMW[a];
                        const int64_t ex = (sMOE[b] - sMOE[a]) > 0 ? X : 0;
                        const bool fit0 = dw + ms * (sMA0[b] - sMA0[a]) + ex <= cap;
                        const bool fit1 = recomp && dw + ms * (sMA1[b] - sMA1[a]) + ex <= cap;
                        if (!(fit0 || fit1)) break;
                        amin = a;
                        if (fit0) a0 = a;
                    }
                    if (bounds[i] != (uint16_t)(amin | (a0 << 8))) C.diff = 1;
                }
                __syncthreads();
                const int differ = C.diff;
                __syncthreads();
                if (differ) break;
                vmax = v2;
            }
            v_prev = vmax;
            auto member = [&](int j) {
                if (j >= nB) return false;
                const int vj = H.micro[j] < PP ? H.micro[j] : PP;
                return vj >= v && vj <= vmax;
            };
            if (tid < nB && member(tid)) {
                inc[tid].obj = kNone;
                inc[tid].M = kNone;
                inc[tid].passes = 0;
            }
            if (tid == 0) C.relax = 0;
            __syncthreads();
            int passes = 0;
            if (shape_ok && !EXACT) {
                pass(kNone, v);
                ++passes;
                if (P.F != kNone) {
                    if (tid < nB && member(tid)) take(tid);
                    if (tid == 0) {
                        C.finf = P.F;
                        C.lastF = P.F;
                        C.t = P.M - 1;
                    }
                    __syncthreads();
                    for (;;) {
                        if (tid == 0) {
                            // thresholds above lim_B cannot reach B's incumbent (F_t >= F_inf)
                            int64_t lim = -1;
                            for (int j = 0; j < nB; ++j) {
                                if (!member(j)) continue;
                                const int64_t B = H.micro[j];
                                const int64_t lj = B > 1 ? (inc[j].obj - C.finf) / (B - 1)
                                                         : (C.lastF == C.finf ? kNone : -1);
                                lim = lj > lim ? lj : lim;
                            }
                            C.t = C.t < lim ? C.t : lim;
                            C.go = C.t >= 0;
                        }
                        __syncthreads();
                        if (!C.go) break;
                        pass(C.t, v);
                        ++passes;
                        if (P.F == kNone) break;
                        if (tid < nB && member(tid)) take(tid);
                        if (tid == 0) {
                            C.lastF = P.F;
                            C.t = P.M - 1;
                        }
                        __syncthreads();
                    }
                }
            }
            if (shape_ok && EXACT) {
                // walk the (max, sum) frontier downwards: the pending point Q is a
                // frontier point once a pass at its max - 1 has a larger sum, and is
                // dropped if the sum is the same (a lower max reaches it)
                pass(kNone, v);
                ++passes;
                if (P.F != kNone) {
                    if (tid == 0) {
                        Q = P;
                        C.t = P.M - 1;
                    }
                    __syncthreads();
                    for (;;) {
                        if (tid == 0) {
                            // every later point has latency >= its sum >= Q.F: stop once no
                            // incumbent can be reached (Q itself included)
                            bool need = false;
                            for (int j = 0; j < nB; ++j)
                                if (member(j)) need = need || !(inc[j].obj < Q.F);
                            C.go = C.t >= 0 && need;
                        }
                        __syncthreads();
                        if (!C.go) break;
                        pass(C.t, v);
                        ++passes;
                        if (P.F == kNone) break;
                        if (P.F > Q.F && tid < nB && member(tid)) take_exact(tid, Q);
                        __syncthreads();
                        if (tid == 0) {
                            Q = P;
                            C.t = P.M - 1;
                        }
                        __syncthreads();
                    }
                    if (tid < nB && member(tid)) take_exact(tid, Q);   // the last point
                }
            }
            __syncthreads();
            // ---- results of the group's candidates in range ----
            if (tid < nB && member(tid)) {
                const int64_t inst = idx0 + tid;
                if (inst >= first && inst < first + count) {
                    const TypeInc &I = inc[tid];
                    hapmoe_dp_result *o = res + (inst - first);
                    uint8_t *ty = types_out + (inst - first) * kMaxStages;
                    const bool ok = I.obj != kNone;
                    const int st = pi->status != HAPMOE_STATUS_OK ? HAPMOE_STATUS_OVERFLOW
                                   : ok                              ? HAPMOE_STATUS_OK
                                                                     : HAPMOE_STATUS_INFEASIBLE;
                    o->objective = ok ? I.obj + ki->dp_const : kNone;
                    o->stage_sum = ok ? I.F : kNone;
                    o->t_max = ok ? I.M : kNone;
                    o->status = st;
                    o->recompute_mask = ok ? I.rmask : 0;
                    for (int i = 0; i < kMaxStages; ++i) {
                        o->layers[i] = ok ? I.layers[i] : 0;
                        ty[i] = ok && i < PP ? (uint8_t)(1u << I.types[i]) : 0;
                    }
                    if (STATS) {
                        int32_t *so = stats + 4 * (inst - first);
                        bool lead = true;   // the group's work is counted once, on its first candidate
                        for (int j = 0; j < tid; ++j) lead = lead && !member(j);
                        so[0] = passes;
                        so[1] = lead ? (int32_t)C.relax : 0;
                        so[2] = 0;
                        so[3] = 0;
                    }
                }
            }
            __syncthreads();
        }
    }
}

__global__ void k_reset_type_queue(uint32_t *q) { q[0] = 0; }

}  // namespace

TypeLds type_dp_lds(int n_layers, int n_types, int n_micro, int umax, int ppmax)
{
    const int W = n_layers + 1;
    TypeLds S;
    S.umax = umax;
    int64_t off = 0;
    auto take = [&](int64_t bytes) {
        const int64_t at = off;
        off = (off + bytes + 15) & ~int64_t(15);
        return (int)at;
    };
    S.off_t0 = take((int64_t)n_types * W * 8);
    S.off_t1 = take((int64_t)n_types * W * 8);
    S.off_mw = take((int64_t)3 * W * 8);
    S.off_moe = take((int64_t)W * 4);
    S.off_inc = take((int64_t)n_micro * sizeof(TypeInc));
    S.off_path = take(2 * sizeof(TypePath));
    S.off_ctl = take(sizeof(TypeCtl));
    S.off_ulist = take((int64_t)umax * 8);
    S.off_bounds = take((int64_t)ppmax * n_types * W * 2);
    S.bytes = (int)off;
    return S;
}

int64_t type_dp_slot_bytes(int n_layers, int n_types, int umax)
{
    const int64_t states = (int64_t)umax * (n_layers + 1) * (n_types + 1);
    return align256(states * 8 + states * 2);
}

int64_t type_dp_slots(int64_t n_keys, int64_t slot_bytes)
{
    int64_t slots = n_keys < kTypeDpMaxSlots ? n_keys : kTypeDpMaxSlots;
    const int64_t cap = kTypeDpMaxSlotBytes / (slot_bytes > 0 ? slot_bytes : 1);
    slots = slots < cap ? slots : cap;
    return slots < 1 ? 1 : slots;
}

hipError_t launch_type_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_layers, int n_types,
                          int n_micro, int umax, int ppmax, const TablesLayout &L, const void *d_tables, int64_t first,
                          int64_t count, hapmoe_dp_result *d_res, uint8_t *d_types, int32_t *d_stats, void *d_ws,
                          bool exact, hipStream_t s)
{
    const int64_t key_lo = first / n_micro, key_hi = (first + count - 1) / n_micro;
    const int64_t n_keys = key_hi - key_lo + 1;
    const TypeLds S = type_dp_lds(n_layers, n_types, n_micro, umax, ppmax);
    const int64_t slot_bytes = type_dp_slot_bytes(n_layers, n_types, umax);
    const int64_t slots = type_dp_slots(L.n_configs, slot_bytes);
    const int64_t grid = slots < n_keys ? slots : n_keys;
    auto *queue = static_cast<uint32_t *>(d_ws);
    auto *slot_base = static_cast<unsigned char *>(d_ws) + 256;
    hipLaunchKernelGGL(k_reset_type_queue, dim3(1), dim3(1), 0, s, queue);
    const auto *img = static_cast<const unsigned char *>(d_image);
    const auto *tab = static_cast<const unsigned char *>(d_tables);
    const dim3 grid3((unsigned)grid), block(kThreads);
    // more than 64 KB of LDS a workgroup (the count states of 32-stage pipelines
    // on four types) has to be allowed per kernel
#define HAPMOE_TYPE_DP(ST, EX)                                                                                 \
    do {                                                                                                       \
        if (S.bytes > 65536) {                                                                                 \
            const hipError_t e_ = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_type_dp<ST, EX>),     \
                                                      hipFuncAttributeMaxDynamicSharedMemorySize, S.bytes);    \
            if (e_ != hipSuccess) return e_;                                                                   \
        }                                                                                                      \
        hipLaunchKernelGGL((k_type_dp<ST, EX>), grid3, block, S.bytes, s, img, d_cand, L, tab, first, count,     \
                           key_lo, n_keys, S, slot_base, slot_bytes, d_res, d_types, d_stats, queue);          \
    } while (0)
    if (d_stats && exact)
        HAPMOE_TYPE_DP(true, true);
    else if (d_stats)
        HAPMOE_TYPE_DP(true, false);
    else if (exact)
        HAPMOE_TYPE_DP(false, true);
    else
        HAPMOE_TYPE_DP(false, false);
#undef HAPMOE_TYPE_DP
    return hipGetLastError();
}

int64_t type_dp_ws_bytes(int n_layers, int n_types, int umax, int64_t n_configs)
{
    const int64_t slot_bytes = type_dp_slot_bytes(n_layers, n_types, umax);
    return 256 + type_dp_slots(n_configs, slot_bytes) * slot_bytes;
}

}  // namespace hapmoe
