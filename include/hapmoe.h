/*
 * hapmoe.h -- C ABI of the MI355X (gfx950) planner hot path of HAPMoE
 * ("Heterogeneity-Aware Automatic Parallelism Planning for Mixture-of-Experts
 * Models Training").
 *
 * The library evaluates the paper's MoE-aware cost model (Section 3.2) over the
 * 6D candidate space (DP, PP, TP, CP, EP, TPE) on a heterogeneous cluster and
 * runs, for every candidate, the pruning-enhanced stage DP of Section 3.4
 * (Algorithm 1) that picks a non-uniform layer-to-stage partition and a
 * per-stage recomputation choice.  Pipeline of calls:
 *
 *   hapmoe_enumerate_candidates   host   the candidate set (pi, device ordering, B)
 *   hapmoe_pack_image             host   flatten the problem for the device
 *   hapmoe_eval_cost_tables       GPU    cost-table kernel
 *   hapmoe_stage_dp               GPU    stage-DP kernel, one result per candidate
 *   hapmoe_best_plan              GPU    segmented arg-min -> the best plan (syncs)
 *
 * Conventions
 *  - Every call returns an int32_t status: HAPMOE_OK (0) or a negative
 *    HAPMOE_E_* code; hapmoe_strerror() names it.  Nothing throws.
 *  - The caller owns all memory.  Pointers named h_* / host structs are host
 *    memory; d_* are device memory of the current HIP device.  The library
 *    never allocates device memory; buffer sizes come from the *_bytes queries.
 *  - `stream` is a hipStream_t passed as void* (0 = the null stream).  GPU calls
 *    enqueue work and return; only hapmoe_best_plan waits for its stream.
 *  - Times are int64 nanoseconds, memory sizes int64 bytes, bandwidths bytes/ns
 *    (= GB/s), latencies ns.  Costs are rounded up to whole ns / bytes once per
 *    modelled term.
 *  - The device calls need a gfx950 device (HAPMOE_E_ARCH otherwise).  The
 *    library caches that answer per device (an atomic flag each, set once); it
 *    holds no other state between calls except the section-clock table of its
 *    diagnostic build.  Concurrent calls from several host threads are safe
 *    as long as they do not share output buffers or a workspace.
 */
#ifndef HAPMOE_H
#define HAPMOE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HAPMOE_MAX_TYPES 4     /* device types |H| */
#define HAPMOE_MAX_STAGES 32   /* pipeline stages PP */
#define HAPMOE_MAX_LAYERS 127  /* transformer layers N */
#define HAPMOE_MAX_MICRO 64    /* entries of the microbatch-count list */

enum {
    HAPMOE_OK = 0,
    HAPMOE_E_INVAL = -1,      /* malformed problem or argument */
    HAPMOE_E_CAPACITY = -2,   /* output array too small; the required count is returned */
    HAPMOE_E_WORKSPACE = -3,  /* device buffer smaller than the *_bytes query says */
    HAPMOE_E_HIP = -4,        /* a HIP runtime call failed */
    HAPMOE_E_ARCH = -5,       /* current device is not gfx950 */
    HAPMOE_E_INFEASIBLE = -6, /* no candidate has a memory-feasible partition */
    HAPMOE_E_RANGE = -7       /* candidate sub-range outside [0, n) */
};

/* Per-candidate status in hapmoe_dp_result.status */
enum {
    HAPMOE_STATUS_OK = 0,
    HAPMOE_STATUS_INFEASIBLE = 1, /* no partition passes the three prunings */
    HAPMOE_STATUS_OVERFLOW = 2    /* a modelled term left the int64 range the DP allows */
};

/* Model and training hyper-parameters (Section 3.1 "Input": N, S, H, E, k,
 * batch sizes, optimizer).  Arrays are host memory, N = n_layers entries. */
typedef struct hapmoe_model {
    int32_t n_layers;          /* N, 1..HAPMOE_MAX_LAYERS */
    int32_t seq_len;           /* S */
    int32_t hidden;            /* H */
    int32_t n_experts;         /* E (0 = dense model) */
    int32_t top_k;             /* k */
    int32_t micro_batch_size;  /* tokens per microbatch = seq_len * micro_batch_size */
    int32_t elem_bytes;        /* beta of Eq. 3 */
    double moe_ffn_mult;       /* the factor 2 of Eq. 2: expert work relative to t_ffn */
    const uint8_t *is_moe;          /* [N] 1 = MoE layer */
    const int64_t *expert_tokens;   /* [N][E] router statistics |T_e| (Section 3.2) */
    const int64_t *params_dense;    /* [N] non-expert parameters */
    const int64_t *params_expert;   /* [N] parameters of all experts of the layer */
    const int64_t *act_bytes;       /* [N] activation bytes of one microbatch at TP = CP = 1 */
} hapmoe_model;

/* Device types (Section 3.1: type h has (P_h, C_h, B_h) and m_h devices) and
 * the profiled tables of Section 3.3. */
typedef struct hapmoe_cluster {
    int32_t n_types;                          /* |H|, 1..4 */
    int32_t count[HAPMOE_MAX_TYPES];          /* m_h */
    int32_t speed[HAPMOE_MAX_TYPES];          /* P_h, relative compute speed (integer) */
    int64_t mem_bytes[HAPMOE_MAX_TYPES];      /* C_h */
    double eff[HAPMOE_MAX_TYPES];             /* eta_h of Eq. 2, in (0, 1] */
    double route_coef[HAPMOE_MAX_TYPES];      /* router ns per (token x hidden) */
    double bw[HAPMOE_MAX_TYPES][HAPMOE_MAX_TYPES];     /* link bandwidth h -> h', bytes/ns */
    double alpha[HAPMOE_MAX_TYPES][HAPMOE_MAX_TYPES];  /* link latency h -> h', ns */
    const int64_t *t_dense;  /* [T][4][4][N] dense layer time at TP = 2^i, CP = 2^j, ns */
    const int64_t *t_ffn;    /* [T][4][4][N] its FFN part (0 <= t_ffn <= t_dense) */
} hapmoe_cluster;

/* Method parameters (Sections 3.2 and 3.4). */
typedef struct hapmoe_params {
    double gamma;            /* load-imbalance weight, [0, 1] */
    double rc_time;          /* recomputation time factor (>= 1) */
    double rc_act;           /* xi(r = 1): activation factor under recomputation, [0, 1] */
    double opt_coef;         /* optimizer step, ns per parameter */
    int32_t delta_num;       /* pruning-1 tolerance delta = delta_num / delta_den */
    int32_t delta_den;
    int32_t eta_prune;       /* pruning-3 factor eta */
    int32_t prune_window;    /* layer windows: 0 none, 1 pruning 1 (Section 3.4), 2 uniform:
                                every stage holds floor(N/PP)..ceil(N/PP) layers (non-uniform
                                assignment disabled, the ablation of the evaluation) */
    int32_t prune_hetero;    /* pruning 3 on/off */
    int32_t allow_recompute; /* r in {0, 1} (1) or r = 0 only (0) */
} hapmoe_params;

/* Candidate space (Section 3.4: configuration set Pi; Algorithm 1 input). */
typedef struct hapmoe_space {
    int32_t pp_max;      /* PP <= pp_max <= HAPMOE_MAX_STAGES */
    int32_t tp_mask;     /* bit i: TP = 2^i allowed (i < 4) */
    int32_t cp_mask;     /* bit i: CP = 2^i allowed */
    int32_t ep_max;      /* EP = powers of two dividing E, <= ep_max */
    int32_t tpe_mask;    /* bit i: TPE = 2^i allowed */
    int32_t mode;        /* 0: EP*TPE folds inside the stage group (DP = group/(TP*CP));
                            1: literal product PP*DP*TP*CP*EP*TPE = sum_h m_h */
    int32_t stage_types; /* 0: device-type orderings -- the devices listed type by type in each
                            of the |H|! orders, stage i takes the i-th group of G/PP (a group
                            may straddle two types);
                            1: free per-stage type (the DP state m of Section 3.4): every stage
                            is one group of a single type h, configurations whose m_h are not
                            all multiples of G/PP are left out, and "order" o is the o-th
                            distinct stage-type sequence (lexicographic over the arrangements
                            of m_h / (G/PP) stages of each type h); n_orders is the most such
                            sequences over the configurations, at most 2^20, and a slot past a
                            configuration's own count is an infeasible candidate;
                            2: free per-stage type chosen by the DP over device counts (the
                            state m of Section 3.4): the same configurations as 1, one order
                            slot each (order 0 lays out the first sequence), solved by
                            hapmoe_stage_dp_types; at most 8192 count states prod_h (k_h + 1)
                            per pipeline, k_h = m_h / (G/PP).
                            3: per-stage data-parallel widths (the non-uniform PP/DP of
                            Section 1): the block orderings of 0, but stage i takes the next
                            w_i half-groups of G/(2 PP) devices, w_i in {1, 2, 3} with sum
                            2 PP, and runs DP_i = w_i DP / 2 replicas, each holding 2 / w_i
                            of the nominal tokens of a micro-batch; the widths are chosen by
                            hapmoe_stage_dp_widths; only configurations with DP even and
                            EP * TPE dividing G/(2 PP) take part.
                            With 1, 2 or 3, a space that leaves no configuration is
                            HAPMOE_E_INVAL */
    int32_t n_micro;     /* entries of micro[] */
    int32_t micro[HAPMOE_MAX_MICRO]; /* microbatch counts B, 1..1024 */
    int32_t global_batch; /* 0: every B of micro[] competes in hapmoe_best_plan's arg-min (each
                             candidate's objective is the latency of its own B micro-batches);
                             > 0: the training batch is fixed (Section 3.1 input) at this many
                             sequences, and the arg-min (per configuration and global) only
                             takes candidates whose B * DP * micro_batch_size equals it.  The
                             stage DP itself is unaffected. */
} hapmoe_space;

typedef struct hapmoe_problem {
    hapmoe_model model;
    hapmoe_cluster cluster;
    hapmoe_params params;
    hapmoe_space space;
} hapmoe_problem;

/* One candidate: the 6D configuration pi (Section 3.1 output), the device-type
 * ordering that places the stages on devices, and the microbatch count B. */
typedef struct hapmoe_candidate {
    int32_t pp, tp, cp, dp, ep, tpe;
    int32_t order;      /* rank of the type permutation in lexicographic order */
    int32_t n_micro;    /* B */
} hapmoe_candidate;     /* 32 bytes */

/* Stage-DP result of one candidate (64 bytes). */
typedef struct hapmoe_dp_result {
    int64_t objective;        /* sum_i c_i + (B-1) max_i c_i + C(pi), INT64_MAX if not OK */
    int64_t stage_sum;        /* sum_i c_i */
    int64_t t_max;            /* max_i c_i (the threshold t*) */
    int32_t status;           /* HAPMOE_STATUS_* */
    uint32_t recompute_mask;  /* bit i = r_i */
    uint8_t layers[HAPMOE_MAX_STAGES]; /* n_i */
} hapmoe_dp_result;

/* The best plan (Section 3.1 output (pi*, L*, {h_i*}, {r_i*})). */
typedef struct hapmoe_plan {
    int64_t instance;         /* index of the winning candidate */
    int64_t objective, stage_sum, t_max, dp_const;
    hapmoe_candidate cand;
    int32_t n_stages;
    uint32_t recompute_mask;
    uint8_t layers[HAPMOE_MAX_STAGES];      /* n_i */
    uint8_t stage_types[HAPMOE_MAX_STAGES]; /* bit h set = stage uses device type h */
} hapmoe_plan;

/* Diagnostics: where the stage-DP kernel's time goes.  Only a library built
 * with HAPMOE_SECTION_CLOCKS defined records it (HAPMOE_E_INVAL otherwise).
 * out[0..4] = shader-clock cycles summed over all waves of the launches since
 * the last clear, spent in key set-up and classification, feasibility scans,
 * the relaxation rounds of the passes, the back-traces, and the sweep control;
 * out[5] = the waves' total cycles; out[6..8] = keys, segment batches and
 * passes.  clear != 0 zeroes the table after reading. */
int32_t hapmoe_section_clocks(uint64_t out[16], int32_t clear);

/* Name of a status code (static string). */
const char *hapmoe_strerror(int32_t code);

/* Check a problem against the limits above.  HAPMOE_OK or HAPMOE_E_INVAL. */
int32_t hapmoe_validate(const hapmoe_problem *p);

/* Candidate set (Section 3.1 output pi; Section 3.4 / Algorithm 1 loop over
 * Pi, device types and the microbatch list).  Order: PP, TP, CP, EP, TPE
 * ascending, then the type ordering, then micro[] in the given order; the index
 * of a candidate is ((config * n_orders) + order) * n_micro + micro_index.
 * Host only.  Writes min(capacity, total) candidates to `out` (may be NULL) and
 * the total to *n_total; returns HAPMOE_E_CAPACITY if out is NULL or too small. */
int32_t hapmoe_enumerate_candidates(const hapmoe_problem *p, hapmoe_candidate *out,
                                    int64_t capacity, int64_t *n_total);

/* Problem image: a flat copy of the problem that the kernels read.  The caller
 * copies the packed host image to device memory once and passes that device
 * pointer to the GPU calls together with the same host problem. */
int32_t hapmoe_image_bytes(const hapmoe_problem *p, int64_t *bytes);
int32_t hapmoe_pack_image(const hapmoe_problem *p, void *h_image, int64_t bytes);

/* Size of the cost-table buffer for the full candidate array, and of the
 * optional fp64 debug buffer (pre-rounding terms). */
int32_t hapmoe_tables_bytes(const hapmoe_problem *p, int64_t *bytes);
int32_t hapmoe_debug_bytes(const hapmoe_problem *p, int64_t *bytes);

/* Cost-table buffer format (for inspection; the stage DP reads it):
 *   out[0..8] = n_configs, n_orders, n_masks (= 2^T - 1), np (prefix stride
 *   >= N + 1), off_pi, off_key, off_mem, off_time, total bytes.
 *   pi   [n_configs] 152-byte records {int64 x_bytes, int64 tbar,
 *        int64 p2p[4][4], int32 status, uint32 used_masks}
 *   key  [n_configs * n_orders] 136-byte records {int64 dp_const,
 *        uint8 mask[32], lo[32], hi[32], bpair[32]}
 *   mem  [n_configs][4][np] int64 prefix sums over layers of weights, r = 0
 *        activations, r = 1 activations, and the count of MoE layers
 *   time [n_configs][n_masks][3][np] int64 prefix sums of the stage time
 *        without / with recomputation and of its communication part, for the
 *        device-type set m at index m - 1 (only sets some stage uses are
 *        written).
 *   then, 256-byte aligned after time, [N] double: every layer's
 *        load-imbalance factor 1 + gamma (rho - 1) (1 for dense layers),
 *        written once per call before the per-configuration tables.
 * Debug buffer (fp64, per configuration, out[0..3] = doubles per
 * configuration, offsets of the type, set and memory blocks):
 *   type [N][T][2] (Eq. 2 compute, expert), set [n_masks][N][3] (all-to-all,
 *   TP, CP), mem [N][2] (weights, activations). */
int32_t hapmoe_tables_layout(const hapmoe_problem *p, int64_t out[9]);
int32_t hapmoe_debug_layout(const hapmoe_problem *p, int64_t out[4]);

/* Cost-table kernel (Section 3.2 Eq. 2, Eq. 3, load imbalance, stage memory;
 * Section 3.3 compute / primitive tables; Section 3.4 pruning windows and the
 * constants of Eq. 4).  Per configuration and device-type set it writes prefix
 * sums over layers of the stage time without (r = 0) and with (r = 1)
 * recomputation and of the communication part, per configuration the weight /
 * activation prefix sums, and per (configuration, ordering) the stage layout.
 * d_cand must be the full array of hapmoe_enumerate_candidates (n_cand
 * entries); d_tables has hapmoe_tables_bytes bytes and is indexed by the
 * global configuration index.  Only the configurations holding candidates
 * [first, first + count) are evaluated (every one of their orderings), so a
 * caller can fill the buffer in chunks before running the stage DP on them;
 * every call also rewrites the per-layer load-imbalance factors.  count = 0
 * enqueues nothing; a range outside [0, n_cand) is HAPMOE_E_RANGE.  d_debug
 * (may be NULL) receives the fp64 terms before rounding of the same
 * configurations (hapmoe_debug_bytes).  Asynchronous. */
int32_t hapmoe_eval_cost_tables(const hapmoe_problem *p, const void *d_image,
                                const hapmoe_candidate *d_cand, int64_t n_cand,
                                int64_t first, int64_t count,
                                void *d_tables, int64_t tables_bytes,
                                double *d_debug, int64_t debug_bytes, void *stream);

/* Workspace of hapmoe_stage_dp (its work-queue counter). */
int32_t hapmoe_stage_dp_ws_bytes(const hapmoe_problem *p, int64_t *bytes);

/* Stage-DP kernel (Section 3.4 DP transition, prunings 1-3, Algorithm 1 with
 * backtrace) for candidates [first, first + count): for each, the partition
 * minimising sum_i c_i + (B-1) max_i c_i subject to every stage fitting its
 * memory with the least recomputation.  Ties: lowest threshold t*, then the
 * smallest split point at each backtrace step (from the last stage).  Writes
 * d_res[0 .. count).  d_stats (may be NULL) receives per candidate four
 * int32: threshold passes of its sweep, DP relaxations, split-point
 * evaluations of the feasibility scan, and the lane slots the relaxation
 * loops issued for the sweep (relaxations / slots is the SIMD-lane
 * utilisation of those loops).  Candidates of one (pi, ordering) whose B
 * gives the same min(B, PP) share one sweep; its relaxations, evaluations
 * and slots are counted once, on the first of them.  d_ws
 * (hapmoe_stage_dp_ws_bytes)
 * holds the kernel's work queue: calls that may overlap need their own d_ws.
 * Problems with stage_types = 2 or 3 are HAPMOE_E_INVAL here
 * (hapmoe_stage_dp_types, hapmoe_stage_dp_widths).
 * Asynchronous. */
int32_t hapmoe_stage_dp(const hapmoe_problem *p, const void *d_image,
                        const hapmoe_candidate *d_cand, int64_t n_cand,
                        const void *d_tables, int64_t tables_bytes,
                        int64_t first, int64_t count,
                        hapmoe_dp_result *d_res, int32_t *d_stats,
                        void *d_ws, int64_t ws_bytes, void *stream);

/* Stage DP with the 1F1B iteration latency of the appendix as the objective
 * (Eq. 4 with its steady-state term, a re-scoring of the threshold DP's
 * frontier).  Same arguments, ranges, workspace and errors as hapmoe_stage_dp.
 * For each candidate the (max, sum) Pareto frontier of its feasible partitions
 * is walked -- the thresholds at which the least stage sum drops, each with the
 * canonical partition of the threshold DP there -- and every frontier point is
 * scored with
 *   T = sum_i c_i + sum_{i <= s} ceil(c_i / 3) + max(0, B - s - 1) * max_i c_i,
 * s the first (1-based) stage of largest cost (a stage's forward part is
 * ceil(c / 3), its backward part the rest).  The result keeps the least T,
 * ties to the lower largest stage: objective = T + C, stage_sum and t_max of the
 * chosen partition, its recomputation mask and stage lengths.  d_stats as for
 * hapmoe_stage_dp (passes = DP passes of the frontier walk).  Not for
 * stage_types = 2 or 3 (HAPMOE_E_INVAL).  Asynchronous. */
int32_t hapmoe_stage_dp_1f1b(const hapmoe_problem *p, const void *d_image,
                             const hapmoe_candidate *d_cand, int64_t n_cand,
                             const void *d_tables, int64_t tables_bytes,
                             int64_t first, int64_t count,
                             hapmoe_dp_result *d_res, int32_t *d_stats,
                             void *d_ws, int64_t ws_bytes, void *stream);

/* The least 1F1B iteration latency over every partition (Appendix B, Eq. 5,
 * with the steady-state term of Eq. 4), exact rather than a re-scoring of the
 * threshold DP's frontier:
 *   T = sum_i c_i + sum_{i <= s} ceil(c_i / 3) + max(0, B - s - 1) * max_i c_i,
 * s the first (1-based) stage of largest cost, minimised over every partition
 * that passes the three prunings (stage costs, recomputation and memory as in
 * hapmoe_stage_dp).  For every distinct stage cost t, ascending from the least
 * possible largest stage (the thresholds below it admit no partition), a DP over
 * (stage, end layer, bottleneck placed yet) gives the least T with largest
 * stage exactly t; the sweep stops once F_inf + ceil(t / 3) +
 * max(0, B - PP - 1) t, F_inf the least stage sum, reaches the best T.  Ties:
 * least T, then the lower largest stage, then the lexicographically smallest
 * (b_PP-1, ..., b_1) of the stage end layers.  For each candidate of
 * [first, first + count) writes d_res[i - first]: objective = T + C, stage_sum
 * and t_max of the chosen partition, its recomputation mask and stage lengths.
 * One workgroup per (configuration, ordering) key, lane j holding the key's
 * j-th candidate, the deepest pipelines first.  Its stage-cost table holds, for
 * every stage, end layer b of the stage's band (the end layers its windows
 * allow) and split point of its window, an 8-byte cost c (kept as
 * c + ceil(c / 3)) and a 1-byte recomputation flag (the flags rounded up to 16
 * bytes), plus 16 bytes of DP state for every (stage, b).
 * Launches in tiers of LDS a workgroup: every candidate with 24 KB, then those
 * whose table did not fit (over 22,784 bytes) with 40, 80 and 160 KB; a
 * candidate whose table exceeds 162,048 bytes gets HAPMOE_STATUS_OVERFLOW.  The candidates of a (configuration, ordering) key
 * with B >= PP + 1 share one sweep (their latencies at a threshold t differ by
 * (B - B') t); d_stats (may be NULL): thresholds swept for the candidate, and
 * DP relaxations counted on the first candidate of each shared sweep (columns
 * 2, 3 zero).  No workspace.  Not for
 * stage_types = 2 or 3 (HAPMOE_E_INVAL); ranges and errors as hapmoe_stage_dp.
 * Asynchronous. */
int32_t hapmoe_stage_dp_latency(const hapmoe_problem *p, const void *d_image,
                                const hapmoe_candidate *d_cand, int64_t n_cand,
                                const void *d_tables, int64_t tables_bytes,
                                int64_t first, int64_t count,
                                hapmoe_dp_result *d_res, int32_t *d_stats, void *stream);

/* Workspace of hapmoe_stage_dp_types: the work-queue counter and one slice of
 * DP states per workgroup (F as int64 and the back-trace pointer as int16 per
 * state (u, b, h')); HAPMOE_E_INVAL unless stage_types = 2. */
int32_t hapmoe_stage_dp_types_ws_bytes(const hapmoe_problem *p, int64_t *bytes);

/* Stage DP over device counts for free per-stage device types (stage_types =
 * 2; Section 3.4 with the DP state m of remaining devices per type, the
 * transitions of Algorithm 1 choosing each stage's type h and its layers,
 * prunings 1-3).  A pipeline of PP stages holds k_h = m_h / (G/PP) stages of
 * type h; a stage of type h is a pure group of that type (window, capacity and
 * speed of h, memory with min(PP - i + 1, B) stored micro-batches), and the
 * transfer to the next stage depends on both types.  For each candidate of
 * [first, first + count) it minimises sum_i c_i + (B-1) max_i c_i over every
 * stage-type sequence and partition.  Ties: lowest threshold t*, then at each
 * back-trace step from the last stage the smallest split point, then the
 * smallest type.  Writes d_res[0 .. count) like hapmoe_stage_dp and
 * d_types[32 * (0 .. count)], the type mask (1 << h_i) of each stage (0 past
 * PP and for infeasible candidates).  d_stats (may be NULL): passes of the
 * candidate's sweep and the relaxations of the sweep on the first candidate
 * that shares it (columns 2, 3 zero).  d_ws (hapmoe_stage_dp_types_ws_bytes)
 * is the kernel's: calls that may overlap need their own.  Asynchronous. */
int32_t hapmoe_stage_dp_types(const hapmoe_problem *p, const void *d_image,
                              const hapmoe_candidate *d_cand, int64_t n_cand,
                              const void *d_tables, int64_t tables_bytes,
                              int64_t first, int64_t count,
                              hapmoe_dp_result *d_res, uint8_t *d_types, int32_t *d_stats,
                              void *d_ws, int64_t ws_bytes, void *stream);

/* The device-count DP with the 1F1B latency of hapmoe_stage_dp_1f1b as the
 * objective: the (max, sum) frontier of each candidate over every stage-type
 * sequence and partition is walked (a threshold at which the least sum drops,
 * with the canonical path there), each point is scored with
 *   T = sum_i c_i + sum_{i <= s} ceil(c_i / 3) + max(0, B - s - 1) * max_i c_i,
 * and the least T wins, ties to the lower largest stage.  Same arguments,
 * outputs, workspace and errors as hapmoe_stage_dp_types (d_stats: passes of
 * the walk).  Asynchronous. */
int32_t hapmoe_stage_dp_types_1f1b(const hapmoe_problem *p, const void *d_image,
                                   const hapmoe_candidate *d_cand, int64_t n_cand,
                                   const void *d_tables, int64_t tables_bytes,
                                   int64_t first, int64_t count,
                                   hapmoe_dp_result *d_res, uint8_t *d_types, int32_t *d_stats,
                                   void *d_ws, int64_t ws_bytes, void *stream);

/* Workspace of hapmoe_stage_dp_widths for a launch over `count` candidates: the
 * work-queue counter and one slice of back-trace pointers per workgroup (at
 * most 1024; the DP values themselves live in the workgroup's LDS).
 * HAPMOE_E_INVAL unless stage_types = 3. */
int32_t hapmoe_stage_dp_widths_ws_bytes(const hapmoe_problem *p, int64_t count, int64_t *bytes);

/* Stage DP with per-stage data-parallel widths (stage_types = 3; the
 * "non-uniform PP/DP partitioning" of Section 1 and the ablation of the
 * evaluation: stage-wise parallelism knobs chosen jointly with the layers).
 * The devices are listed type by type in the candidate's ordering; stage i takes
 * the next w_i half-groups of G/(2 PP) devices, w_i in {1, 2, 3}, sum w_i = 2 PP,
 * so it runs DP_i = w_i DP / 2 replicas; every stage processes the same global
 * micro-batch, a replica holding r = 2 / w_i of the nominal tokens.  The stage's
 * cost is the Section 3.2 model at that token count (compute tables scaled by r,
 * router and collectives at the scaled activation), its memory the ZeRO-1 state
 * over DP_i plus activations and MoE buffers at r, its outgoing transfer the
 * sender's per-rank activation over the boundary link; pruning 1 uses the
 * stage's share w_i P_i (G/(2 PP)) / sum_h m_h P_h of the cluster's compute,
 * pruning 3 and the constant of Eq. 4 their nominal values (the constant of the
 * uniform layout).  For each candidate of [first, first + count) it minimises
 * sum_i c_i + (B-1) max_i c_i over the width sequences and partitions.  Ties:
 * lowest threshold t*, then at each back-trace step from the last stage the
 * smallest split point, then the smallest width.  Writes d_res[0 .. count)
 * like hapmoe_stage_dp, d_types[32 * (0 .. count)] the device-type set of each
 * stage and d_widths[32 * (0 .. count)] each w_i (0 past PP and for infeasible
 * candidates).  d_stats (may be NULL): passes of the candidate's sweep and its
 * relaxations, counted on the first candidate of the key that shares the sweep
 * (those with equal min(B, PP) share every pass; columns 2, 3 zero).  The tables must come from
 * hapmoe_eval_cost_tables on the same problem (which adds the width tables).
 * d_ws (hapmoe_stage_dp_widths_ws_bytes for count) is the kernel's: calls that
 * may overlap need their own.  Asynchronous. */
int32_t hapmoe_stage_dp_widths(const hapmoe_problem *p, const void *d_image,
                               const hapmoe_candidate *d_cand, int64_t n_cand,
                               const void *d_tables, int64_t tables_bytes,
                               int64_t first, int64_t count,
                               hapmoe_dp_result *d_res, uint8_t *d_types, uint8_t *d_widths,
                               int32_t *d_stats, void *d_ws, int64_t ws_bytes, void *stream);

/* Workspace of hapmoe_best_plan for n results. */
int32_t hapmoe_best_plan_ws_bytes(const hapmoe_problem *p, int64_t n, int64_t *bytes);

/* Segmented arg-min (Eq. 1 objective): per configuration pi the best of its
 * candidates (d_config_best, n_configs int64 entries: candidate index or -1;
 * may be NULL), then the global best by (objective, candidate index).  d_res
 * holds the results of candidates [0, n); with stage_types = 2 or 3, d_types
 * holds their stage types (hapmoe_stage_dp_types / _widths; the winner's widths
 * are d_widths[32 * instance]), otherwise it must be NULL.
 * Waits for `stream`, fills *h_plan.  Returns HAPMOE_E_INFEASIBLE if no
 * candidate is feasible. */
int32_t hapmoe_best_plan(const hapmoe_problem *p, const hapmoe_candidate *d_cand,
                         const void *d_tables, int64_t tables_bytes,
                         const hapmoe_dp_result *d_res, const uint8_t *d_types, int64_t n,
                         int64_t *d_config_best, void *d_ws, int64_t ws_bytes,
                         hapmoe_plan *h_plan, void *stream);

/* hapmoe_best_plan without a caller workspace, for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, outputs and errors as
 * hapmoe_best_plan minus d_ws / ws_bytes: the workspace is a fixed array of
 * HAPMOE_BEST_PLAN_SCRATCH_BYTES in the library's device image, which each GPU
 * holds until the process ends.  A problem whose hapmoe_best_plan_ws_bytes(p, n)
 * exceeds it is HAPMOE_E_WORKSPACE (checked before any device work).  The call
 * allocates nothing; nothing in the array has to start at zero.  Every call on
 * one GPU shares that GPU's array, so calls that may overlap on one GPU (other
 * host threads, other streams) race and must be serialised by the caller.
 * Waits for `stream`, fills *h_plan. */
#define HAPMOE_BEST_PLAN_SCRATCH_BYTES 262144
int32_t hapmoe_best_plan_noalloc(const hapmoe_problem *p, const hapmoe_candidate *d_cand,
                                 const void *d_tables, int64_t tables_bytes,
                                 const hapmoe_dp_result *d_res, const uint8_t *d_types, int64_t n,
                                 int64_t *d_config_best, hapmoe_plan *h_plan, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* HAPMOE_H */
