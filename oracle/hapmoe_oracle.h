/*
 * Reference oracle for the HAPMoE planner hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU implementation of what the planner
 * computes: the 6D candidate enumeration, the MoE-aware per-layer cost model
 * (Section 3.2: Eq. 2 compute, Eq. 3 dispatch volume, the load-imbalance
 * factor, the stage memory model), the stage constants (Section 3.3: the 1F1B
 * iteration model, Eq. 4), the three prunings of Section 3.4, and the stage
 * DP of Section 3.4 / Algorithm 1 in its threshold form
 *     minimise  sum_i c_i + (B-1) * max_i c_i  over layer partitions,
 * solved by sweeping every distinct stage cost ascending as the threshold.
 *
 * A second objective re-scores the partitions of the (max, sum) Pareto frontier
 * with the 1F1B iteration latency of the appendix (the steady-state term with
 * the bottleneck stage's position, Eq. 4 and its appendix expansion); see
 * orc_dp_exact for the readings it takes.
 *
 * Only the test-suite, the smoke check and the CPU-baseline leg of the bench
 * may load this code.  It shares no code, header or table with the HIP library
 * and reads its own flat problem struct.  Everything is fp64 with IEEE
 * + - * / and ceil only, compiled with -ffp-contract=off.
 *
 * Parity status: the enumeration, the cost-model closed forms and the DP are
 * pinned by tests against hand-worked values, closed forms, invariants and
 * brute force.  The absolute accuracy of the modelled latencies against real
 * hardware is parity unpinned (the paper's profiled tables are not available).
 */
#ifndef HAPMOE_ORACLE_H
#define HAPMOE_ORACLE_H
#include <stdint.h>

#define ORC_MAX_TYPES 4
#define ORC_MAX_STAGES 64
#define ORC_MAX_MICRO 64
#define ORC_INF INT64_MAX

/* Flat problem description (Section 3.1 "Input"). */
typedef struct orc_problem {
    /* model parameters (N, S, H, E, k) and training hyper-parameters */
    int32_t n_layers, seq_len, hidden, n_experts, top_k, micro_batch_size, elem_bytes;
    double moe_ffn_mult;             /* the factor 2 of Eq. 2 (top-k x expert/FFN size) */
    const uint8_t *is_moe;           /* [N] */
    const int64_t *expert_tokens;    /* [N][E] router statistics |T_e| */
    const int64_t *params_dense;     /* [N] non-expert parameters of each layer */
    const int64_t *params_expert;    /* [N] parameters of all experts of each layer */
    const int64_t *act_bytes;        /* [N] activation bytes of one micro-batch, TP=CP=1 */
    /* hardware inventory {m_h}, (P_h, C_h, B_h) */
    int32_t n_types;
    int32_t count[ORC_MAX_TYPES];
    int32_t speed[ORC_MAX_TYPES];
    int64_t mem_bytes[ORC_MAX_TYPES];
    double eff[ORC_MAX_TYPES];        /* eta_h of Eq. 2 */
    double route_coef[ORC_MAX_TYPES]; /* router ns per (token x hidden) */
    double bw[ORC_MAX_TYPES * ORC_MAX_TYPES];     /* bytes per ns, [h][h'] */
    double alpha[ORC_MAX_TYPES * ORC_MAX_TYPES];  /* ns, [h][h'] */
    const int64_t *t_dense;          /* [T][4 tp][4 cp][N] ns */
    const int64_t *t_ffn;            /* [T][4 tp][4 cp][N] ns */
    /* method parameters */
    double gamma, rc_time, rc_act, opt_coef;
    int32_t delta_num, delta_den, eta_prune;
    int32_t prune_window;          /* 0 none, 1 pruning-1 windows, 2 uniform floor/ceil(N/PP) */
    int32_t prune_hetero, allow_recompute;
    /* search space */
    int32_t pp_max, tp_mask, cp_mask, ep_max, tpe_mask, mode;
    int32_t stage_types;           /* 0: block orderings of the types; 1: free per-stage type, one
                                      candidate per stage-type sequence; 2: free per-stage type
                                      chosen by the DP over device counts (one order slot);
                                      3: block orderings with per-stage data-parallel widths
                                      chosen by the DP (w_i half-groups, w_i in {1, 2, 3}) */
    int32_t n_micro;
    int32_t micro[ORC_MAX_MICRO];
} orc_problem;

typedef struct orc_config { int32_t pp, tp, cp, dp, ep, tpe; } orc_config;

/* one pipeline stage of an instance (device layout, Section 3.4) */
typedef struct orc_stage {
    int32_t mask;          /* device types present in the stage */
    int32_t speed;         /* min P_h over the stage */
    int32_t lo, hi;        /* load-balance window on n_i (pruning 1) */
    int32_t mixed;         /* more than one device type in the stage */
    int32_t bdiff;         /* next stage starts on another device type */
    int32_t first_type, last_type;
    int64_t cap;           /* min C_h over the stage */
    int64_t p2p;           /* inter-stage activation + gradient transfer, 0 for the last */
    int64_t m_store;       /* micro-batches whose activations the stage keeps (1F1B) */
    double alpha, bw;      /* max latency / min bandwidth over type pairs of the stage */
} orc_stage;

typedef struct orc_type_terms {
    double comp, expert;           /* fp64 before rounding */
    int64_t q_comp, q_expert;
} orc_type_terms;

typedef struct orc_mask_terms {
    double a2a, tp, cp;            /* fp64 before rounding */
    int64_t q_a2a, q_tp, q_cp;
    int64_t comm, t_r0, t_r1;      /* comm = sum of rounded terms; stage times, r = 0 / 1 */
} orc_mask_terms;

typedef struct orc_mem_terms {
    double w, a0;                  /* fp64 before rounding */
    int64_t q_w, q_a0, q_a1;
} orc_mem_terms;

typedef struct orc_pi_terms {
    double p_avg, dp_const_f, x_f;
    int64_t x_bytes;               /* MoE dispatch/combine buffers + routing metadata */
    int64_t tbar;                  /* mean per-stage compute bound used by pruning 3 */
} orc_pi_terms;

typedef struct orc_result {
    int32_t status;                /* 0 = feasible, 1 = infeasible */
    int32_t pp;
    int64_t opt, sum, tmax, dp_const;
    int64_t thresholds;            /* thresholds swept */
    uint8_t layers[ORC_MAX_STAGES];
    uint8_t recompute[ORC_MAX_STAGES];
    uint8_t stage_mask[ORC_MAX_STAGES];
    uint8_t width[ORC_MAX_STAGES];   /* per-stage widths (stage_types = 3): half-groups of stage i */
} orc_result;

int32_t orc_validate(const orc_problem *p);
int64_t orc_enumerate(const orc_problem *p, orc_config *out, int64_t cap);
int32_t orc_n_orders(const orc_problem *p);
/* Free per-stage types: the o-th stage-type sequence of a pipeline of pp
 * stages (lexicographic over the distinct arrangements of the multiset with
 * m_h / (G / pp) stages of type h); -1 if o is past the last one. */
int32_t orc_sequence(const orc_problem *p, int32_t pp, int32_t o, int32_t *seq);
void orc_order(const orc_problem *p, int32_t o, int32_t *perm);
int64_t orc_n_instances(const orc_problem *p);
int32_t orc_instance(const orc_problem *p, int64_t idx, orc_config *cfg, int32_t *order, int32_t *micro);

void orc_type_terms_eval(const orc_problem *p, const orc_config *c, int32_t layer, int32_t h, orc_type_terms *o);
void orc_mask_terms_eval(const orc_problem *p, const orc_config *c, int32_t layer, int32_t mask, orc_mask_terms *o);
void orc_mem_terms_eval(const orc_problem *p, const orc_config *c, int32_t layer, orc_mem_terms *o);
void orc_pi_terms_eval(const orc_problem *p, const orc_config *c, orc_pi_terms *o);
int64_t orc_p2p(const orc_problem *p, const orc_config *c, int32_t h_from, int32_t h_to);
int64_t orc_dp_const(const orc_problem *p, const orc_config *c, int32_t order);
int32_t orc_stages(const orc_problem *p, const orc_config *c, int32_t order, int32_t micro, orc_stage *st);

/* segment costs of an instance: cost[i][a][b] (INF = infeasible), rflag[i][a][b] */
int32_t orc_segment_costs(const orc_problem *p, int64_t idx, int64_t *cost, uint8_t *rflag);

/* DP core on an explicit cost tensor [pp][n+1][n+1] */
int32_t orc_dp(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r);
int32_t orc_brute(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r);

int32_t orc_solve(const orc_problem *p, int64_t idx, orc_result *r);
int32_t orc_solve_many(const orc_problem *p, const int64_t *idx, int64_t n, orc_result *r);
int32_t orc_solve_brute(const orc_problem *p, int64_t idx, orc_result *r);

/* 1F1B iteration latency of a partition given its stage costs c[0..pp): with
 * t_f = ceil(c/3), t_b = c - t_f and s the first (1-based) stage of largest c,
 *   T = sum c + sum_{i <= s} t_f,i + max(0, B - s - 1) * max c. */
int64_t orc_latency_1f1b(int32_t pp, const int64_t *c, int64_t micro);
/* Exact re-scoring over the (max, sum) Pareto frontier: r->opt = least T, ties
 * to the lower max; r->sum / r->tmax / layers describe the chosen point's
 * canonical partition (the threshold DP's back-trace at t = its max);
 * r->thresholds = frontier points scored. */
int32_t orc_dp_exact(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r);
int32_t orc_brute_exact(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r);
int32_t orc_solve_exact(const orc_problem *p, int64_t idx, orc_result *r);
int32_t orc_solve_exact_many(const orc_problem *p, const int64_t *idx, int64_t n, orc_result *r);
int32_t orc_solve_exact_brute(const orc_problem *p, int64_t idx, orc_result *r);

/* Per-stage data-parallel widths (stage_types = 3): cost tensor
 * [pp][2pp + 1][3][n + 1][n + 1], entry (s, u, w - 1, a, b) = the cost of stage
 * s on half-groups [u, u + w) and layers [a, b); the threshold DP over (stage,
 * end layer, half-groups used) and its brute force over every width sequence
 * and composition; r->width gets w_i. */
int32_t orc_width_costs(const orc_problem *p, int64_t idx, int64_t *cost, uint8_t *rflag);
/* the width-w terms of one layer (type_out[T]) and the layout of a width stage */
void orc_width_terms(const orc_problem *p, const orc_config *c, int32_t layer, int32_t mask, int32_t w,
                     orc_type_terms *type_out, orc_mask_terms *mask_out, orc_mem_terms *mem_out, int64_t *x_bytes);
int32_t orc_width_stage(const orc_problem *p, const orc_config *c, int32_t order, int32_t s, int32_t u, int32_t w,
                        int32_t micro, orc_stage *x);
int32_t orc_dp_widths(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r);
int32_t orc_brute_widths(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r);

/* The least 1F1B latency over every partition (not only the frontier's): r->opt
 * = least orc_latency_1f1b, ties to the lower largest stage, then the
 * lexicographically smallest (b_{pp-1}, ..., b_1); r->thresholds = thresholds
 * swept (orc_dp_latency) or compositions scored (orc_brute_latency). */
int32_t orc_dp_latency(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r);
int32_t orc_brute_latency(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r);
int32_t orc_solve_latency(const orc_problem *p, int64_t idx, orc_result *r);
int32_t orc_solve_latency_brute(const orc_problem *p, int64_t idx, orc_result *r);
int32_t orc_solve_latency_many(const orc_problem *p, const int64_t *idx, int64_t n, orc_result *r);

/* Free per-stage device types by the DP over device counts (stage_types = 2):
 * cost tensor [pp][T][T + 1][n + 1][n + 1], entry (s, h, h', a, b) = the cost
 * of a type-h stage s on layers [a, b) followed by a type-h' stage (h' = T:
 * the last stage); k[h] = stages of type h.  r->stage_mask gets 1 << h_i. */
int32_t orc_type_costs(const orc_problem *p, int64_t idx, int64_t *cost, uint8_t *rflag);
int32_t orc_dp_types(int32_t pp, int32_t T, const int32_t *k, int32_t n, int64_t micro, const int64_t *cost,
                     orc_result *r);
int32_t orc_brute_types(int32_t pp, int32_t T, const int32_t *k, int32_t n, int64_t micro, const int64_t *cost,
                        orc_result *r);
/* ... and its 1F1B re-scoring of the (max, sum) frontier (as orc_dp_exact) */
int32_t orc_dp_types_exact(int32_t pp, int32_t T, const int32_t *k, int32_t n, int64_t micro, const int64_t *cost,
                           orc_result *r);
int32_t orc_brute_types_exact(int32_t pp, int32_t T, const int32_t *k, int32_t n, int64_t micro,
                              const int64_t *cost, orc_result *r);

#endif
