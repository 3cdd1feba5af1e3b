/*
 * Sanitizer driver for the oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Built by the test-suite with AddressSanitizer and UndefinedBehaviorSanitizer
 * and run as a plain executable: it builds small seeded problems (inputs only,
 * a fixed linear congruential generator) and calls every oracle entry point on
 * every candidate, in the fixed-type, sequence and device-count modes, so that
 * an out-of-bounds access, a leak or undefined arithmetic anywhere in the
 * oracle fails the run.  Prints one line per problem; exit status 0 on success.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "hapmoe_oracle.h"

static uint64_t lcg_state;
static uint32_t next_u32(void)
{
    lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(lcg_state >> 33);
}
static int64_t uniform(int64_t lo, int64_t hi) { return lo + (int64_t)(next_u32() % (uint32_t)(hi - lo + 1)); }

typedef struct arrays {
    uint8_t is_moe[16];
    int64_t tokens[16 * 8], pd[16], pe[16], act[16];
    int64_t td[4 * 16 * 16], tf[4 * 16 * 16];
} arrays;

static void make_problem(orc_problem *p, arrays *A, uint64_t seed, int n_layers, int n_types, const int *count,
                         int stage_types)
{
    lcg_state = seed;
    memset(p, 0, sizeof(*p));
    memset(A, 0, sizeof(*A));
    int E = 8;
    p->n_layers = n_layers;
    p->seq_len = 1024;
    p->hidden = 512;
    p->n_experts = E;
    p->top_k = 2;
    p->micro_batch_size = 1;
    p->elem_bytes = 2;
    p->moe_ffn_mult = 2.0;
    for (int l = 0; l < n_layers; l++) {
        A->is_moe[l] = (uint8_t)(l % 3 != 0);
        for (int e = 0; e < E; e++) A->tokens[l * E + e] = A->is_moe[l] ? uniform(10, 600) : 0;
        A->pd[l] = uniform(1000000, 30000000);
        A->pe[l] = A->is_moe[l] ? uniform(1000000, 90000000) : 0;
        A->act[l] = uniform(10000000, 900000000);
    }
    p->n_types = n_types;
    for (int h = 0; h < n_types; h++) {
        p->count[h] = count[h];
        p->speed[h] = (int32_t)uniform(60, 250);
        p->mem_bytes[h] = uniform(2, 30) * 1000000000ll;
        p->eff[h] = 0.5 + 0.1 * (double)h;
        p->route_coef[h] = 1e-5;
        for (int g = 0; g < n_types; g++) {
            p->bw[h * ORC_MAX_TYPES + g] = h == g ? 400.0 : (double)uniform(20, 80);
            p->alpha[h * ORC_MAX_TYPES + g] = h == g ? 5000.0 : 20000.0;
        }
        for (int i = 0; i < 16 * n_layers; i++) {
            int64_t d = uniform(2000, 200000);
            A->td[h * 16 * n_layers + i] = d;
            A->tf[h * 16 * n_layers + i] = d / 2;
        }
    }
    p->is_moe = A->is_moe;
    p->expert_tokens = A->tokens;
    p->params_dense = A->pd;
    p->params_expert = A->pe;
    p->act_bytes = A->act;
    p->t_dense = A->td;
    p->t_ffn = A->tf;
    p->gamma = 0.5;
    p->rc_time = 1.33;
    p->rc_act = 0.4;
    p->opt_coef = 0.01;
    p->delta_num = 1;
    p->delta_den = 5;
    p->eta_prune = 2;
    p->prune_window = (int32_t)(seed % 3);
    p->prune_hetero = 1;
    p->allow_recompute = 1;
    p->pp_max = 4;
    p->tp_mask = 0xF;
    p->cp_mask = 0xF;
    p->ep_max = 8;
    p->tpe_mask = 0xF;
    p->mode = 0;
    p->stage_types = stage_types;
    p->n_micro = 3;
    p->micro[0] = 1;
    p->micro[1] = 2;
    p->micro[2] = 8;
}

static int run_problem(const orc_problem *p, const char *name)
{
    if (orc_validate(p)) {
        printf("%s: invalid\n", name);
        return 1;
    }
    int64_t n = orc_n_instances(p), feasible = 0;
    int W = p->n_layers + 1, T = p->n_types;
    int64_t ncfg = orc_enumerate(p, NULL, 0);
    orc_config *cfgs = malloc(sizeof(orc_config) * (size_t)(ncfg > 0 ? ncfg : 1));
    orc_enumerate(p, cfgs, ncfg);
    int64_t *cost = malloc(sizeof(int64_t) * (size_t)ORC_MAX_STAGES * (T + 1) * T * W * W);
    uint8_t *rf = malloc((size_t)ORC_MAX_STAGES * (T + 1) * T * W * W);
    const int widths = p->stage_types == 3;
    int64_t *wcost = malloc(sizeof(int64_t) * (size_t)p->pp_max * (2 * p->pp_max + 1) * 3 * W * W);
    uint8_t *wrf = malloc((size_t)p->pp_max * (2 * p->pp_max + 1) * 3 * W * W);
    for (int64_t i = 0; i < n; i++) {
        orc_result a, b, c, d;
        if (orc_solve(p, i, &a) || orc_solve_brute(p, i, &b) ||
            (!widths && (orc_solve_exact(p, i, &c) || orc_solve_exact_brute(p, i, &d)))) {
            printf("%s: solve failed at %lld\n", name, (long long)i);
            return 1;
        }
        if (a.status != b.status || a.opt != b.opt || (!widths && (c.status != d.status || c.opt != d.opt))) {
            printf("%s: dp and brute force differ at %lld\n", name, (long long)i);
            return 1;
        }
        if (p->stage_types == 0) {   /* the least 1F1B latency and its brute force */
            if (orc_solve_latency(p, i, &c) || orc_solve_latency_brute(p, i, &d) || c.status != d.status ||
                c.opt != d.opt) {
                printf("%s: least latency differs at %lld\n", name, (long long)i);
                return 1;
            }
        }
        feasible += a.status == 0;
        if (p->stage_types == 2)
            orc_type_costs(p, i, cost, rf);
        else if (widths)
            orc_width_costs(p, i, wcost, wrf);
        else
            orc_segment_costs(p, i, cost, rf);
    }
    free(wcost);
    free(wrf);
    for (int64_t k = 0; k < ncfg; k++) {
        orc_pi_terms pt;
        orc_pi_terms_eval(p, &cfgs[k], &pt);
        for (int o = 0; o < orc_n_orders(p); o++) {
            orc_stage st[ORC_MAX_STAGES];
            orc_stages(p, &cfgs[k], o, 2, st);
            (void)orc_dp_const(p, &cfgs[k], o);
        }
        for (int l = 0; l < p->n_layers; l++) {
            orc_mem_terms mt;
            orc_mem_terms_eval(p, &cfgs[k], l, &mt);
            for (int h = 0; h < T; h++) {
                orc_type_terms tt;
                orc_type_terms_eval(p, &cfgs[k], l, h, &tt);
            }
            for (int m = 1; m < (1 << T); m++) {
                orc_mask_terms mk;
                orc_mask_terms_eval(p, &cfgs[k], l, m, &mk);
            }
        }
    }
    free(cost);
    free(rf);
    free(cfgs);
    printf("%s: %lld candidates, %lld feasible, dp = brute force\n", name, (long long)n, (long long)feasible);
    return 0;
}

int main(void)
{
    static const int c2[2] = {2, 2}, c3[3] = {2, 1, 1}, c1[1] = {4};
    arrays A;
    orc_problem p;
    int bad = 0;
    for (int seed = 1; seed <= 3; seed++)
        for (int mode = 0; mode <= 3; mode++) {
            char name[64];
            snprintf(name, sizeof(name), "two types, seed %d, stage_types %d", seed, mode);
            make_problem(&p, &A, (uint64_t)seed, 6, 2, c2, mode);
            bad |= run_problem(&p, name);
            snprintf(name, sizeof(name), "three types, seed %d, stage_types %d", seed, mode);
            make_problem(&p, &A, (uint64_t)seed + 10, 5, 3, c3, mode);
            bad |= run_problem(&p, name);
        }
    make_problem(&p, &A, 7, 7, 1, c1, 0);
    bad |= run_problem(&p, "one type");
    return bad;
}
