/*
 * Reference oracle for the HAPMoE planner hot path -- TEST INFRASTRUCTURE ONLY.
 * (Only tests, the smoke check and the bench's CPU-baseline leg use it.)
 *
 * Plain single-threaded C, fp64, IEEE + - * / and ceil only; build with
 * -O2 -ffp-contract=off -fno-fast-math.  Each function names the passage of the
 * paper it restates.  Readings of passages the paper leaves open are listed in
 * the design notes of the repository and restated next to the code here.
 */
#include "hapmoe_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

static int64_t q(double x) { return (int64_t)ceil(x); }   /* ns / bytes are whole numbers, rounded up */
static int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }
static int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }
static int lg2(int v) { int r = 0; while ((1 << r) < v) r++; return r; }
static int popc(int v) { int c = 0; while (v) { c += v & 1; v >>= 1; } return c; }
/* free per-stage device types (stage_types 1 and 2): every stage one type's group */
static int free_types(const orc_problem *p) { return p->stage_types == 1 || p->stage_types == 2; }

int32_t orc_validate(const orc_problem *p)
{
    int N = p->n_layers, T = p->n_types;
    if (N < 1 || N > 255 || T < 1 || T > ORC_MAX_TYPES) return -1;
    if (p->seq_len < 1 || p->hidden < 1 || p->micro_batch_size < 1 || p->elem_bytes < 0) return -1;
    if (p->n_experts < 0 || (p->n_experts > 0 && (p->top_k < 1 || p->top_k > p->n_experts))) return -1;
    for (int l = 0; l < N; l++)
        if (p->is_moe[l] && p->n_experts == 0) return -1;
    for (int h = 0; h < T; h++) {
        if (p->count[h] < 1 || p->speed[h] < 1 || p->mem_bytes[h] < 0 || !(p->eff[h] > 0.0)) return -1;
        if (!(p->route_coef[h] >= 0.0)) return -1;
        for (int g = 0; g < T; g++)
            if (!(p->bw[h * ORC_MAX_TYPES + g] > 0.0) || !(p->alpha[h * ORC_MAX_TYPES + g] >= 0.0)) return -1;
    }
    for (int64_t i = 0; i < (int64_t)T * 16 * N; i++)
        if (p->t_ffn[i] < 0 || p->t_ffn[i] > p->t_dense[i]) return -1;
    if (!(p->rc_time >= 1.0) || !(p->rc_act >= 0.0 && p->rc_act <= 1.0)) return -1;
    if (!(p->gamma >= 0.0 && p->gamma <= 1.0) || !(p->opt_coef >= 0.0) || !(p->moe_ffn_mult >= 0.0)) return -1;
    if (p->delta_den < 1 || p->delta_num < 0 || p->delta_num >= p->delta_den || p->eta_prune < 0) return -1;
    if (p->prune_window < 0 || p->prune_window > 2) return -1;
    if (p->n_micro < 1 || p->n_micro > ORC_MAX_MICRO) return -1;
    if (p->pp_max < 1 || p->pp_max > ORC_MAX_STAGES || p->mode < 0 || p->mode > 1) return -1;
    if (p->stage_types < 0 || p->stage_types > 3) return -1;
    for (int i = 0; i < p->n_micro; i++)
        if (p->micro[i] < 1 || p->micro[i] > (1 << 20)) return -1;
    return 0;
}

/* ------------------------------------------------------------------------
 * Candidate set.  Section 3.1 output pi = (PP, TP, DP, EP, TPE, CP); the
 * search of Section 3.4 / Algorithm 1 runs over a configuration set Pi.
 * Reading: every stage is a group of G/PP devices (G = sum_h m_h); TP and CP
 * split a stage group, DP = group / (TP*CP); the expert dimensions fold
 * inside the group (EP*TPE divides it).  mode 1 instead takes the literal
 * product PP*DP*TP*CP*EP*TPE = G.  Dense models use EP = TPE = 1.
 * Loop order PP, TP, CP, EP, TPE ascending; candidate index
 * ((config * n_orders) + order) * n_micro + micro_index.
 * ---------------------------------------------------------------------- */
int64_t orc_enumerate(const orc_problem *p, orc_config *out, int64_t cap)
{
    int G = 0;
    for (int h = 0; h < p->n_types; h++) G += p->count[h];
    int dense = (p->n_experts == 0);
    int64_t n = 0;
    for (int PP = 1; PP <= G; PP++) {
        if (G % PP != 0 || PP > p->pp_max || PP > p->n_layers) continue;
        int g = G / PP;
        if (free_types(p)) {   /* free per-stage type: every stage is one type's group */
            int whole = 1;
            for (int h = 0; h < p->n_types; h++) whole &= p->count[h] % g == 0;
            if (!whole) continue;
        }
        for (int i = 0; i < 4; i++) {
            int TP = 1 << i;
            if (!((p->tp_mask >> i) & 1) || g % TP != 0 || p->hidden % TP != 0) continue;
            for (int j = 0; j < 4; j++) {
                int CP = 1 << j;
                if (!((p->cp_mask >> j) & 1) || p->seq_len % CP != 0) continue;
                for (int EP = 1; EP <= (dense ? 1 : p->ep_max); EP *= 2) {
                    if (!dense && p->n_experts % EP != 0) continue;
                    for (int m = 0; m < 4; m++) {
                        int TPE = 1 << m;
                        if (dense ? (TPE != 1) : !((p->tpe_mask >> m) & 1)) continue;
                        int DP;
                        if (p->mode == 0) {
                            if (g % (TP * CP) != 0 || g % (EP * TPE) != 0) continue;
                            DP = g / (TP * CP);
                        } else {
                            int prod = TP * CP * EP * TPE;
                            if (g % prod != 0) continue;
                            DP = g / prod;
                        }
                        /* per-stage widths: half a group must hold whole replicas and
                         * whole expert groups (DP even, EP * TPE | g / 2) */
                        if (p->stage_types == 3 && (DP % 2 != 0 || (g / 2) % (EP * TPE) != 0)) continue;
                        if (out && n < cap) {
                            orc_config c = {PP, TP, CP, DP, EP, TPE};
                            out[n] = c;
                        }
                        n++;
                    }
                }
            }
        }
    }
    return n;
}

/* number of distinct stage-type sequences of a pp-stage pipeline: the
 * multinomial pp! / prod_h k_h! with k_h = m_h / g, built one stage at a time
 * (each step multiplies by r / i >= 1, so it never falls); capped at INT32_MAX */
static int64_t n_sequences(const orc_problem *p, int pp)
{
    int G = 0;
    for (int h = 0; h < p->n_types; h++) G += p->count[h];
    int g = G / pp, r = 0;
    int64_t n = 1;
    for (int h = 0; h < p->n_types; h++)
        for (int i = 1; i <= p->count[h] / g; i++) {
            r++;
            n = n * r / i;
            if (n > INT32_MAX) return INT32_MAX;
        }
    return n;
}

/* Device-type orderings: all permutations of the type indices, lexicographic;
 * with free per-stage types, the largest number of stage-type sequences over
 * the configurations (a configuration with fewer has empty slots). */
int32_t orc_n_orders(const orc_problem *p)
{
    if (p->stage_types == 2) return 1;   /* the DP over device counts picks the sequence */
    if (p->stage_types == 1) {
        int64_t ncfg = orc_enumerate(p, NULL, 0), best = 1;
        orc_config *all = (orc_config *)malloc(sizeof(orc_config) * (size_t)(ncfg > 0 ? ncfg : 1));
        orc_enumerate(p, all, ncfg);
        for (int64_t i = 0; i < ncfg; i++) {
            int64_t n = n_sequences(p, all[i].pp);
            if (n > best) best = n;
        }
        free(all);
        return (int32_t)best;
    }
    int f = 1;
    for (int i = 2; i <= p->n_types; i++) f *= i;
    return f;
}

/* next arrangement of a multiset in lexicographic order; 0 after the last */
static int next_arrangement(int32_t *v, int n)
{
    int i = n - 2;
    while (i >= 0 && v[i] >= v[i + 1]) i--;
    if (i < 0) return 0;
    int j = n - 1;
    while (v[j] <= v[i]) j--;
    int32_t t = v[i];
    v[i] = v[j];
    v[j] = t;
    for (int a = i + 1, b = n - 1; a < b; a++, b--) {
        t = v[a];
        v[a] = v[b];
        v[b] = t;
    }
    return 1;
}

int32_t orc_sequence(const orc_problem *p, int32_t pp, int32_t o, int32_t *seq)
{
    int G = 0;
    for (int h = 0; h < p->n_types; h++) G += p->count[h];
    int g = G / pp, k = 0;
    for (int h = 0; h < p->n_types; h++)
        for (int i = 0; i < p->count[h] / g; i++) seq[k++] = h;
    for (int32_t i = 0; i < o; i++)
        if (!next_arrangement(seq, pp)) return -1;
    return 0;
}

void orc_order(const orc_problem *p, int32_t o, int32_t *perm)
{
    /* o-th permutation in lexicographic order (factorial number system) */
    int T = p->n_types, used[ORC_MAX_TYPES] = {0};
    int fact = orc_n_orders(p);
    for (int pos = 0; pos < T; pos++) {
        fact /= (T - pos);
        int k = o / fact;
        o %= fact;
        for (int h = 0; h < T; h++) {
            if (used[h]) continue;
            if (k == 0) { perm[pos] = h; used[h] = 1; break; }
            k--;
        }
    }
}

int64_t orc_n_instances(const orc_problem *p)
{
    return orc_enumerate(p, NULL, 0) * orc_n_orders(p) * p->n_micro;
}

int32_t orc_instance(const orc_problem *p, int64_t idx, orc_config *cfg, int32_t *order, int32_t *micro)
{
    int64_t ncfg = orc_enumerate(p, NULL, 0);
    int64_t per = (int64_t)orc_n_orders(p) * p->n_micro;
    if (idx < 0 || idx >= ncfg * per) return -1;
    orc_config *all = (orc_config *)malloc(sizeof(orc_config) * (size_t)ncfg);
    orc_enumerate(p, all, ncfg);
    *cfg = all[idx / per];
    free(all);
    *order = (int32_t)((idx / p->n_micro) % orc_n_orders(p));
    *micro = p->micro[idx % p->n_micro];
    return 0;
}

/* ------------------------------------------------------------------------
 * Link model.  Section 3.2: collective time is a primitive-specific function
 * of (bytes, world, link type).  Reading: an alpha-beta model per pair of
 * device types; a group spanning several types runs at the slowest pair
 * (largest latency, smallest bandwidth).  Ring all-reduce over w ranks moves
 * 2(w-1)/w of the buffer in 2(w-1) steps.
 * ---------------------------------------------------------------------- */
static void mask_link(const orc_problem *p, int mask, double *alpha, double *bw)
{
    double a = 0.0, b = 0.0;
    int first = 1;
    for (int h = 0; h < p->n_types; h++) {
        if (!((mask >> h) & 1)) continue;
        for (int g = 0; g < p->n_types; g++) {
            if (!((mask >> g) & 1)) continue;
            double al = p->alpha[h * ORC_MAX_TYPES + g], bb = p->bw[h * ORC_MAX_TYPES + g];
            if (first || al > a) a = al;
            if (first || bb < b) b = bb;
            first = 0;
        }
    }
    *alpha = a;
    *bw = b;
}

static double ring_allreduce(double bytes, int w, double alpha, double bw)
{
    if (w == 1) return 0.0;
    double steps = (double)(2 * (w - 1));
    return steps * alpha + ((steps * bytes) / (double)w) / bw;
}

/* tokens per rank of one micro-batch: S * micro_batch_size / CP */
static double tokens(const orc_problem *p, const orc_config *c)
{
    return (double)((int64_t)p->seq_len * p->micro_batch_size / c->cp);
}

/* activation bytes of one micro-batch on one rank: tokens * H * beta */
static double act_tensor(const orc_problem *p, const orc_config *c)
{
    return (tokens(p, c) * (double)p->hidden) * (double)p->elem_bytes;
}

/* Load-imbalance factor (Section 3.2): rho = max_e |T_e| / mean_e |T_e|,
 * applied as 1 + gamma (rho - 1). */
static double skew(const orc_problem *p, int layer)
{
    int E = p->n_experts;
    int64_t sum = 0, mx = 0;
    for (int e = 0; e < E; e++) {
        int64_t v = p->expert_tokens[(int64_t)layer * E + e];
        sum += v;
        if (v > mx) mx = v;
    }
    double rho = sum > 0 ? (double)(mx * E) / (double)sum : 1.0;
    return 1.0 + p->gamma * (rho - 1.0);
}

/* Eq. 2 (Section 3.2): per-layer compute on device type h,
 *   t = t_base - t_ffn + mult * t_ffn / (eta_h * EP * TPE) + t_route(h),
 * with t_route = route_coef_h * tokens * H and the expert part scaled by the
 * load-imbalance factor.  Dense layers take t_base from the table. */
void orc_type_terms_eval(const orc_problem *p, const orc_config *c, int32_t layer, int32_t h, orc_type_terms *o)
{
    int64_t off = (((int64_t)h * 4 + lg2(c->tp)) * 4 + lg2(c->cp)) * p->n_layers + layer;
    double td = (double)p->t_dense[off], tf = (double)p->t_ffn[off];
    if (!p->is_moe[layer]) {
        o->comp = td;
        o->expert = 0.0;
    } else {
        double route = p->route_coef[h] * (tokens(p, c) * (double)p->hidden);
        o->comp = (td - tf) + route;
        double xexp = (p->moe_ffn_mult * tf) / ((p->eff[h] * (double)c->ep) * (double)c->tpe);
        o->expert = skew(p, layer) * xexp;
    }
    o->q_comp = q(o->comp);
    o->q_expert = q(o->expert);
}

/* Communication of one layer on a stage whose devices span type set `mask`.
 *  - dispatch/combine (Eq. 3): D_moe = tokens * H * beta * k * (1 - 1/EP) per
 *    all-to-all; the all-gather dispatcher moves tokens * H * beta * (EP-1);
 *    the cheaper primitive is used (all-to-all on ties), 4 transfers per
 *    micro-batch (dispatch + combine, forward + backward), scaled by the
 *    load-imbalance factor (the MoE critical path);
 *  - TP: 4 ring all-reduces of the activation (2 for MoE layers, plus 2 over
 *    the TPE group);
 *  - CP: CP-1 ring steps exchanging K and V, forward + 2x backward. */
void orc_mask_terms_eval(const orc_problem *p, const orc_config *c, int32_t layer, int32_t mask, orc_mask_terms *o)
{
    double alpha, bw;
    mask_link(p, mask, &alpha, &bw);
    double D = act_tensor(p, c);
    if (!p->is_moe[layer]) {
        o->a2a = 0.0;
        o->tp = 4.0 * ring_allreduce(D, c->tp, alpha, bw);
    } else {
        double s = skew(p, layer);
        double dm = (D * (double)p->top_k) * (1.0 - 1.0 / (double)c->ep);
        double f_a2a = (double)(c->ep - 1) * alpha + dm / bw;
        double f_ag = (double)(c->ep - 1) * alpha + (D * (double)(c->ep - 1)) / bw;
        double sel = f_ag < f_a2a ? f_ag : f_a2a;
        o->a2a = s * (4.0 * sel);
        o->tp = 2.0 * ring_allreduce(D, c->tp, alpha, bw) + 2.0 * ring_allreduce(D, c->tpe, alpha, bw);
    }
    o->cp = c->cp == 1 ? 0.0 : 3.0 * ((double)(c->cp - 1) * (alpha + ((2.0 * D) / (double)c->tp) / bw));
    o->q_a2a = q(o->a2a);
    o->q_tp = q(o->tp);
    o->q_cp = q(o->cp);
    o->comm = o->q_a2a + o->q_tp + o->q_cp;
    /* a stage spanning several types runs at its slowest type */
    int64_t ce = -1;
    for (int h = 0; h < p->n_types; h++) {
        if (!((mask >> h) & 1)) continue;
        orc_type_terms t;
        orc_type_terms_eval(p, c, layer, h, &t);
        if (t.q_comp + t.q_expert > ce) ce = t.q_comp + t.q_expert;
    }
    o->t_r0 = ce + o->comm;
    o->t_r1 = q(p->rc_time * (double)o->t_r0);   /* recomputation: time x rc_time */
}

/* Stage memory model (Section 3.2): weights + gradients + optimizer states
 * sharded by (TP, DP, EP, TPE); ZeRO-1 bf16 training keeps 2 + 4 bytes per
 * parameter plus 12 bytes of fp32 optimizer state split over DP; activations
 * split by TP and CP, times xi(r) = rc_act under recomputation. */
void orc_mem_terms_eval(const orc_problem *p, const orc_config *c, int32_t layer, orc_mem_terms *o)
{
    double beta_opt = 6.0 + 12.0 / (double)c->dp;
    o->w = ((double)p->params_dense[layer] / (double)c->tp +
            (double)p->params_expert[layer] / (double)(c->ep * c->tpe)) * beta_opt;
    o->a0 = (double)p->act_bytes[layer] / (double)(c->tp * c->cp);
    o->q_w = q(o->w);
    o->q_a0 = q(o->a0);
    o->q_a1 = q(p->rc_act * (double)o->q_a0);
}

/* Per-configuration terms:
 *  - X: routing metadata (8 bytes per token and choice) plus the dispatch
 *    and combine buffers (2 D_moe), held once by a stage with an MoE layer;
 *  - tbar: mean compute per stage, ceil(sum_l max_h (comp + expert) / PP),
 *    the T_comp-bar of pruning 3 bounded independently of the partition;
 *  - p_avg: parameters per device, averaged over stages. */
void orc_pi_terms_eval(const orc_problem *p, const orc_config *c, orc_pi_terms *o)
{
    int64_t pd = 0, pe = 0;
    for (int l = 0; l < p->n_layers; l++) {
        pd += p->params_dense[l];
        pe += p->params_expert[l];
    }
    o->p_avg = ((double)pd / (double)c->tp + (double)pe / (double)(c->ep * c->tpe)) / (double)c->pp;
    double D = act_tensor(p, c);
    double dm = (D * (double)p->top_k) * (1.0 - 1.0 / (double)c->ep);
    o->x_f = ((8.0 * tokens(p, c)) * (double)p->top_k) + 2.0 * dm;
    o->x_bytes = q(o->x_f);
    int64_t s = 0;
    for (int l = 0; l < p->n_layers; l++) {
        int64_t m = 0;
        for (int h = 0; h < p->n_types; h++) {
            orc_type_terms t;
            orc_type_terms_eval(p, c, l, h, &t);
            m = max64(m, t.q_comp + t.q_expert);
        }
        s += m;
    }
    o->tbar = (s + c->pp - 1) / c->pp;
    o->dp_const_f = 0.0;
}

/* T_comm(h, h', k, j) of the DP transition (Section 3.4): the activation sent
 * forward and its gradient sent back between adjacent stages, one message of
 * tokens * H * beta / TP bytes each way over the boundary link. */
int64_t orc_p2p(const orc_problem *p, const orc_config *c, int32_t h_from, int32_t h_to)
{
    double al = p->alpha[h_from * ORC_MAX_TYPES + h_to], bw = p->bw[h_from * ORC_MAX_TYPES + h_to];
    return q(2.0 * (al + (act_tensor(p, c) / (double)c->tp) / bw));
}

/* device type of device d under an ordering */
static int dev_type(const orc_problem *p, const int *perm, int d)
{
    int start = 0;
    for (int j = 0; j < p->n_types; j++) {
        int h = perm[j];
        if (d < start + p->count[h]) return h;
        start += p->count[h];
    }
    return perm[p->n_types - 1];
}

/* Device layout of a (configuration, ordering): the devices are listed type by
 * type in the ordering (m_h devices each) and stage i takes the i-th group of
 * G/PP consecutive devices.  This fixes {h_i} per candidate (the state m of
 * the DP of Section 3.4 is enumerated through the orderings instead). */
int32_t orc_stages(const orc_problem *p, const orc_config *c, int32_t order, int32_t micro, orc_stage *st)
{
    int perm[ORC_MAX_TYPES];
    int32_t seq[ORC_MAX_STAGES];
    if (free_types(p)) {   /* free per-stage type: stage s is one group of type seq[s] */
        if (orc_sequence(p, c->pp, order, seq)) return -1;
    } else {
        orc_order(p, order, perm);
    }
    int G = 0;
    for (int h = 0; h < p->n_types; h++) G += p->count[h];
    int PP = c->pp, g = G / PP;
    int64_t sum_speed = 0;
    for (int s = 0; s < PP; s++) {
        orc_stage *x = &st[s];
        int lo = s * g, hi = lo + g;
        x->mask = 0;
        if (free_types(p)) {
            x->mask = 1 << seq[s];
            x->first_type = x->last_type = seq[s];
        } else {
            for (int d = lo; d < hi; d++) x->mask |= 1 << dev_type(p, perm, d);
            x->first_type = dev_type(p, perm, lo);
            x->last_type = dev_type(p, perm, hi - 1);
        }
        x->cap = -1;
        x->speed = 0;
        for (int h = 0; h < p->n_types; h++) {
            if (!((x->mask >> h) & 1)) continue;
            if (x->cap < 0 || p->mem_bytes[h] < x->cap) x->cap = p->mem_bytes[h];
            if (x->speed == 0 || p->speed[h] < x->speed) x->speed = p->speed[h];
        }
        mask_link(p, x->mask, &x->alpha, &x->bw);
        x->mixed = popc(x->mask) > 1;
        if (s < PP - 1) {
            int nt = free_types(p) ? seq[s + 1] : dev_type(p, perm, hi);
            x->bdiff = nt != x->last_type;
            x->p2p = orc_p2p(p, c, x->last_type, nt);
        } else {
            x->bdiff = 0;
            x->p2p = 0;
        }
        /* 1F1B: stage i (1-based) holds the activations of PP - i + 1 micro-batches */
        x->m_store = min64(PP - s, micro);
        sum_speed += x->speed;
    }
    /* Pruning 1 (Section 3.4): n_i within [(1-delta) w_i N, (1+delta) w_i N],
     * w_i = the stage's share of the summed stage speeds; integer floor / ceil. */
    int64_t dn = p->delta_num, dd = p->delta_den, N = p->n_layers;
    for (int s = 0; s < PP; s++) {
        if (!p->prune_window) {
            st[s].lo = 1;
            st[s].hi = (int32_t)N;
            continue;
        }
        if (p->prune_window == 2) {   /* uniform assignment (the ablation): floor / ceil of N / PP */
            st[s].lo = (int32_t)(N / PP);
            st[s].hi = (int32_t)((N + PP - 1) / PP);
            continue;
        }
        int64_t den = dd * sum_speed;
        int64_t lo = ((dd - dn) * st[s].speed * N) / den;
        int64_t hi = ((dd + dn) * st[s].speed * N + den - 1) / den;
        st[s].lo = (int32_t)max64(1, lo);
        st[s].hi = (int32_t)min64(N, hi);
    }
    return 0;
}

/* T_dp-sync + T_opt of Eq. 4: a ring all-reduce of fp32 gradients over DP at
 * the slowest link of the candidate's stages plus an optimizer step
 * proportional to the parameters each rank updates.  Partition-independent. */
int64_t orc_dp_const(const orc_problem *p, const orc_config *c, int32_t order)
{
    orc_stage st[ORC_MAX_STAGES];
    if (orc_stages(p, c, order, 1, st)) return 0;   /* an empty slot of the free stage types */
    double al = 0.0, bw = 0.0;
    for (int s = 0; s < c->pp; s++) {
        if (s == 0 || st[s].alpha > al) al = st[s].alpha;
        if (s == 0 || st[s].bw < bw) bw = st[s].bw;
    }
    orc_pi_terms t;
    orc_pi_terms_eval(p, c, &t);
    return q(ring_allreduce(4.0 * t.p_avg, c->dp, al, bw) + (p->opt_coef * t.p_avg) / (double)c->dp);
}

/* ------------------------------------------------------------------------
 * Segment cost c_i(a, b) of putting layers [a, b) on stage i (Algorithm 1 inner
 * body): pruning 1 window; the smallest recomputation choice that fits the
 * stage's memory (pruning 2); pruning 3 on cross-type communication; then
 * T_stage + T_comm.
 * ---------------------------------------------------------------------- */
/* layer prefix sums of one configuration: memory terms, and the stage-time
 * terms of one device-type set */
typedef struct prefixes {
    int n;
    int64_t *w, *a0, *a1, *moe, *t0, *t1, *comm;
} prefixes;

static void prefixes_init(const orc_problem *p, const orc_config *c, prefixes *P)
{
    int N = p->n_layers, W = N + 1;
    P->n = N;
    P->w = calloc((size_t)W, 8);
    P->a0 = calloc((size_t)W, 8);
    P->a1 = calloc((size_t)W, 8);
    P->moe = calloc((size_t)W, 8);
    P->t0 = calloc((size_t)W, 8);
    P->t1 = calloc((size_t)W, 8);
    P->comm = calloc((size_t)W, 8);
    for (int l = 0; l < N; l++) {
        orc_mem_terms m;
        orc_mem_terms_eval(p, c, l, &m);
        P->w[l + 1] = P->w[l] + m.q_w;
        P->a0[l + 1] = P->a0[l] + m.q_a0;
        P->a1[l + 1] = P->a1[l] + m.q_a1;
        P->moe[l + 1] = P->moe[l] + (p->is_moe[l] ? 1 : 0);
    }
}

static void prefixes_time(const orc_problem *p, const orc_config *c, int mask, prefixes *P)
{
    for (int l = 0; l < P->n; l++) {
        orc_mask_terms m;
        orc_mask_terms_eval(p, c, l, mask, &m);
        P->t0[l + 1] = P->t0[l] + m.t_r0;
        P->t1[l + 1] = P->t1[l] + m.t_r1;
        P->comm[l + 1] = P->comm[l] + m.comm;
    }
}

static void prefixes_free(prefixes *P)
{
    free(P->w); free(P->a0); free(P->a1); free(P->moe); free(P->t0); free(P->t1); free(P->comm);
}

/* c_i(a, b) of one stage (ORC_INF if pruned), *r = the recomputation choice */
static int64_t segment_cost(const orc_problem *p, const orc_pi_terms *pt, const orc_stage *st,
                            const prefixes *P, int a, int b, uint8_t *r)
{
    *r = 0;
    if (b <= a) return ORC_INF;
    int n = b - a;
    if (n < st->lo || n > st->hi) return ORC_INF;                              /* pruning 1 */
    int64_t extra = (P->moe[b] - P->moe[a]) > 0 ? pt->x_bytes : 0;
    int64_t m0 = (P->w[b] - P->w[a]) + st->m_store * (P->a0[b] - P->a0[a]) + extra;
    int64_t m1 = (P->w[b] - P->w[a]) + st->m_store * (P->a1[b] - P->a1[a]) + extra;
    int64_t t;
    if (m0 <= st->cap) {
        t = P->t0[b] - P->t0[a];
    } else if (p->allow_recompute && m1 <= st->cap) {
        t = P->t1[b] - P->t1[a];
        *r = 1;
    } else {
        return ORC_INF;                                                          /* pruning 2 */
    }
    if (p->prune_hetero) {
        int64_t hc = (st->mixed ? P->comm[b] - P->comm[a] : 0) + (st->bdiff ? st->p2p : 0);
        if (hc > (int64_t)p->eta_prune * pt->tbar) {                             /* pruning 3 */
            *r = 0;
            return ORC_INF;
        }
    }
    return t + st->p2p;
}

int32_t orc_segment_costs(const orc_problem *p, int64_t idx, int64_t *cost, uint8_t *rflag)
{
    orc_config c;
    int32_t order, micro;
    if (orc_instance(p, idx, &c, &order, &micro)) return -1;
    int N = p->n_layers, PP = c.pp, W = N + 1;
    orc_stage st[ORC_MAX_STAGES];
    if (orc_stages(p, &c, order, micro, st)) {   /* an empty slot: no partition */
        for (int64_t i = 0; i < (int64_t)PP * W * W; i++) {
            cost[i] = ORC_INF;
            rflag[i] = 0;
        }
        return 0;
    }
    orc_pi_terms pt;
    orc_pi_terms_eval(p, &c, &pt);
    prefixes P;
    prefixes_init(p, &c, &P);
    for (int i = 0; i < PP; i++) {
        prefixes_time(p, &c, st[i].mask, &P);
        for (int a = 0; a < W; a++)
            for (int b = 0; b < W; b++) {
                int64_t at = ((int64_t)i * W + a) * W + b;
                cost[at] = segment_cost(p, &pt, &st[i], &P, a, b, &rflag[at]);
            }
    }
    prefixes_free(&P);
    return 0;
}

/* ------------------------------------------------------------------------
 * Stage DP (Section 3.4 transition; Algorithm 1).  F[i][b] = the least sum of
 * stage costs placing layers [0, b) on stages 1..i, every stage cost <= t.
 * Ties keep the smallest split point a.
 * ---------------------------------------------------------------------- */
static int64_t dp_pass(int pp, int n, const int64_t *cost, int64_t t, int64_t *F, int16_t *arg)
{
    int W = n + 1;
    for (int b = 0; b < W; b++) F[b] = b == 0 ? 0 : ORC_INF;
    for (int i = 1; i <= pp; i++) {
        for (int b = 0; b < W; b++) {
            int64_t best = ORC_INF;
            int ba = -1;
            for (int a = 0; a < b; a++) {
                int64_t prev = F[(int64_t)(i - 1) * W + a];
                int64_t c = cost[((int64_t)(i - 1) * W + a) * W + b];
                if (prev == ORC_INF || c == ORC_INF || c > t) continue;
                if (prev + c < best) {
                    best = prev + c;
                    ba = a;
                }
            }
            F[(int64_t)i * W + b] = best;
            arg[(int64_t)i * W + b] = (int16_t)ba;
        }
    }
    return F[(int64_t)pp * W + n];
}

static int cmp_i64(const void *x, const void *y)
{
    int64_t a = *(const int64_t *)x, b = *(const int64_t *)y;
    return (a > b) - (a < b);
}

/* Threshold form of the 1F1B objective: with every stage <= t,
 *   score(t) = F_t + (B-1) t,  OPT = min_t score(t)
 * over t in the set of distinct finite stage costs, ascending; t* is the
 * smallest t reaching OPT and the partition is the back-trace of F at t*.
 * The sweep stops once F_inf + (B-1) t >= best (no larger t can do better). */
int32_t orc_dp(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r)
{
    int W = n + 1;
    int64_t ncost = (int64_t)pp * W * W;
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    int64_t *theta = malloc(sizeof(int64_t) * (size_t)(ncost + 1));
    int64_t nt = 0;
    for (int64_t i = 0; i < ncost; i++)
        if (cost[i] != ORC_INF) theta[nt++] = cost[i];
    qsort(theta, (size_t)nt, sizeof(int64_t), cmp_i64);
    int64_t u = 0;
    for (int64_t i = 0; i < nt; i++)
        if (u == 0 || theta[i] != theta[u - 1]) theta[u++] = theta[i];
    int64_t *F = malloc(sizeof(int64_t) * (size_t)(pp + 1) * W);
    int16_t *arg = malloc(sizeof(int16_t) * (size_t)(pp + 1) * W);

    int64_t finf = dp_pass(pp, n, cost, ORC_INF, F, arg);
    int64_t best = ORC_INF, tstar = -1, swept = 0;
    if (finf != ORC_INF) {
        for (int64_t k = 0; k < u; k++) {
            int64_t t = theta[k];
            if (finf + (micro - 1) * t >= best) break;
            int64_t f = dp_pass(pp, n, cost, t, F, arg);
            swept++;
            if (f == ORC_INF) continue;
            int64_t score = f + (micro - 1) * t;
            if (score < best) {
                best = score;
                tstar = t;
            }
        }
    }
    r->thresholds = swept;
    if (tstar < 0) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
    } else {
        r->sum = dp_pass(pp, n, cost, tstar, F, arg);
        r->tmax = tstar;
        r->opt = best;
        int b = n;
        for (int i = pp; i >= 1; i--) {
            int a = arg[(int64_t)i * W + b];
            r->layers[i - 1] = (uint8_t)(b - a);
            b = a;
        }
    }
    free(theta);
    free(F);
    free(arg);
    return 0;
}

/* Brute force over every composition of n layers into pp non-empty stages.
 * Order: (sum + (B-1) max, max, b_{pp-1}, b_{pp-2}, ..., b_1) ascending, where
 * b_i is the end layer of stage i -- the same canonical choice as orc_dp. */
typedef struct brute_state {
    int pp, n, W;
    int64_t micro;
    const int64_t *cost;
    int b[ORC_MAX_STAGES + 1];
    int best_b[ORC_MAX_STAGES + 1];
    int64_t best_obj, best_max, best_sum;
    int found;
} brute_state;

static int brute_better(const brute_state *s, int64_t obj, int64_t mx)
{
    if (!s->found) return 1;
    if (obj != s->best_obj) return obj < s->best_obj;
    if (mx != s->best_max) return mx < s->best_max;
    for (int i = s->pp - 1; i >= 1; i--)
        if (s->b[i] != s->best_b[i]) return s->b[i] < s->best_b[i];
    return 0;
}

static void brute_rec(brute_state *s, int i)
{
    if (i == s->pp) {
        int64_t sum = 0, mx = 0;
        for (int k = 0; k < s->pp; k++) {
            int64_t c = s->cost[((int64_t)k * s->W + s->b[k]) * s->W + s->b[k + 1]];
            if (c == ORC_INF) return;
            sum += c;
            if (c > mx) mx = c;
        }
        int64_t obj = sum + (s->micro - 1) * mx;
        if (brute_better(s, obj, mx)) {
            s->found = 1;
            s->best_obj = obj;
            s->best_max = mx;
            s->best_sum = sum;
            memcpy(s->best_b, s->b, sizeof(s->b));
        }
        return;
    }
    if (i == s->pp - 1) {
        s->b[i + 1] = s->n;
        if (s->b[i] < s->n) brute_rec(s, i + 1);
        return;
    }
    for (int e = s->b[i] + 1; e <= s->n - (s->pp - 1 - i); e++) {
        s->b[i + 1] = e;
        brute_rec(s, i + 1);
    }
}

int32_t orc_brute(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r)
{
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    brute_state s;
    memset(&s, 0, sizeof(s));
    s.pp = pp;
    s.n = n;
    s.W = n + 1;
    s.micro = micro;
    s.cost = cost;
    s.b[0] = 0;
    if (pp <= n) brute_rec(&s, 0);
    if (!s.found) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
        return 0;
    }
    r->opt = s.best_obj;
    r->sum = s.best_sum;
    r->tmax = s.best_max;
    for (int i = 0; i < pp; i++) r->layers[i] = (uint8_t)(s.best_b[i + 1] - s.best_b[i]);
    return 0;
}

/* ------------------------------------------------------------------------
 * 1F1B re-scoring (Eq. 4 with the appendix's steady-state term).  The
 * appendix gives, for stage forward / backward times t_f,i and t_b,i and the
 * bottleneck stage s (largest t_f + t_b), the iteration latency
 *   sum_i (t_f,i + t_b,i) + sum_{i <= s} t_f,i + (M - s - 1) max_i (t_f,i + t_b,i)
 * with M micro-batches.  Readings: a stage cost c splits as t_f = ceil(c/3),
 * t_b = c - t_f (backward twice the forward); s is the first (1-based) stage
 * of largest cost; the count M - s - 1 is taken as max(0, M - s - 1), as the
 * steady state has no full cycle when B <= s.
 * ---------------------------------------------------------------------- */
int64_t orc_latency_1f1b(int32_t pp, const int64_t *c, int64_t micro)
{
    int64_t sum = 0, mx = -1;
    int s = 0;
    for (int i = 0; i < pp; i++) {
        sum += c[i];
        if (c[i] > mx) {
            mx = c[i];
            s = i + 1;
        }
    }
    int64_t fwd = 0;
    for (int i = 0; i < s; i++) fwd += (c[i] + 2) / 3;
    int64_t steady = micro - s - 1;
    if (steady < 0) steady = 0;
    return sum + fwd + steady * mx;
}

/* The candidates are the (max, sum) Pareto frontier: the thresholds t at which
 * F_t drops (F_t < F_t' for every t' < t), each with the canonical partition of
 * the threshold DP at t, whose largest stage is then t.  The least latency
 * wins; ties go to the lower max (the earlier frontier point, ascending). */
int32_t orc_dp_exact(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r)
{
    int W = n + 1;
    int64_t ncost = (int64_t)pp * W * W;
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    int64_t *theta = malloc(sizeof(int64_t) * (size_t)(ncost + 1));
    int64_t nt = 0;
    for (int64_t i = 0; i < ncost; i++)
        if (cost[i] != ORC_INF) theta[nt++] = cost[i];
    qsort(theta, (size_t)nt, sizeof(int64_t), cmp_i64);
    int64_t u = 0;
    for (int64_t i = 0; i < nt; i++)
        if (u == 0 || theta[i] != theta[u - 1]) theta[u++] = theta[i];
    int64_t *F = malloc(sizeof(int64_t) * (size_t)(pp + 1) * W);
    int16_t *arg = malloc(sizeof(int16_t) * (size_t)(pp + 1) * W);
    int64_t best = ORC_INF, prev = ORC_INF, points = 0;
    for (int64_t k = 0; k < u; k++) {
        int64_t t = theta[k];
        int64_t f = dp_pass(pp, n, cost, t, F, arg);
        if (f == ORC_INF || f >= prev) continue;   /* not a frontier point */
        prev = f;
        points++;
        int64_t c[ORC_MAX_STAGES];
        uint8_t len[ORC_MAX_STAGES];
        int b = n;
        int64_t mx = 0;
        for (int i = pp; i >= 1; i--) {
            int a = arg[(int64_t)i * W + b];
            c[i - 1] = cost[((int64_t)(i - 1) * W + a) * W + b];
            len[i - 1] = (uint8_t)(b - a);
            if (c[i - 1] > mx) mx = c[i - 1];
            b = a;
        }
        int64_t lat = orc_latency_1f1b(pp, c, micro);
        if (lat < best) {
            best = lat;
            r->sum = f;
            r->tmax = mx;
            memcpy(r->layers, len, (size_t)pp);
        }
    }
    r->thresholds = points;
    if (best == ORC_INF) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
    } else {
        r->opt = best;
    }
    free(theta);
    free(F);
    free(arg);
    return 0;
}

/* Brute force for the same objective: every composition, the Pareto-optimal
 * (max, sum) pairs, per pair the partition with the smallest
 * (b_{pp-1}, b_{pp-2}, ..., b_1), then the least latency, ties to the lower max. */
typedef struct part_rec {
    int64_t mx, sum;
    int b[ORC_MAX_STAGES + 1];
} part_rec;

typedef struct part_list {
    int pp, n, W;
    const int64_t *cost;
    int b[ORC_MAX_STAGES + 1];
    part_rec *v;
    int64_t len, cap;
} part_list;

static void collect(part_list *L, int i)
{
    if (i == L->pp) {
        part_rec rec;
        rec.mx = 0;
        rec.sum = 0;
        for (int k = 0; k < L->pp; k++) {
            int64_t c = L->cost[((int64_t)k * L->W + L->b[k]) * L->W + L->b[k + 1]];
            if (c == ORC_INF) return;
            rec.sum += c;
            if (c > rec.mx) rec.mx = c;
        }
        memcpy(rec.b, L->b, sizeof(rec.b));
        if (L->len == L->cap) {
            L->cap = L->cap ? 2 * L->cap : 64;
            L->v = realloc(L->v, sizeof(part_rec) * (size_t)L->cap);
        }
        L->v[L->len++] = rec;
        return;
    }
    if (i == L->pp - 1) {
        L->b[i + 1] = L->n;
        if (L->b[i] < L->n) collect(L, i + 1);
        return;
    }
    for (int e = L->b[i] + 1; e <= L->n - (L->pp - 1 - i); e++) {
        L->b[i + 1] = e;
        collect(L, i + 1);
    }
}

static int lex_smaller(int pp, const int *x, const int *y)   /* (b_{pp-1}, ..., b_1) */
{
    for (int i = pp - 1; i >= 1; i--)
        if (x[i] != y[i]) return x[i] < y[i];
    return 0;
}

int32_t orc_brute_exact(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r)
{
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    part_list L;
    memset(&L, 0, sizeof(L));
    L.pp = pp;
    L.n = n;
    L.W = n + 1;
    L.cost = cost;
    if (pp <= n) collect(&L, 0);
    int64_t best = ORC_INF, best_mx = ORC_INF, points = 0;
    for (int64_t i = 0; i < L.len; i++) {
        const part_rec *x = &L.v[i];
        int keep = 1;
        for (int64_t j = 0; j < L.len && keep; j++) {
            const part_rec *y = &L.v[j];
            if (y->mx <= x->mx && y->sum <= x->sum && (y->mx < x->mx || y->sum < x->sum)) keep = 0;   /* dominated */
            else if (y->mx == x->mx && y->sum == x->sum && lex_smaller(pp, y->b, x->b)) keep = 0;    /* not canonical */
        }
        if (!keep) continue;
        points++;
        int64_t c[ORC_MAX_STAGES];
        for (int k = 0; k < pp; k++) c[k] = cost[((int64_t)k * L.W + x->b[k]) * L.W + x->b[k + 1]];
        int64_t lat = orc_latency_1f1b(pp, c, micro);
        if (lat < best || (lat == best && x->mx < best_mx)) {
            best = lat;
            best_mx = x->mx;
            r->sum = x->sum;
            r->tmax = x->mx;
            for (int k = 0; k < pp; k++) r->layers[k] = (uint8_t)(x->b[k + 1] - x->b[k]);
        }
    }
    r->thresholds = points;
    if (best == ORC_INF) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
    } else {
        r->opt = best;
    }
    free(L.v);
    return 0;
}

/* ------------------------------------------------------------------------
 * The least 1F1B latency itself (Eq. 4 with the appendix's steady-state term,
 * orc_latency_1f1b) over every partition -- not only the partitions of the
 * (max, sum) frontier that orc_dp_exact re-scores.  The latency of a partition
 * depends on where its first largest stage s sits, so it is not a function of
 * (max, sum): a partition off the frontier can have a lower latency.
 *
 * Exact minimisation: every partition has one largest cost t and one first
 * stage s reaching it, and then its latency is the sum of per-stage weights
 *   stages i < s:  c_i < t,   weight c_i + ceil(c_i / 3)   (its forward time counts)
 *   stage s:       c_s = t,   weight t + ceil(t / 3) + max(0, B - s - 1) t
 *   stages i > s:  c_i <= t,  weight c_i.
 * For each threshold t (every distinct finite stage cost, ascending) a DP over
 * (stage, end layer, z) -- z = 1 once the bottleneck stage is placed -- finds
 * the least weight sum with the largest stage exactly t.  The sweep stops once
 * F_inf + ceil(t/3) + max(0, B - pp - 1) t (a lower bound for every larger t)
 * reaches the best latency.  Ties: least latency, then the lower largest
 * stage, then the lexicographically smallest (b_{pp-1}, ..., b_1).
 * ---------------------------------------------------------------------- */
typedef struct lat_dp {
    int pp, n, W;
    int64_t micro, t;
    const int64_t *cost;
    int64_t *V;   /* [pp + 1][W][2] least weight sums */
} lat_dp;

static int64_t *lat_at(const lat_dp *d, int i, int b, int z) { return &d->V[((int64_t)i * d->W + b) * 2 + z]; }

/* weight of stage i (1-based) on [a, b) moving from z0 to z1 (ORC_INF if not allowed) */
static int64_t lat_weight(const lat_dp *d, int i, int a, int b, int z0, int z1)
{
    int64_t c = d->cost[((int64_t)(i - 1) * d->W + a) * d->W + b];
    if (c == ORC_INF) return ORC_INF;
    if (z0 == 0 && z1 == 0) return c < d->t ? c + (c + 2) / 3 : ORC_INF;
    if (z0 == 0 && z1 == 1) {
        if (c != d->t) return ORC_INF;
        int64_t steady = d->micro - i - 1;
        return c + (c + 2) / 3 + (steady > 0 ? steady : 0) * c;
    }
    if (z0 == 1 && z1 == 1) return c <= d->t ? c : ORC_INF;
    return ORC_INF;
}

static void lat_pass(lat_dp *d)
{
    for (int i = 0; i <= d->pp; i++)
        for (int b = 0; b < d->W; b++)
            for (int z = 0; z < 2; z++) *lat_at(d, i, b, z) = (i == 0 && b == 0 && z == 0) ? 0 : ORC_INF;
    for (int i = 1; i <= d->pp; i++)
        for (int b = 1; b < d->W; b++)
            for (int z = 0; z < 2; z++) {
                int64_t best = ORC_INF;
                for (int a = 0; a < b; a++)
                    for (int z0 = 0; z0 <= z; z0++) {
                        int64_t v = *lat_at(d, i - 1, a, z0), w = lat_weight(d, i, a, b, z0, z);
                        if (v != ORC_INF && w != ORC_INF && v + w < best) best = v + w;
                    }
                *lat_at(d, i, b, z) = best;
            }
}

/* The lexicographically smallest (b_{pp-1}, ..., b_1) among the optimal paths
 * into (pp, n, z = 1): walking back from the last stage, keep the set of states
 * (one end layer, z in {0, 1}) on some optimal path, take the smallest split
 * point a through which one continues optimally, and move to those states. */
static void lat_trace(const lat_dp *d, uint8_t *len)
{
    int b = d->n;
    int live[2] = {0, 1};   /* live[z]: state (i, b, z) is on an optimal path */
    for (int i = d->pp; i >= 1; i--) {
        int na = -1, nl[2] = {0, 0};
        for (int a = 0; a < b && na < 0; a++)
            for (int z0 = 0; z0 < 2; z0++)
                for (int z = z0; z < 2; z++) {
                    if (!live[z]) continue;
                    int64_t v = *lat_at(d, i - 1, a, z0), w = lat_weight(d, i, a, b, z0, z);
                    if (v != ORC_INF && w != ORC_INF && v + w == *lat_at(d, i, b, z)) {
                        na = a;
                        nl[z0] = 1;
                    }
                }
        len[i - 1] = (uint8_t)(b - na);
        b = na;
        live[0] = nl[0];
        live[1] = nl[1];
    }
}

int32_t orc_dp_latency(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r)
{
    int W = n + 1;
    int64_t ncost = (int64_t)pp * W * W;
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    int64_t *theta = malloc(sizeof(int64_t) * (size_t)(ncost + 1));
    int64_t nt = 0;
    for (int64_t i = 0; i < ncost; i++)
        if (cost[i] != ORC_INF) theta[nt++] = cost[i];
    qsort(theta, (size_t)nt, sizeof(int64_t), cmp_i64);
    int64_t u = 0;
    for (int64_t i = 0; i < nt; i++)
        if (u == 0 || theta[i] != theta[u - 1]) theta[u++] = theta[i];
    int64_t *F = malloc(sizeof(int64_t) * (size_t)(pp + 1) * W);
    int16_t *arg = malloc(sizeof(int16_t) * (size_t)(pp + 1) * W);
    lat_dp d;
    d.pp = pp;
    d.n = n;
    d.W = W;
    d.micro = micro;
    d.cost = cost;
    d.V = malloc(sizeof(int64_t) * (size_t)(pp + 1) * W * 2);
    int64_t finf = pp <= n ? dp_pass(pp, n, cost, ORC_INF, F, arg) : ORC_INF;
    int64_t best = ORC_INF, swept = 0, steady_min = micro - pp - 1;
    if (steady_min < 0) steady_min = 0;
    for (int64_t k = 0; k < u && finf != ORC_INF; k++) {
        d.t = theta[k];
        if (finf + (d.t + 2) / 3 + steady_min * d.t >= best) break;
        lat_pass(&d);
        swept++;
        int64_t v = *lat_at(&d, pp, n, 1);
        if (v < best) {
            best = v;
            r->tmax = d.t;
            lat_trace(&d, r->layers);
        }
    }
    r->thresholds = swept;
    if (best == ORC_INF) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
        memset(r->layers, 0, sizeof(r->layers));
    } else {
        r->opt = best;
        r->sum = 0;
        for (int i = 0, a = 0; i < pp; i++) {
            r->sum += cost[((int64_t)i * W + a) * W + a + r->layers[i]];
            a += r->layers[i];
        }
    }
    free(theta);
    free(F);
    free(arg);
    free(d.V);
    return 0;
}

/* Brute force of the same minimum: every composition, key (latency, largest
 * stage, b_{pp-1}, ..., b_1) ascending. */
int32_t orc_brute_latency(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r)
{
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    part_list L;
    memset(&L, 0, sizeof(L));
    L.pp = pp;
    L.n = n;
    L.W = n + 1;
    L.cost = cost;
    if (pp <= n) collect(&L, 0);
    int64_t best = ORC_INF, best_mx = ORC_INF;
    const part_rec *win = NULL;
    for (int64_t i = 0; i < L.len; i++) {
        const part_rec *x = &L.v[i];
        int64_t c[ORC_MAX_STAGES];
        for (int k = 0; k < pp; k++) c[k] = cost[((int64_t)k * L.W + x->b[k]) * L.W + x->b[k + 1]];
        int64_t lat = orc_latency_1f1b(pp, c, micro);
        if (lat < best || (lat == best && (x->mx < best_mx || (x->mx == best_mx && lex_smaller(pp, x->b, win->b))))) {
            best = lat;
            best_mx = x->mx;
            win = x;
        }
    }
    r->thresholds = L.len;
    if (!win) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
    } else {
        r->opt = best;
        r->sum = win->sum;
        r->tmax = win->mx;
        for (int k = 0; k < pp; k++) r->layers[k] = (uint8_t)(win->b[k + 1] - win->b[k]);
    }
    free(L.v);
    return 0;
}

/* ------------------------------------------------------------------------
 * Free per-stage device types by the DP over device counts (Section 3.4: the
 * DP state carries the remaining devices of each type, and every transition
 * picks the type h and the layers of one more stage; Algorithm 1).
 *
 * A pipeline of pp stages with g = G / pp devices a stage holds k_h = m_h / g
 * stages of type h.  State (u, b, h): u_h stages of type h placed so far
 * (s = sum u of them), layers [0, b) covered, and the next stage -- number s --
 * of type h.  A type-h stage on [a, b) followed by a type-h' stage costs
 * c[s][h][h'](a, b) (h' = T: it is the last stage), the segment cost of a pure
 * stage at position s; the transfer to the next stage, and pruning 3 on it,
 * depend on h'.  Threshold form as in orc_dp:
 *     F_t(u + e_h, b, h') = min over (a, h) of F_t(u, a, h) + c[s][h][h'](a, b)
 * over costs <= t, starting from F(0, 0, h) = 0 for every type with k_h > 0.
 * Ties keep the smallest a, then the smallest h.  OPT = min_t F_t + (B-1) t,
 * t* the smallest threshold reaching it, and the back-trace at t* gives the
 * lexicographically smallest (b_{pp-1}, h_{pp-1}, ..., b_1, h_1, h_0) among
 * the optima (b_i = first layer of stage i, h_i = its type).
 * ---------------------------------------------------------------------- */
typedef struct type_space {
    int pp, T, n, W, U;
    int k[ORC_MAX_TYPES], rad[ORC_MAX_TYPES];
} type_space;

static void type_space_init(type_space *S, int pp, int T, const int32_t *k, int n)
{
    S->pp = pp;
    S->T = T;
    S->n = n;
    S->W = n + 1;
    S->U = 1;
    for (int h = 0; h < T; h++) {
        S->k[h] = k[h];
        S->rad[h] = S->U;
        S->U *= k[h] + 1;
    }
}

static int digit(const type_space *S, int u, int h) { return (u / S->rad[h]) % (S->k[h] + 1); }

static int64_t cost_at(const type_space *S, const int64_t *cost, int s, int h, int hn, int a, int b)
{
    return cost[((((int64_t)s * S->T + h) * (S->T + 1) + hn) * S->W + a) * S->W + b];
}

/* one pass at threshold t: F and arg over [U][W][T + 1]; returns F at the end state */
static int64_t type_pass(const type_space *S, const int64_t *cost, int64_t t, int64_t *F, int32_t *arg)
{
    int W = S->W, T1 = S->T + 1;
    for (int64_t i = 0; i < (int64_t)S->U * W * T1; i++) {
        F[i] = ORC_INF;
        arg[i] = -1;
    }
    for (int h = 0; h < S->T; h++)
        if (S->k[h] > 0) F[h] = 0;   /* u = 0, b = 0 */
    for (int u = 1; u < S->U; u++) {   /* u - e_h < u: increasing index is a topological order */
        int done = 0;
        for (int h = 0; h < S->T; h++) done += digit(S, u, h);
        int s = done - 1;   /* the stage that ends at b */
        for (int b = 0; b < W; b++)
            for (int hn = 0; hn < T1; hn++) {
                if (done == S->pp ? hn != S->T : (hn == S->T || digit(S, u, hn) >= S->k[hn])) continue;
                int64_t best = ORC_INF;
                int32_t ba = -1;
                for (int a = 0; a < b; a++)
                    for (int h = 0; h < S->T; h++) {
                        if (digit(S, u, h) == 0) continue;
                        int64_t prev = F[((int64_t)(u - S->rad[h]) * W + a) * T1 + h];
                        int64_t c = cost_at(S, cost, s, h, hn, a, b);
                        if (prev == ORC_INF || c == ORC_INF || c > t) continue;
                        if (prev + c < best) {
                            best = prev + c;
                            ba = a * 8 + h;
                        }
                    }
                F[((int64_t)u * W + b) * T1 + hn] = best;
                arg[((int64_t)u * W + b) * T1 + hn] = ba;
            }
    }
    return F[((int64_t)(S->U - 1) * W + S->n) * T1 + S->T];
}

int32_t orc_dp_types(int32_t pp, int32_t T, const int32_t *k, int32_t n, int64_t micro, const int64_t *cost,
                     orc_result *r)
{
    type_space S;
    type_space_init(&S, pp, T, k, n);
    int W = S.W, T1 = T + 1;
    int64_t ncost = (int64_t)pp * T * T1 * W * W;
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    int64_t *theta = malloc(sizeof(int64_t) * (size_t)(ncost + 1));
    int64_t nt = 0;
    for (int64_t i = 0; i < ncost; i++)
        if (cost[i] != ORC_INF) theta[nt++] = cost[i];
    qsort(theta, (size_t)nt, sizeof(int64_t), cmp_i64);
    int64_t nu = 0;
    for (int64_t i = 0; i < nt; i++)
        if (nu == 0 || theta[i] != theta[nu - 1]) theta[nu++] = theta[i];
    int64_t *F = malloc(sizeof(int64_t) * (size_t)S.U * W * T1);
    int32_t *arg = malloc(sizeof(int32_t) * (size_t)S.U * W * T1);

    int64_t finf = type_pass(&S, cost, ORC_INF, F, arg);
    int64_t best = ORC_INF, tstar = -1, swept = 0;
    if (finf != ORC_INF) {
        for (int64_t i = 0; i < nu; i++) {
            int64_t t = theta[i];
            if (finf + (micro - 1) * t >= best) break;
            int64_t f = type_pass(&S, cost, t, F, arg);
            swept++;
            if (f == ORC_INF) continue;
            if (f + (micro - 1) * t < best) {
                best = f + (micro - 1) * t;
                tstar = t;
            }
        }
    }
    r->thresholds = swept;
    if (tstar < 0) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
    } else {
        r->sum = type_pass(&S, cost, tstar, F, arg);
        r->tmax = tstar;
        r->opt = best;
        int u = S.U - 1, b = n, hn = T;
        for (int i = pp - 1; i >= 0; i--) {
            int32_t x = arg[((int64_t)u * W + b) * T1 + hn];
            int a = x / 8, h = x % 8;
            r->layers[i] = (uint8_t)(b - a);
            r->stage_mask[i] = (uint8_t)(1 << h);
            u -= S.rad[h];
            b = a;
            hn = h;
        }
    }
    free(theta);
    free(F);
    free(arg);
    return 0;
}

/* Brute force: every stage-type sequence (arrangement of the multiset) and
 * every composition, ordered by (objective, largest stage, b_{pp-1}, h_{pp-1},
 * ..., b_1, h_1, h_0) -- the canonical choice of orc_dp_types. */
typedef struct type_brute {
    const type_space *S;
    const int64_t *cost;
    int64_t micro;
    int seq[ORC_MAX_STAGES], b[ORC_MAX_STAGES + 1];
    int best_seq[ORC_MAX_STAGES], best_b[ORC_MAX_STAGES + 1];
    int64_t best_obj, best_max, best_sum;
    int found;
} type_brute;

static int type_brute_better(const type_brute *x, int64_t obj, int64_t mx)
{
    if (!x->found) return 1;
    if (obj != x->best_obj) return obj < x->best_obj;
    if (mx != x->best_max) return mx < x->best_max;
    for (int i = x->S->pp - 1; i >= 1; i--) {
        if (x->b[i] != x->best_b[i]) return x->b[i] < x->best_b[i];
        if (x->seq[i] != x->best_seq[i]) return x->seq[i] < x->best_seq[i];
    }
    return x->seq[0] < x->best_seq[0];
}

static void type_brute_parts(type_brute *x, int i)
{
    const type_space *S = x->S;
    if (i == S->pp) {
        int64_t sum = 0, mx = 0;
        for (int j = 0; j < S->pp; j++) {
            int hn = j + 1 < S->pp ? x->seq[j + 1] : S->T;
            int64_t c = cost_at(S, x->cost, j, x->seq[j], hn, x->b[j], x->b[j + 1]);
            if (c == ORC_INF) return;
            sum += c;
            if (c > mx) mx = c;
        }
        int64_t obj = sum + (x->micro - 1) * mx;
        if (type_brute_better(x, obj, mx)) {
            x->found = 1;
            x->best_obj = obj;
            x->best_max = mx;
            x->best_sum = sum;
            memcpy(x->best_seq, x->seq, sizeof(x->seq));
            memcpy(x->best_b, x->b, sizeof(x->b));
        }
        return;
    }
    if (i == S->pp - 1) {
        x->b[S->pp] = S->n;
        if (x->b[i] < S->n) type_brute_parts(x, S->pp);
        return;
    }
    for (int e = x->b[i] + 1; e <= S->n - (S->pp - 1 - i); e++) {
        x->b[i + 1] = e;
        type_brute_parts(x, i + 1);
    }
}

static void type_brute_seq(type_brute *x, int i, int *left)
{
    if (i == x->S->pp) {
        x->b[0] = 0;
        type_brute_parts(x, 0);
        return;
    }
    for (int h = 0; h < x->S->T; h++) {
        if (left[h] == 0) continue;
        left[h]--;
        x->seq[i] = h;
        type_brute_seq(x, i + 1, left);
        left[h]++;
    }
}

int32_t orc_brute_types(int32_t pp, int32_t T, const int32_t *k, int32_t n, int64_t micro, const int64_t *cost,
                        orc_result *r)
{
    type_space S;
    type_space_init(&S, pp, T, k, n);
    type_brute x;
    memset(&x, 0, sizeof(x));
    x.S = &S;
    x.cost = cost;
    x.micro = micro;
    int left[ORC_MAX_TYPES];
    for (int h = 0; h < T; h++) left[h] = k[h];
    type_brute_seq(&x, 0, left);
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    if (!x.found) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
        return 0;
    }
    r->opt = x.best_obj;
    r->sum = x.best_sum;
    r->tmax = x.best_max;
    for (int i = 0; i < pp; i++) {
        r->layers[i] = (uint8_t)(x.best_b[i + 1] - x.best_b[i]);
        r->stage_mask[i] = (uint8_t)(1 << x.best_seq[i]);
    }
    return 0;
}

/* 1F1B re-scoring over the device-count DP (stage_types = 2): the frontier
 * points are the thresholds at which F_t drops, each with the canonical path
 * at t (whose largest stage is then t); each is scored with
 * orc_latency_1f1b of its stage costs in pipeline order.  Least latency, ties
 * to the lower largest stage. */
int32_t orc_dp_types_exact(int32_t pp, int32_t T, const int32_t *k, int32_t n, int64_t micro, const int64_t *cost,
                           orc_result *r)
{
    type_space S;
    type_space_init(&S, pp, T, k, n);
    int W = S.W, T1 = T + 1;
    int64_t ncost = (int64_t)pp * T * T1 * W * W;
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    int64_t *theta = malloc(sizeof(int64_t) * (size_t)(ncost + 1));
    int64_t nt = 0;
    for (int64_t i = 0; i < ncost; i++)
        if (cost[i] != ORC_INF) theta[nt++] = cost[i];
    qsort(theta, (size_t)nt, sizeof(int64_t), cmp_i64);
    int64_t nu = 0;
    for (int64_t i = 0; i < nt; i++)
        if (nu == 0 || theta[i] != theta[nu - 1]) theta[nu++] = theta[i];
    int64_t *F = malloc(sizeof(int64_t) * (size_t)S.U * W * T1);
    int32_t *arg = malloc(sizeof(int32_t) * (size_t)S.U * W * T1);
    int64_t best = ORC_INF, prev = ORC_INF, points = 0;
    for (int64_t i = 0; i < nu; i++) {
        int64_t t = theta[i];
        int64_t f = type_pass(&S, cost, t, F, arg);
        if (f == ORC_INF || f >= prev) continue;   /* not a frontier point */
        prev = f;
        points++;
        int64_t c[ORC_MAX_STAGES], mx = 0;
        uint8_t len[ORC_MAX_STAGES], mask[ORC_MAX_STAGES];
        int u = S.U - 1, b = n, hn = T;
        for (int j = pp - 1; j >= 0; j--) {
            int32_t x = arg[((int64_t)u * W + b) * T1 + hn];
            int a = x / 8, h = x % 8;
            c[j] = cost_at(&S, cost, j, h, hn, a, b);
            len[j] = (uint8_t)(b - a);
            mask[j] = (uint8_t)(1 << h);
            if (c[j] > mx) mx = c[j];
            u -= S.rad[h];
            b = a;
            hn = h;
        }
        int64_t lat = orc_latency_1f1b(pp, c, micro);
        if (lat < best) {
            best = lat;
            r->sum = f;
            r->tmax = mx;
            memcpy(r->layers, len, (size_t)pp);
            memcpy(r->stage_mask, mask, (size_t)pp);
        }
    }
    r->thresholds = points;
    if (best == ORC_INF) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
        memset(r->stage_mask, 0, sizeof(r->stage_mask));
    } else {
        r->opt = best;
    }
    free(theta);
    free(F);
    free(arg);
    return 0;
}

/* Brute force of the same: every (sequence, composition), the Pareto-optimal
 * (max, sum) pairs, per pair the smallest (b_{pp-1}, h_{pp-1}, ..., b_1, h_1,
 * h_0), then the least latency, ties to the lower max. */
typedef struct type_rec {
    int64_t mx, sum, c[ORC_MAX_STAGES];
    int seq[ORC_MAX_STAGES], b[ORC_MAX_STAGES + 1];
} type_rec;

typedef struct type_recs {
    const type_space *S;
    const int64_t *cost;
    int seq[ORC_MAX_STAGES], b[ORC_MAX_STAGES + 1];
    type_rec *v;
    int64_t len, cap;
} type_recs;

static void recs_parts(type_recs *x, int i)
{
    const type_space *S = x->S;
    if (i == S->pp) {
        type_rec r;
        r.mx = 0;
        r.sum = 0;
        for (int j = 0; j < S->pp; j++) {
            int hn = j + 1 < S->pp ? x->seq[j + 1] : S->T;
            int64_t c = cost_at(S, x->cost, j, x->seq[j], hn, x->b[j], x->b[j + 1]);
            if (c == ORC_INF) return;
            r.c[j] = c;
            r.sum += c;
            if (c > r.mx) r.mx = c;
        }
        memcpy(r.seq, x->seq, sizeof(r.seq));
        memcpy(r.b, x->b, sizeof(r.b));
        if (x->len == x->cap) {
            x->cap = x->cap ? 2 * x->cap : 256;
            x->v = realloc(x->v, sizeof(type_rec) * (size_t)x->cap);
        }
        x->v[x->len++] = r;
        return;
    }
    if (i == S->pp - 1) {
        x->b[S->pp] = S->n;
        if (x->b[i] < S->n) recs_parts(x, S->pp);
        return;
    }
    for (int e = x->b[i] + 1; e <= S->n - (S->pp - 1 - i); e++) {
        x->b[i + 1] = e;
        recs_parts(x, i + 1);
    }
}

static void recs_seq(type_recs *x, int i, int *left)
{
    if (i == x->S->pp) {
        x->b[0] = 0;
        recs_parts(x, 0);
        return;
    }
    for (int h = 0; h < x->S->T; h++) {
        if (left[h] == 0) continue;
        left[h]--;
        x->seq[i] = h;
        recs_seq(x, i + 1, left);
        left[h]++;
    }
}

static int rec_key_less(const type_rec *p, const type_rec *q, int pp)
{
    for (int i = pp - 1; i >= 1; i--) {
        if (p->b[i] != q->b[i]) return p->b[i] < q->b[i];
        if (p->seq[i] != q->seq[i]) return p->seq[i] < q->seq[i];
    }
    return p->seq[0] < q->seq[0];
}

int32_t orc_brute_types_exact(int32_t pp, int32_t T, const int32_t *k, int32_t n, int64_t micro,
                              const int64_t *cost, orc_result *r)
{
    type_space S;
    type_space_init(&S, pp, T, k, n);
    type_recs x;
    memset(&x, 0, sizeof(x));
    x.S = &S;
    x.cost = cost;
    int left[ORC_MAX_TYPES];
    for (int h = 0; h < T; h++) left[h] = k[h];
    recs_seq(&x, 0, left);
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    int64_t best = ORC_INF, best_mx = ORC_INF;
    const type_rec *win = NULL;
    for (int64_t i = 0; i < x.len; i++) {
        const type_rec *a = &x.v[i];
        int pareto = 1, first = 1;   /* first: the smallest key of its (max, sum) pair */
        for (int64_t j = 0; j < x.len && pareto; j++) {
            const type_rec *o = &x.v[j];
            if (o->mx <= a->mx && o->sum <= a->sum && (o->mx < a->mx || o->sum < a->sum)) pareto = 0;
            if (o->mx == a->mx && o->sum == a->sum && rec_key_less(o, a, pp)) first = 0;
        }
        if (!pareto || !first) continue;
        r->thresholds++;
        int64_t lat = orc_latency_1f1b(pp, a->c, micro);
        if (lat < best || (lat == best && a->mx < best_mx)) {
            best = lat;
            best_mx = a->mx;
            win = a;
        }
    }
    if (!win) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
    } else {
        r->opt = best;
        r->sum = win->sum;
        r->tmax = win->mx;
        for (int i = 0; i < pp; i++) {
            r->layers[i] = (uint8_t)(win->b[i + 1] - win->b[i]);
            r->stage_mask[i] = (uint8_t)(1 << win->seq[i]);
        }
    }
    free(x.v);
    return 0;
}

/* stage counts k_h of a configuration under free per-stage types */
static void type_counts(const orc_problem *p, const orc_config *c, int32_t *k)
{
    int G = 0;
    for (int h = 0; h < p->n_types; h++) G += p->count[h];
    int g = G / c->pp;
    for (int h = 0; h < p->n_types; h++) k[h] = p->count[h] / g;
}

int32_t orc_type_costs(const orc_problem *p, int64_t idx, int64_t *cost, uint8_t *rflag)
{
    orc_config c;
    int32_t order, micro;
    if (p->stage_types != 2 || orc_instance(p, idx, &c, &order, &micro)) return -1;
    int N = p->n_layers, PP = c.pp, W = N + 1, T = p->n_types;
    int32_t k[ORC_MAX_TYPES];
    type_counts(p, &c, k);
    /* the first sequence's stages give every type's stage description
     * (cap, speed, links, pruning-1 window); position and neighbour set the rest */
    orc_stage st0[ORC_MAX_STAGES], of_type[ORC_MAX_TYPES];
    int32_t seq[ORC_MAX_STAGES];
    orc_stages(p, &c, 0, micro, st0);
    orc_sequence(p, PP, 0, seq);
    for (int s = 0; s < PP; s++) of_type[seq[s]] = st0[s];
    orc_pi_terms pt;
    orc_pi_terms_eval(p, &c, &pt);
    prefixes P;
    prefixes_init(p, &c, &P);
    for (int h = 0; h < T; h++) {
        if (k[h] > 0) prefixes_time(p, &c, 1 << h, &P);
        for (int s = 0; s < PP; s++)
            for (int hn = 0; hn <= T; hn++) {
                int64_t base = (((int64_t)s * T + h) * (T + 1) + hn) * W * W;
                int ok = k[h] > 0 && (s == PP - 1 ? hn == T : hn < T && k[hn] > 0);
                orc_stage x;
                if (ok) {
                    x = of_type[h];
                    x.m_store = min64(PP - s, micro);
                    x.bdiff = hn < T && hn != h;
                    x.p2p = hn < T ? orc_p2p(p, &c, h, hn) : 0;
                }
                for (int a = 0; a < W; a++)
                    for (int b = 0; b < W; b++) {
                        if (!ok) {
                            cost[base + (int64_t)a * W + b] = ORC_INF;
                            rflag[base + (int64_t)a * W + b] = 0;
                            continue;
                        }
                        cost[base + (int64_t)a * W + b] = segment_cost(p, &pt, &x, &P, a, b,
                                                                       &rflag[base + (int64_t)a * W + b]);
                    }
            }
    }
    prefixes_free(&P);
    return 0;
}

/* ------------------------------------------------------------------------
 * Per-stage data-parallel widths (stage_types = 3): the non-uniform PP/DP
 * partitioning of the paper's contributions and its ablation ("stage-wise
 * parallelism knobs" chosen jointly with the layers).  The cost model of
 * Section 3.2 has no terms for stages of unequal width; the readings here:
 *  - the devices are listed type by type in the ordering, as for the block
 *    layout, and stage i takes the next w_i half-groups (g/2 devices each,
 *    g = G/PP), w_i in {1, 2, 3}, sum w_i = 2 PP: every device is used and the
 *    stage has DP_i = w_i DP / 2 replicas (TP, CP, EP, TPE as in pi; the
 *    configurations with DP even and EP * TPE | g/2);
 *  - every stage processes the same global micro-batch of DP * mbs sequences,
 *    split over its DP_i replicas: a replica holds r = 2 / w_i of the nominal
 *    tokens, so every per-layer term is evaluated at T = (S mbs / CP) r tokens
 *    per rank -- compute and expert tables scaled by r (they are profiled per
 *    micro-batch of mbs sequences), router and collectives at that token count;
 *  - memory: ZeRO-1 optimizer state over DP_i (beta_opt = 6 + 12 / DP_i),
 *    activations and MoE buffers at r;
 *  - the boundary transfer is the sender's per-rank activation over the link
 *    of the boundary's two device types;
 *  - pruning-1 windows from the stage's share of the cluster's compute,
 *    w_i P_i (g/2) / sum_h m_h P_h (the share among the stages when every stage
 *    is of one type); pruning 3 with the nominal T-bar; T_dp-sync + T_opt at
 *    the nominal width (the gradient sync folded into the constant, as in the
 *    uniform model).
 * A candidate's DP chooses the widths with the layers: state (stage, end
 * layer, half-groups used).
 * ---------------------------------------------------------------------- */
static double w_tokens(const orc_problem *p, const orc_config *c, double r) { return tokens(p, c) * r; }

static double w_act(const orc_problem *p, const orc_config *c, double r)
{
    return (w_tokens(p, c, r) * (double)p->hidden) * (double)p->elem_bytes;
}

/* Eq. 2 at r times the nominal tokens (compute and expert tables scale with them) */
static void w_type_terms(const orc_problem *p, const orc_config *c, int layer, int h, double r, orc_type_terms *o)
{
    int64_t off = (((int64_t)h * 4 + lg2(c->tp)) * 4 + lg2(c->cp)) * p->n_layers + layer;
    double td = (double)p->t_dense[off], tf = (double)p->t_ffn[off];
    if (!p->is_moe[layer]) {
        o->comp = td * r;
        o->expert = 0.0;
    } else {
        double route = p->route_coef[h] * (w_tokens(p, c, r) * (double)p->hidden);
        o->comp = (td - tf) * r + route;
        double xexp = (p->moe_ffn_mult * (tf * r)) / ((p->eff[h] * (double)c->ep) * (double)c->tpe);
        o->expert = skew(p, layer) * xexp;
    }
    o->q_comp = q(o->comp);
    o->q_expert = q(o->expert);
}

/* dispatch / TP / CP terms and stage times of one layer at r (as orc_mask_terms_eval) */
static void w_mask_terms(const orc_problem *p, const orc_config *c, int layer, int mask, double r, orc_mask_terms *o)
{
    double alpha, bw;
    mask_link(p, mask, &alpha, &bw);
    double D = w_act(p, c, r);
    if (!p->is_moe[layer]) {
        o->a2a = 0.0;
        o->tp = 4.0 * ring_allreduce(D, c->tp, alpha, bw);
    } else {
        double sk = skew(p, layer);
        double dm = (D * (double)p->top_k) * (1.0 - 1.0 / (double)c->ep);
        double f_a2a = (double)(c->ep - 1) * alpha + dm / bw;
        double f_ag = (double)(c->ep - 1) * alpha + (D * (double)(c->ep - 1)) / bw;
        o->a2a = sk * (4.0 * (f_ag < f_a2a ? f_ag : f_a2a));
        o->tp = 2.0 * ring_allreduce(D, c->tp, alpha, bw) + 2.0 * ring_allreduce(D, c->tpe, alpha, bw);
    }
    o->cp = c->cp == 1 ? 0.0 : 3.0 * ((double)(c->cp - 1) * (alpha + ((2.0 * D) / (double)c->tp) / bw));
    o->q_a2a = q(o->a2a);
    o->q_tp = q(o->tp);
    o->q_cp = q(o->cp);
    o->comm = o->q_a2a + o->q_tp + o->q_cp;
    int64_t ce = -1;
    for (int h = 0; h < p->n_types; h++) {
        if (!((mask >> h) & 1)) continue;
        orc_type_terms t;
        w_type_terms(p, c, layer, h, r, &t);
        if (t.q_comp + t.q_expert > ce) ce = t.q_comp + t.q_expert;
    }
    o->t_r0 = ce + o->comm;
    o->t_r1 = q(p->rc_time * (double)o->t_r0);
}

/* memory of one layer on a stage of dp_i replicas at r */
static void w_mem_terms(const orc_problem *p, const orc_config *c, int layer, int dp_i, double r, orc_mem_terms *o)
{
    double beta_opt = 6.0 + 12.0 / (double)dp_i;
    o->w = ((double)p->params_dense[layer] / (double)c->tp +
            (double)p->params_expert[layer] / (double)(c->ep * c->tpe)) * beta_opt;
    o->a0 = ((double)p->act_bytes[layer] * r) / (double)(c->tp * c->cp);
    o->q_w = q(o->w);
    o->q_a0 = q(o->a0);
    o->q_a1 = q(p->rc_act * (double)o->q_a0);
}

static int64_t w_x_bytes(const orc_problem *p, const orc_config *c, double r)
{
    double dm = (w_act(p, c, r) * (double)p->top_k) * (1.0 - 1.0 / (double)c->ep);
    return q(((8.0 * w_tokens(p, c, r)) * (double)p->top_k) + 2.0 * dm);
}

static int64_t w_p2p(const orc_problem *p, const orc_config *c, int h_from, int h_to, double r)
{
    double al = p->alpha[h_from * ORC_MAX_TYPES + h_to], bw = p->bw[h_from * ORC_MAX_TYPES + h_to];
    return q(2.0 * (al + (w_act(p, c, r) / (double)c->tp) / bw));
}

/* token share of a replica of a width-w stage: r = 2 / w */
static double w_ratio(int w) { return 2.0 / (double)w; }

/* the stage of half-groups [u, u + w) as stage s of the pipeline */
static void w_stage(const orc_problem *p, const orc_config *c, const int *perm, int s, int u, int w, int micro,
                    orc_stage *x)
{
    int G = 0;
    int64_t total_speed = 0;
    for (int h = 0; h < p->n_types; h++) {
        G += p->count[h];
        total_speed += (int64_t)p->count[h] * p->speed[h];
    }
    int PP = c->pp, half = G / PP / 2, lo = u * half, hi = (u + w) * half;
    x->mask = 0;
    for (int d = lo; d < hi; d++) x->mask |= 1 << dev_type(p, perm, d);
    x->first_type = dev_type(p, perm, lo);
    x->last_type = dev_type(p, perm, hi - 1);
    x->cap = -1;
    x->speed = 0;
    for (int h = 0; h < p->n_types; h++) {
        if (!((x->mask >> h) & 1)) continue;
        if (x->cap < 0 || p->mem_bytes[h] < x->cap) x->cap = p->mem_bytes[h];
        if (x->speed == 0 || p->speed[h] < x->speed) x->speed = p->speed[h];
    }
    mask_link(p, x->mask, &x->alpha, &x->bw);
    x->mixed = popc(x->mask) > 1;
    if (u + w < 2 * PP) {
        int nt = dev_type(p, perm, hi);
        x->bdiff = nt != x->last_type;
        x->p2p = w_p2p(p, c, x->last_type, nt, w_ratio(w));
    } else {
        x->bdiff = 0;
        x->p2p = 0;
    }
    x->m_store = min64(PP - s, micro);
    int64_t N = p->n_layers, dn = p->delta_num, dd = p->delta_den;
    if (p->prune_window == 1) {
        /* share w P (g/2) / sum_h m_h P_h of the cluster's compute */
        int64_t num = (int64_t)w * x->speed * half * N, den = dd * total_speed;
        x->lo = (int32_t)max64(1, ((dd - dn) * num) / den);
        x->hi = (int32_t)min64(N, ((dd + dn) * num + den - 1) / den);
    } else if (p->prune_window == 2) {
        x->lo = (int32_t)(N / PP);
        x->hi = (int32_t)((N + PP - 1) / PP);
    } else {
        x->lo = 1;
        x->hi = (int32_t)N;
    }
}

/* the width-scaled terms of one layer, for the tests */
void orc_width_terms(const orc_problem *p, const orc_config *c, int32_t layer, int32_t mask, int32_t w,
                     orc_type_terms *type_out, orc_mask_terms *mask_out, orc_mem_terms *mem_out, int64_t *x_bytes)
{
    double r = w_ratio(w);
    for (int h = 0; h < p->n_types; h++) w_type_terms(p, c, layer, h, r, &type_out[h]);
    w_mask_terms(p, c, layer, mask, r, mask_out);
    w_mem_terms(p, c, layer, c->dp * w / 2, r, mem_out);
    *x_bytes = w_x_bytes(p, c, r);
}

/* the stage of half-groups [u, u + w) as stage s (layout, window, boundary), for the tests */
int32_t orc_width_stage(const orc_problem *p, const orc_config *c, int32_t order, int32_t s, int32_t u, int32_t w,
                        int32_t micro, orc_stage *x)
{
    if (w < 1 || w > 3 || u < 0 || u + w > 2 * c->pp) return -1;
    int perm[ORC_MAX_TYPES];
    orc_order(p, order, perm);
    w_stage(p, c, perm, s, u, w, micro, x);
    return 0;
}

/* Cost tensor of a width-mode candidate: [pp][2pp + 1][3][n + 1][n + 1], entry
 * (s, u, w - 1, a, b) = c_s(a, b) of stage s on half-groups [u, u + w) */
int32_t orc_width_costs(const orc_problem *p, int64_t idx, int64_t *cost, uint8_t *rflag)
{
    orc_config c;
    int32_t order, micro;
    if (p->stage_types != 3 || orc_instance(p, idx, &c, &order, &micro)) return -1;
    int perm[ORC_MAX_TYPES];
    orc_order(p, order, perm);
    int N = p->n_layers, W = N + 1, PP = c.pp, U = 2 * PP;
    orc_pi_terms pt;
    orc_pi_terms_eval(p, &c, &pt);   /* the nominal T-bar */
    prefixes P;
    for (int w = 1; w <= 3; w++) {
        double r = w_ratio(w);
        orc_pi_terms ptw = pt;
        ptw.x_bytes = w_x_bytes(p, &c, r);
        int dp_i = c.dp * w / 2;
        P.n = N;
        P.w = calloc((size_t)W, 8);
        P.a0 = calloc((size_t)W, 8);
        P.a1 = calloc((size_t)W, 8);
        P.moe = calloc((size_t)W, 8);
        P.t0 = calloc((size_t)W, 8);
        P.t1 = calloc((size_t)W, 8);
        P.comm = calloc((size_t)W, 8);
        for (int l = 0; l < N; l++) {
            orc_mem_terms m;
            w_mem_terms(p, &c, l, dp_i, r, &m);
            P.w[l + 1] = P.w[l] + m.q_w;
            P.a0[l + 1] = P.a0[l] + m.q_a0;
            P.a1[l + 1] = P.a1[l] + m.q_a1;
            P.moe[l + 1] = P.moe[l] + (p->is_moe[l] ? 1 : 0);
        }
        for (int s = 0; s < PP; s++)
            for (int u = 0; u <= U; u++) {
                int64_t base = (((int64_t)s * (U + 1) + u) * 3 + (w - 1)) * W * W;
                int ok = u + w <= U;
                orc_stage x;
                if (ok) {
                    w_stage(p, &c, perm, s, u, w, micro, &x);
                    for (int l = 0; l < N; l++) {
                        orc_mask_terms m;
                        w_mask_terms(p, &c, l, x.mask, r, &m);
                        P.t0[l + 1] = P.t0[l] + m.t_r0;
                        P.t1[l + 1] = P.t1[l] + m.t_r1;
                        P.comm[l + 1] = P.comm[l] + m.comm;
                    }
                }
                for (int a = 0; a < W; a++)
                    for (int b = 0; b < W; b++) {
                        uint8_t rr = 0;
                        cost[base + (int64_t)a * W + b] = ok ? segment_cost(p, &ptw, &x, &P, a, b, &rr) : ORC_INF;
                        rflag[base + (int64_t)a * W + b] = rr;
                    }
            }
        prefixes_free(&P);
    }
    return 0;
}

/* Threshold DP over (stage, end layer, half-groups used): F_t[i][b][u] = the
 * least stage sum placing layers [0, b) on stages 1..i that use u half-groups,
 * every stage cost <= t; ties keep the smallest split point a, then the
 * smallest width.  OPT = min over t of F_t[pp][n][2pp] + (B-1) t, the sweep and
 * t* as in orc_dp; the back-trace at t* gives the lexicographically smallest
 * ((b_{pp-1}, w_pp), (b_{pp-2}, w_{pp-1}), ..., (0, w_1)) among the optima. */
static int64_t w_pass(int pp, int n, const int64_t *cost, int64_t t, int64_t *F, int16_t *arg)
{
    int W = n + 1, U = 2 * pp;
    for (int i = 0; i <= pp; i++)
        for (int b = 0; b < W; b++)
            for (int u = 0; u <= U; u++) F[((int64_t)i * W + b) * (U + 1) + u] = (i == 0 && b == 0 && u == 0) ? 0 : ORC_INF;
    for (int i = 1; i <= pp; i++)
        for (int b = 1; b < W; b++)
            for (int u = 1; u <= U; u++) {
                int64_t best = ORC_INF;
                int arg_best = -1;
                for (int a = 0; a < b; a++)
                    for (int w = 1; w <= 3 && w <= u; w++) {
                        int64_t prev = F[((int64_t)(i - 1) * W + a) * (U + 1) + (u - w)];
                        int64_t cst = cost[((((int64_t)(i - 1) * (U + 1) + (u - w)) * 3 + (w - 1)) * W + a) * W + b];
                        if (prev == ORC_INF || cst == ORC_INF || cst > t) continue;
                        if (prev + cst < best) {
                            best = prev + cst;
                            arg_best = a * 4 + w;
                        }
                    }
                F[((int64_t)i * W + b) * (U + 1) + u] = best;
                arg[((int64_t)i * W + b) * (U + 1) + u] = (int16_t)arg_best;
            }
    return F[((int64_t)pp * W + n) * (U + 1) + U];
}

int32_t orc_dp_widths(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r)
{
    int W = n + 1, U = 2 * pp;
    int64_t ncost = (int64_t)pp * (U + 1) * 3 * W * W, nstate = (int64_t)(pp + 1) * W * (U + 1);
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    int64_t *theta = malloc(sizeof(int64_t) * (size_t)(ncost + 1));
    int64_t nt = 0;
    for (int64_t i = 0; i < ncost; i++)
        if (cost[i] != ORC_INF) theta[nt++] = cost[i];
    qsort(theta, (size_t)nt, sizeof(int64_t), cmp_i64);
    int64_t u = 0;
    for (int64_t i = 0; i < nt; i++)
        if (u == 0 || theta[i] != theta[u - 1]) theta[u++] = theta[i];
    int64_t *F = malloc(sizeof(int64_t) * (size_t)nstate);
    int16_t *arg = malloc(sizeof(int16_t) * (size_t)nstate);
    int64_t finf = pp <= n ? w_pass(pp, n, cost, ORC_INF, F, arg) : ORC_INF;
    int64_t best = ORC_INF, tstar = -1, swept = 0;
    for (int64_t k = 0; k < u && finf != ORC_INF; k++) {
        int64_t t = theta[k];
        if (finf + (micro - 1) * t >= best) break;
        int64_t f = w_pass(pp, n, cost, t, F, arg);
        swept++;
        if (f == ORC_INF) continue;
        if (f + (micro - 1) * t < best) {
            best = f + (micro - 1) * t;
            tstar = t;
        }
    }
    r->thresholds = swept;
    if (tstar < 0) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
    } else {
        r->sum = w_pass(pp, n, cost, tstar, F, arg);
        r->tmax = tstar;
        r->opt = best;
        int b = n, uu = U;
        for (int i = pp; i >= 1; i--) {
            int x = arg[((int64_t)i * W + b) * (U + 1) + uu], a = x / 4, w = x % 4;
            r->layers[i - 1] = (uint8_t)(b - a);
            r->width[i - 1] = (uint8_t)w;
            b = a;
            uu -= w;
        }
    }
    free(theta);
    free(F);
    free(arg);
    return 0;
}

/* Brute force: every width sequence (w_i in {1, 2, 3}, sum 2 pp) and every
 * composition; key (sum + (B-1) max, max, then (b_{pp-1}, w_pp), (b_{pp-2},
 * w_{pp-1}), ...) ascending. */
typedef struct w_brute {
    int pp, n, W, U;
    int64_t micro;
    const int64_t *cost;
    int b[ORC_MAX_STAGES + 1], w[ORC_MAX_STAGES];
    int best_b[ORC_MAX_STAGES + 1], best_w[ORC_MAX_STAGES];
    int64_t best_obj, best_max, best_sum;
    int found;
} w_brute;

static int w_brute_better(const w_brute *x, int64_t obj, int64_t mx)
{
    if (!x->found) return 1;
    if (obj != x->best_obj) return obj < x->best_obj;
    if (mx != x->best_max) return mx < x->best_max;
    for (int i = x->pp - 1; i >= 0; i--) {
        if (x->b[i] != x->best_b[i]) return x->b[i] < x->best_b[i];
        if (x->w[i] != x->best_w[i]) return x->w[i] < x->best_w[i];
    }
    return 0;
}

static void w_brute_parts(w_brute *x, int i)
{
    if (i == x->pp) {
        int64_t sum = 0, mx = 0;
        int u = 0;
        for (int k = 0; k < x->pp; k++) {
            int64_t c = x->cost[((((int64_t)k * (x->U + 1) + u) * 3 + (x->w[k] - 1)) * x->W + x->b[k]) * x->W + x->b[k + 1]];
            if (c == ORC_INF) return;
            sum += c;
            if (c > mx) mx = c;
            u += x->w[k];
        }
        int64_t obj = sum + (x->micro - 1) * mx;
        if (w_brute_better(x, obj, mx)) {
            x->found = 1;
            x->best_obj = obj;
            x->best_max = mx;
            x->best_sum = sum;
            memcpy(x->best_b, x->b, sizeof(x->b));
            memcpy(x->best_w, x->w, sizeof(x->w));
        }
        return;
    }
    if (i == x->pp - 1) {
        x->b[i + 1] = x->n;
        if (x->b[i] < x->n) w_brute_parts(x, i + 1);
        return;
    }
    for (int e = x->b[i] + 1; e <= x->n - (x->pp - 1 - i); e++) {
        x->b[i + 1] = e;
        w_brute_parts(x, i + 1);
    }
}

static void w_brute_seq(w_brute *x, int i, int used)
{
    if (i == x->pp) {
        if (used == x->U) w_brute_parts(x, 0);
        return;
    }
    for (int w = 1; w <= 3; w++) {
        x->w[i] = w;
        w_brute_seq(x, i + 1, used + w);
    }
}

int32_t orc_brute_widths(int32_t pp, int32_t n, int64_t micro, const int64_t *cost, orc_result *r)
{
    memset(r, 0, sizeof(*r));
    r->pp = pp;
    w_brute x;
    memset(&x, 0, sizeof(x));
    x.pp = pp;
    x.n = n;
    x.W = n + 1;
    x.U = 2 * pp;
    x.micro = micro;
    x.cost = cost;
    if (pp <= n) w_brute_seq(&x, 0, 0);
    if (!x.found) {
        r->status = 1;
        r->opt = r->sum = r->tmax = ORC_INF;
        return 0;
    }
    r->opt = x.best_obj;
    r->sum = x.best_sum;
    r->tmax = x.best_max;
    for (int i = 0; i < pp; i++) {
        r->layers[i] = (uint8_t)(x.best_b[i + 1] - x.best_b[i]);
        r->width[i] = (uint8_t)x.best_w[i];
    }
    return 0;
}

static int32_t solve_widths(const orc_problem *p, int64_t idx, orc_result *r, int mode)
{
    orc_config c;
    int32_t order, micro;
    if (mode > 1 || orc_instance(p, idx, &c, &order, &micro)) return -1;
    int W = p->n_layers + 1, U = 2 * c.pp;
    int64_t ncost = (int64_t)c.pp * (U + 1) * 3 * W * W;
    int64_t *cost = malloc(sizeof(int64_t) * (size_t)ncost);
    uint8_t *rf = malloc((size_t)ncost);
    orc_width_costs(p, idx, cost, rf);
    if (mode == 0)
        orc_dp_widths(c.pp, p->n_layers, micro, cost, r);
    else
        orc_brute_widths(c.pp, p->n_layers, micro, cost, r);
    /* T_dp-sync + T_opt of the uniform layout of the same (pi, ordering) */
    orc_problem q0 = *p;
    q0.stage_types = 0;
    r->dp_const = orc_dp_const(&q0, &c, order);
    if (r->status == 0) {
        r->opt += r->dp_const;
        int perm[ORC_MAX_TYPES];
        orc_order(p, order, perm);
        int a = 0, u = 0;
        for (int i = 0; i < c.pp; i++) {
            int b = a + r->layers[i], w = r->width[i];
            orc_stage x;
            w_stage(p, &c, perm, i, u, w, micro, &x);
            r->stage_mask[i] = (uint8_t)x.mask;
            r->recompute[i] = rf[((((int64_t)i * (U + 1) + u) * 3 + (w - 1)) * W + a) * W + b];
            a = b;
            u += w;
        }
    }
    free(cost);
    free(rf);
    return 0;
}

/* mode: 0 threshold DP, 1 its brute force, 2 1F1B re-scoring, 3 its brute force */
static int32_t solve_types(const orc_problem *p, int64_t idx, orc_result *r, int mode)
{
    orc_config c;
    int32_t order, micro;
    if (orc_instance(p, idx, &c, &order, &micro)) return -1;
    int T = p->n_types, W = p->n_layers + 1;
    int32_t k[ORC_MAX_TYPES];
    type_counts(p, &c, k);
    int64_t ncost = (int64_t)c.pp * T * (T + 1) * W * W;
    int64_t *cost = malloc(sizeof(int64_t) * (size_t)ncost);
    uint8_t *rf = malloc((size_t)ncost);
    orc_type_costs(p, idx, cost, rf);
    if (mode == 0)
        orc_dp_types(c.pp, T, k, p->n_layers, micro, cost, r);
    else if (mode == 1)
        orc_brute_types(c.pp, T, k, p->n_layers, micro, cost, r);
    else if (mode == 2)
        orc_dp_types_exact(c.pp, T, k, p->n_layers, micro, cost, r);
    else
        orc_brute_types_exact(c.pp, T, k, p->n_layers, micro, cost, r);
    r->dp_const = orc_dp_const(p, &c, 0);
    if (r->status == 0) {
        r->opt += r->dp_const;
        int a = 0;
        for (int i = 0; i < c.pp; i++) {
            int b = a + r->layers[i], h = 0, hn = T;
            while (!((r->stage_mask[i] >> h) & 1)) h++;
            if (i + 1 < c.pp)
                for (hn = 0; !((r->stage_mask[i + 1] >> hn) & 1); hn++) {}
            r->recompute[i] = rf[((((int64_t)i * T + h) * (T + 1) + hn) * W + a) * W + b];
            a = b;
        }
    }
    free(cost);
    free(rf);
    return 0;
}

/* mode: 0 threshold DP, 1 its brute force, 2 1F1B frontier re-scoring, 3 its
 * brute force, 4 the least 1F1B latency, 5 its brute force */
static int32_t solve_with(const orc_problem *p, int64_t idx, orc_result *r, int mode)
{
    if (p->stage_types == 2) {   /* the device-count DP (no least-latency mode) */
        if (mode > 3) return -1;
        return solve_types(p, idx, r, mode);
    }
    if (p->stage_types == 3) return solve_widths(p, idx, r, mode);   /* per-stage widths */
    orc_config c;
    int32_t order, micro;
    if (orc_instance(p, idx, &c, &order, &micro)) return -1;
    int W = p->n_layers + 1;
    int64_t *cost = malloc(sizeof(int64_t) * (size_t)c.pp * W * W);
    uint8_t *rf = malloc((size_t)c.pp * W * W);
    orc_segment_costs(p, idx, cost, rf);
    if (mode == 0)
        orc_dp(c.pp, p->n_layers, micro, cost, r);
    else if (mode == 1)
        orc_brute(c.pp, p->n_layers, micro, cost, r);
    else if (mode == 2)
        orc_dp_exact(c.pp, p->n_layers, micro, cost, r);
    else if (mode == 3)
        orc_brute_exact(c.pp, p->n_layers, micro, cost, r);
    else if (mode == 4)
        orc_dp_latency(c.pp, p->n_layers, micro, cost, r);
    else
        orc_brute_latency(c.pp, p->n_layers, micro, cost, r);
    orc_stage st[ORC_MAX_STAGES];
    const int laid = orc_stages(p, &c, order, micro, st) == 0;
    for (int i = 0; i < c.pp; i++) r->stage_mask[i] = laid ? (uint8_t)st[i].mask : 0;
    r->dp_const = orc_dp_const(p, &c, order);
    if (r->status == 0) {
        r->opt += r->dp_const;
        int a = 0;
        for (int i = 0; i < c.pp; i++) {
            int b = a + r->layers[i];
            r->recompute[i] = rf[((int64_t)i * W + a) * W + b];
            a = b;
        }
    }
    free(cost);
    free(rf);
    return 0;
}

int32_t orc_solve(const orc_problem *p, int64_t idx, orc_result *r) { return solve_with(p, idx, r, 0); }
int32_t orc_solve_brute(const orc_problem *p, int64_t idx, orc_result *r) { return solve_with(p, idx, r, 1); }

int32_t orc_solve_many(const orc_problem *p, const int64_t *idx, int64_t n, orc_result *r)
{
    for (int64_t i = 0; i < n; i++)
        if (orc_solve(p, idx[i], &r[i])) return -1;
    return 0;
}

int32_t orc_solve_exact(const orc_problem *p, int64_t idx, orc_result *r) { return solve_with(p, idx, r, 2); }
int32_t orc_solve_exact_brute(const orc_problem *p, int64_t idx, orc_result *r) { return solve_with(p, idx, r, 3); }

int32_t orc_solve_exact_many(const orc_problem *p, const int64_t *idx, int64_t n, orc_result *r)
{
    for (int64_t i = 0; i < n; i++)
        if (orc_solve_exact(p, idx[i], &r[i])) return -1;
    return 0;
}

int32_t orc_solve_latency(const orc_problem *p, int64_t idx, orc_result *r) { return solve_with(p, idx, r, 4); }
int32_t orc_solve_latency_brute(const orc_problem *p, int64_t idx, orc_result *r) { return solve_with(p, idx, r, 5); }

int32_t orc_solve_latency_many(const orc_problem *p, const int64_t *idx, int64_t n, orc_result *r)
{
    for (int64_t i = 0; i < n; i++)
        if (orc_solve_latency(p, idx[i], &r[i])) return -1;
    return 0;
}
