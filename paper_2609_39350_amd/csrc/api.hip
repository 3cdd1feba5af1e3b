// Host side of the C ABI declared in include/hapmoe.h: argument checks, the
// candidate enumeration, the device problem image, buffer-size queries and the
// kernel launches.  No device memory is allocated here.
#include <algorithm>
#include <array>
#include <atomic>
#include <cmath>
#include <cstring>
#include <vector>

#include "internal.h"

using namespace hapmoe;

namespace {

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

int32_t check_fields(const hapmoe_problem *p)
{
    if (!p) return HAPMOE_E_INVAL;
    const hapmoe_model &m = p->model;
    const hapmoe_cluster &c = p->cluster;
    const hapmoe_params &q = p->params;
    const hapmoe_space &s = p->space;
    const int N = m.n_layers, T = c.n_types;
    if (N < 1 || N > kMaxLayers || T < 1 || T > kMaxTypes) return HAPMOE_E_INVAL;
    if (m.seq_len < 1 || m.hidden < 1 || m.micro_batch_size < 1 || m.elem_bytes < 0) return HAPMOE_E_INVAL;
    if ((int64_t)m.seq_len * m.micro_batch_size > (int64_t(1) << 31)) return HAPMOE_E_INVAL;
    if (m.n_experts < 0 || m.n_experts > 65536) return HAPMOE_E_INVAL;
    if (m.n_experts > 0 && (m.top_k < 1 || m.top_k > m.n_experts)) return HAPMOE_E_INVAL;
    if (!finite_nonneg(m.moe_ffn_mult)) return HAPMOE_E_INVAL;
    if (!m.is_moe || !m.params_dense || !m.params_expert || !m.act_bytes) return HAPMOE_E_INVAL;
    if (m.n_experts > 0 && !m.expert_tokens) return HAPMOE_E_INVAL;
    const int64_t big = int64_t(1) << 50;
    for (int l = 0; l < N; ++l) {
        if (m.is_moe[l] > 1 || (m.is_moe[l] && m.n_experts == 0)) return HAPMOE_E_INVAL;
        if (m.params_dense[l] < 0 || m.params_dense[l] > big) return HAPMOE_E_INVAL;
        if (m.params_expert[l] < 0 || m.params_expert[l] > big) return HAPMOE_E_INVAL;
        if (m.act_bytes[l] < 0 || m.act_bytes[l] > big) return HAPMOE_E_INVAL;
        for (int e = 0; e < m.n_experts; ++e) {
            const int64_t v = m.expert_tokens[(int64_t)l * m.n_experts + e];
            if (v < 0 || v > (int64_t(1) << 40)) return HAPMOE_E_INVAL;
        }
    }
    int64_t G = 0;
    for (int h = 0; h < T; ++h) {
        if (c.count[h] < 1 || c.speed[h] < 1 || c.speed[h] > 1000000 || c.mem_bytes[h] < 0) return HAPMOE_E_INVAL;
        if (!(std::isfinite(c.eff[h]) && c.eff[h] > 0.0) || !finite_nonneg(c.route_coef[h])) return HAPMOE_E_INVAL;
        for (int g = 0; g < T; ++g)
            if (!(std::isfinite(c.bw[h][g]) && c.bw[h][g] > 0.0) || !finite_nonneg(c.alpha[h][g]))
                return HAPMOE_E_INVAL;
        G += c.count[h];
    }
    if (G > (1 << 20)) return HAPMOE_E_INVAL;
    if (!c.t_dense || !c.t_ffn) return HAPMOE_E_INVAL;
    for (int64_t i = 0; i < (int64_t)T * 16 * N; ++i)
        if (c.t_dense[i] < 0 || c.t_dense[i] > (int64_t(1) << 40) || c.t_ffn[i] < 0 || c.t_ffn[i] > c.t_dense[i])
            return HAPMOE_E_INVAL;
    if (!(q.rc_time >= 1.0 && q.rc_time <= 16.0) || !(q.rc_act >= 0.0 && q.rc_act <= 1.0)) return HAPMOE_E_INVAL;
    if (!(q.gamma >= 0.0 && q.gamma <= 1.0) || !finite_nonneg(q.opt_coef)) return HAPMOE_E_INVAL;
    if (q.delta_den < 1 || q.delta_den > 1000000 || q.delta_num < 0 || q.delta_num >= q.delta_den)
        return HAPMOE_E_INVAL;
    if (q.eta_prune < 0 || q.eta_prune > 1000000) return HAPMOE_E_INVAL;
    if (q.prune_window < 0 || q.prune_window > 2) return HAPMOE_E_INVAL;
    if (s.pp_max < 1 || s.pp_max > kMaxStages || s.mode < 0 || s.mode > 1 || s.ep_max < 1) return HAPMOE_E_INVAL;
    if (s.tp_mask < 0 || s.tp_mask > 15 || s.cp_mask < 0 || s.cp_mask > 15 || s.tpe_mask < 0 || s.tpe_mask > 15)
        return HAPMOE_E_INVAL;
    if (s.n_micro < 1 || s.n_micro > HAPMOE_MAX_MICRO) return HAPMOE_E_INVAL;
    for (int i = 0; i < s.n_micro; ++i)
        if (s.micro[i] < 1 || s.micro[i] > kMaxMicroValue) return HAPMOE_E_INVAL;
    if (s.stage_types < 0 || s.stage_types > 3) return HAPMOE_E_INVAL;
    if (s.global_batch < 0) return HAPMOE_E_INVAL;
    return HAPMOE_OK;
}

// The configuration set, the type orderings and the LDS bounds of the DP kernel.
struct Space {
    std::vector<std::array<int32_t, 6>> cfg;   // pp, tp, cp, dp, ep, tpe
    std::vector<std::array<int8_t, kMaxTypes>> perm;   // block orderings (stage_types = 0)
    int64_t n_orders = 1;   // orderings, or the most stage-type sequences (stage_types = 1)
    int kmax = 1;    // distinct device-type sets over the stages of any candidate
    int ppmax = 1;
    int umax = 1;    // device-count DP: most states u = prod_h (k_h + 1) of a pipeline
};

constexpr int64_t kMaxFreeOrders = int64_t(1) << 20;
constexpr int64_t kMaxKeys = int64_t(1) << 31;   // (configuration, order) keys: a 32-bit work queue

// distinct arrangements of k_h = m_h / g stages of each type h, pp! / prod k_h!,
// built one stage at a time: the running multinomial never falls, so it can
// stop at a cap above every accepted count and stay exact below it
int64_t arrangements(const hapmoe_cluster &c, int g)
{
    constexpr int64_t cap = int64_t(1) << 40;
    int64_t n = 1;
    int r = 0;
    for (int h = 0; h < c.n_types; ++h)
        for (int i = 1; i <= c.count[h] / g; ++i) {
            n = n * ++r / i;
            if (n > cap) return cap;
        }
    return n;
}

void build_space(const hapmoe_problem *p, Space &S)
{
    const hapmoe_model &m = p->model;
    const hapmoe_cluster &c = p->cluster;
    const hapmoe_space &sp = p->space;
    const int T = c.n_types;
    int G = 0;
    for (int h = 0; h < T; ++h) G += c.count[h];

    std::vector<int> tps, cps, tpes, eps;
    for (int i = 0; i < 4; ++i) {
        if ((sp.tp_mask >> i) & 1) tps.push_back(1 << i);
        if ((sp.cp_mask >> i) & 1) cps.push_back(1 << i);
        if ((sp.tpe_mask >> i) & 1) tpes.push_back(1 << i);
    }
    const bool dense = m.n_experts == 0;
    if (dense) {
        eps = {1};
        tpes = {1};
    } else {
        for (int e = 1; e <= sp.ep_max && e <= m.n_experts; e *= 2)
            if (m.n_experts % e == 0) eps.push_back(e);
    }
    S.cfg.clear();
    S.cfg.reserve(4096);
    S.kmax = 1;
    S.ppmax = 1;
    S.umax = 1;
    const bool free_types = sp.stage_types == 1 || sp.stage_types == 2;
    const bool widths = sp.stage_types == 3;
    S.n_orders = 1;
    for (int PP = 1; PP <= std::min(G, std::min(sp.pp_max, m.n_layers)); ++PP) {
        if (G % PP) continue;
        const int g = G / PP;
        if (free_types) {   // every stage one group of a single type
            bool whole = true;
            for (int h = 0; h < T; ++h) whole &= c.count[h] % g == 0;
            if (!whole) continue;
        }
        bool any = false;
        // TP, CP, EP and TPE are powers of two, so every divisibility test below is
        // a mask test: x % d == (x & (d - 1)) for x >= 0
        for (int TP : tps) {
            if ((g & (TP - 1)) || (m.hidden & (TP - 1))) continue;
            for (int CP : cps) {
                if (m.seq_len & (CP - 1)) continue;
                for (int EP : eps)
                    for (int TPE : tpes) {
                        int DP;
                        if (sp.mode == 0) {
                            if ((g & (TP * CP - 1)) || (g & (EP * TPE - 1))) continue;
                            DP = g / (TP * CP);
                        } else {
                            const int prod = TP * CP * EP * TPE;
                            if (g & (prod - 1)) continue;
                            DP = g / prod;
                        }
                        // per-stage widths: half a group holds whole replicas and expert groups
                        if (widths && ((DP & 1) || ((g / 2) & (EP * TPE - 1)))) continue;
                        S.cfg.push_back({PP, TP, CP, DP, EP, TPE});
                        any = true;
                    }
            }
        }
        if (any) {
            // pure stages use at most T sets; a stage straddling a type boundary
            // (possible only if some m_h is not a multiple of the group) adds at most T-1
            bool straddle = false;
            for (int h = 0; h < T; ++h) straddle |= (c.count[h] % g) != 0;
            S.kmax = std::max(S.kmax, std::min(PP, T + (straddle ? T - 1 : 0)));
            S.ppmax = std::max(S.ppmax, PP);
            if (sp.stage_types == 1) S.n_orders = std::max(S.n_orders, arrangements(c, g));
            if (sp.stage_types == 2) {
                int64_t U = 1;
                for (int h = 0; h < T; ++h) U *= c.count[h] / g + 1;
                S.umax = (int)std::min<int64_t>(std::max<int64_t>(S.umax, U), int64_t(1) << 30);
            }
        }
    }
    std::array<int8_t, kMaxTypes> cur{};
    for (int h = 0; h < T; ++h) cur[h] = (int8_t)h;
    S.perm.clear();
    if (free_types) return;
    do {
        S.perm.push_back(cur);
    } while (std::next_permutation(cur.begin(), cur.begin() + T));
    S.n_orders = (int64_t)S.perm.size();
}

int32_t check_problem(const hapmoe_problem *p)
{
    if (const int32_t e = check_fields(p)) return e;
    if (p->space.stage_types) {   // the sequence count, the key queue and the DP states stay in range
        Space S;
        build_space(p, S);
        if (S.cfg.empty() || S.n_orders > kMaxFreeOrders || (int64_t)S.cfg.size() * S.n_orders > kMaxKeys)
            return HAPMOE_E_INVAL;
        if (p->space.stage_types == 2 &&
            (S.umax > kMaxTypeStates ||
             type_dp_lds(p->model.n_layers, p->cluster.n_types, p->space.n_micro, S.umax, S.ppmax).bytes >
                 kTypeDpMaxLds))
            return HAPMOE_E_INVAL;
    }
    return HAPMOE_OK;
}

// The architecture check runs on every device call; its answer per device is
// cached.  Each slot is an atomic written with the same value by whichever
// thread gets there first, so concurrent callers on any devices are safe.
int check_arch()
{
    static std::atomic<int> cache[64];   // 0 unknown, 1 gfx950, 2 other (zero-initialised)
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return HAPMOE_E_HIP;
    const bool slot = dev >= 0 && dev < 64;
    const int known = slot ? cache[dev].load(std::memory_order_relaxed) : 0;
    if (known) return known == 1 ? HAPMOE_OK : HAPMOE_E_ARCH;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return HAPMOE_E_HIP;
    const bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    if (slot) cache[dev].store(ok ? 1 : 2, std::memory_order_relaxed);
    return ok ? HAPMOE_OK : HAPMOE_E_ARCH;
}

struct ImageLayout {
    int64_t off_is_moe, off_tokens, off_pdense, off_pexp, off_act, off_tdense, off_tffn, total;
};

ImageLayout image_layout(const hapmoe_problem *p)
{
    const int64_t N = p->model.n_layers, E = p->model.n_experts, T = p->cluster.n_types;
    ImageLayout I;
    I.off_is_moe = align256((int64_t)sizeof(ImageHeader));
    I.off_tokens = align256(I.off_is_moe + N);
    I.off_pdense = align256(I.off_tokens + N * E * 8);
    I.off_pexp = align256(I.off_pdense + N * 8);
    I.off_act = align256(I.off_pexp + N * 8);
    I.off_tdense = align256(I.off_act + N * 8);
    I.off_tffn = align256(I.off_tdense + T * 16 * N * 8);
    I.total = align256(I.off_tffn + T * 16 * N * 8);
    return I;
}

int64_t per_config(const hapmoe_problem *p, const Space &S)
{
    return S.n_orders * p->space.n_micro;
}

}  // namespace

extern "C" {

int32_t hapmoe_section_clocks(uint64_t out[16], int32_t clear)
{
    if (!out) return HAPMOE_E_INVAL;
    for (int i = 0; i < 16; ++i) out[i] = 0;
    static_assert(kSectionClocks <= 16, "section table");
    return stage_dp_section_clocks(out, clear != 0);
}

const char *hapmoe_strerror(int32_t code)
{
    switch (code) {
    case HAPMOE_OK: return "ok";
    case HAPMOE_E_INVAL: return "invalid problem or argument";
    case HAPMOE_E_CAPACITY: return "output array too small";
    case HAPMOE_E_WORKSPACE: return "device buffer too small";
    case HAPMOE_E_HIP: return "HIP runtime error";
    case HAPMOE_E_ARCH: return "current device is not gfx950";
    case HAPMOE_E_INFEASIBLE: return "no candidate has a feasible partition";
    case HAPMOE_E_RANGE: return "candidate range out of bounds";
    default: return "unknown status";
    }
}

int32_t hapmoe_validate(const hapmoe_problem *p) { return check_problem(p); }

int32_t hapmoe_enumerate_candidates(const hapmoe_problem *p, hapmoe_candidate *out, int64_t capacity,
                                    int64_t *n_total)
{
    if (n_total) *n_total = 0;
    if (const int32_t e = check_problem(p)) return e;
    if (!n_total || capacity < 0) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    const int64_t total = (int64_t)S.cfg.size() * per_config(p, S);
    *n_total = total;
    if (out) {
        int64_t k = 0;
        for (const auto &cf : S.cfg)
            for (int o = 0; o < (int)S.n_orders; ++o)
                for (int b = 0; b < p->space.n_micro; ++b) {
                    if (k >= capacity) break;
                    hapmoe_candidate &x = out[k++];
                    x.pp = cf[0];
                    x.tp = cf[1];
                    x.cp = cf[2];
                    x.dp = cf[3];
                    x.ep = cf[4];
                    x.tpe = cf[5];
                    x.order = o;
                    x.n_micro = p->space.micro[b];
                }
    }
    return (!out || capacity < total) ? HAPMOE_E_CAPACITY : HAPMOE_OK;
}

int32_t hapmoe_image_bytes(const hapmoe_problem *p, int64_t *bytes)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!bytes) return HAPMOE_E_INVAL;
    *bytes = image_layout(p).total;
    return HAPMOE_OK;
}

int32_t hapmoe_pack_image(const hapmoe_problem *p, void *h_image, int64_t bytes)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!h_image) return HAPMOE_E_INVAL;
    const ImageLayout I = image_layout(p);
    if (bytes < I.total) return HAPMOE_E_WORKSPACE;
    Space S;
    build_space(p, S);
    unsigned char *base = static_cast<unsigned char *>(h_image);
    std::memset(base, 0, (size_t)I.total);
    ImageHeader &H = *reinterpret_cast<ImageHeader *>(base);
    const hapmoe_model &m = p->model;
    const hapmoe_cluster &c = p->cluster;
    const hapmoe_params &q = p->params;
    H.n_layers = m.n_layers;
    H.seq_len = m.seq_len;
    H.hidden = m.hidden;
    H.n_experts = m.n_experts;
    H.top_k = m.top_k;
    H.mbs = m.micro_batch_size;
    H.elem_bytes = m.elem_bytes;
    H.n_types = c.n_types;
    H.total_devices = 0;
    for (int h = 0; h < kMaxTypes; ++h) {
        const bool on = h < c.n_types;
        H.count[h] = on ? c.count[h] : 0;
        H.speed[h] = on ? c.speed[h] : 0;
        H.mem_bytes[h] = on ? c.mem_bytes[h] : 0;
        H.eff[h] = on ? c.eff[h] : 1.0;
        H.route_coef[h] = on ? c.route_coef[h] : 0.0;
        H.total_devices += H.count[h];
        for (int g = 0; g < kMaxTypes; ++g) {
            const bool on2 = on && g < c.n_types;
            H.bw[h * kMaxTypes + g] = on2 ? c.bw[h][g] : 1.0;
            H.alpha[h * kMaxTypes + g] = on2 ? c.alpha[h][g] : 0.0;
        }
    }
    H.moe_ffn_mult = m.moe_ffn_mult;
    H.gamma = q.gamma;
    H.rc_time = q.rc_time;
    H.rc_act = q.rc_act;
    H.opt_coef = q.opt_coef;
    H.delta_num = q.delta_num;
    H.delta_den = q.delta_den;
    H.eta_prune = q.eta_prune;
    H.prune_window = q.prune_window;   // 0, 1 or 2 (checked)
    H.prune_hetero = q.prune_hetero ? 1 : 0;
    H.allow_recompute = q.allow_recompute ? 1 : 0;
    H.n_orders = (int32_t)S.n_orders;
    H.stage_types = p->space.stage_types;
    H.n_micro = p->space.n_micro;
    H.n_configs = (int32_t)S.cfg.size();
    for (size_t o = 0; o < S.perm.size(); ++o)
        for (int j = 0; j < kMaxTypes; ++j) H.perm[o][j] = S.perm[o][j];
    for (int i = 0; i < p->space.n_micro; ++i) H.micro[i] = p->space.micro[i];
    H.off_is_moe = I.off_is_moe;
    H.off_tokens = I.off_tokens;
    H.off_pdense = I.off_pdense;
    H.off_pexp = I.off_pexp;
    H.off_act = I.off_act;
    H.off_tdense = I.off_tdense;
    H.off_tffn = I.off_tffn;
    H.image_bytes = I.total;
    const int64_t N = m.n_layers, E = m.n_experts, T = c.n_types;
    std::memcpy(base + I.off_is_moe, m.is_moe, (size_t)N);
    if (E > 0) std::memcpy(base + I.off_tokens, m.expert_tokens, (size_t)(N * E * 8));
    std::memcpy(base + I.off_pdense, m.params_dense, (size_t)(N * 8));
    std::memcpy(base + I.off_pexp, m.params_expert, (size_t)(N * 8));
    std::memcpy(base + I.off_act, m.act_bytes, (size_t)(N * 8));
    std::memcpy(base + I.off_tdense, c.t_dense, (size_t)(T * 16 * N * 8));
    std::memcpy(base + I.off_tffn, c.t_ffn, (size_t)(T * 16 * N * 8));
    return HAPMOE_OK;
}

int32_t hapmoe_tables_bytes(const hapmoe_problem *p, int64_t *bytes)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!bytes) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    *bytes = tables_layout((int64_t)S.cfg.size(), (int)S.n_orders, p->cluster.n_types, p->model.n_layers, p->space.stage_types == 3).total;
    return HAPMOE_OK;
}

int32_t hapmoe_tables_layout(const hapmoe_problem *p, int64_t out[9])
{
    if (const int32_t e = check_problem(p)) return e;
    if (!out) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    const TablesLayout L = tables_layout((int64_t)S.cfg.size(), (int)S.n_orders, p->cluster.n_types, p->model.n_layers, p->space.stage_types == 3);
    const int64_t v[9] = {L.n_configs, L.n_orders, L.n_masks, L.np, L.off_pi, L.off_key, L.off_mem, L.off_time,
                          L.total};
    for (int i = 0; i < 9; ++i) out[i] = v[i];
    return HAPMOE_OK;
}

int32_t hapmoe_debug_layout(const hapmoe_problem *p, int64_t out[4])
{
    if (const int32_t e = check_problem(p)) return e;
    if (!out) return HAPMOE_E_INVAL;
    const DebugLayout D = debug_layout(p->cluster.n_types, p->model.n_layers);
    out[0] = D.per_cfg;
    out[1] = D.off_type;
    out[2] = D.off_mask;
    out[3] = D.off_mem;
    return HAPMOE_OK;
}

int32_t hapmoe_debug_bytes(const hapmoe_problem *p, int64_t *bytes)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!bytes) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    *bytes = (int64_t)S.cfg.size() * debug_layout(p->cluster.n_types, p->model.n_layers).per_cfg * 8;
    return HAPMOE_OK;
}

int32_t hapmoe_eval_cost_tables(const hapmoe_problem *p, const void *d_image, const hapmoe_candidate *d_cand,
                                int64_t n_cand, int64_t first, int64_t count, void *d_tables, int64_t tables_bytes,
                                double *d_debug, int64_t debug_bytes, void *stream)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!d_image || !d_cand || !d_tables) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    const int64_t per = per_config(p, S);
    if (n_cand != (int64_t)S.cfg.size() * per) return HAPMOE_E_INVAL;
    if (first < 0 || count < 0 || first + count > n_cand) return HAPMOE_E_RANGE;
    const TablesLayout L = tables_layout((int64_t)S.cfg.size(), (int)S.n_orders, p->cluster.n_types, p->model.n_layers, p->space.stage_types == 3);
    if (tables_bytes < L.total) return HAPMOE_E_WORKSPACE;
    const DebugLayout D = debug_layout(p->cluster.n_types, p->model.n_layers);
    if (d_debug && debug_bytes < (int64_t)S.cfg.size() * D.per_cfg * 8) return HAPMOE_E_WORKSPACE;
    if (const int e = check_arch()) return e;
    if (count == 0) return HAPMOE_OK;
    // the configurations holding candidates [first, first + count)
    const int64_t cfg_lo = first / per, cfg_hi = (first + count - 1) / per;
    if (launch_cost_tables(d_image, d_cand, per, p->model.n_layers, L, cfg_lo, cfg_hi - cfg_lo + 1, d_tables,
                           d_debug, D, (hipStream_t)stream) != hipSuccess)
        return HAPMOE_E_HIP;
    if (p->space.stage_types == 3 &&
        launch_width_tables(d_image, d_cand, per, L, cfg_lo, cfg_hi - cfg_lo + 1, d_tables, (hipStream_t)stream) !=
            hipSuccess)
        return HAPMOE_E_HIP;
    return HAPMOE_OK;
}

int32_t hapmoe_stage_dp_ws_bytes(const hapmoe_problem *p, int64_t *bytes)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!bytes) return HAPMOE_E_INVAL;
    *bytes = stage_dp_ws_bytes();
    return HAPMOE_OK;
}

namespace {

int32_t stage_dp_any(const hapmoe_problem *p, const void *d_image, const hapmoe_candidate *d_cand, int64_t n_cand,
                     const void *d_tables, int64_t tables_bytes, int64_t first, int64_t count,
                     hapmoe_dp_result *d_res, int32_t *d_stats, void *d_ws, int64_t ws_bytes, void *stream,
                     bool exact)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!d_image || !d_cand || !d_tables || !d_res || !d_ws) return HAPMOE_E_INVAL;
    if (p->space.stage_types >= 2) return HAPMOE_E_INVAL;   // hapmoe_stage_dp_types / _widths
    Space S;
    build_space(p, S);
    const int64_t per = per_config(p, S);
    if (n_cand != (int64_t)S.cfg.size() * per) return HAPMOE_E_INVAL;
    if (first < 0 || count < 0 || first + count > n_cand || count > INT32_MAX) return HAPMOE_E_RANGE;
    const TablesLayout L = tables_layout((int64_t)S.cfg.size(), (int)S.n_orders, p->cluster.n_types, p->model.n_layers, p->space.stage_types == 3);
    if (tables_bytes < L.total || ws_bytes < stage_dp_ws_bytes()) return HAPMOE_E_WORKSPACE;
    if (const int e = check_arch()) return e;
    std::vector<int32_t> cfg_pp(S.cfg.size());
    for (size_t i = 0; i < S.cfg.size(); ++i) cfg_pp[i] = S.cfg[i][0];
    if (launch_stage_dp(d_image, d_cand, p->model.n_layers, p->space.n_micro, cfg_pp, (int)S.n_orders, L,
                        d_tables, first, count, S.kmax, S.ppmax, d_res, d_stats, d_ws, p->space.micro, exact,
                        (hipStream_t)stream) != hipSuccess)
        return HAPMOE_E_HIP;
    return HAPMOE_OK;
}

}  // namespace

int32_t hapmoe_stage_dp(const hapmoe_problem *p, const void *d_image, const hapmoe_candidate *d_cand,
                        int64_t n_cand, const void *d_tables, int64_t tables_bytes, int64_t first, int64_t count,
                        hapmoe_dp_result *d_res, int32_t *d_stats, void *d_ws, int64_t ws_bytes, void *stream)
{
    return stage_dp_any(p, d_image, d_cand, n_cand, d_tables, tables_bytes, first, count, d_res, d_stats, d_ws,
                        ws_bytes, stream, false);
}

int32_t hapmoe_stage_dp_1f1b(const hapmoe_problem *p, const void *d_image, const hapmoe_candidate *d_cand,
                             int64_t n_cand, const void *d_tables, int64_t tables_bytes, int64_t first,
                             int64_t count, hapmoe_dp_result *d_res, int32_t *d_stats, void *d_ws,
                             int64_t ws_bytes, void *stream)
{
    return stage_dp_any(p, d_image, d_cand, n_cand, d_tables, tables_bytes, first, count, d_res, d_stats, d_ws,
                        ws_bytes, stream, true);
}

int32_t hapmoe_stage_dp_latency(const hapmoe_problem *p, const void *d_image, const hapmoe_candidate *d_cand,
                                int64_t n_cand, const void *d_tables, int64_t tables_bytes, int64_t first,
                                int64_t count, hapmoe_dp_result *d_res, int32_t *d_stats, void *stream)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!d_image || !d_cand || !d_tables || !d_res) return HAPMOE_E_INVAL;
    if (p->space.stage_types >= 2) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    const int64_t per = per_config(p, S);
    if (n_cand != (int64_t)S.cfg.size() * per) return HAPMOE_E_INVAL;
    if (first < 0 || count < 0 || first + count > n_cand) return HAPMOE_E_RANGE;
    const TablesLayout L = tables_layout((int64_t)S.cfg.size(), (int)S.n_orders, p->cluster.n_types,
                                         p->model.n_layers);
    if (tables_bytes < L.total) return HAPMOE_E_WORKSPACE;
    if (const int e = check_arch()) return e;
    if (launch_latency_dp(d_image, d_cand, p->space.n_micro, L, d_tables, first, count, d_res, d_stats,
                          (hipStream_t)stream) != hipSuccess)
        return HAPMOE_E_HIP;
    return HAPMOE_OK;
}

int32_t hapmoe_stage_dp_types_ws_bytes(const hapmoe_problem *p, int64_t *bytes)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!bytes || p->space.stage_types != 2) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    *bytes = type_dp_ws_bytes(p->model.n_layers, p->cluster.n_types, S.umax, (int64_t)S.cfg.size());
    return HAPMOE_OK;
}

namespace {

int32_t stage_dp_types_any(const hapmoe_problem *p, const void *d_image, const hapmoe_candidate *d_cand,
                           int64_t n_cand, const void *d_tables, int64_t tables_bytes, int64_t first, int64_t count,
                           hapmoe_dp_result *d_res, uint8_t *d_types, int32_t *d_stats, void *d_ws,
                           int64_t ws_bytes, void *stream, bool exact)
{
    if (const int32_t e = check_problem(p)) return e;
    if (p->space.stage_types != 2 || !d_image || !d_cand || !d_tables || !d_res || !d_types || !d_ws)
        return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    const int64_t ncfg = (int64_t)S.cfg.size(), per = per_config(p, S);
    if (n_cand != ncfg * per) return HAPMOE_E_INVAL;
    if (first < 0 || count < 0 || first + count > n_cand || count > INT32_MAX) return HAPMOE_E_RANGE;
    const TablesLayout L = tables_layout(ncfg, (int)S.n_orders, p->cluster.n_types, p->model.n_layers, p->space.stage_types == 3);
    if (tables_bytes < L.total ||
        ws_bytes < type_dp_ws_bytes(p->model.n_layers, p->cluster.n_types, S.umax, ncfg))
        return HAPMOE_E_WORKSPACE;
    if (const int e = check_arch()) return e;
    if (count == 0) return HAPMOE_OK;
    if (launch_type_dp(d_image, d_cand, p->model.n_layers, p->cluster.n_types, p->space.n_micro, S.umax, S.ppmax, L,
                       d_tables, first, count, d_res, d_types, d_stats, d_ws, exact,
                       (hipStream_t)stream) != hipSuccess)
        return HAPMOE_E_HIP;
    return HAPMOE_OK;
}

}  // namespace

int32_t hapmoe_stage_dp_types(const hapmoe_problem *p, const void *d_image, const hapmoe_candidate *d_cand,
                              int64_t n_cand, const void *d_tables, int64_t tables_bytes, int64_t first,
                              int64_t count, hapmoe_dp_result *d_res, uint8_t *d_types, int32_t *d_stats,
                              void *d_ws, int64_t ws_bytes, void *stream)
{
    return stage_dp_types_any(p, d_image, d_cand, n_cand, d_tables, tables_bytes, first, count, d_res, d_types,
                              d_stats, d_ws, ws_bytes, stream, false);
}

int32_t hapmoe_stage_dp_types_1f1b(const hapmoe_problem *p, const void *d_image, const hapmoe_candidate *d_cand,
                                   int64_t n_cand, const void *d_tables, int64_t tables_bytes, int64_t first,
                                   int64_t count, hapmoe_dp_result *d_res, uint8_t *d_types, int32_t *d_stats,
                                   void *d_ws, int64_t ws_bytes, void *stream)
{
    return stage_dp_types_any(p, d_image, d_cand, n_cand, d_tables, tables_bytes, first, count, d_res, d_types,
                              d_stats, d_ws, ws_bytes, stream, true);
}

int32_t hapmoe_stage_dp_widths_ws_bytes(const hapmoe_problem *p, int64_t count, int64_t *bytes)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!bytes || count < 0 || p->space.stage_types != 3) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    *bytes = width_dp_ws_bytes(p->model.n_layers, S.ppmax, count);
    return HAPMOE_OK;
}

int32_t hapmoe_stage_dp_widths(const hapmoe_problem *p, const void *d_image, const hapmoe_candidate *d_cand,
                               int64_t n_cand, const void *d_tables, int64_t tables_bytes, int64_t first,
                               int64_t count, hapmoe_dp_result *d_res, uint8_t *d_types, uint8_t *d_widths,
                               int32_t *d_stats, void *d_ws, int64_t ws_bytes, void *stream)
{
    if (const int32_t e = check_problem(p)) return e;
    if (p->space.stage_types != 3 || !d_image || !d_cand || !d_tables || !d_res || !d_types || !d_widths || !d_ws)
        return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    const int64_t ncfg = (int64_t)S.cfg.size(), per = per_config(p, S);
    if (n_cand != ncfg * per) return HAPMOE_E_INVAL;
    if (first < 0 || count < 0 || first + count > n_cand || count > INT32_MAX) return HAPMOE_E_RANGE;
    const TablesLayout L = tables_layout(ncfg, (int)S.n_orders, p->cluster.n_types, p->model.n_layers, true);
    if (tables_bytes < L.total || ws_bytes < width_dp_ws_bytes(p->model.n_layers, S.ppmax, count))
        return HAPMOE_E_WORKSPACE;
    if (const int e = check_arch()) return e;
    if (launch_width_dp(d_image, d_cand, p->model.n_layers, S.ppmax, L, d_tables, first, count, d_res, d_types, d_widths,
                        d_stats, d_ws, (hipStream_t)stream) != hipSuccess)
        return HAPMOE_E_HIP;
    return HAPMOE_OK;
}

int32_t hapmoe_best_plan_ws_bytes(const hapmoe_problem *p, int64_t n, int64_t *bytes)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!bytes || n < 0) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    *bytes = best_plan_ws_bytes(n, per_config(p, S), (int64_t)S.cfg.size());
    return HAPMOE_OK;
}

}  // extern "C"

namespace {

// hapmoe_best_plan with its workspace [d_ws, d_ws + ws_bytes); `noalloc`: the
// workspace is the library's fixed array (its size checked before any device work)
int32_t best_plan_any(const hapmoe_problem *p, const hapmoe_candidate *d_cand, const void *d_tables,
                      int64_t tables_bytes, const hapmoe_dp_result *d_res, const uint8_t *d_types, int64_t n,
                      int64_t *d_config_best, void *d_ws, int64_t ws_bytes, hapmoe_plan *h_plan, void *stream,
                      bool noalloc)
{
    if (const int32_t e = check_problem(p)) return e;
    if (!d_cand || !d_tables || !d_res || (!noalloc && !d_ws) || !h_plan) return HAPMOE_E_INVAL;
    if (p->space.stage_types >= 2 ? !d_types : d_types != nullptr) return HAPMOE_E_INVAL;
    Space S;
    build_space(p, S);
    const int64_t per = per_config(p, S), ncfg = (int64_t)S.cfg.size();
    if (n < 1 || n > ncfg * per) return HAPMOE_E_RANGE;
    const TablesLayout L = tables_layout(ncfg, (int)S.n_orders, p->cluster.n_types, p->model.n_layers, p->space.stage_types == 3);
    if (tables_bytes < L.total) return HAPMOE_E_WORKSPACE;
    const int64_t need = best_plan_ws_bytes(n, per, ncfg);
    if (noalloc ? need > HAPMOE_BEST_PLAN_SCRATCH_BYTES : ws_bytes < need) return HAPMOE_E_WORKSPACE;
    if (const int e = check_arch()) return e;
    if (noalloc) {
        int64_t have = 0;
        if (best_plan_scratch(&d_ws, &have) != hipSuccess) return HAPMOE_E_HIP;
        if (have < need) return HAPMOE_E_WORKSPACE;
    }
    hipStream_t s = (hipStream_t)stream;
    const auto *tab = static_cast<const unsigned char *>(d_tables);
    if (launch_best_plan(d_res, d_cand, tab + L.off_key, d_types, p->space.n_micro, n, per, ncfg,
                         p->space.global_batch, p->model.micro_batch_size, d_config_best,
                         d_ws, s) != hipSuccess)
        return HAPMOE_E_HIP;
    // one copy: the global (objective, index) pair and the winner's records
    struct {
        int64_t best[2];
        hapmoe_dp_result r;
        hapmoe_candidate cd;
        KeyInfo ki;
        unsigned char pad[kWinnerBytes - sizeof(hapmoe_dp_result) - sizeof(hapmoe_candidate) - sizeof(KeyInfo)];
    } h;
    static_assert(sizeof(h) == 16 + kWinnerBytes, "winner layout");
    if (hipMemcpyAsync(&h, d_ws, sizeof(h), hipMemcpyDeviceToHost, s) != hipSuccess) return HAPMOE_E_HIP;
    if (hipStreamSynchronize(s) != hipSuccess) return HAPMOE_E_HIP;
    std::memset(h_plan, 0, sizeof(*h_plan));
    h_plan->instance = -1;
    if (h.best[0] == kInf) return HAPMOE_E_INFEASIBLE;
    const int64_t idx = h.best[1];
    const hapmoe_dp_result &r = h.r;
    const hapmoe_candidate &cd = h.cd;
    const KeyInfo &ki = h.ki;
    h_plan->instance = idx;
    h_plan->objective = r.objective;
    h_plan->stage_sum = r.stage_sum;
    h_plan->t_max = r.t_max;
    h_plan->dp_const = ki.dp_const;
    h_plan->cand = cd;
    h_plan->n_stages = cd.pp;
    h_plan->recompute_mask = r.recompute_mask;
    for (int i = 0; i < kMaxStages; ++i) {
        h_plan->layers[i] = i < cd.pp ? r.layers[i] : 0;
        h_plan->stage_types[i] = i < cd.pp ? ki.mask[i] : 0;
    }
    return HAPMOE_OK;
}

}  // namespace

extern "C" {

int32_t hapmoe_best_plan(const hapmoe_problem *p, const hapmoe_candidate *d_cand, const void *d_tables,
                         int64_t tables_bytes, const hapmoe_dp_result *d_res, const uint8_t *d_types, int64_t n,
                         int64_t *d_config_best, void *d_ws, int64_t ws_bytes, hapmoe_plan *h_plan, void *stream)
{
    return best_plan_any(p, d_cand, d_tables, tables_bytes, d_res, d_types, n, d_config_best, d_ws, ws_bytes, h_plan,
                         stream, false);
}

int32_t hapmoe_best_plan_noalloc(const hapmoe_problem *p, const hapmoe_candidate *d_cand, const void *d_tables,
                                 int64_t tables_bytes, const hapmoe_dp_result *d_res, const uint8_t *d_types,
                                 int64_t n, int64_t *d_config_best, hapmoe_plan *h_plan, void *stream)
{
    return best_plan_any(p, d_cand, d_tables, tables_bytes, d_res, d_types, n, d_config_best, nullptr, 0, h_plan,
                         stream, true);
}

}  // extern "C"
