// Sanitizer driver for the library's host code (test infrastructure).
//
// Built by the test-suite from every library source with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host side only, and run as a plain
// executable on a machine without a GPU: it calls every entry point that does
// not touch the device -- validation, enumeration, image packing, the size and
// layout queries -- on seeded problems of each stage-type mode, then the bad
// inputs each must refuse (the device calls included, which must return their
// error before any HIP call).  Exit status 0 on success.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "hapmoe.h"

namespace {

uint64_t lcg_state;
uint32_t next_u32()
{
    lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(lcg_state >> 33);
}
int64_t uniform(int64_t lo, int64_t hi) { return lo + (int64_t)(next_u32() % (uint32_t)(hi - lo + 1)); }

struct Inputs {
    std::vector<uint8_t> is_moe;
    std::vector<int64_t> tokens, pd, pe, act, td, tf;
};

void make_problem(hapmoe_problem &p, Inputs &A, uint64_t seed, int N, int T, const int *count, int stage_types)
{
    lcg_state = seed;
    std::memset(&p, 0, sizeof(p));
    const int E = 8;
    A.is_moe.assign(N, 0);
    A.tokens.assign((size_t)N * E, 0);
    A.pd.assign(N, 0);
    A.pe.assign(N, 0);
    A.act.assign(N, 0);
    A.td.assign((size_t)T * 16 * N, 0);
    A.tf.assign((size_t)T * 16 * N, 0);
    for (int l = 0; l < N; ++l) {
        A.is_moe[l] = (uint8_t)(l % 3 != 0);
        for (int e = 0; e < E; ++e) A.tokens[(size_t)l * E + e] = A.is_moe[l] ? uniform(10, 600) : 0;
        A.pd[l] = uniform(1000000, 30000000);
        A.pe[l] = A.is_moe[l] ? uniform(1000000, 90000000) : 0;
        A.act[l] = uniform(10000000, 900000000);
    }
    for (size_t i = 0; i < A.td.size(); ++i) {
        A.td[i] = uniform(2000, 200000);
        A.tf[i] = A.td[i] / 2;
    }
    hapmoe_model &m = p.model;
    m.n_layers = N;
    m.seq_len = 1024;
    m.hidden = 512;
    m.n_experts = E;
    m.top_k = 2;
    m.micro_batch_size = 1;
    m.elem_bytes = 2;
    m.moe_ffn_mult = 2.0;
    m.is_moe = A.is_moe.data();
    m.expert_tokens = A.tokens.data();
    m.params_dense = A.pd.data();
    m.params_expert = A.pe.data();
    m.act_bytes = A.act.data();
    hapmoe_cluster &c = p.cluster;
    c.n_types = T;
    for (int h = 0; h < T; ++h) {
        c.count[h] = count[h];
        c.speed[h] = (int32_t)uniform(60, 250);
        c.mem_bytes[h] = uniform(2, 30) * 1000000000ll;
        c.eff[h] = 0.5 + 0.1 * h;
        c.route_coef[h] = 1e-5;
        for (int g = 0; g < T; ++g) {
            c.bw[h][g] = h == g ? 400.0 : (double)uniform(20, 80);
            c.alpha[h][g] = h == g ? 5000.0 : 20000.0;
        }
    }
    c.t_dense = A.td.data();
    c.t_ffn = A.tf.data();
    hapmoe_params &q = p.params;
    q.gamma = 0.5;
    q.rc_time = 1.33;
    q.rc_act = 0.4;
    q.opt_coef = 0.01;
    q.delta_num = 1;
    q.delta_den = 5;
    q.eta_prune = 2;
    q.prune_window = (int32_t)(seed % 3);
    q.prune_hetero = 1;
    q.allow_recompute = 1;
    hapmoe_space &s = p.space;
    s.pp_max = 8;
    s.tp_mask = s.cp_mask = s.tpe_mask = 0xF;
    s.ep_max = 8;
    s.mode = (int32_t)(seed % 2);
    s.stage_types = stage_types;
    s.n_micro = 3;
    s.micro[0] = 1;
    s.micro[1] = 4;
    s.micro[2] = 16;
}

int fail(const char *what, int code)
{
    std::printf("FAIL %s: %d (%s)\n", what, code, hapmoe_strerror(code));
    return 1;
}

int run_problem(const hapmoe_problem &p, const char *name)
{
    int bad = 0;
    if (int e = hapmoe_validate(&p)) return fail(name, e);
    int64_t n = 0;
    if (hapmoe_enumerate_candidates(&p, nullptr, 0, &n) != HAPMOE_E_CAPACITY || n < 1) return fail("count", -1);
    std::vector<hapmoe_candidate> cand((size_t)n);
    if (int e = hapmoe_enumerate_candidates(&p, cand.data(), n, &n)) bad |= fail("enumerate", e);
    if (n > 3) {   // a short array: the first entries, and the required count
        int64_t m = 0;
        std::vector<hapmoe_candidate> few(3);
        if (hapmoe_enumerate_candidates(&p, few.data(), 3, &m) != HAPMOE_E_CAPACITY || m != n)
            bad |= fail("short array", -1);
    }
    int64_t img = 0, tab = 0, dbg = 0, ws = 0, bws = 0;
    if (int e = hapmoe_image_bytes(&p, &img)) bad |= fail("image bytes", e);
    std::vector<unsigned char> image((size_t)img);
    if (int e = hapmoe_pack_image(&p, image.data(), img)) bad |= fail("pack", e);
    if (hapmoe_pack_image(&p, image.data(), img - 1) == HAPMOE_OK) bad |= fail("pack short", 0);
    if (int e = hapmoe_tables_bytes(&p, &tab)) bad |= fail("tables bytes", e);
    if (int e = hapmoe_debug_bytes(&p, &dbg)) bad |= fail("debug bytes", e);
    int64_t lay[9], dlay[4];
    if (int e = hapmoe_tables_layout(&p, lay)) bad |= fail("tables layout", e);
    if (lay[8] != tab) bad |= fail("layout total", -1);
    if (int e = hapmoe_debug_layout(&p, dlay)) bad |= fail("debug layout", e);
    if (p.space.stage_types == 2) {
        if (int e = hapmoe_stage_dp_types_ws_bytes(&p, &ws)) bad |= fail("types ws", e);
    } else if (p.space.stage_types == 3) {
        if (int e = hapmoe_stage_dp_widths_ws_bytes(&p, n, &ws)) bad |= fail("widths ws", e);
        if (hapmoe_stage_dp_widths(&p, nullptr, nullptr, n, nullptr, 0, 0, n, nullptr, nullptr, nullptr, nullptr,
                                   nullptr, 0, nullptr) == HAPMOE_OK)
            bad |= fail("widths null", 0);
    } else if (int e = hapmoe_stage_dp_ws_bytes(&p, &ws)) {
        bad |= fail("dp ws", e);
    }
    if (int e = hapmoe_best_plan_ws_bytes(&p, n, &bws)) bad |= fail("plan ws", e);
    // device calls with missing buffers: refused before any device work
    if (hapmoe_eval_cost_tables(&p, nullptr, nullptr, n, 0, n, nullptr, 0, nullptr, 0, nullptr) == HAPMOE_OK)
        bad |= fail("tables null", 0);
    if (hapmoe_stage_dp(&p, nullptr, nullptr, n, nullptr, 0, 0, n, nullptr, nullptr, nullptr, 0, nullptr) ==
        HAPMOE_OK)
        bad |= fail("dp null", 0);
    if (hapmoe_stage_dp_types(&p, nullptr, nullptr, n, nullptr, 0, 0, n, nullptr, nullptr, nullptr, nullptr, 0,
                              nullptr) == HAPMOE_OK)
        bad |= fail("types null", 0);
    if (hapmoe_stage_dp_latency(&p, nullptr, nullptr, n, nullptr, 0, 0, n, nullptr, nullptr, nullptr) ==
        HAPMOE_OK)
        bad |= fail("latency null", 0);
    {   // range and table-size checks with stand-in pointers (never dereferenced)
        void *fake = reinterpret_cast<void *>(uintptr_t(1) << 20);
        const auto *fc = static_cast<const hapmoe_candidate *>(fake);
        auto *fr = static_cast<hapmoe_dp_result *>(fake);
        if (p.space.stage_types < 2) {
            if (hapmoe_stage_dp_latency(&p, fake, fc, n, fake, tab, n, 1, fr, nullptr, nullptr) != HAPMOE_E_RANGE)
                bad |= fail("latency range", 0);
            if (hapmoe_stage_dp_latency(&p, fake, fc, n, fake, tab - 1, 0, 1, fr, nullptr, nullptr) !=
                HAPMOE_E_WORKSPACE)
                bad |= fail("latency tables", 0);
        } else if (hapmoe_stage_dp_latency(&p, fake, fc, n, fake, tab, 0, 1, fr, nullptr, nullptr) !=
                   HAPMOE_E_INVAL) {
            bad |= fail("latency mode", 0);
        }
    }
    hapmoe_plan plan;
    if (hapmoe_best_plan(&p, nullptr, nullptr, 0, nullptr, nullptr, n, nullptr, nullptr, 0, &plan, nullptr) ==
        HAPMOE_OK)
        bad |= fail("plan null", 0);
    std::printf("%s: %lld candidates, image %lld B, tables %lld B, dp workspace %lld B\n", name, (long long)n,
                (long long)img, (long long)tab, (long long)ws);
    return bad;
}

}  // namespace

int main()
{
    static const int c2[2] = {4, 4}, c3[3] = {4, 2, 2}, c4[4] = {2, 2, 2, 2};
    Inputs A;
    hapmoe_problem p;
    int bad = 0;
    for (int seed = 1; seed <= 4; ++seed)
        for (int st = 0; st <= 3; ++st) {
            char name[80];
            std::snprintf(name, sizeof(name), "2 types seed %d stage_types %d", seed, st);
            make_problem(p, A, (uint64_t)seed, 12, 2, c2, st);
            bad |= run_problem(p, name);
            std::snprintf(name, sizeof(name), "3 types seed %d stage_types %d", seed, st);
            make_problem(p, A, (uint64_t)seed + 10, 9, 3, c3, st);
            bad |= run_problem(p, name);
            std::snprintf(name, sizeof(name), "4 types seed %d stage_types %d", seed, st);
            make_problem(p, A, (uint64_t)seed + 20, 16, 4, c4, st);
            bad |= run_problem(p, name);
        }
    // malformed problems: every one refused with HAPMOE_E_INVAL
    make_problem(p, A, 1, 12, 2, c2, 0);
    const hapmoe_problem base = p;
    int refused = 0, cases = 0;
    auto expect_inval = [&](const hapmoe_problem &q) {
        ++cases;
        refused += hapmoe_validate(&q) == HAPMOE_E_INVAL;
    };
    p = base; p.model.n_layers = 0; expect_inval(p);
    p = base; p.model.top_k = 9; expect_inval(p);
    p = base; p.cluster.n_types = 5; expect_inval(p);
    p = base; p.cluster.count[0] = 0; expect_inval(p);
    p = base; p.params.rc_time = 0.5; expect_inval(p);
    p = base; p.params.delta_num = 5; expect_inval(p);
    p = base; p.params.prune_window = 3; expect_inval(p);
    p = base; p.space.pp_max = 33; expect_inval(p);
    p = base; p.space.n_micro = 0; expect_inval(p);
    p = base; p.space.micro[0] = 5000; expect_inval(p);
    p = base; p.space.stage_types = 4; expect_inval(p);
    p = base; p.space.global_batch = -1; expect_inval(p);
    p = base; p.model.is_moe = nullptr; expect_inval(p);
    if (hapmoe_validate(nullptr) != HAPMOE_E_INVAL) bad |= fail("null problem", 0);
    if (refused != cases) bad |= fail("malformed problems accepted", cases - refused);
    std::printf("%d malformed problems refused\n", refused);
    return bad;
}
