// Internal layouts of the HAPMoE planner library: the device problem image and
// the cost-table buffer.  Shared by the host API and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "hapmoe.h"

namespace hapmoe {

constexpr int kMaxTypes = HAPMOE_MAX_TYPES;
constexpr int kMaxStages = HAPMOE_MAX_STAGES;
constexpr int kMaxLayers = HAPMOE_MAX_LAYERS;
constexpr int kMaxMasks = (1 << kMaxTypes) - 1;   // non-empty device-type sets
constexpr int kMaxOrders = 24;                      // 4!
constexpr int64_t kInf = INT64_MAX;
// Every rounded per-layer term must stay below 2^44 so that prefix sums,
// memory totals (x M_store <= 32) and (B-1) * t_max (B <= 1024) fit in int64.
constexpr int64_t kTermLimit = int64_t(1) << 44;
constexpr int kMaxMicroValue = 1024;

// Flat problem image (host packs it, device reads it).  Arrays follow the
// header at the offsets below (bytes from the image start, 256-byte aligned).
struct ImageHeader {
    int32_t n_layers, seq_len, hidden, n_experts, top_k, mbs, elem_bytes, n_types;
    int32_t count[kMaxTypes];
    int32_t speed[kMaxTypes];
    int64_t mem_bytes[kMaxTypes];
    double eff[kMaxTypes];
    double route_coef[kMaxTypes];
    double bw[kMaxTypes * kMaxTypes];
    double alpha[kMaxTypes * kMaxTypes];
    double moe_ffn_mult, gamma, rc_time, rc_act, opt_coef;
    int32_t delta_num, delta_den, eta_prune, prune_window, prune_hetero, allow_recompute;
    int32_t n_orders, n_micro, n_configs, total_devices;
    int32_t stage_types, pad_st;          // 1: free per-stage type sequences (perm unused)
    int8_t perm[kMaxOrders][kMaxTypes];   // orderings, lexicographic
    int32_t micro[HAPMOE_MAX_MICRO];
    int64_t off_is_moe, off_tokens, off_pdense, off_pexp, off_act, off_tdense, off_tffn;
    int64_t image_bytes;
};

// Per configuration pi.
struct PiInfo {
    int64_t x_bytes;                 // MoE buffers of a stage holding an MoE layer
    int64_t tbar;                    // pruning-3 compute bound
    int64_t p2p[kMaxTypes * kMaxTypes];  // boundary transfer cost, [from][to]
    int32_t status;                  // HAPMOE_STATUS_OK or _OVERFLOW
    uint32_t used_masks;             // bit (m-1): device-type set m occurs in some stage
};

// Per (configuration, ordering): the stage layout.
struct KeyInfo {
    int64_t dp_const;                // T_dp-sync + T_opt
    uint8_t mask[kMaxStages];        // device types of stage s
    uint8_t lo[kMaxStages];          // pruning-1 window on n_s
    uint8_t hi[kMaxStages];
    uint8_t bpair[kMaxStages];       // (type of last device << 2) | type of next stage's first
};

// Byte layout of the cost-table buffer.  np = prefix stride (>= N + 1).
//   pi   [n_configs] PiInfo
//   key  [n_configs * n_orders] KeyInfo
//   mem  [n_configs][4][np] int64   W, A0, A1 prefix sums and MoE-layer count
//   time [n_configs][n_masks][3][np] int64   T0, T1, comm prefix sums
//   layer [N] double   load-imbalance factor 1 + gamma (rho - 1) of every layer
//   with per-stage widths (stage_types = 3), after the layer factors:
//   wmem  [n_configs][3 widths][4][np] int64   W, A0, A1 prefix sums, MoE-layer count
//   wtime [n_configs][n_masks][3 widths][3][np] int64   T0, T1, comm prefix sums
//   wx    [n_configs][4] int64   MoE buffers of a stage of width 1, 2, 3 (and padding)
struct TablesLayout {
    int64_t n_configs, n_orders, n_masks, np;
    int64_t off_pi, off_key, off_mem, off_time, off_layer, total;
    int64_t off_wmem, off_wtime, off_wx;   // 0 without per-stage widths
};

// fp64 debug buffer: per configuration
//   type [N][T][2] (comp, expert), mask [n_masks][N][3] (a2a, tp, cp), mem [N][2] (w, a0)
struct DebugLayout {
    int64_t per_cfg, off_type, off_mask, off_mem;
};

static_assert(sizeof(PiInfo) == 152, "PiInfo layout is part of the documented table format");
static_assert(sizeof(KeyInfo) == 136, "KeyInfo layout is part of the documented table format");
static_assert(offsetof(KeyInfo, mask) == 8, "stage type masks at words 2..9");
static_assert(sizeof(hapmoe_candidate) == 32 && sizeof(hapmoe_dp_result) == 64, "ABI record sizes");

inline int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

inline TablesLayout tables_layout(int64_t n_configs, int n_orders, int n_types, int n_layers, bool widths = false)
{
    TablesLayout L;
    L.n_configs = n_configs;
    L.n_orders = n_orders;
    L.n_masks = (1 << n_types) - 1;
    L.np = (n_layers + 1 + 7) & ~7;
    L.off_pi = 0;
    L.off_key = align256(L.off_pi + n_configs * (int64_t)sizeof(PiInfo));
    L.off_mem = align256(L.off_key + n_configs * n_orders * (int64_t)sizeof(KeyInfo));
    L.off_time = align256(L.off_mem + n_configs * 4 * L.np * 8);
    L.off_layer = align256(L.off_time + n_configs * L.n_masks * 3 * L.np * 8);
    L.total = align256(L.off_layer + (int64_t)n_layers * 8);
    L.off_wmem = L.off_wtime = L.off_wx = 0;
    if (widths) {
        L.off_wmem = L.total;
        L.off_wtime = align256(L.off_wmem + n_configs * 3 * 4 * L.np * 8);
        L.off_wx = align256(L.off_wtime + n_configs * L.n_masks * 3 * 3 * L.np * 8);
        L.total = align256(L.off_wx + n_configs * 4 * 8);
    }
    return L;
}

inline DebugLayout debug_layout(int n_types, int n_layers)
{
    DebugLayout D;
    int64_t M = (1 << n_types) - 1;
    D.off_type = 0;
    D.off_mask = D.off_type + (int64_t)n_layers * n_types * 2;
    D.off_mem = D.off_mask + M * n_layers * 3;
    D.per_cfg = D.off_mem + (int64_t)n_layers * 2;
    return D;
}

// Kernel launchers (stream = hipStream_t).
hipError_t launch_cost_tables(const void *d_image, const hapmoe_candidate *d_cand, int64_t per_config,
                              int n_layers, const TablesLayout &L, int64_t cfg_lo, int64_t n_cfg, void *d_tables,
                              double *d_debug, const DebugLayout &D, hipStream_t s);
hipError_t launch_stage_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_layers, int n_micro,
                           const std::vector<int32_t> &config_pp, int n_orders, const TablesLayout &L,
                           const void *d_tables, int64_t first, int64_t count, int kmax, int ppmax,
                           hapmoe_dp_result *d_res, int32_t *d_stats, void *d_ws, const int32_t *micro,
                           bool exact, hipStream_t s);
int64_t stage_dp_ws_bytes();
// the least 1F1B latency over every partition: one workgroup per candidate
hipError_t launch_latency_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_micro,
                             const TablesLayout &L, const void *d_tables, int64_t first, int64_t count,
                             hapmoe_dp_result *d_res, int32_t *d_stats, hipStream_t stream);
// section clocks of the stage-DP kernel (libraries built with HAPMOE_SECTION_CLOCKS)
enum {
    kClockSetup, kClockScan, kClockRelax, kClockTrace, kClockControl, kClockTotal,
    kCountKeys, kCountBatches, kCountPasses,
    // wall-clock (constant-rate counter) records: the longest key of any wave
    // (ticks << 6 | its pipeline depth), the earliest wave start and end
    // (stored complemented, so that all three are maxima), the latest wave end
    kKeyMax, kWaveStartMinC, kWaveEndMinC, kWaveEndMax, kWallClockKHz, kSectionClocks
};
int32_t stage_dp_section_clocks(uint64_t *out, bool clear);

// Device-count DP (free per-stage device types by the DP state of device counts).
constexpr int kMaxTypeStates = 8192;                        // states u = prod_h (k_h + 1) per pipeline
constexpr int64_t kTypeDpMaxSlots = 512;                    // workgroups with a state slice each
constexpr int64_t kTypeDpMaxSlotBytes = int64_t(8) << 30;   // all slices together
constexpr int kTypeDpMaxLds = 160 * 1024;                   // the LDS of one gfx950 CU
struct TypeLds {
    int umax;
    int off_t0, off_t1, off_mw, off_moe, off_inc, off_path, off_ctl, off_ulist, off_bounds, bytes;
};
TypeLds type_dp_lds(int n_layers, int n_types, int n_micro, int umax, int ppmax);
int64_t type_dp_slot_bytes(int n_layers, int n_types, int umax);
int64_t type_dp_slots(int64_t n_keys, int64_t slot_bytes);
int64_t type_dp_ws_bytes(int n_layers, int n_types, int umax, int64_t n_configs);
hipError_t launch_type_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_layers, int n_types,
                          int n_micro, int umax, int ppmax, const TablesLayout &L, const void *d_tables, int64_t first,
                          int64_t count, hapmoe_dp_result *d_res, uint8_t *d_types, int32_t *d_stats, void *d_ws,
                          bool exact, hipStream_t s);
// Per-stage data-parallel widths (stage_types = 3): the width tables (run after
// the cost tables on the same stream) and the DP over (stage, end layer,
// half-groups used).
constexpr int64_t kWidthDpMaxSlots = 1024;   // workgroups with a state slice each
hipError_t launch_width_tables(const void *d_image, const hapmoe_candidate *d_cand, int64_t per_config,
                               const TablesLayout &L, int64_t cfg_lo, int64_t n_cfg, void *d_tables, hipStream_t s);
int64_t width_dp_slot_bytes(int n_layers, int ppmax);
int64_t width_dp_ws_bytes(int n_layers, int ppmax, int64_t n_cand);
hipError_t launch_width_dp(const void *d_image, const hapmoe_candidate *d_cand, int n_layers, int ppmax,
                           const TablesLayout &L, const void *d_tables, int64_t first, int64_t count,
                           hapmoe_dp_result *d_res, uint8_t *d_types, uint8_t *d_widths, int32_t *d_stats, void *d_ws,
                           hipStream_t s);
// bytes of the winner record in the best-plan workspace (result, candidate, stage layout)
constexpr int64_t kWinnerBytes = 256;
static_assert(sizeof(hapmoe_dp_result) + sizeof(hapmoe_candidate) + sizeof(KeyInfo) <= kWinnerBytes, "winner");
static_assert(sizeof(hapmoe_dp_result) % 4 == 0 && sizeof(hapmoe_candidate) % 4 == 0 && sizeof(KeyInfo) % 4 == 0,
              "word copies");
hipError_t launch_best_plan(const hapmoe_dp_result *d_res, const hapmoe_candidate *d_cand,
                            const unsigned char *d_key_info, const uint8_t *d_types, int64_t n_micro, int64_t n,
                            int64_t per_config, int64_t n_configs, int64_t global_batch, int64_t mbs,
                            int64_t *d_config_best, void *d_ws, hipStream_t s);
int64_t best_plan_ws_bytes(int64_t n, int64_t per_config, int64_t n_configs);
// device address and size of the fixed workspace of hapmoe_best_plan_noalloc on the current device
hipError_t best_plan_scratch(void **ptr, int64_t *bytes);

}  // namespace hapmoe
