// Segmented arg-min over the stage-DP results (the outer min of Eq. 1 over pi
// and the candidate's ordering and B): per configuration pi the best of its
// candidates, then the global best.  Order: objective, then candidate index.
// Reading the 8-byte objective of every 64-byte result record, this is a
// streaming (HBM-bound) reduction.
#include "internal.h"

namespace hapmoe {
namespace {

struct Best {
    int64_t obj;
    int64_t idx;
};

constexpr int kThreads = 256;
constexpr int64_t kChunk = 4096;   // candidates per workgroup of the first level

__device__ inline bool better(const Best &a, const Best &b)
{
    return a.obj < b.obj || (a.obj == b.obj && a.idx < b.idx);
}

__device__ inline Best shfl_best(const Best &v, int d)
{
    Best o;
    o.obj = __shfl_xor(v.obj, d, 64);
    o.idx = __shfl_xor(v.idx, d, 64);
    return o;
}

__device__ inline Best block_min(Best v, Best *sh)
{
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const Best o = shfl_best(v, d);
        if (better(o, v)) v = o;
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    if (lane == 0) sh[wave] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < nw; ++w)
            if (better(sh[w], v)) v = sh[w];
        sh[0] = v;
    }
    __syncthreads();
    return sh[0];
}

// level 1: chunk ch of configuration cfg -> partial[cfg * chunks + ch]
__global__ __launch_bounds__(kThreads) void k_seg_partial(const hapmoe_dp_result *__restrict__ res, int64_t n,
                                                          int64_t per, int64_t chunks, Best *__restrict__ partial)
{
    __shared__ Best sh[kThreads / 64];
    const int64_t cfg = blockIdx.x, ch = blockIdx.y;
    const int64_t seg_lo = cfg * per, seg_hi = seg_lo + per < n ? seg_lo + per : n;
    const int64_t lo = seg_lo + ch * kChunk;
    const int64_t hi = lo + kChunk < seg_hi ? lo + kChunk : seg_hi;
    Best v = {kInf, INT64_MAX};
    for (int64_t i = lo + threadIdx.x; i < hi; i += kThreads) {
        const hapmoe_dp_result &r = res[i];
        const Best o = {r.status == HAPMOE_STATUS_OK ? r.objective : kInf, i};
        if (better(o, v)) v = o;
    }
    v = block_min(v, sh);
    if (threadIdx.x == 0) partial[cfg * chunks + ch] = v;
}

// level 2: per configuration over its chunks
__global__ __launch_bounds__(kThreads) void k_seg_final(const Best *__restrict__ partial, int64_t n_configs,
                                                        int64_t chunks, Best *__restrict__ cfg_best,
                                                        int64_t *__restrict__ config_best)
{
    const int64_t cfg = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (cfg >= n_configs) return;
    Best v = {kInf, INT64_MAX};
    for (int64_t k = 0; k < chunks; ++k) {
        const Best o = partial[cfg * chunks + k];
        if (better(o, v)) v = o;
    }
    cfg_best[cfg] = v;
    if (config_best) config_best[cfg] = v.obj == kInf ? -1 : v.idx;
}

// level 3: global best over configurations (one workgroup)
__global__ __launch_bounds__(1024) void k_global(const Best *__restrict__ cfg_best, int64_t n_configs,
                                                 Best *__restrict__ out)
{
    __shared__ Best sh[1024 / 64];
    Best v = {kInf, INT64_MAX};
    for (int64_t i = threadIdx.x; i < n_configs; i += blockDim.x) {
        const Best o = cfg_best[i];
        if (better(o, v)) v = o;
    }
    v = block_min(v, sh);
    if (threadIdx.x == 0) *out = v;
}

int64_t chunks_per_config(int64_t per) { return (per + kChunk - 1) / kChunk; }

}  // namespace

// workspace: [global Best][cfg_best n_configs][partial n_configs * chunks]
int64_t best_plan_ws_bytes(int64_t n, int64_t per_config, int64_t n_configs)
{
    (void)n;
    const int64_t chunks = chunks_per_config(per_config);
    return (int64_t)sizeof(Best) * (1 + n_configs + n_configs * chunks);
}

hipError_t launch_best_plan(const hapmoe_dp_result *d_res, int64_t n, int64_t per_config, int64_t n_configs,
                            int64_t *d_config_best, void *d_ws, hipStream_t s)
{
    const int64_t chunks = chunks_per_config(per_config);
    Best *glob = static_cast<Best *>(d_ws);
    Best *cfg_best = glob + 1;
    Best *partial = cfg_best + n_configs;
    hipLaunchKernelGGL(k_seg_partial, dim3((unsigned)n_configs, (unsigned)chunks), dim3(kThreads), 0, s, d_res, n,
                       per_config, chunks, partial);
    hipLaunchKernelGGL(k_seg_final, dim3((unsigned)((n_configs + kThreads - 1) / kThreads)), dim3(kThreads), 0, s,
                       partial, n_configs, chunks, cfg_best, d_config_best);
    hipLaunchKernelGGL(k_global, dim3(1), dim3(1024), 0, s, cfg_best, n_configs, glob);
    return hipGetLastError();
}

}  // namespace hapmoe
