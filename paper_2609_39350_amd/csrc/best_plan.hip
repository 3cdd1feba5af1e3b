// Segmented arg-min over the stage-DP results (the outer min of Eq. 1 over pi
// and the candidate's ordering and B): per configuration pi the best of its
// candidates, then the global best.  Order: objective, then candidate index.
// Two kernels: the streaming partial minima over 4,096-candidate chunks, then
// one workgroup for the per-configuration and global minima and the winner.
// Reading the 8-byte objective of every 64-byte result record, this is a
// streaming (HBM-bound) reduction.
#include <mutex>

#include "internal.h"

namespace hapmoe {
namespace {

// Workspace of hapmoe_best_plan_noalloc: a fixed device array that every call
// on a GPU shares (each GPU that loads the library holds its own copy until the
// process ends).  Host code never passes `scratch` itself to a kernel -- in
// host code it names a host-side stand-in -- but the device address that
// hipGetSymbolAddress returns for the current device.
constexpr int64_t kScratchBytes = HAPMOE_BEST_PLAN_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];   // per device, looked up once with that device current

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
// (with a fixed global batch gbs > 0 only the candidates whose B * DP * mbs equals it)
__global__ __launch_bounds__(kThreads) void k_seg_partial(const hapmoe_dp_result *__restrict__ res,
                                                          const hapmoe_candidate *__restrict__ cand, int64_t n,
                                                          int64_t per, int64_t chunks, int64_t gbs, int64_t mbs,
                                                          Best *__restrict__ partial)
{
    __shared__ Best sh[kThreads / 64];
    const int64_t cfg = blockIdx.x, ch = blockIdx.y;
    const int64_t seg_lo = cfg * per, seg_hi = seg_lo + per < n ? seg_lo + per : n;
    const int64_t lo = seg_lo + ch * kChunk;
    const int64_t hi = lo + kChunk < seg_hi ? lo + kChunk : seg_hi;
    Best v = {kInf, INT64_MAX};
    for (int64_t i = lo + threadIdx.x; i < hi; i += kThreads) {
        const hapmoe_dp_result &r = res[i];
        bool take = r.status == HAPMOE_STATUS_OK;
        if (gbs > 0) take = take && (int64_t)cand[i].n_micro * cand[i].dp * mbs == gbs;
        const Best o = {take ? r.objective : kInf, i};
        if (better(o, v)) v = o;
    }
    v = block_min(v, sh);
    if (threadIdx.x == 0) partial[cfg * chunks + ch] = v;
}

int64_t chunks_per_config(int64_t per) { return (per + kChunk - 1) / kChunk; }

constexpr int kFinishThreads = 1024;

// levels 2 and 3 in one workgroup: per configuration over its chunks (into
// config_best), the global best over configurations, then the winner's result,
// candidate and stage layout copied next to it, so that the host reads
// everything with one copy.
__global__ __launch_bounds__(kFinishThreads) void k_finish(const Best *__restrict__ partial, int64_t n_configs,
                                                           int64_t chunks, int64_t *__restrict__ config_best,
                                                           const hapmoe_dp_result *__restrict__ res,
                                                           const hapmoe_candidate *__restrict__ cand,
                                                           const unsigned char *__restrict__ key_info,
                                                           const uint8_t *__restrict__ types, int64_t n_micro,
                                                           Best *__restrict__ glob, uint32_t *__restrict__ out)
{
    __shared__ Best sh[kFinishThreads / 64];
    Best v = {kInf, INT64_MAX};
    for (int64_t cfg = threadIdx.x; cfg < n_configs; cfg += kFinishThreads) {
        Best c = {kInf, INT64_MAX};
        for (int64_t k = 0; k < chunks; ++k) {
            const Best o = partial[cfg * chunks + k];
            if (better(o, c)) c = o;
        }
        if (config_best) config_best[cfg] = c.obj == kInf ? -1 : c.idx;
        if (better(c, v)) v = c;
    }
    const Best b = block_min(v, sh);
    if (threadIdx.x == 0) *glob = b;
    if (b.obj == kInf || threadIdx.x >= 64) return;
    const int w = threadIdx.x;
    constexpr int kRes = (int)sizeof(hapmoe_dp_result) / 4, kCand = (int)sizeof(hapmoe_candidate) / 4;
    constexpr int kKey = (int)sizeof(KeyInfo) / 4;
    if (w < kRes) out[w] = reinterpret_cast<const uint32_t *>(res + b.idx)[w];
    if (w < kCand) out[kRes + w] = reinterpret_cast<const uint32_t *>(cand + b.idx)[w];
    const auto *ki = reinterpret_cast<const uint32_t *>(key_info + (b.idx / n_micro) * (int64_t)sizeof(KeyInfo));
    // the device-count DP chooses each candidate's stage types: they replace the
    // layout's type masks (KeyInfo words 2..9)
    const auto *ty = types ? reinterpret_cast<const uint32_t *>(types + b.idx * kMaxStages) : nullptr;
    for (int i = w; i < kKey; i += 64) out[kRes + kCand + i] = (ty && i >= 2 && i < 2 + kMaxStages / 4) ? ty[i - 2] : ki[i];
}

}  // namespace

// The device address of `scratch` on the current device: looked up with
// hipGetSymbolAddress on the first call per device, then reused.
hipError_t best_plan_scratch(void **ptr, int64_t *bytes)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    *bytes = kScratchBytes;
    return hipSuccess;
}

// workspace: [global Best][winner: result | candidate | stage layout][partial
// n_configs * chunks]
int64_t best_plan_ws_bytes(int64_t n, int64_t per_config, int64_t n_configs)
{
    (void)n;
    const int64_t chunks = chunks_per_config(per_config);
    return (int64_t)sizeof(Best) * (1 + n_configs * chunks) + kWinnerBytes;
}

hipError_t launch_best_plan(const hapmoe_dp_result *d_res, const hapmoe_candidate *d_cand,
                            const unsigned char *d_key_info, const uint8_t *d_types, int64_t n_micro, int64_t n,
                            int64_t per_config, int64_t n_configs, int64_t global_batch, int64_t mbs,
                            int64_t *d_config_best, void *d_ws, hipStream_t s)
{
    const int64_t chunks = chunks_per_config(per_config);
    Best *glob = static_cast<Best *>(d_ws);
    auto *winner = reinterpret_cast<uint32_t *>(static_cast<unsigned char *>(d_ws) + sizeof(Best));
    Best *partial = reinterpret_cast<Best *>(static_cast<unsigned char *>(d_ws) + sizeof(Best) + kWinnerBytes);
    hipLaunchKernelGGL(k_seg_partial, dim3((unsigned)n_configs, (unsigned)chunks), dim3(kThreads), 0, s, d_res,
                       d_cand, n, per_config, chunks, global_batch, mbs, partial);
    hipLaunchKernelGGL(k_finish, dim3(1), dim3(kFinishThreads), 0, s, partial, n_configs, chunks, d_config_best,
                       d_res, d_cand, d_key_info, d_types, n_micro, glob, winner);
    return hipGetLastError();
}

}  // namespace hapmoe
