// scram_patchmatch_noalloc: the PatchMatch entry point for callers that
// cannot allocate device memory.  The sweeps' ping-pong buffers live in a
// fixed device array of this file instead of a caller-given workspace; the
// kernels and the launch plan are scram_patchmatch's own.

#include <mutex>

#include <hip/hip_runtime.h>

#include "scram.h"
#include "scram_launch.h"

namespace {

static_assert(SCRAM_NOALLOC_SCRATCH_BYTES == 3 * 4 * SCRAM_NOALLOC_MAX_QUERIES,
              "one int32 map and two fp32 score maps of the largest call");

// Each GPU the library runs on holds its own copy, until the process ends.
// In host code `scratch` is only a handle for the symbol lookup below, never
// an address: the kernels get the device address that lookup returns.
static __device__ __align__(256) unsigned char scratch[SCRAM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_scratch[kMaxDevices];  // device address of `scratch` on each device (null: not looked up yet)

// The device address of `scratch` on the device `stream` belongs to (the
// current device for the null stream), looked up with that device current on
// the first call there.
int scratch_address(hipStream_t stream, void** out)
{
    int dev = 0, cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return SCRAM_ERR_HIP;
    dev = cur;
    if (stream && hipStreamGetDevice(stream, &dev) != hipSuccess) return SCRAM_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return SCRAM_ERR_HIP;
    std::lock_guard<std::mutex> hold(g_lock);
    if (!g_scratch[dev]) {
        if (dev != cur && hipSetDevice(dev) != hipSuccess) return SCRAM_ERR_HIP;
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (dev != cur && hipSetDevice(cur) != hipSuccess) return SCRAM_ERR_HIP;
        if (e != hipSuccess || !p) return SCRAM_ERR_HIP;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return SCRAM_OK;
}

}  // namespace

extern "C" int scram_patchmatch_noalloc(const void* Q, const void* K, int dtype, int S, int Hq, int Wq, int Hk,
                                        int Wk, int d, int iters, uint64_t seed, const int32_t* init,
                                        const float* init_score, int t0, uint32_t flags, const int32_t* prev,
                                        int n_prev, int sep, int32_t* argmax_out, float* score_out,
                                        hipEvent_t* events, hipStream_t stream)
{
    // every argument check before any HIP call, the scratch limit among them
    int rc = scram::patchmatch_check(Q, K, dtype, S, Hq, Wq, Hk, Wk, d, iters, init, init_score, t0, flags, prev,
                                     n_prev, sep, argmax_out, score_out, nullptr, 0);
    if (rc) return rc;
    if (int64_t(S) * Hq * Wq > SCRAM_NOALLOC_MAX_QUERIES) return SCRAM_ERR_SCRATCH;
    const size_t need = scram_patchmatch_workspace_bytes(S, Hq, Wq);
    if (need > SCRAM_NOALLOC_SCRATCH_BYTES) return SCRAM_ERR_SCRATCH;
    void* ws = nullptr;
    if ((rc = scratch_address(stream, &ws))) return rc;
    return scram_patchmatch(Q, K, dtype, S, Hq, Wq, Hk, Wk, d, iters, seed, init, init_score, t0, flags, prev,
                            n_prev, sep, argmax_out, score_out, ws, SCRAM_NOALLOC_SCRATCH_BYTES, events, stream);
}
