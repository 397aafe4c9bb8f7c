// C-ABI front end of the SCRAM library: argument validation (host only, no
// HIP call before every check has passed), ping-pong buffer planning for the
// Jacobi sweeps, and the launches.  The contract is documented in scram.h.

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <hip/hip_runtime.h>

#include "scram.h"
#include "scram_launch.h"

namespace {

constexpr int64_t kMaxSide = int64_t(1) << 30;
constexpr int64_t kMaxCount = int64_t(1) << 31;
constexpr uint64_t kMaxBlocks = 0xFFFFFFFFull / 256;  // one dispatch: at most 2^32 - 1 work-items

size_t round256(size_t b) { return (b + 255) & ~size_t(255); }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

struct Range {
    uintptr_t lo, hi;  // [lo, hi)
};

Range range(const void* p, size_t bytes)
{
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    return Range{a, a + bytes};
}

bool overlap(const Range& a, const Range& b)
{
    return a.lo != a.hi && b.lo != b.hi && a.lo < b.hi && b.lo < a.hi;
}

bool supported_width(int d) { return d == 16 || d == 32 || d == 64 || d == 128; }

size_t elem_bytes(int dtype) { return dtype == SCRAM_BF16 ? 2 : 4; }

int check_grid(int S, int Hq, int Wq, int Hk, int Wk)
{
    if (S <= 0 || Hq <= 0 || Wq <= 0 || Hk <= 0 || Wk <= 0) return SCRAM_ERR_SHAPE;
    if (Hq > kMaxSide || Wq > kMaxSide || Hk > kMaxSide || Wk > kMaxSide) return SCRAM_ERR_SHAPE;
    if (int64_t(S) * Hq * Wq >= kMaxCount || int64_t(Hk) * Wk >= kMaxCount) return SCRAM_ERR_SHAPE;
    return SCRAM_OK;
}

int check_type(int dtype, int d)
{
    if (dtype != SCRAM_F32 && dtype != SCRAM_BF16) return SCRAM_ERR_UNSUPPORTED;
    if (!supported_width(d)) return SCRAM_ERR_UNSUPPORTED;
    return SCRAM_OK;
}

}  // namespace

namespace scram {

// Every check of scram_patchmatch's arguments, on the host (no HIP call).  A
// null workspace is the library's own scratch (scram_patchmatch_noalloc):
// its presence, size and overlap are then not checked here.
int patchmatch_check(const void* Q, const void* K, int dtype, int S, int Hq, int Wq, int Hk, int Wk, int d,
                     int iters, const int32_t* init, const float* init_score, int t0, uint32_t flags,
                     const int32_t* prev, int n_prev, int sep, const int32_t* argmax_out, const float* score_out,
                     const void* workspace, size_t workspace_bytes)
{
    if (!Q || !K || !argmax_out) return SCRAM_ERR_NULL;
    if (n_prev > 0 && !prev) return SCRAM_ERR_NULL;
    int rc = check_grid(S, Hq, Wq, Hk, Wk);
    if (rc) return rc;
    if (iters < 0 || t0 < 1 || int64_t(t0) + iters > int64_t(0xFFFFFFFFu)) return SCRAM_ERR_SHAPE;
    if (n_prev < 0 || n_prev > SCRAM_MAX_PREV || sep < 1) return SCRAM_ERR_SHAPE;
    if ((rc = check_type(dtype, d))) return rc;
    if (patchmatch_max_blocks(dtype, Grid{S, Hq, Wq, Hk, Wk, d}) > kMaxBlocks) return SCRAM_ERR_SHAPE;
    if (flags & ~uint32_t(SCRAM_PM_NO_PROPAGATION | SCRAM_PM_NO_RANDOM_SEARCH | SCRAM_CAUSAL))
        return SCRAM_ERR_UNSUPPORTED;
    const bool causal = (flags & SCRAM_CAUSAL) != 0;
    if (causal && (Hq != Hk || Wq != Wk)) return SCRAM_ERR_SHAPE;
    if (!init) init_score = nullptr;
    if (n_prev == 0) prev = nullptr;
    if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(argmax_out, 4) || (workspace && !aligned(workspace, 256)) ||
        (score_out && !aligned(score_out, 4)) || (init && !aligned(init, 4)) ||
        (init_score && !aligned(init_score, 4)) || (prev && !aligned(prev, 4)))
        return SCRAM_ERR_ALIGN;
    const size_t n = size_t(S) * Hq * Wq;
    const size_t need = scram_patchmatch_workspace_bytes(S, Hq, Wq);
    if (workspace && workspace_bytes < need) return SCRAM_ERR_WORKSPACE;

    const size_t eb = elem_bytes(dtype);
    const Range rQ = range(Q, n * d * eb), rK = range(K, size_t(S) * Hk * Wk * d * eb);
    const Range rJ = range(argmax_out, 4 * n), rW = workspace ? range(workspace, need) : Range{0, 0};
    const Range rS = score_out ? range(score_out, 4 * n) : Range{0, 0};
    const Range rI = init ? range(init, 4 * n) : Range{0, 0};
    const Range rIS = init_score ? range(init_score, 4 * n) : Range{0, 0};
    const Range rP = prev ? range(prev, 4 * n * size_t(n_prev)) : Range{0, 0};
    for (const Range& out : {rJ, rS, rW}) {
        for (const Range& other : {rQ, rK, rI, rIS, rP}) {
            if (overlap(out, other)) return SCRAM_ERR_ALIAS;
        }
    }
    if (overlap(rJ, rS) || overlap(rJ, rW) || overlap(rS, rW)) return SCRAM_ERR_ALIAS;
    return SCRAM_OK;
}

}  // namespace scram

extern "C" {

size_t scram_patchmatch_workspace_bytes(int S, int Hq, int Wq)
{
    if (S <= 0 || Hq <= 0 || Wq <= 0) return 0;
    const size_t n = size_t(S) * size_t(Hq) * size_t(Wq);
    return 3 * round256(4 * n);
}

int scram_patchmatch(const void* Q, const void* K, int dtype, int S, int Hq, int Wq, int Hk, int Wk,
                     int d, int iters, uint64_t seed, const int32_t* init, const float* init_score,
                     int t0, uint32_t flags, const int32_t* prev, int n_prev, int sep, int32_t* argmax_out,
                     float* score_out, void* workspace, size_t workspace_bytes, hipEvent_t* events,
                     hipStream_t stream)
{
    // ---- validation (no HIP call above this line) ----
    if (Q && K && argmax_out && !(n_prev > 0 && !prev) && !workspace) return SCRAM_ERR_WORKSPACE;
    int rc = scram::patchmatch_check(Q, K, dtype, S, Hq, Wq, Hk, Wk, d, iters, init, init_score, t0, flags, prev,
                                     n_prev, sep, argmax_out, score_out, workspace, workspace_bytes);
    if (rc) return rc;
    const bool causal = (flags & SCRAM_CAUSAL) != 0;
    if (!init) init_score = nullptr;
    if (n_prev == 0) prev = nullptr;
    const size_t n = size_t(S) * Hq * Wq;

    // ---- plan the ping-pong buffers ----
    // The map after sweep k (k = 0 is the initial map) lives in buffer
    // (iters - k) % 2, so the last sweep writes buffer 0 = the caller's
    // outputs and no sweep reads the buffer it writes.
    char* ws = static_cast<char*>(workspace);
    int32_t* Jbuf[2] = {argmax_out, reinterpret_cast<int32_t*>(ws)};
    float* s_ws0 = reinterpret_cast<float*>(ws + round256(4 * n));
    float* s_ws1 = reinterpret_cast<float*>(ws + 2 * round256(4 * n));
    float* sbuf[2] = {score_out ? score_out : s_ws0, s_ws1};
    const scram::Grid grid{S, Hq, Wq, Hk, Wk, d};
    const scram::RunSpec run{prev, n_prev, sep, causal};
    flags &= ~uint32_t(SCRAM_CAUSAL);

    const int p0 = iters % 2;
    const int32_t* Jcur;
    const float* scur;
    hipEvent_t* ev = events;  // 2 per launch: start, stop
    hipError_t e = hipSuccess;
    if (init) {
        Jcur = init;
        if (init_score) {
            scur = init_score;
            if (ev) {  // nothing to launch: the first pair brackets no work
                e = hipEventRecord(ev[0], stream);
                if (e == hipSuccess) e = hipEventRecord(ev[1], stream);
            }
        } else {
            e = scram::launch_pm_init(dtype, Q, K, grid, seed, run, init, nullptr, sbuf[p0], stream,
                                      ev ? ev[0] : nullptr, ev ? ev[1] : nullptr);
            scur = sbuf[p0];
        }
        if (e == hipSuccess && iters == 0) {
            e = hipMemcpyAsync(argmax_out, init, 4 * n, hipMemcpyDeviceToDevice, stream);
            if (e == hipSuccess && score_out && init_score)
                e = hipMemcpyAsync(score_out, init_score, 4 * n, hipMemcpyDeviceToDevice, stream);
        }
    } else if (iters > 0 && flags == 0) {
        // the first sweep recomputes the random initial field itself: no
        // init launch, and the init's event pair brackets no work
        Jcur = nullptr;
        scur = nullptr;
        if (ev) {
            e = hipEventRecord(ev[0], stream);
            if (e == hipSuccess) e = hipEventRecord(ev[1], stream);
        }
    } else {
        e = scram::launch_pm_init(dtype, Q, K, grid, seed, run, nullptr, Jbuf[p0], sbuf[p0], stream,
                                  ev ? ev[0] : nullptr, ev ? ev[1] : nullptr);
        Jcur = Jbuf[p0];
        scur = sbuf[p0];
    }
    for (int k = 1; k <= iters && e == hipSuccess; ++k) {
        const int pk = (iters - k) % 2;
        // maps between two sweeps of this call carry the stable-entry mark;
        // the caller's init and the final map do not
        e = scram::launch_pm_iter(dtype, Q, K, grid, seed, run, uint32_t(t0 + k - 1), flags, Jcur, scur, k > 1,
                                  k < iters, Jbuf[pk], sbuf[pk], stream, ev ? ev[2 * k] : nullptr,
                                  ev ? ev[2 * k + 1] : nullptr);
        Jcur = Jbuf[pk];
        scur = sbuf[pk];
    }
    return e == hipSuccess ? SCRAM_OK : SCRAM_ERR_HIP;
}

int scram_sparse_attend(const void* Q, const void* K, const void* V, int dtype, const int32_t* argmax, int kappa,
                        int S, int Hq, int Wq, int Hk, int Wk, int d, int dv, int window, float scale,
                        uint32_t flags, void* out, hipEvent_t* events, hipStream_t stream)
{
    if (!Q || !K || !V || !argmax || !out) return SCRAM_ERR_NULL;
    int rc = check_grid(S, Hq, Wq, Hk, Wk);
    if (rc) return rc;
    if (window < 1 || window % 2 == 0 || window > 32767) return SCRAM_ERR_SHAPE;
    if (kappa < 1 || kappa > SCRAM_MAX_KAPPA) return SCRAM_ERR_SHAPE;
    if (!isfinite(scale)) return SCRAM_ERR_SHAPE;
    if ((rc = check_type(dtype, d))) return rc;
    if (scram::attend_max_blocks(dtype, scram::Grid{S, Hq, Wq, Hk, Wk, d}) > kMaxBlocks) return SCRAM_ERR_SHAPE;
    if (dv != d) return SCRAM_ERR_UNSUPPORTED;
    if (flags & ~uint32_t(SCRAM_CAUSAL)) return SCRAM_ERR_UNSUPPORTED;
    const bool causal = (flags & SCRAM_CAUSAL) != 0;
    if (causal && (Hq != Hk || Wq != Wk)) return SCRAM_ERR_SHAPE;
    if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(out, 16) || !aligned(argmax, 4))
        return SCRAM_ERR_ALIGN;
    const size_t n = size_t(S) * Hq * Wq, eb = elem_bytes(dtype);
    const Range rO = range(out, n * dv * eb);
    for (const Range& other : {range(Q, n * d * eb), range(K, size_t(S) * Hk * Wk * d * eb),
                               range(V, size_t(S) * Hk * Wk * dv * eb), range(argmax, 4 * n * size_t(kappa))}) {
        if (overlap(rO, other)) return SCRAM_ERR_ALIAS;
    }
    const scram::Grid grid{S, Hq, Wq, Hk, Wk, d};
    const hipError_t e = scram::launch_attend(dtype, Q, K, V, argmax, kappa, grid, window, scale, causal, out, stream,
                                              events ? events[0] : nullptr, events ? events[1] : nullptr);
    return e == hipSuccess ? SCRAM_OK : SCRAM_ERR_HIP;
}

size_t scram_sparse_attend_backward_workspace_bytes(int S, int Hq, int Wq, int Hk, int Wk, int d, int dtype,
                                                    int kappa)
{
    if (check_grid(S, Hq, Wq, Hk, Wk) || kappa < 1 || kappa > SCRAM_MAX_KAPPA || check_type(dtype, d)) return 0;
    return scram::attend_backward_workspace_bytes(S, Hq, Wq, Hk, Wk, d, dtype, kappa);
}

int scram_sparse_attend_backward(const void* Q, const void* K, const void* V, int dtype, const int32_t* argmax,
                                 int kappa, int S, int Hq, int Wq, int Hk, int Wk, int d, int dv, int window,
                                 float scale, uint32_t flags, const void* dO, float* dQ, float* dK, float* dV,
                                 void* workspace, size_t workspace_bytes, hipEvent_t* events, hipStream_t stream)
{
    if (!Q || !K || !V || !argmax || !dO || !dQ || !dK || !dV) return SCRAM_ERR_NULL;
    int rc = check_grid(S, Hq, Wq, Hk, Wk);
    if (rc) return rc;
    // the inverse map codes (match, query) pairs as e * n + i in an int32, and
    // keys are numbered across slices (s * Hk * Wk + j)
    if (int64_t(S) * Hq * Wq * (kappa < 1 ? 1 : kappa) >= kMaxCount) return SCRAM_ERR_SHAPE;
    if (int64_t(S) * Hk * Wk >= kMaxCount) return SCRAM_ERR_SHAPE;
    if (window < 1 || window % 2 == 0 || window > 32767) return SCRAM_ERR_SHAPE;
    if (kappa < 1 || kappa > SCRAM_MAX_KAPPA) return SCRAM_ERR_SHAPE;
    if (!isfinite(scale)) return SCRAM_ERR_SHAPE;
    if ((rc = check_type(dtype, d))) return rc;
    if (scram::attend_backward_max_blocks(dtype, scram::Grid{S, Hq, Wq, Hk, Wk, d}, kappa) > kMaxBlocks)
        return SCRAM_ERR_SHAPE;
    if (dv != d) return SCRAM_ERR_UNSUPPORTED;
    if (flags & ~uint32_t(SCRAM_CAUSAL)) return SCRAM_ERR_UNSUPPORTED;
    const bool causal = (flags & SCRAM_CAUSAL) != 0;
    if (causal && (Hq != Hk || Wq != Wk)) return SCRAM_ERR_SHAPE;
    if (!workspace) return SCRAM_ERR_WORKSPACE;
    if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(dO, 16) || !aligned(argmax, 4) ||
        !aligned(dQ, 16) || !aligned(dK, 16) || !aligned(dV, 16) || !aligned(workspace, 256))
        return SCRAM_ERR_ALIGN;
    const size_t need = scram::attend_backward_workspace_bytes(S, Hq, Wq, Hk, Wk, d, dtype, kappa);
    if (workspace_bytes < need) return SCRAM_ERR_WORKSPACE;
    const size_t n = size_t(S) * Hq * Wq, nk = size_t(S) * Hk * Wk, eb = elem_bytes(dtype);
    const Range rQ = range(dQ, 4 * n * d), rK = range(dK, 4 * nk * d), rV = range(dV, 4 * nk * dv);
    const Range rW = range(workspace, need);
    for (const Range& o : {rQ, rK, rV, rW}) {
        for (const Range& other : {range(Q, n * d * eb), range(K, nk * d * eb), range(V, nk * dv * eb),
                                   range(argmax, 4 * n * size_t(kappa)), range(dO, n * dv * eb)}) {
            if (overlap(o, other)) return SCRAM_ERR_ALIAS;
        }
    }
    if (overlap(rQ, rK) || overlap(rQ, rV) || overlap(rK, rV) || overlap(rW, rQ) || overlap(rW, rK) ||
        overlap(rW, rV))
        return SCRAM_ERR_ALIAS;
    const scram::Grid grid{S, Hq, Wq, Hk, Wk, d};
    const hipError_t e = scram::launch_attend_backward(dtype, Q, K, V, argmax, kappa, grid, window, scale, causal, dO,
                                                       dQ, dK, dV, workspace, stream, events);
    return e == hipSuccess ? SCRAM_OK : SCRAM_ERR_HIP;
}

int scram_snis_attend(const void* Q, const void* K, const void* V, int dtype, const int32_t* modes, int kappa, int S,
                      int Hq, int Wq, int Hk, int Wk, int d, int dv, int samples, float alpha, int radius, float scale,
                      uint64_t seed, uint32_t flags, void* out, float* ess_out, float* var_out, hipEvent_t* events,
                      hipStream_t stream)
{
    if (!Q || !K || !V || !modes || !out) return SCRAM_ERR_NULL;
    int rc = check_grid(S, Hq, Wq, Hk, Wk);
    if (rc) return rc;
    if (kappa < 1 || kappa > SCRAM_MAX_KAPPA) return SCRAM_ERR_SHAPE;
    if (samples < 1 || samples > SCRAM_SNIS_MAX_SAMPLES) return SCRAM_ERR_SHAPE;
    if (!(alpha >= 0.f && alpha <= 1.f)) return SCRAM_ERR_SHAPE;  // also rejects NaN
    if (radius < 0 || radius > SCRAM_SNIS_MAX_RADIUS) return SCRAM_ERR_SHAPE;
    if (!isfinite(scale)) return SCRAM_ERR_SHAPE;
    if ((rc = check_type(dtype, d))) return rc;
    if (scram::snis_max_blocks(dtype, scram::Grid{S, Hq, Wq, Hk, Wk, d}) > kMaxBlocks) return SCRAM_ERR_SHAPE;
    if (dv != d) return SCRAM_ERR_UNSUPPORTED;
    if (flags & ~uint32_t(SCRAM_CAUSAL)) return SCRAM_ERR_UNSUPPORTED;
    const bool causal = (flags & SCRAM_CAUSAL) != 0;
    if (causal && (Hq != Hk || Wq != Wk)) return SCRAM_ERR_SHAPE;
    if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(out, 16) || !aligned(modes, 4) ||
        (ess_out && !aligned(ess_out, 4)) || (var_out && !aligned(var_out, 16)))
        return SCRAM_ERR_ALIGN;
    const size_t n = size_t(S) * Hq * Wq, eb = elem_bytes(dtype);
    const Range rO = range(out, n * dv * eb);
    const Range rE = ess_out ? range(ess_out, 4 * n) : Range{0, 0};
    const Range rV = var_out ? range(var_out, 4 * n * dv) : Range{0, 0};
    for (const Range& o : {rO, rE, rV}) {
        for (const Range& other : {range(Q, n * d * eb), range(K, size_t(S) * Hk * Wk * d * eb),
                                   range(V, size_t(S) * Hk * Wk * dv * eb), range(modes, 4 * n * size_t(kappa))}) {
            if (overlap(o, other)) return SCRAM_ERR_ALIAS;
        }
    }
    if (overlap(rO, rE) || overlap(rO, rV) || overlap(rE, rV)) return SCRAM_ERR_ALIAS;
    const scram::Grid grid{S, Hq, Wq, Hk, Wk, d};
    const scram::SnisSpec spec{samples, alpha, radius, scale, seed};
    const hipError_t e = scram::launch_snis(dtype, Q, K, V, modes, kappa, grid, spec, causal, out, ess_out, var_out,
                                            stream, events ? events[0] : nullptr, events ? events[1] : nullptr);
    return e == hipSuccess ? SCRAM_OK : SCRAM_ERR_HIP;
}

const char* scram_status_string(int status)
{
    switch (status) {
        case SCRAM_OK: return "ok";
        case SCRAM_ERR_NULL: return "a required pointer is NULL";
        case SCRAM_ERR_SHAPE: return "a size or count is out of range";
        case SCRAM_ERR_UNSUPPORTED: return "unsupported dtype, channel count or flag";
        case SCRAM_ERR_ALIGN: return "a pointer is not aligned as required";
        case SCRAM_ERR_ALIAS: return "an output overlaps an input or another output";
        case SCRAM_ERR_HIP: return "a HIP launch or copy failed";
        case SCRAM_ERR_WORKSPACE: return "workspace missing or too small";
        case SCRAM_ERR_SCRATCH: return "more queries than the no-allocation entry point's fixed scratch holds";
        default: return "unknown status";
    }
}

int scram_abi_version(void) { return SCRAM_ABI_VERSION; }

}  // extern "C"
