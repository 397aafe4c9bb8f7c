// Internal interface between the C-ABI front end (scram_api.cpp) and the
// kernels (scram_pm.hip, scram_attend.hip, scram_backward.hip,
// scram_snis.hip).  Arguments reaching these functions have been
// validated by the front end.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace scram {

struct Grid {
    int S, Hq, Wq, Hk, Wk, d;
};

// Constraints of one PatchMatch run: the maps of the n_prev previous runs
// (n_prev is also this run's index), their minimum separation, causality.
struct RunSpec {
    const int32_t* prev;
    int n_prev;
    int sep;
    bool causal;
};

// Host-side validation of scram_patchmatch's arguments (no HIP call); a null
// workspace stands for the library's own scratch and is not checked.
int patchmatch_check(const void* Q, const void* K, int dtype, int S, int Hq, int Wq, int Hk, int Wk, int d,
                     int iters, const int32_t* init, const float* init_score, int t0, uint32_t flags,
                     const int32_t* prev, int n_prev, int sep, const int32_t* argmax_out, const float* score_out,
                     const void* workspace, size_t workspace_bytes);

// Every launch takes optional start/stop events that the dispatch itself
// stamps with the kernel's start and end times (null: plain launch).

// Random initial map (init == nullptr) or the scores of a given map.
// J may be nullptr when init is given (the map is not copied).
hipError_t launch_pm_init(int dtype, const void* Q, const void* K, const Grid& g, uint64_t seed,
                          const RunSpec& run, const int32_t* init, int32_t* J, float* s, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop);

// One Jacobi sweep t: (Jp, sp) -> (Jn, sn).  Jp == sp == nullptr: the first
// sweep of a run from the random initial field (flags must be 0), which the
// sweep recomputes instead of reading.  marked_in: Jp was written by the
// previous sweep of the same call with mark_out, so its entries carry the
// stable mark (bit 31) that lets this sweep skip candidates it already
// scored; mark_out: write that mark (never into a map the caller reads).
hipError_t launch_pm_iter(int dtype, const void* Q, const void* K, const Grid& g, uint64_t seed,
                          const RunSpec& run, uint32_t t, uint32_t flags, const int32_t* Jp, const float* sp,
                          bool marked_in, bool mark_out, int32_t* Jn, float* sn, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop);

// Window softmax + value gather around the kappa maps in J ([kappa, n]).
hipError_t launch_attend(int dtype, const void* Q, const void* K, const void* V, const int32_t* J, int kappa,
                         const Grid& g, int window, float scale, bool causal, void* out, hipStream_t stream,
                         hipEvent_t start, hipEvent_t stop);

// Gradients of the attend step with the maps held fixed.  The workspace
// (attend_backward_workspace_bytes) holds the inverse map, per-query
// softmax statistics and the entry-ordered copies of q, dO and those
// statistics.  events: null or 6 (inverse map's scan and fill start/stop,
// query side (clearing the counts, then the query kernel, which counts the
// inverse map's entries) start/stop, key side start/stop).
size_t attend_backward_workspace_bytes(int S, int Hq, int Wq, int Hk, int Wk, int d, int dtype, int kappa);
hipError_t launch_attend_backward(int dtype, const void* Q, const void* K, const void* V, const int32_t* J, int kappa,
                                  const Grid& g, int window, float scale, bool causal, const void* dO, float* dQ,
                                  float* dK, float* dV, void* workspace, hipStream_t stream, hipEvent_t* events);

// Self-normalised importance sampling around the kappa maps in modes
// ([kappa, n]): samples per query, mixture weight, binomial radius m,
// softmax scale and Philox seed.
struct SnisSpec {
    int samples;
    float alpha;
    int radius;
    float scale;
    uint64_t seed;
};

hipError_t launch_snis(int dtype, const void* Q, const void* K, const void* V, const int32_t* modes, int kappa,
                       const Grid& g, const SnisSpec& spec, bool causal, void* out, float* ess, float* var,
                       hipStream_t stream, hipEvent_t start, hipEvent_t stop);

// Blocks (of 256 threads) of the largest dispatch an entry point makes for
// this shape; 0 for an unsupported (dtype, d).  One dispatch holds at most
// 2^32 - 1 work-items, so the front end rejects shapes above that.
uint64_t patchmatch_max_blocks(int dtype, const Grid& g);
uint64_t attend_max_blocks(int dtype, const Grid& g);
uint64_t snis_max_blocks(int dtype, const Grid& g);
uint64_t attend_backward_max_blocks(int dtype, const Grid& g, int kappa);

}  // namespace scram
