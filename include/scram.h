/*
 * scram.h -- C ABI of the SCRAM hot path on AMD Instinct MI355X (gfx950).
 *
 * SCRAM ("Spatially Coherent Randomized Attention Maps", Calian et al. 2019)
 * approximates one attention / non-local-mean layer over an image in two
 * steps, both exported here:
 *
 *   1. scram_patchmatch -- PatchMatch (Algorithm 1, run once: kappa = 1)
 *      estimates for every query pixel the key pixel with the largest q.k
 *      (Equation 7 at kappa = 1): random initialisation, then T synchronous
 *      sweeps of propagation from neighbours at distances 8, 4, 2, 1 and
 *      random search at distances R, R/2, ..., 1.
 *   2. scram_sparse_attend -- the sparse non-local mean (Algorithm 2,
 *      Equations 8-9): a softmax of scale * q.k over the (2b+1) x (2b+1)
 *      window of keys around each query's match, then the weighted sum of
 *      the values of those keys.
 *
 * Several matches per query (kappa > 1, Section 4.2 and Algorithm 2's first
 * step) come from kappa runs of scram_patchmatch, run c receiving the maps of
 * runs 0..c-1 (Algorithm 1's input J) and a separation L: is_index_valid
 * keeps a key only if its Chebyshev distance max(|du|, |dv|) to each earlier
 * match is at least L (L = 1: distinct keys, the top-kappa-max variant;
 * L > 1: separated modes, top-kappa-mode).  scram_sparse_attend then takes
 * the union of the kappa windows, each key once.  SCRAM_CAUSAL (Section
 * 4.2.1) restricts both steps to keys at or before the query in raster order.
 *
 * scram_sparse_attend_backward gives the gradients of step 2 with respect to
 * Q, K and V with the maps held fixed.
 *
 * scram_snis_attend replaces the window of step 2 by the self-normalised
 * importance-sampling estimator of Section 4.2 (Monte Carlo estimators,
 * Equations 11-17): T keys per query drawn from a mixture of local densities
 * around the kappa matches and a uniform distribution, weighted by
 * exp(a_ij) / r_i(j).
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 * - Data layout: row-major, channels innermost.  Q is [S, Hq, Wq, d], K is
 *   [S, Hk, Wk, d], V is [S, Hk, Wk, dv], the output of the attend step is
 *   [S, Hq, Wq, dv]; S counts independent slices (batch x heads).  Index maps
 *   are int32 [S, Hq, Wq] holding the flat key index u * Wk + v of key pixel
 *   (u, v) inside the query's own slice.  Query (s, x, y) has the global id
 *   g = (s * Hq + x) * Wq + y.  Self-attention is the case Hq = Hk, Wq = Wk;
 *   different grids give a general non-local mean (Equation 4).
 * - Element types: SCRAM_F32 (fp32) or SCRAM_BF16 (bfloat16) storage for Q,
 *   K, V and the attend output; all arithmetic accumulates in fp32.
 * - Supported sizes: d in {16, 32, 64, 128}; dv == d; S*Hq*Wq < 2^31 and
 *   Hk*Wk < 2^31.  One kernel dispatch holds at most 2^32 - 1 work-items, and
 *   the kernels give each query (or key) d * elem_bytes / 32 lanes (at least
 *   one), so a call is also rejected with SCRAM_ERR_SHAPE when its largest
 *   grid, rounded up to whole tiles of the query or key grid, would exceed
 *   that -- roughly when the query (or key) tensor passes 128 GiB.
 * - Pointers are device pointers (HIP) owned by the caller.  Q, K, V and the
 *   attend output must be 16-byte aligned; index and score buffers 4-byte
 *   aligned; the workspace 256-byte aligned.  The library allocates no memory
 *   and keeps no state between calls; calls are re-entrant.  (The one
 *   exception is scram_patchmatch_noalloc, whose buffers are a fixed device
 *   array the library holds; see there.)
 * - Every call only enqueues work on `stream` (0 = the null stream) and
 *   returns without synchronising.  Arguments are validated on the host
 *   before any HIP call; a non-zero status means nothing was enqueued
 *   (SCRAM_ERR_HIP: a launch failed; work enqueued before it by the same call
 *   may still run).  Device faults surface at the caller's next
 *   synchronisation.  Nothing else crosses the ABI: no exceptions, no abort.
 * - Index values read from device memory (init, argmax) are clamped into
 *   [0, Hk*Wk) before use, so an out-of-range entry gives an unspecified
 *   result but never an out-of-bounds access.
 */
#ifndef SCRAM_H
#define SCRAM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* storage type of Q, K, V and the attend output */
typedef enum { SCRAM_F32 = 0, SCRAM_BF16 = 1 } scram_dtype;

/* status codes */
enum {
    SCRAM_OK = 0,
    SCRAM_ERR_NULL = -1,        /* a required pointer is NULL */
    SCRAM_ERR_SHAPE = -2,       /* a size or count is out of range */
    SCRAM_ERR_UNSUPPORTED = -3, /* dtype, d or dv not supported, unknown flag */
    SCRAM_ERR_ALIGN = -4,       /* a pointer is not aligned as required */
    SCRAM_ERR_ALIAS = -5,       /* an output overlaps an input or another output */
    SCRAM_ERR_HIP = -6,         /* a HIP call failed */
    SCRAM_ERR_WORKSPACE = -7,   /* workspace missing or smaller than required */
    SCRAM_ERR_SCRATCH = -8      /* more queries than scram_patchmatch_noalloc's fixed scratch holds */
};

/* flags of scram_patchmatch: switch one step of an iteration off (tests) */
enum { SCRAM_PM_NO_PROPAGATION = 1u, SCRAM_PM_NO_RANDOM_SEARCH = 2u };

/* flag of both entry points: autoregressive masking (query grid == key grid) */
enum { SCRAM_CAUSAL = 4u };

/* most previous runs one PatchMatch run may be constrained by, and most maps
 * one attend call may unite */
enum { SCRAM_MAX_PREV = 7, SCRAM_MAX_KAPPA = 8 };

/* limits of scram_snis_attend: samples per query, binomial radius m */
enum { SCRAM_SNIS_MAX_SAMPLES = 1 << 20, SCRAM_SNIS_MAX_RADIUS = 16 };

/*
 * Bytes of workspace scram_patchmatch needs for S*Hq*Wq queries: one int32
 * index map and two fp32 score maps, each rounded up to 256 bytes.
 */
size_t scram_patchmatch_workspace_bytes(int S, int Hq, int Wq);

/*
 * PatchMatch argmax (Algorithm 1 with kappa = 1, so is_index_valid reduces to
 * "inside the key grid"; the attend window size b is not used here).
 *
 * Initialisation (Algorithm 1, first loop): when `init` is NULL, query g
 * draws J0[g] = u * Wk + v with u = floor(w0 * Hk / 2^32),
 * v = floor(w1 * Wk / 2^32), where (w0, w1, ., .) is the Philox4x32-10 block
 * (Salmon et al., SC 2011) of counter (g, 0, 0, n_prev) and key
 * (seed mod 2^32, seed div 2^32); with SCRAM_CAUSAL, J0[g] =
 * floor(w0 * (i + 1) / 2^32) for the query's raster index i in its slice.  When `init` is given it is J0 (not
 * modified; entries clamped into the key grid).  The incumbent scores s0 are
 * the fp32 dot products q_g . k_J0[g], or `init_score` when given (which
 * must then hold exactly what this library computed for that map, e.g. a
 * previous call's score_out).
 *
 * Iterations t = t0, ..., t0 + iters - 1 (the "parallel foreach" over query
 * pixels), each reading only the previous iteration's map (a Jacobi sweep):
 *   - propagation: for jump in 8, 4, 2, 1 and each axis direction delta, the
 *     neighbour p' = p + jump * delta (skipped outside the query grid)
 *     offers its match shifted back by jump * delta (skipped outside the key
 *     grid) -- a shift in query is an equal shift in key (Section 4.1);
 *   - random search: with D = R = max(Hk, Wk), halved (integer) down to 1,
 *     a key drawn uniformly from the square of half-side D around the
 *     running best, clipped to the key grid; step k uses the Philox block of
 *     counter (g, t, k div 2, n_prev), words 2(k mod 2) and 2(k mod 2) + 1
 *     mapped like the initial draw onto the clipped rows and columns;
 *   - a candidate replaces the incumbent iff it is valid (see the several
 *     matches and causal notes above) and its unscaled fp32 score q.k is
 *     larger, or equal with a lower flat key index.  An incumbent that is
 *     not valid counts as minus infinity.
 *
 * Arguments:
 *   Q, K        inputs, layouts above, element type `dtype`
 *   S, Hq, Wq   slices and query grid; Hk, Wk key grid; d channels
 *   iters       T >= 0 sweeps (0 returns the initial map)
 *   seed        64-bit Philox key
 *   init        nullable int32 [S, Hq, Wq] initial map
 *   init_score  nullable fp32 [S, Hq, Wq] scores of `init` (ignored when
 *               init is NULL)
 *   t0          index of the first sweep, >= 1 (1 for a fresh run; a run
 *               split as (T1 sweeps) then (init = its map, t0 = T1 + 1)
 *               equals the unsplit run bit for bit)
 *   flags       0, or SCRAM_PM_NO_PROPAGATION / SCRAM_PM_NO_RANDOM_SEARCH /
 *               SCRAM_CAUSAL
 *   prev        int32 [n_prev, S, Hq, Wq] maps of the previous runs (NULL
 *               when n_prev = 0); read only
 *   n_prev      0 <= n_prev <= SCRAM_MAX_PREV: previous runs, and this run's
 *               index in the Philox counter (0 for a single-match run)
 *   sep         separation L >= 1 from the previous runs' matches
 *   argmax_out  int32 [S, Hq, Wq] final map J_T (written)
 *   score_out   nullable fp32 [S, Hq, Wq] final scores q . k_{J_T} (unscaled;
 *               minus infinity where no valid key was found)
 *   workspace   >= scram_patchmatch_workspace_bytes(S, Hq, Wq) bytes of
 *               device memory, contents ignored and overwritten
 *   events      nullable array of 2 * (iters + 1) caller-created HIP
 *               events, for timing the kernels: the dispatch of launch k
 *               stamps events[2k] with its start and events[2k + 1] with its
 *               end (k = 0: the initial map or its scores; k = 1..iters:
 *               sweep k).  When init and init_score are both given nothing
 *               is launched for k = 0 and events[0], events[1] are recorded
 *               back to back.  The library does not create, wait on or
 *               destroy them.
 * Outputs must not overlap each other, the inputs or the workspace
 * (SCRAM_ERR_ALIAS).  Returns a status code.
 */
int scram_patchmatch(const void* Q, const void* K, int dtype, int S, int Hq, int Wq, int Hk, int Wk,
                     int d, int iters, uint64_t seed, const int32_t* init, const float* init_score,
                     int t0, uint32_t flags, const int32_t* prev, int n_prev, int sep, int32_t* argmax_out,
                     float* score_out, void* workspace, size_t workspace_bytes, hipEvent_t* events,
                     hipStream_t stream);

/*
 * scram_patchmatch without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  The sweeps' ping-pong buffers (one int32
 * map and two fp32 score maps) live in a fixed array of
 * SCRAM_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it has
 * run this entry point on, from that first call until the process ends; the
 * call itself allocates nothing.
 *
 * Arguments, outputs, events and semantics are those of scram_patchmatch
 * (results bit for bit equal to it), minus workspace and workspace_bytes.
 * Limit: S * Hq * Wq <= SCRAM_NOALLOC_MAX_QUERIES, else SCRAM_ERR_SCRATCH;
 * like every other argument error, this is found on the host before any
 * HIP call.  The first call on a device looks up that device's copy of the
 * array (the device of `stream`, or the current device for the null
 * stream); a failure there is SCRAM_ERR_HIP.  The scratch needs no
 * clearing: every buffer in it is written before it is read.
 *
 * All calls on one GPU share its array, which keeps the last call's
 * contents: calls ordered on one stream are safe, but calls that may
 * overlap in time on one GPU (several streams, or host threads without an
 * ordering between their streams) race on it and give undefined results.
 */
enum {
    SCRAM_NOALLOC_MAX_QUERIES = 1 << 20,
    SCRAM_NOALLOC_SCRATCH_BYTES = 3 * 4 * SCRAM_NOALLOC_MAX_QUERIES /* 12 MiB */
};

int scram_patchmatch_noalloc(const void* Q, const void* K, int dtype, int S, int Hq, int Wq, int Hk, int Wk, int d,
                             int iters, uint64_t seed, const int32_t* init, const float* init_score, int t0,
                             uint32_t flags, const int32_t* prev, int n_prev, int sep, int32_t* argmax_out,
                             float* score_out, hipEvent_t* events, hipStream_t stream);

/*
 * Sparse attention around the matches (Algorithm 2, Equations 8-9).  For
 * query g with matches (u_e, v_e) = divmod(argmax[e][g], Wk), e < kappa: the
 * set W_g = union over e of {(u_e + a, v_e + c) : |a|, |c| <= b} with
 * b = (window - 1)/2, each key once, keys outside the key grid dropped (and,
 * with SCRAM_CAUSAL, keys after the query in raster order);
 * out[g] = sum_{j in W_g} softmax_j(scale * q_g . k_j) v_j, computed with an
 * fp32 online softmax and written in `dtype` (a zero row if W_g is empty,
 * which cannot happen without SCRAM_CAUSAL).
 *
 * Arguments:
 *   Q, K, V   inputs, layouts above; V has dv channels (dv == d); finite
 *             values (with bf16 storage and d of 32 or 64, the keys of
 *             neighbouring queries' windows are read in shared blocks in
 *             which a key outside a query's window has weight 0, and
 *             0 * inf would reach that query)
 *   argmax    int32 [kappa, S, Hq, Wq] flat key indices (e.g. kappa runs of
 *             scram_patchmatch)
 *   kappa     1 <= kappa <= SCRAM_MAX_KAPPA
 *   window    odd side 2b + 1 >= 1 of the square window (<= 32767)
 *   scale     softmax temperature, 1/sqrt(d_k) for Equation 1; finite
 *   flags     0 or SCRAM_CAUSAL
 *   out       [S, Hq, Wq, dv] in `dtype` (written; must not overlap inputs)
 *   events    nullable array of 2 caller-created HIP events stamped with the
 *             kernel's start and end (as in scram_patchmatch)
 * Returns a status code.
 */
int scram_sparse_attend(const void* Q, const void* K, const void* V, int dtype, const int32_t* argmax, int kappa,
                        int S, int Hq, int Wq, int Hk, int Wk, int d, int dv, int window, float scale,
                        uint32_t flags, void* out, hipEvent_t* events, hipStream_t stream);

/*
 * Backward of scram_sparse_attend with the maps held fixed (the key sets
 * W_i depend only on argmax, window and flags, so they carry no gradient).
 * With p_ij the softmax weights of query i over W_i, dp_ij = dO_i . v_j and
 * D_i = sum_j p_ij dp_ij:
 *   dQ_i = scale * sum_j p_ij (dp_ij - D_i) k_j
 *   dK_j = scale * sum_i p_ij (dp_ij - D_i) q_i
 *   dV_j = sum_i p_ij dO_i
 * (the derivative of Equations 8-9).  fp32 throughout; the scores and
 * weights are recomputed from Q, K, V (the forward output is not needed).
 * Key j lies in W_i exactly when a match of query i lies in the
 * (2b+1) x (2b+1) neighbourhood of j, so dK_j and dV_j gather over the
 * queries found through the inverse of the maps (kept in the workspace; for
 * fp32 storage and for windows of side 1 or above 15 the key side also copies
 * those queries' q, dO rows there in the inverse map's order).
 * Every gradient row has a single writer; the order in which the queries of
 * one match key are summed is the order the inverse map was filled in,
 * which may differ between calls (dK, dV may differ in the last bits; dQ is
 * deterministic).  A query with an empty set (causal only) contributes
 * nothing and gets dQ = 0.
 *
 * Arguments: as scram_sparse_attend, plus
 *   dO        [S, Hq, Wq, dv] in `dtype`: gradient of the output
 *   dQ        fp32 [S, Hq, Wq, d] (written)
 *   dK        fp32 [S, Hk, Wk, d] (written)
 *   dV        fp32 [S, Hk, Wk, dv] (written)
 *   workspace device scratch of at least
 *             scram_sparse_attend_backward_workspace_bytes(S, Hq, Wq, Hk, Wk,
 *             d, dtype, kappa) bytes, 256-byte aligned; contents undefined
 *             on return (about 2 * kappa * S*Hq*Wq rows of d elements plus
 *             a few int32 / fp32 per key and query)
 *   events    NULL or 6 events: start/stop of the inverse map's scan and
 *             fill, of the query side (clearing the counts, then the
 *             per-query kernel, which also counts the inverse map's entries)
 *             and of the key side
 * Also requires S*Hq*Wq*kappa < 2^31 and S*Hk*Wk < 2^31.  dQ, dK, dV must be 16-byte aligned;
 * no output or the workspace may overlap an input or another output.
 * Returns a status code.
 */
size_t scram_sparse_attend_backward_workspace_bytes(int S, int Hq, int Wq, int Hk, int Wk, int d, int dtype,
                                                    int kappa);

int scram_sparse_attend_backward(const void* Q, const void* K, const void* V, int dtype, const int32_t* argmax,
                                 int kappa, int S, int Hq, int Wq, int Hk, int Wk, int d, int dv, int window,
                                 float scale, uint32_t flags, const void* dO, float* dQ, float* dK, float* dV,
                                 void* workspace, size_t workspace_bytes, hipEvent_t* events, hipStream_t stream);

/*
 * Self-normalised importance sampling around the matches (Section 4.2,
 * Monte Carlo estimators, Equations 11-17).  For query i with matches
 * (u_e, v_e) = divmod(modes[e][i], Wk), e < kappa:
 *   - importance distribution (Equation 17):
 *       r_i(j) = alpha' / kappa * sum_e g(j; u_e, v_e) + (1 - alpha') / (Hk Wk)
 *     with alpha' = round(alpha * 65536) / 65536 and g the product over the
 *     two axes of a centred binomial offset (the number of ones among 2m fair
 *     bits, minus m: a discrete Gaussian of variance m / 2), the coordinate
 *     clamped to the grid (the edge row or column holds that side's tail);
 *   - sample t (Equation 12) of query g uses the Philox4x32-10 block
 *     (w0, w1, w2, w3) of counter (g, t, 0, 0x534E4953) and key (seed mod 2^32,
 *     seed div 2^32): if (w0 >> 16) < round(alpha * 65536), mode
 *     e = floor(w1 * kappa / 2^32) and offsets popcount(w2 & (2^2m - 1)) - m,
 *     popcount(w3 & (2^2m - 1)) - m; otherwise row floor(w2 * Hk / 2^32) and
 *     column floor(w3 * Wk / 2^32);
 *   - weights w_t = exp(scale * q_i . k_j_t) / r_i(j_t) (Equation 13; with
 *     SCRAM_CAUSAL a key after the query has weight 0);
 *   - out[i] = sum_t w_t v_j_t / sum_t w_t (Equation 14), written in `dtype`;
 *   - ess_out[i] = (sum_t w_t)^2 / sum_t w_t^2 (Equation 16);
 *   - var_out[i][e] = sum_t (w_t / sum_s w_s)^2 (v_j_t,e - out[i][e])^2
 *     (Equation 15 with self-normalised weights).
 * All in fp32, with weights kept relative to their running maximum (ratios
 * unchanged).  A query whose weights are all 0 gets a zero row, ESS 0 and
 * variance 0.  The variance takes a second pass over the same samples.  Sums
 * over more than 256 samples are compensated (Kahan), so the estimate, ESS and
 * variance keep fp32 accuracy up to SCRAM_SNIS_MAX_SAMPLES.
 *
 * Arguments:
 *   Q, K, V   inputs, layouts above; dv == d
 *   modes     int32 [kappa, S, Hq, Wq] flat key indices (e.g. PatchMatch maps)
 *   kappa     1 <= kappa <= SCRAM_MAX_KAPPA
 *   samples   T, 1 <= T <= SCRAM_SNIS_MAX_SAMPLES
 *   alpha     mixture weight of the local densities, 0 <= alpha <= 1
 *   radius    m, 0 <= m <= SCRAM_SNIS_MAX_RADIUS (m = 0: the mode itself)
 *   scale     softmax temperature (1/sqrt(d_k)); finite
 *   seed      Philox key
 *   flags     0 or SCRAM_CAUSAL
 *   out       [S, Hq, Wq, dv] in `dtype` (written)
 *   ess_out   nullable fp32 [S, Hq, Wq] (written)
 *   var_out   nullable fp32 [S, Hq, Wq, dv], 16-byte aligned (written)
 *   events    NULL or 2 events, as for scram_sparse_attend
 * Outputs must not overlap the inputs or each other.  Returns a status code.
 */
int scram_snis_attend(const void* Q, const void* K, const void* V, int dtype, const int32_t* modes, int kappa, int S,
                      int Hq, int Wq, int Hk, int Wk, int d, int dv, int samples, float alpha, int radius, float scale,
                      uint64_t seed, uint32_t flags, void* out, float* ess_out, float* var_out, hipEvent_t* events,
                      hipStream_t stream);

/* Static, NUL-terminated description of a status code. */
const char* scram_status_string(int status);

/* ABI version of this header: (major << 16) | minor. */
int scram_abi_version(void);

#define SCRAM_ABI_VERSION ((2 << 16) | 6)

#ifdef __cplusplus
}
#endif

#endif /* SCRAM_H */
