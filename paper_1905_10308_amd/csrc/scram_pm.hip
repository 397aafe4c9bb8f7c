// PatchMatch kernels (Algorithm 1): the random initial field and one
// synchronous sweep of propagation and random search.

#include "scram_device.h"

namespace scram {
namespace {

struct PmParams {
    const void* Q;
    const void* K;
    const int32_t* init;  // init kernel: optional given map
    const int32_t* Jp;    // sweep: previous map and scores
    const float* sp;
    int32_t* Jn;          // output map (init kernel: may be null)
    float* sn;            // output scores
    uint32_t n;           // S * Hq * Wq
    int Hq, Wq, Hk, Wk;
    uint32_t plane_q;     // Hq * Wq
    uint32_t nkeys;       // Hk * Wk
    Div div_plane, div_wq, div_wk;
    uint32_t key0, key1;  // Philox key
    uint32_t t;           // sweep index (Philox counter word 1)
    int R;                // max(Hk, Wk)
    int rs_steps;         // floor(log2 R) + 1
    const int32_t* prev;  // [n_prev, n] maps of the previous runs (validity variant)
    int n_prev;           // also this run's index: Philox counter word 3
    int sep;              // minimum Chebyshev distance to every previous match
    int causal;           // keys after the query (raster order) are not valid
    int first;            // the sweep recomputes the random initial field (Jp, sp unused)
    int marked_in;        // Jp entries carry kStable (Jp was written by a sweep with mark_out)
    int mark_out;         // set kStable on Jn entries whose match did not change
    Tiling tq;            // sweep blocks -> tiles of the query grid
};


constexpr int kMaxPrev = 7;  // previous runs a PatchMatch run may be constrained by

// Between two sweeps of one call the map entries carry a mark in bit 31:
// set when the sweep that wrote the entry kept its incumbent.  A query's
// propagation candidate from a marked neighbour is the candidate that query
// already scored in the previous sweep (same neighbour match, same offset),
// and that sweep ended on a running best at least as good in the strict
// total order; the best only improves, so the candidate cannot win again and
// is not gathered.  The result is identical with or without the mark.
constexpr uint32_t kStable = 0x80000000u;

// is_index_valid for one query: not after the query when causal, and at
// Chebyshev distance >= sep from each previous run's match (at most NP of
// them, a compile-time bound so the matches live in registers).
template <int NP>
struct Validity {
    static constexpr int kSlots = NP > 0 ? NP : 1;
    int n, sep;
    bool causal;
    uint32_t local;  // the query's raster index in its slice
    uint32_t pu[kSlots], pv[kSlots];

    __device__ bool ok(uint32_t r, uint32_t c, int32_t idx) const
    {
        bool v = !(causal && static_cast<uint32_t>(idx) > local);
#pragma unroll
        for (int i = 0; i < NP; ++i) {
            if (i < n) {
                const int du = abs(static_cast<int>(r) - static_cast<int>(pu[i]));
                const int dv = abs(static_cast<int>(c) - static_cast<int>(pv[i]));
                v = v && max(du, dv) >= sep;
            }
        }
        return v;
    }
};

// ---------------------------------------------------------------------------
// K1: initial field and its scores
// ---------------------------------------------------------------------------

// The random initial match of query g (raster index rem in its slice): the
// Philox block (g, 0, 0, run) mapped onto the key grid, or, with the causal
// mask, onto the keys up to the query.  The first sweep of a fresh run
// recomputes its neighbours' initial matches with this same function.
__device__ __forceinline__ int32_t initial_draw(const PmParams& p, uint32_t g, uint32_t rem)
{
    const uint4 w = philox4x32_10(g, 0u, 0u, static_cast<uint32_t>(p.n_prev), p.key0, p.key1);
    if (p.causal) return static_cast<int32_t>(__umulhi(w.x, rem + 1u));
    const uint32_t u = __umulhi(w.x, static_cast<uint32_t>(p.Hk));
    const uint32_t v = __umulhi(w.y, static_cast<uint32_t>(p.Wk));
    return static_cast<int32_t>(u * p.Wk + v);
}
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void pm_init_kernel(PmParams p)
{
    using RW = Row<T, D, G>;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t g = blockIdx.x * RW::kQpb + threadIdx.x / G;
    if (g >= p.n) return;  // whole lane groups leave together
    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);

    const int32_t idx = p.init ? clamp_index(p.init[g], p.nkeys) : initial_draw(p, g, rem);
    const T* Ks = static_cast<const T*>(p.K) + static_cast<size_t>(s) * p.nkeys * D;
    uint4 q[RW::kCh], k[RW::kCh];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    load_row<T, D, G>(Ks, idx, lane, k);
    const float sc = row_score<T, D, G>(q, k);
    if (lane == 0) {
        if (p.Jn) p.Jn[g] = idx;
        p.sn[g] = sc;
    }
}

// ---------------------------------------------------------------------------
// K2: one Jacobi sweep (propagation + random search), (Jp, sp) -> (Jn, sn)
//
// Each lane group carries QPG queries whose gathers are interleaved, so a
// wave keeps several independent loads in flight.  A sweep has two stages:
//   1. a batch of candidates that do not depend on each other: the 16
//      propagation candidates and random-search step 0 -- at distance R the
//      clipped search window is the whole key grid, so that draw does not
//      depend on the running best.  Candidates outside the grids or equal to
//      the incumbent (which cannot win) are dropped, the rest compacted per
//      query in shared memory via wave ballots and gathered kNb at a time.
//   2. random-search steps 1, 2, ...: each window is centred on the running
//      best, so they form a dependent chain (interleaved across the QPG
//      queries).
// Because "better" is a strict total order, visiting the candidates of
// stage 1 in any order gives the same result as the order of Algorithm 1.
// ---------------------------------------------------------------------------
// NP < 0: no validity test (a single-match run without masking); NP >= 0:
// causal masking and/or up to NP previous runs.  FIRST: the first sweep of a
// run started from the random initial field, which is not read from memory:
// each query recomputes its own initial match and those of its neighbours
// (initial_draw) and scores its own.
template <typename T, int D, int G, int QPG, int kNb, bool PROP, bool RS, int NP, bool FIRST = false>
__global__ __launch_bounds__(kBlock) void pm_iter_kernel(PmParams p)
{
    constexpr bool VALID = NP >= 0;
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int kGroups = RW::kQpb;           // lane groups per block
    constexpr int kQpb = kGroups * QPG;         // queries per block
    constexpr int kList = 17;                   // 16 propagation candidates + random-search step 0
    constexpr int kSlots = (kList + G - 1) / G; // candidate slots per lane
    static_assert(16 % G == 0, "step 0's Philox block and its candidate slot must share lane 0");
    __shared__ int32_t s_list[kGroups * QPG * kList];

    const int lane = threadIdx.x & (G - 1);
    const int qslot = threadIdx.x / G;
    const int gbase = (threadIdx.x & 63) - lane;  // wave lane of the group's first lane
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);

    uint32_t g[QPG], s[QPG], x[QPG], y[QPG];
    bool live[QPG];
    const T* Ks[QPG];
    uint4 q[QPG][CH];
    int32_t cur[QPG], cur0[QPG];
    float best[QPG];
#pragma unroll
    for (int j = 0; j < QPG; ++j) {
        uint32_t gr;
        live[j] = tile_item<kQpb>(p.tq, blk, j * kGroups + qslot, gr);
        // groups past the grid's edge work on the last query and write nothing, so
        // every lane reaches the block barrier below
        g[j] = live[j] ? gr : p.n - 1;
        uint32_t rem;
        divmod(g[j], p.div_plane, s[j], rem);
        divmod(rem, p.div_wq, x[j], y[j]);
        Ks[j] = static_cast<const T*>(p.K) + static_cast<size_t>(s[j]) * p.nkeys * D;
        load_row<T, D, G>(static_cast<const T*>(p.Q), g[j], lane, q[j]);
        if constexpr (FIRST) {
            cur[j] = initial_draw(p, g[j], x[j] * p.Wq + y[j]);
        } else {
            const int32_t raw = p.Jp[g[j]];
            cur[j] = clamp_index(p.marked_in ? static_cast<int32_t>(raw & ~kStable) : raw, p.nkeys);
            best[j] = p.sp[g[j]];
        }
        cur0[j] = cur[j];
    }
    // FIRST: the incumbent's row, scored once stage 1's candidates are built
    uint4 kinc[QPG][CH];
    if constexpr (FIRST) {
#pragma unroll
        for (int j = 0; j < QPG; ++j) load_row<T, D, G>(Ks[j], cur[j], lane, kinc[j]);
    }
    // validity variant: the previous runs' matches of each query; an invalid
    // incumbent counts as minus infinity
    Validity<NP> val[QPG];
    if constexpr (VALID) {
#pragma unroll
        for (int j = 0; j < QPG; ++j) {
            val[j].n = p.n_prev;
            val[j].sep = p.sep;
            val[j].causal = p.causal != 0;
            val[j].local = x[j] * p.Wq + y[j];
#pragma unroll
            for (int i = 0; i < Validity<NP>::kSlots; ++i) {
                val[j].pu[i] = val[j].pv[i] = 0u;
                if (i < p.n_prev)
                    divmod(static_cast<uint32_t>(clamp_index(p.prev[static_cast<size_t>(i) * p.n + g[j]], p.nkeys)),
                           p.div_wk, val[j].pu[i], val[j].pv[i]);
            }
            if constexpr (!FIRST) {
                uint32_t u0, v0;
                divmod(static_cast<uint32_t>(cur[j]), p.div_wk, u0, v0);
                if (!val[j].ok(u0, v0, cur[j])) best[j] = -INFINITY;
            }
        }
    }

    // Philox blocks of this sweep: block m serves random-search steps 2m and
    // 2m+1; lane l draws block l (the first round; later rounds below).
    const int nblk = RS ? (p.rs_steps + 1) >> 1 : 0;
    uint4 w0[QPG];
#pragma unroll
    for (int j = 0; j < QPG; ++j) {
        w0[j] = make_uint4(0u, 0u, 0u, 0u);
        if (lane < nblk)
            w0[j] = philox4x32_10(g[j], p.t, static_cast<uint32_t>(lane), static_cast<uint32_t>(p.n_prev), p.key0,
                                  p.key1);
    }

    // ---- stage 1 ----
    int count[QPG];
    const int32_t* Jp = p.Jp;
#pragma unroll
    for (int j = 0; j < QPG; ++j) {
        count[j] = 0;
        int32_t* list = s_list + (j * kGroups + qslot) * kList;
#pragma unroll
        for (int m = 0; m < kSlots; ++m) {
            const int i = lane + m * G;
            int32_t c = -1;
            if (PROP && i < 16) {
                // jump index i/4 over 8,4,2,1; direction i%4 over row-1, row+1,
                // col-1, col+1: the neighbour's match shifted back by the offset
                const int jump = 8 >> (i >> 2);
                const int dir = i & 3;
                const int ox = dir == 0 ? -jump : (dir == 1 ? jump : 0);
                const int oy = dir == 2 ? -jump : (dir == 3 ? jump : 0);
                const int nx = static_cast<int>(x[j]) + ox, ny = static_cast<int>(y[j]) + oy;
                if (nx >= 0 && nx < p.Hq && ny >= 0 && ny < p.Wq) {
                    const uint32_t ng = static_cast<uint32_t>((static_cast<size_t>(s[j]) * p.Hq + nx) * p.Wq + ny);
                    uint32_t nb;
                    bool seen = false;  // scored by this query in the previous sweep
                    if constexpr (FIRST) {
                        nb = static_cast<uint32_t>(initial_draw(p, ng, static_cast<uint32_t>(nx * p.Wq + ny)));
                    } else {
                        int32_t raw = Jp[ng];
                        if (p.marked_in) {
                            seen = (static_cast<uint32_t>(raw) & kStable) != 0u;
                            raw = static_cast<int32_t>(raw & ~kStable);
                        }
                        nb = clamp_index(raw, p.nkeys);
                    }
                    uint32_t nu, nv;
                    divmod(nb, p.div_wk, nu, nv);
                    const int r = static_cast<int>(nu) - ox, cc = static_cast<int>(nv) - oy;
                    if (!seen && r >= 0 && r < p.Hk && cc >= 0 && cc < p.Wk) {
                        c = r * p.Wk + cc;
                        if (VALID && !val[j].ok(r, cc, c)) c = -1;
                    }
                }
            } else if (RS && i == 16) {
                // random-search step 0: uniform over the whole key grid
                const uint32_t r = __umulhi(w0[j].x, static_cast<uint32_t>(p.Hk));
                const uint32_t cc = __umulhi(w0[j].y, static_cast<uint32_t>(p.Wk));
                c = static_cast<int32_t>(r * p.Wk + cc);
                if (VALID && !val[j].ok(r, cc, c)) c = -1;
            }
            const bool keep = c >= 0 && c != cur0[j];
            const uint64_t bal = __ballot(keep);
            const uint32_t grp = static_cast<uint32_t>(bal >> gbase) & (G == 32 ? 0xFFFFFFFFu : ((1u << G) - 1u));
            if (keep) list[count[j] + __popc(grp & ((1u << lane) - 1u))] = c;
            count[j] += __popc(grp);
        }
    }
    if constexpr (FIRST) {
#pragma unroll
        for (int j = 0; j < QPG; ++j) {
            best[j] = row_score<T, D, G>(q[j], kinc[j]);
            if constexpr (VALID) {
                uint32_t u0, v0;
                divmod(static_cast<uint32_t>(cur[j]), p.div_wk, u0, v0);
                if (!val[j].ok(u0, v0, cur[j])) best[j] = -INFINITY;
            }
        }
    }
    __syncthreads();

    {
        // gather kNb list entries of every query per batch: all loads in
        // flight, then the dot products (independent chains), then the
        // comparisons.  Slots past the end of a list keep stale data whose
        // score is never used.
        uint4 raw[QPG][kNb][CH];
#pragma unroll
        for (int j = 0; j < QPG; ++j)
#pragma unroll
            for (int e = 0; e < kNb; ++e)
#pragma unroll
                for (int c = 0; c < CH; ++c) raw[j][e][c] = make_uint4(0u, 0u, 0u, 0u);
        int most = count[0];
#pragma unroll
        for (int j = 1; j < QPG; ++j) most = max(most, count[j]);
        for (int k0 = 0; __any(k0 < most); k0 += kNb) {
            int32_t idx[QPG][kNb];
#pragma unroll
            for (int j = 0; j < QPG; ++j) {
                const int32_t* list = s_list + (j * kGroups + qslot) * kList;
#pragma unroll
                for (int e = 0; e < kNb; ++e) {
                    const int kk = k0 + e;
                    const int32_t entry = list[min(kk, kList - 1)];  // in bounds; stale past the end
                    idx[j][e] = kk < count[j] ? entry : cur0[j];
                    if (kk < count[j]) load_row<T, D, G>(Ks[j], idx[j][e], lane, raw[j][e]);
                }
            }
            float sc[QPG][kNb];
#pragma unroll
            for (int j = 0; j < QPG; ++j)
#pragma unroll
                for (int e = 0; e < kNb; ++e) sc[j][e] = row_score<T, D, G>(q[j], raw[j][e]);
#pragma unroll
            for (int j = 0; j < QPG; ++j)
#pragma unroll
                for (int e = 0; e < kNb; ++e) {
                    const bool take = (k0 + e < count[j]) & better(sc[j][e], idx[j][e], best[j], cur[j]);
                    best[j] = take ? sc[j][e] : best[j];
                    cur[j] = take ? idx[j][e] : cur[j];
                }
        }
    }

    // ---- stage 2: random-search steps 1, 2, ... around the running best ----
    // Step k uses words 2(k mod 2), 2(k mod 2)+1 of Philox block k/2, held by
    // lane (k/2) mod G of the group; a new round of blocks is drawn every 2G
    // steps.  A draw equal to the incumbent scores bit-identically and is not
    // "better", so it needs no special case.
    if constexpr (RS) {
        uint32_t cu[QPG], cv[QPG];
        uint4 w[QPG];
#pragma unroll
        for (int j = 0; j < QPG; ++j) {
            divmod(static_cast<uint32_t>(cur[j]), p.div_wk, cu[j], cv[j]);
            w[j] = w0[j];
        }
        for (int k = 1; k < p.rs_steps; ++k) {
            const int m = k >> 1;
            if ((k & 1) == 0 && m % G == 0) {
#pragma unroll
                for (int j = 0; j < QPG; ++j) {
                    w[j] = make_uint4(0u, 0u, 0u, 0u);
                    if (m + lane < nblk)
                        w[j] = philox4x32_10(g[j], p.t, static_cast<uint32_t>(m + lane),
                                             static_cast<uint32_t>(p.n_prev), p.key0, p.key1);
                }
            }
            const int src = gbase + m % G;
            const int dk = p.R >> k;
            int32_t idx[QPG];
            uint32_t rr[QPG], rc[QPG];
            uint4 kr[QPG][CH];
#pragma unroll
            for (int j = 0; j < QPG; ++j) {
                const uint32_t wr = __shfl((k & 1) ? w[j].z : w[j].x, src);
                const uint32_t wc = __shfl((k & 1) ? w[j].w : w[j].y, src);
                const int lo_r = max(static_cast<int>(cu[j]) - dk, 0);
                const int hi_r = min(static_cast<int>(cu[j]) + dk, p.Hk - 1);
                const int lo_c = max(static_cast<int>(cv[j]) - dk, 0);
                const int hi_c = min(static_cast<int>(cv[j]) + dk, p.Wk - 1);
                rr[j] = lo_r + __umulhi(wr, static_cast<uint32_t>(hi_r - lo_r + 1));
                rc[j] = lo_c + __umulhi(wc, static_cast<uint32_t>(hi_c - lo_c + 1));
                idx[j] = static_cast<int32_t>(rr[j] * p.Wk + rc[j]);
                load_row<T, D, G>(Ks[j], idx[j], lane, kr[j]);
            }
#pragma unroll
            for (int j = 0; j < QPG; ++j) {
                const float sc = row_score<T, D, G>(q[j], kr[j]);
                const bool ok = !VALID || val[j].ok(rr[j], rc[j], idx[j]);
                const bool gain = better(sc, idx[j], best[j], cur[j]);
                const bool take = ok && gain;
                best[j] = take ? sc : best[j];
                cur[j] = take ? idx[j] : cur[j];
                cu[j] = take ? rr[j] : cu[j];
                cv[j] = take ? rc[j] : cv[j];
            }
        }
    }

#pragma unroll
    for (int j = 0; j < QPG; ++j) {
        if (live[j] && lane == 0) {
            p.Jn[g[j]] = static_cast<int32_t>(static_cast<uint32_t>(cur[j]) |
                                              (p.mark_out && cur[j] == cur0[j] ? kStable : 0u));
            p.sn[g[j]] = best[j];
        }
    }
}

PmParams make_pm_params(const void* Q, const void* K, const Grid& gr, uint64_t seed)
{
    PmParams p{};
    p.Q = Q;
    p.K = K;
    p.n = static_cast<uint32_t>(gr.S) * gr.Hq * gr.Wq;
    p.Hq = gr.Hq;
    p.Wq = gr.Wq;
    p.Hk = gr.Hk;
    p.Wk = gr.Wk;
    p.plane_q = static_cast<uint32_t>(gr.Hq) * gr.Wq;
    p.nkeys = static_cast<uint32_t>(gr.Hk) * gr.Wk;
    p.div_plane = make_div(p.plane_q);
    p.div_wq = make_div(gr.Wq);
    p.div_wk = make_div(gr.Wk);
    p.key0 = static_cast<uint32_t>(seed & 0xFFFFFFFFu);
    p.key1 = static_cast<uint32_t>(seed >> 32);
    p.R = gr.Hk > gr.Wk ? gr.Hk : gr.Wk;
    int steps = 1;
    for (int r = p.R; r > 1; r >>= 1) ++steps;
    p.rs_steps = steps;
    return p;
}

template <typename T, int D>
hipError_t run_init(const PmParams& p, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kPm;
    const uint64_t blocks = (uint64_t(p.n) + Row<T, D, G>::kQpb - 1) / Row<T, D, G>::kQpb;
    return launch(pm_init_kernel<T, D, G>, blocks, st, e0, e1, p);
}

#ifndef SCRAM_PM_QPG
#define SCRAM_PM_QPG 1
#endif
#ifndef SCRAM_PM_BATCH
#define SCRAM_PM_BATCH 3
#endif

template <typename T, int D, int NP>
hipError_t run_iter_v(const PmParams& p, uint32_t flags, uint64_t blocks, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kPm;
    constexpr int QPG = SCRAM_PM_QPG;
    constexpr int NB = SCRAM_PM_BATCH;
    const bool prop = !(flags & SCRAM_PM_NO_PROPAGATION);
    const bool rs = !(flags & SCRAM_PM_NO_RANDOM_SEARCH);
    if (p.first) return launch(pm_iter_kernel<T, D, G, QPG, NB, true, true, NP, true>, blocks, st, e0, e1, p);
    if (prop && rs) return launch(pm_iter_kernel<T, D, G, QPG, NB, true, true, NP>, blocks, st, e0, e1, p);
    if (prop) return launch(pm_iter_kernel<T, D, G, QPG, NB, true, false, NP>, blocks, st, e0, e1, p);
    if (rs) return launch(pm_iter_kernel<T, D, G, QPG, NB, false, true, NP>, blocks, st, e0, e1, p);
    return launch(pm_iter_kernel<T, D, G, QPG, NB, false, false, NP>, blocks, st, e0, e1, p);
}

template <typename T, int D>
hipError_t run_iter(const PmParams& p0, uint32_t flags, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kPm;
    PmParams p = p0;
    p.tq = make_tiling(p.Hq, p.Wq, Row<T, D, G>::kQpb * SCRAM_PM_QPG, kLaneSkew);
    const uint64_t blocks = tiling_blocks(p.tq, p.n / p.plane_q);
    // the smallest register budget that holds this run's previous matches
    if (p.n_prev == 0) {
        return p.causal ? run_iter_v<T, D, 0>(p, flags, blocks, st, e0, e1)
                        : run_iter_v<T, D, -1>(p, flags, blocks, st, e0, e1);
    }
    if (p.n_prev <= 1) return run_iter_v<T, D, 1>(p, flags, blocks, st, e0, e1);
    if (p.n_prev <= 3) return run_iter_v<T, D, 3>(p, flags, blocks, st, e0, e1);
    return run_iter_v<T, D, kMaxPrev>(p, flags, blocks, st, e0, e1);
}

}  // namespace

hipError_t launch_pm_init(int dtype, const void* Q, const void* K, const Grid& g, uint64_t seed,
                          const RunSpec& run, const int32_t* init, int32_t* J, float* s, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop)
{
    PmParams p = make_pm_params(Q, K, g, seed);
    p.init = init;
    p.Jn = J;
    p.sn = s;
    p.n_prev = run.n_prev;
    p.causal = run.causal ? 1 : 0;
    return dispatch(dtype, g.d, [&](auto t, auto d) {
        return run_init<decltype(t), decltype(d)::value>(p, stream, start, stop);
    });
}

hipError_t launch_pm_iter(int dtype, const void* Q, const void* K, const Grid& g, uint64_t seed,
                          const RunSpec& run, uint32_t t, uint32_t flags, const int32_t* Jp, const float* sp,
                          bool marked_in, bool mark_out, int32_t* Jn, float* sn, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop)
{
    PmParams p = make_pm_params(Q, K, g, seed);
    p.marked_in = marked_in && Jp != nullptr ? 1 : 0;
    p.mark_out = mark_out ? 1 : 0;
    // no previous map: the first sweep of a fresh run (propagation and random
    // search both on) starts from the random initial field it recomputes
    p.first = Jp == nullptr ? 1 : 0;
    p.t = t;
    p.Jp = Jp;
    p.sp = sp;
    p.Jn = Jn;
    p.sn = sn;
    p.prev = run.prev;
    p.n_prev = run.n_prev;
    p.sep = run.sep;
    p.causal = run.causal ? 1 : 0;
    return dispatch(dtype, g.d, [&](auto ty, auto d) {
        return run_iter<decltype(ty), decltype(d)::value>(p, flags, stream, start, stop);
    });
}

uint64_t patchmatch_max_blocks(int dtype, const Grid& g)
{
    return dispatch_value(dtype, g.d, uint64_t(0), [&](auto t, auto d) {
        using T = decltype(t);
        constexpr int D = decltype(d)::value;
        constexpr uint32_t kQpb = Row<T, D, Lanes<T, D>::kPm>::kQpb;
        const uint64_t init = (uint64_t(g.S) * g.Hq * g.Wq + kQpb - 1) / kQpb;
        const uint64_t iter = tiling_blocks(make_tiling(g.Hq, g.Wq, kQpb * SCRAM_PM_QPG, kLaneSkew), g.S);
        return init > iter ? init : iter;
    });
}

}  // namespace scram
