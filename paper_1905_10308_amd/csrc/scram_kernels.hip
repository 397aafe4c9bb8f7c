// HIP kernels of the SCRAM hot path for gfx950 (MI355X).
//
//   pm_init_kernel   -- random initial nearest-neighbour field (Algorithm 1,
//                       first loop) or the scores of a given field
//   pm_iter_kernel   -- one synchronous (Jacobi) sweep of Algorithm 1:
//                       propagation from neighbours at jumps 8, 4, 2, 1 and
//                       random search at distances R, R/2, ..., 1
//   attend_kernel    -- Algorithm 2 (Equations 8-9): online softmax over the
//                       (2b+1)^2 windows around the matches, fused with the
//                       gather of the values
//   snis_kernel      -- self-normalised importance sampling around the
//                       matches (Section 4.2, Equations 11-17)
//
// Work decomposition.  Every kernel gives one query pixel to a "lane group"
// of G lanes of a 64-wide wavefront.  A feature row (d channels) is split
// into 16-byte chunks; lane l of the group owns chunks l, l+G, l+2G, ... so
// each load instruction of the group reads one contiguous G*16-byte span of
// the row (fully coalesced), and q stays in registers in its storage format.
// A dot product is a per-lane chain in a fixed order -- v_dot2_f32_bf16 on
// packed bf16 pairs, or fp32 FMAs -- then a fixed butterfly across the group
// (DPP row permutes).  Every lane of the group ends with the bit-identical
// sum, so decisions are taken redundantly in registers, and the init and
// sweep kernels use the same order: a score never depends on which kernel
// computed it.
//
// Candidate gathers are not a dense contraction, so there is no MFMA here.
// Blocks are remapped so that consecutive query ranges land on the same XCD
// and share its L2.

#include <math.h>
#include <stdint.h>

#include <type_traits>

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "scram.h"
#include "scram_launch.h"

namespace scram {
namespace {

constexpr int kBlock = 256;  // threads per block: four wave64s
constexpr int kXcds = 8;     // XCDs per MI355X; blocks are dealt round-robin

// ---------------------------------------------------------------------------
// integer helpers
// ---------------------------------------------------------------------------

// x / d and x % d for x < 2^31 with a multiply-high by m = floor((2^32-1)/d).
// The estimate floor(x*m / 2^32) is floor(x/d) or one less (x < 2^31 keeps
// the error of m below one unit), so a single correction step is exact.
struct Div {
    uint32_t d, m;
};

Div make_div(uint32_t d) { return Div{d, 0xFFFFFFFFu / d}; }

__device__ __forceinline__ void divmod(uint32_t x, Div f, uint32_t& q, uint32_t& r)
{
    q = __umulhi(x, f.m);
    r = x - q * f.d;
    if (r >= f.d) {
        q += 1;
        r -= f.d;
    }
}

__device__ __forceinline__ int32_t clamp_index(int32_t j, uint32_t nkeys)
{
    return j < 0 ? 0 : (static_cast<uint32_t>(j) >= nkeys ? static_cast<int32_t>(nkeys - 1) : j);
}

// Block b of nb runs on XCD b % 8.  Give XCD x the contiguous logical range
// [start(x), start(x) + count(x)) so that neighbouring queries -- which read
// neighbouring keys -- share one L2.  A bijection for every nb.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t b, uint32_t nb)
{
    const uint32_t x = b % kXcds, local = b / kXcds;
    const uint32_t q = nb / kXcds, r = nb % kXcds;
    const uint32_t start = x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q;
    return start + local;
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds of two
// 32x32->64 multiplies mixed with the other two words and the round key; the
// key advances by the two Weyl increments after every round.
__device__ __forceinline__ uint4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                               uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int i = 0; i < 10; ++i) {
        const uint32_t a_hi = __umulhi(0xD2511F53u, c0), a_lo = 0xD2511F53u * c0;
        const uint32_t b_hi = __umulhi(0xCD9E8D57u, c2), b_lo = 0xCD9E8D57u * c2;
        const uint32_t n0 = b_hi ^ c1 ^ k0;
        const uint32_t n2 = a_hi ^ c3 ^ k1;
        c0 = n0;
        c1 = b_lo;
        c2 = n2;
        c3 = a_lo;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return make_uint4(c0, c1, c2, c3);
}

// ---------------------------------------------------------------------------
// rows: storage type T (float, or bfloat16 held as uint16_t), D channels,
// G lanes per query
// ---------------------------------------------------------------------------
template <typename T, int D, int G>
struct Row {
    static constexpr int kBytes = D * static_cast<int>(sizeof(T));
    static constexpr int kCh = kBytes / (16 * G);  // 16-byte chunks per lane
    static constexpr int kEpc = 16 / static_cast<int>(sizeof(T));  // channels per chunk
    static constexpr int kQpb = kBlock / G;        // queries per block
    static_assert(G >= 1 && G <= 32 && (G & (G - 1)) == 0, "lane group must be 1..32 lanes");
    static_assert(kCh >= 1 && kCh * 16 * G == kBytes, "row must split into whole chunks per lane");
};

// The lane's chunks of row `row` of a [rows, D] array.
template <typename T, int D, int G>
__device__ __forceinline__ void load_row(const T* base, uint32_t row, int lane, uint4 (&v)[Row<T, D, G>::kCh])
{
    const uint4* p = reinterpret_cast<const uint4*>(base + static_cast<size_t>(row) * D) + lane;
#pragma unroll
    for (int c = 0; c < Row<T, D, G>::kCh; ++c) v[c] = p[c * G];
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c,
                                           false);
}

// Per-lane partial dot product in a fixed order.
template <typename T, int CH>
__device__ __forceinline__ float lane_dot(const uint4 (&q)[CH], const uint4 (&k)[CH])
{
    if constexpr (std::is_same<T, uint16_t>::value) {
        float acc = 0.f;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            acc = dot2_bf16(q[c].x, k[c].x, acc);
            acc = dot2_bf16(q[c].y, k[c].y, acc);
            acc = dot2_bf16(q[c].z, k[c].z, acc);
            acc = dot2_bf16(q[c].w, k[c].w, acc);
        }
        return acc;
    } else {
        float acc = __uint_as_float(q[0].x) * __uint_as_float(k[0].x);
        acc = fmaf(__uint_as_float(q[0].y), __uint_as_float(k[0].y), acc);
        acc = fmaf(__uint_as_float(q[0].z), __uint_as_float(k[0].z), acc);
        acc = fmaf(__uint_as_float(q[0].w), __uint_as_float(k[0].w), acc);
#pragma unroll
        for (int c = 1; c < CH; ++c) {
            acc = fmaf(__uint_as_float(q[c].x), __uint_as_float(k[c].x), acc);
            acc = fmaf(__uint_as_float(q[c].y), __uint_as_float(k[c].y), acc);
            acc = fmaf(__uint_as_float(q[c].z), __uint_as_float(k[c].z), acc);
            acc = fmaf(__uint_as_float(q[c].w), __uint_as_float(k[c].w), acc);
        }
        return acc;
    }
}

// Value of a partner lane inside the row (every pattern used here stays
// inside the group, so bound_ctrl never applies).
template <int CTRL>
__device__ __forceinline__ float dpp(float x)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}

// Sum over an aligned group of G lanes.  Each step adds the value of a
// partner lane (xor 1, xor 2 inside a quad; mirror inside 8; mirror inside
// 16; xor 16).  a + b == b + a exactly, so every lane of the group gets the
// bit-identical total.
template <int G>
__device__ __forceinline__ float group_sum(float x)
{
    if constexpr (G >= 2) x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
    if constexpr (G >= 4) x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
    if constexpr (G >= 8) x += dpp<0x141>(x);  // row_half_mirror
    if constexpr (G >= 16) x += dpp<0x140>(x); // row_mirror
    if constexpr (G >= 32) x += __shfl_xor(x, 16);
    return x;
}

template <typename T, int D, int G>
__device__ __forceinline__ float row_score(const uint4 (&q)[Row<T, D, G>::kCh], const uint4 (&k)[Row<T, D, G>::kCh])
{
    return group_sum<G>(lane_dot<T, Row<T, D, G>::kCh>(q, k));
}

// Higher score wins; equal scores go to the lower flat key index.
__device__ __forceinline__ bool better(float s, int32_t i, float bs, int32_t bi)
{
    return s > bs || (s == bs && i < bi);
}

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

// Lanes per query: a row is split so that each lane holds kLaneBytes of it
// (one lane per query when the row is shorter).  Fewer lanes per query means
// fewer per-query instructions replicated across the group; more lanes means
// fewer distinct cache lines per load instruction.
#ifndef SCRAM_PM_LANE_BYTES
#define SCRAM_PM_LANE_BYTES 32
#endif
#ifndef SCRAM_ATTEND_LANE_BYTES
#define SCRAM_ATTEND_LANE_BYTES 32
#endif

template <typename T, int D, int LANE_BYTES>
struct LanesFor {
    static constexpr int kBytes = D * static_cast<int>(sizeof(T));
    static constexpr int kG0 = kBytes > LANE_BYTES ? kBytes / LANE_BYTES : 1;
    static constexpr int kG = kG0 > 32 ? 32 : kG0;
};

template <typename T, int D>
struct Lanes {
    static constexpr int kPm = LanesFor<T, D, SCRAM_PM_LANE_BYTES>::kG;
    static constexpr int kAttend = LanesFor<T, D, SCRAM_ATTEND_LANE_BYTES>::kG;
};

// ---------------------------------------------------------------------------
// kernel parameters
// ---------------------------------------------------------------------------
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
};

struct AttParams {
    const void* Q;
    const void* K;
    const void* V;
    const int32_t* J;
    void* out;
    uint32_t n;
    int Hk, Wk;
    uint32_t nkeys;
    Div div_plane, div_wk;
    int b;                // window half-width
    float scale_log2e;    // scale * log2(e): scores live in the base-2 domain
    int kappa;            // maps in J ([kappa, n]): the union of their windows
    int causal;           // drop keys after the query (raster order)
};

constexpr int kMaxPrev = 7;   // previous runs a PatchMatch run may be constrained by
constexpr int kMaxKappa = 8;  // maps whose windows attend may unite

// is_index_valid for one query: not after the query when causal, and at
// Chebyshev distance >= sep from each previous run's match.
struct Validity {
    int n, sep;
    bool causal;
    uint32_t local;  // the query's raster index in its slice
    uint32_t pu[kMaxPrev], pv[kMaxPrev];

    __device__ bool ok(uint32_t r, uint32_t c, int32_t idx) const
    {
        bool v = !(causal && static_cast<uint32_t>(idx) > local);
#pragma unroll
        for (int i = 0; i < kMaxPrev; ++i) {
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
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void pm_init_kernel(PmParams p)
{
    using RW = Row<T, D, G>;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t g = blockIdx.x * RW::kQpb + threadIdx.x / G;
    if (g >= p.n) return;  // whole lane groups leave together
    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);

    int32_t idx;
    if (p.init) {
        idx = clamp_index(p.init[g], p.nkeys);
    } else {
        const uint4 w = philox4x32_10(g, 0u, 0u, static_cast<uint32_t>(p.n_prev), p.key0, p.key1);
        if (p.causal) {  // uniform over the keys up to the query's raster index
            idx = static_cast<int32_t>(__umulhi(w.x, rem + 1u));
        } else {
            const uint32_t u = __umulhi(w.x, static_cast<uint32_t>(p.Hk));
            const uint32_t v = __umulhi(w.y, static_cast<uint32_t>(p.Wk));
            idx = static_cast<int32_t>(u * p.Wk + v);
        }
    }
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
template <typename T, int D, int G, int QPG, int kNb, bool PROP, bool RS, bool VALID>
__global__ __launch_bounds__(kBlock) void pm_iter_kernel(PmParams p)
{
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
        const uint32_t gr = blk * kQpb + j * kGroups + qslot;
        live[j] = gr < p.n;
        // groups past the end work on the last query and write nothing, so
        // every lane reaches the block barrier below
        g[j] = live[j] ? gr : p.n - 1;
        uint32_t rem;
        divmod(g[j], p.div_plane, s[j], rem);
        divmod(rem, p.div_wq, x[j], y[j]);
        Ks[j] = static_cast<const T*>(p.K) + static_cast<size_t>(s[j]) * p.nkeys * D;
        load_row<T, D, G>(static_cast<const T*>(p.Q), g[j], lane, q[j]);
        cur[j] = clamp_index(p.Jp[g[j]], p.nkeys);
        cur0[j] = cur[j];
        best[j] = p.sp[g[j]];
    }
    // validity variant: the previous runs' matches of each query; an invalid
    // incumbent counts as minus infinity
    Validity val[QPG];
    if constexpr (VALID) {
#pragma unroll
        for (int j = 0; j < QPG; ++j) {
            val[j].n = p.n_prev;
            val[j].sep = p.sep;
            val[j].causal = p.causal != 0;
            val[j].local = x[j] * p.Wq + y[j];
#pragma unroll
            for (int i = 0; i < kMaxPrev; ++i) {
                val[j].pu[i] = val[j].pv[i] = 0u;
                if (i < p.n_prev)
                    divmod(static_cast<uint32_t>(clamp_index(p.prev[static_cast<size_t>(i) * p.n + g[j]], p.nkeys)),
                           p.div_wk, val[j].pu[i], val[j].pv[i]);
            }
            uint32_t u0, v0;
            divmod(static_cast<uint32_t>(cur[j]), p.div_wk, u0, v0);
            if (!val[j].ok(u0, v0, cur[j])) best[j] = -INFINITY;
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
                    const uint32_t nb = clamp_index(Jp[(static_cast<size_t>(s[j]) * p.Hq + nx) * p.Wq + ny], p.nkeys);
                    uint32_t nu, nv;
                    divmod(nb, p.div_wk, nu, nv);
                    const int r = static_cast<int>(nu) - ox, cc = static_cast<int>(nv) - oy;
                    if (r >= 0 && r < p.Hk && cc >= 0 && cc < p.Wk) {
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
            p.Jn[g[j]] = cur[j];
            p.sn[g[j]] = best[j];
        }
    }
}

// ---------------------------------------------------------------------------
// K4: window softmax + value gather
// ---------------------------------------------------------------------------

// acc[e] += pj * v[e] over the lane's channels of one value row.
template <typename T, int CH>
__device__ __forceinline__ void accumulate_row(float* acc, float pj, const uint4 (&vr)[CH])
{
#pragma unroll
    for (int cc = 0; cc < CH; ++cc) {
        const uint32_t w[4] = {vr[cc].x, vr[cc].y, vr[cc].z, vr[cc].w};
        if constexpr (std::is_same<T, uint16_t>::value) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                acc[cc * 8 + 2 * i] = fmaf(pj, __uint_as_float(w[i] << 16), acc[cc * 8 + 2 * i]);
                acc[cc * 8 + 2 * i + 1] = fmaf(pj, __uint_as_float(w[i] & 0xFFFF0000u), acc[cc * 8 + 2 * i + 1]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[cc * 4 + i] = fmaf(pj, __uint_as_float(w[i]), acc[cc * 4 + i]);
        }
    }
}

// The lane's channels of one value row as floats (the channel order of
// accumulate_row).
template <typename T, int CH>
__device__ __forceinline__ void unpack_row(const uint4 (&vr)[CH], float* out)
{
#pragma unroll
    for (int cc = 0; cc < CH; ++cc) {
        const uint32_t w[4] = {vr[cc].x, vr[cc].y, vr[cc].z, vr[cc].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (std::is_same<T, uint16_t>::value) {
                out[cc * 8 + 2 * i] = __uint_as_float(w[i] << 16);
                out[cc * 8 + 2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
            } else {
                out[cc * 4 + i] = __uint_as_float(w[i]);
            }
        }
    }
}

// out row slice = acc * inv in the storage type.
template <typename T, int D, int G>
__device__ __forceinline__ void store_row(void* out, uint32_t g, int lane, const float* acc, float inv)
{
    constexpr int CH = Row<T, D, G>::kCh;
    uint4* o = reinterpret_cast<uint4*>(static_cast<T*>(out) + static_cast<size_t>(g) * D) + lane;
#pragma unroll
    for (int cc = 0; cc < CH; ++cc) {
        if constexpr (std::is_same<T, uint16_t>::value) {
            uint32_t w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                w[i] = f32_to_bf16_rne(acc[cc * 8 + 2 * i] * inv) |
                       (f32_to_bf16_rne(acc[cc * 8 + 2 * i + 1] * inv) << 16);
            o[cc * G] = make_uint4(w[0], w[1], w[2], w[3]);
        } else {
            o[cc * G] = make_uint4(__float_as_uint(acc[cc * 4] * inv), __float_as_uint(acc[cc * 4 + 1] * inv),
                                   __float_as_uint(acc[cc * 4 + 2] * inv), __float_as_uint(acc[cc * 4 + 3] * inv));
        }
    }
}

// Several windows and/or the causal mask: the centres of all kappa windows
// and the query's raster index.  skip(e, r, c): key (r, c) of window e is
// left out because an earlier window already holds it or it comes after the
// query.
struct WindowSet {
    int kappa, b;
    bool causal;
    uint32_t local, Wk;
    int cu[kMaxKappa], cv[kMaxKappa];

    __device__ bool skip(int e, int r, int c) const
    {
        bool s = causal && static_cast<uint32_t>(r) * Wk + static_cast<uint32_t>(c) > local;
#pragma unroll
        for (int f = 0; f < kMaxKappa; ++f)
            if (f < e) s = s || (abs(r - cu[f]) <= b && abs(c - cv[f]) <= b);
        return s;
    }
};

template <typename P>
__device__ __forceinline__ WindowSet make_window_set(const P& p, uint32_t g, uint32_t rem)
{
    WindowSet ws;
    ws.kappa = p.kappa;
    ws.b = p.b;
    ws.causal = p.causal != 0;
    ws.local = rem;
    ws.Wk = static_cast<uint32_t>(p.Wk);
#pragma unroll
    for (int e = 0; e < kMaxKappa; ++e) {
        uint32_t u = 0, v = 0;
        if (e < p.kappa)
            divmod(static_cast<uint32_t>(clamp_index(p.J[static_cast<size_t>(e) * p.n + g], p.nkeys)), p.div_wk, u, v);
        ws.cu[e] = static_cast<int>(u);
        ws.cv[e] = static_cast<int>(v);
    }
    return ws;
}

// Fixed window side W (odd), one window row per step: the W key rows and W
// value rows of a window row are gathered together (2W loads in flight),
// then the W scores (base-2 domain), one online-softmax rescale, and the
// value accumulation.  Keys outside the grid read a clamped (valid) row and
// get weight 0; window rows entirely outside the grid are skipped.
template <typename T, int D, int G, int W, bool MULTI>
__global__ __launch_bounds__(kBlock) void attend_window_kernel(AttParams p)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;  // channels per lane
    constexpr int B = W / 2;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    const uint32_t g = blk * RW::kQpb + threadIdx.x / G;
    if (g >= p.n) return;

    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);
    const size_t slice = static_cast<size_t>(s) * p.nkeys * D;
    const T* Ks = static_cast<const T*>(p.K) + slice;
    const T* Vs = static_cast<const T*>(p.V) + slice;
    uint4 q[CH];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    WindowSet wset;
    if constexpr (MULTI) wset = make_window_set(p, g, rem);
    const int nwin = MULTI ? p.kappa : 1;

    float m = -INFINITY, l = 0.f;
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;

    for (int e = 0; e < nwin; ++e) {
        uint32_t u, v;
        if constexpr (MULTI) {
            u = static_cast<uint32_t>(wset.cu[0]);
            v = static_cast<uint32_t>(wset.cv[0]);
#pragma unroll
            for (int f = 1; f < kMaxKappa; ++f)
                if (f == e) {
                    u = static_cast<uint32_t>(wset.cu[f]);
                    v = static_cast<uint32_t>(wset.cv[f]);
                }
        } else {
            divmod(static_cast<uint32_t>(clamp_index(p.J[g], p.nkeys)), p.div_wk, u, v);
        }
        // column of each window column, clamped, and whether it is inside
        int cols[W];
        bool col_ok[W];
#pragma unroll
        for (int c = 0; c < W; ++c) {
            const int col = static_cast<int>(v) + c - B;
            col_ok[c] = col >= 0 && col < p.Wk;
            cols[c] = min(max(col, 0), p.Wk - 1);
        }
        for (int a = 0; a < W; ++a) {
            const int r = static_cast<int>(u) + a - B;
            if (r < 0 || r >= p.Hk) continue;
            const uint32_t row0 = static_cast<uint32_t>(r * p.Wk);
            uint4 kr[W][CH], vr[W][CH];
#pragma unroll
            for (int c = 0; c < W; ++c) {
                load_row<T, D, G>(Ks, row0 + cols[c], lane, kr[c]);
                load_row<T, D, G>(Vs, row0 + cols[c], lane, vr[c]);
            }
            float sc[W];
            float mb = m;
#pragma unroll
            for (int c = 0; c < W; ++c) {
                bool use = col_ok[c];
                if constexpr (MULTI) use = use && !wset.skip(e, r, cols[c]);
                sc[c] = use ? row_score<T, D, G>(q, kr[c]) * p.scale_log2e : -INFINITY;
                mb = fmaxf(mb, sc[c]);
            }
            if (mb == -INFINITY) continue;  // nothing of this row is in the set
            const float alpha = __builtin_amdgcn_exp2f(m - mb);  // 0 on the first row
            l *= alpha;
#pragma unroll
            for (int i = 0; i < E; ++i) acc[i] *= alpha;
#pragma unroll
            for (int c = 0; c < W; ++c) {
                const float pj = __builtin_amdgcn_exp2f(sc[c] - mb);  // exp2(-inf) = 0
                l += pj;
                accumulate_row<T, CH>(acc, pj, vr[c]);
            }
            m = mb;
        }
    }
    store_row<T, D, G>(p.out, g, lane, acc, l > 0.f ? 1.f / l : 0.f);  // an empty set gives a zero row
}

// Any window side: the clipped window is visited in row order, kNb keys at a
// time with their key and value loads in flight together; an online softmax
// keeps (running max m, running sum l, accumulator) in the base-2 domain.
template <typename T, int D, int G, bool MULTI>
__global__ __launch_bounds__(kBlock) void attend_kernel(AttParams p)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;
    constexpr int kNb = CH >= 2 ? 4 : 8;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    const uint32_t g = blk * RW::kQpb + threadIdx.x / G;
    if (g >= p.n) return;

    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);
    const size_t slice = static_cast<size_t>(s) * p.nkeys * D;
    const T* Ks = static_cast<const T*>(p.K) + slice;
    const T* Vs = static_cast<const T*>(p.V) + slice;
    uint4 q[CH];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    WindowSet wset;
    if constexpr (MULTI) wset = make_window_set(p, g, rem);
    const int nsets = MULTI ? p.kappa : 1;

    float m = -INFINITY, l = 0.f;
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;

    for (int e = 0; e < nsets; ++e) {
        uint32_t u, v;
        if constexpr (MULTI) {
            u = static_cast<uint32_t>(wset.cu[0]);
            v = static_cast<uint32_t>(wset.cv[0]);
#pragma unroll
            for (int f = 1; f < kMaxKappa; ++f)
                if (f == e) {
                    u = static_cast<uint32_t>(wset.cu[f]);
                    v = static_cast<uint32_t>(wset.cv[f]);
                }
        } else {
            divmod(static_cast<uint32_t>(clamp_index(p.J[g], p.nkeys)), p.div_wk, u, v);
        }
        const int r0 = max(static_cast<int>(u) - p.b, 0), r1 = min(static_cast<int>(u) + p.b, p.Hk - 1);
        const int c0 = max(static_cast<int>(v) - p.b, 0), c1 = min(static_cast<int>(v) + p.b, p.Wk - 1);
        const int nwin = (r1 - r0 + 1) * (c1 - c0 + 1);
        const uint32_t centre = u * p.Wk + v;

        // (r, c) walks the clipped window in row order; slots past its end read
        // the centre row and get weight 0
        int r = r0, c = c0;
        for (int k0 = 0; k0 < nwin; k0 += kNb) {
            uint4 kr[kNb][CH], vr[kNb][CH];
            bool ok[kNb];
#pragma unroll
            for (int j = 0; j < kNb; ++j) {
                ok[j] = k0 + j < nwin;
                if constexpr (MULTI) ok[j] = ok[j] && !wset.skip(e, r, c);
                const uint32_t row = k0 + j < nwin ? static_cast<uint32_t>(r * p.Wk + c) : centre;
                load_row<T, D, G>(Ks, row, lane, kr[j]);
                load_row<T, D, G>(Vs, row, lane, vr[j]);
                if (k0 + j < nwin && ++c > c1) {
                    c = c0;
                    ++r;
                }
            }
            float sc[kNb];
            float mb = m;
#pragma unroll
            for (int j = 0; j < kNb; ++j) {
                sc[j] = ok[j] ? row_score<T, D, G>(q, kr[j]) * p.scale_log2e : -INFINITY;
                mb = fmaxf(mb, sc[j]);
            }
            if (mb == -INFINITY) continue;
            const float alpha = __builtin_amdgcn_exp2f(m - mb);
            l *= alpha;
#pragma unroll
            for (int i = 0; i < E; ++i) acc[i] *= alpha;
#pragma unroll
            for (int j = 0; j < kNb; ++j) {
                const float pj = __builtin_amdgcn_exp2f(sc[j] - mb);
                l += pj;
                accumulate_row<T, CH>(acc, pj, vr[j]);
            }
            m = mb;
        }
    }
    store_row<T, D, G>(p.out, g, lane, acc, l > 0.f ? 1.f / l : 0.f);  // an empty set gives a zero row
}

// ---------------------------------------------------------------------------
// K6: backward of the sparse attention, maps held fixed
//
// For query i with key set W_i (as in the forward), p_ij its softmax
// weights, dp_ij = dO_i . v_j and D_i = sum_j p_ij dp_ij:
//   dQ_i = scale sum_j p_ij (dp_ij - D_i) k_j
//   dK_j = scale sum_i p_ij (dp_ij - D_i) q_i,   dV_j = sum_i p_ij dO_i
// Query side (one lane group per query): pass A walks W_i for the running
// max, the normaliser and D_i and stores log2 of the normaliser (with the
// max) and D_i; pass B walks it again for dQ_i.  Key side (one lane group
// per key): key j lies in W_i exactly when a match of i lies in the
// (2b+1)^2 neighbourhood of j, so the queries are found through the inverse
// map -- the (query, match) entries sorted by match key (a counting sort).
// The keys of one neighbourhood row are consecutive, so their entries form
// one contiguous range.  No float atomics: every gradient row has one
// writer.
// ---------------------------------------------------------------------------
constexpr int kScanItems = 8;                          // counts per thread in the scan
constexpr int kScanTile = kBlock * kScanItems;         // counts per scan block

struct BwdParams {
    const void* Q;
    const void* K;
    const void* V;
    const int32_t* J;      // [kappa, n]
    const void* dO;
    float* dQ;
    float* dK;
    float* dV;
    float* lse2;           // [n] max + log2(normaliser), base-2 scores
    float* Dq;             // [n] D_i
    const int32_t* offsets;  // [S * nkeys + 1] start of each key's entries
    const int32_t* entries;  // [kappa * n] e * n + i, grouped by match key
    uint32_t n;
    uint32_t keys_total;   // S * nkeys
    int Hq, Wq, Hk, Wk;
    uint32_t nkeys;
    Div div_plane, div_wk, div_n, div_keys;
    int b;
    float scale;
    float scale_log2e;
    int kappa;
    int causal;
};

__global__ __launch_bounds__(kBlock) void zero_i32_kernel(int32_t* a, size_t count)
{
    for (size_t i = static_cast<size_t>(blockIdx.x) * kBlock + threadIdx.x; i < count;
         i += static_cast<size_t>(gridDim.x) * kBlock)
        a[i] = 0;
}

// counts[s * nkeys + J[e][i]] += 1 for every (query, match)
__global__ __launch_bounds__(kBlock) void bwd_count_kernel(BwdParams p, int32_t* counts)
{
    const size_t total = static_cast<size_t>(p.kappa) * p.n;
    for (size_t x = static_cast<size_t>(blockIdx.x) * kBlock + threadIdx.x; x < total;
         x += static_cast<size_t>(gridDim.x) * kBlock) {
        const uint32_t g = static_cast<uint32_t>(x % p.n);
        const uint32_t s = g / (static_cast<uint32_t>(p.Hq) * p.Wq);
        atomicAdd(counts + static_cast<size_t>(s) * p.nkeys + clamp_index(p.J[x], p.nkeys), 1);
    }
}

// Exclusive scan, step 1: each block scans a tile of kScanTile counts into
// out (tile-local prefixes) and writes the tile's total to sums[tile].
__global__ __launch_bounds__(kBlock) void scan_tiles_kernel(const int32_t* in, int32_t* out, int32_t* sums, size_t count)
{
    __shared__ int32_t wave_tot[kBlock / 64];
    const size_t base = static_cast<size_t>(blockIdx.x) * kScanTile + static_cast<size_t>(threadIdx.x) * kScanItems;
    int32_t v[kScanItems];
    int32_t run = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        v[i] = base + i < count ? in[base + i] : 0;
        const int32_t x = v[i];
        v[i] = run;  // exclusive within the thread
        run += x;
    }
    // exclusive prefix of the thread totals: within the wave, then across waves
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int32_t incl = run;
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) {
        const int32_t y = __shfl_up(incl, k, 64);
        if (lane >= k) incl += y;
    }
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int32_t before = incl - run;
    for (int w = 0; w < wave; ++w) before += wave_tot[w];
#pragma unroll
    for (int i = 0; i < kScanItems; ++i)
        if (base + i < count) out[base + i] = before + v[i];
    if (threadIdx.x == kBlock - 1) {
        int32_t tot = 0;
        for (int w = 0; w < kBlock / 64; ++w) tot += wave_tot[w];
        sums[blockIdx.x] = tot;
    }
}

// Exclusive scan, step 2 (one block): sums[0..tiles) in place, total in sums[tiles].
__global__ __launch_bounds__(kBlock) void scan_sums_kernel(int32_t* sums, uint32_t tiles)
{
    __shared__ int32_t wave_tot[kBlock / 64];
    __shared__ int32_t carry_s;
    if (threadIdx.x == 0) carry_s = 0;
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (uint32_t c0 = 0; c0 < tiles; c0 += kBlock) {
        const uint32_t i = c0 + threadIdx.x;
        const int32_t x = i < tiles ? sums[i] : 0;
        int32_t incl = x;
#pragma unroll
        for (int k = 1; k < 64; k <<= 1) {
            const int32_t y = __shfl_up(incl, k, 64);
            if (lane >= k) incl += y;
        }
        if (lane == 63) wave_tot[wave] = incl;
        __syncthreads();
        int32_t before = carry_s + incl - x;
        for (int w = 0; w < wave; ++w) before += wave_tot[w];
        if (i < tiles) sums[i] = before;
        __syncthreads();  // every thread has read carry_s and wave_tot
        if (threadIdx.x == kBlock - 1) carry_s = before + x;
        __syncthreads();
    }
    if (threadIdx.x == 0) sums[tiles] = carry_s;
}

// Exclusive scan, step 3: add each tile's offset; out[count] = total.
__global__ __launch_bounds__(kBlock) void scan_add_kernel(int32_t* out, const int32_t* sums, size_t count,
                                                          uint32_t tiles)
{
    const size_t base = static_cast<size_t>(blockIdx.x) * kScanTile;
    const int32_t add = sums[blockIdx.x];
    for (int i = threadIdx.x; i < kScanTile; i += kBlock)
        if (base + i < count) out[base + i] += add;
    if (blockIdx.x == 0 && threadIdx.x == 0) out[count] = sums[tiles];
}

// entries[offsets[key] + (a slot of that key)] = e * n + i; counts end at 0
__global__ __launch_bounds__(kBlock) void bwd_fill_kernel(BwdParams p, int32_t* counts, int32_t* entries)
{
    const size_t total = static_cast<size_t>(p.kappa) * p.n;
    for (size_t x = static_cast<size_t>(blockIdx.x) * kBlock + threadIdx.x; x < total;
         x += static_cast<size_t>(gridDim.x) * kBlock) {
        const uint32_t g = static_cast<uint32_t>(x % p.n);
        const uint32_t s = g / (static_cast<uint32_t>(p.Hq) * p.Wq);
        const size_t key = static_cast<size_t>(s) * p.nkeys + clamp_index(p.J[x], p.nkeys);
        const int32_t slot = atomicSub(counts + key, 1) - 1;
        entries[p.offsets[key] + slot] = static_cast<int32_t>(x);
    }
}

template <typename T, int D, int G, bool MULTI>
__global__ __launch_bounds__(kBlock) void bwd_query_kernel(BwdParams p)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;
    constexpr int kEpc = RW::kEpc;
    constexpr int kNb = CH >= 2 ? 4 : 8;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    const uint32_t g = blk * RW::kQpb + threadIdx.x / G;
    if (g >= p.n) return;

    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);
    const size_t slice = static_cast<size_t>(s) * p.nkeys * D;
    const T* Ks = static_cast<const T*>(p.K) + slice;
    const T* Vs = static_cast<const T*>(p.V) + slice;
    uint4 q[CH], go[CH];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    load_row<T, D, G>(static_cast<const T*>(p.dO), g, lane, go);
    WindowSet wset;
    if constexpr (MULTI) wset = make_window_set(p, g, rem);
    const int nsets = MULTI ? p.kappa : 1;

    // visit(fn): every key of the set, kNb at a time with their key and
    // value rows loaded together; fn(ok[], kr, vr) per batch
    auto visit = [&](auto&& fn) {
        for (int e = 0; e < nsets; ++e) {
            uint32_t u, v;
            if constexpr (MULTI) {
                u = static_cast<uint32_t>(wset.cu[0]);
                v = static_cast<uint32_t>(wset.cv[0]);
#pragma unroll
                for (int f = 1; f < kMaxKappa; ++f)
                    if (f == e) {
                        u = static_cast<uint32_t>(wset.cu[f]);
                        v = static_cast<uint32_t>(wset.cv[f]);
                    }
            } else {
                divmod(static_cast<uint32_t>(clamp_index(p.J[g], p.nkeys)), p.div_wk, u, v);
            }
            const int r0 = max(static_cast<int>(u) - p.b, 0), r1 = min(static_cast<int>(u) + p.b, p.Hk - 1);
            const int c0 = max(static_cast<int>(v) - p.b, 0), c1 = min(static_cast<int>(v) + p.b, p.Wk - 1);
            const int nwin = (r1 - r0 + 1) * (c1 - c0 + 1);
            const uint32_t centre = u * p.Wk + v;
            int r = r0, c = c0;
            for (int k0 = 0; k0 < nwin; k0 += kNb) {
                uint4 kr[kNb][CH], vr[kNb][CH];
                bool ok[kNb];
#pragma unroll
                for (int j = 0; j < kNb; ++j) {
                    ok[j] = k0 + j < nwin;
                    if constexpr (MULTI) ok[j] = ok[j] && !wset.skip(e, r, c);
                    const uint32_t row = k0 + j < nwin ? static_cast<uint32_t>(r * p.Wk + c) : centre;
                    load_row<T, D, G>(Ks, row, lane, kr[j]);
                    load_row<T, D, G>(Vs, row, lane, vr[j]);
                    if (k0 + j < nwin && ++c > c1) {
                        c = c0;
                        ++r;
                    }
                }
                fn(ok, kr, vr);
            }
        }
    };

    // pass A: running max m, normaliser l, sum of e^(a - m) dp (base-2 scores)
    float m = -INFINITY, l = 0.f, dn = 0.f;
    visit([&](const bool (&ok)[kNb], const uint4 (&kr)[kNb][CH], const uint4 (&vr)[kNb][CH]) {
        float sc[kNb], dp[kNb];
        float mb = m;
#pragma unroll
        for (int j = 0; j < kNb; ++j) {
            sc[j] = ok[j] ? row_score<T, D, G>(q, kr[j]) * p.scale_log2e : -INFINITY;
            dp[j] = row_score<T, D, G>(go, vr[j]);
            mb = fmaxf(mb, sc[j]);
        }
        if (mb == -INFINITY) return;
        const float alpha = __builtin_amdgcn_exp2f(m - mb);
        l *= alpha;
        dn *= alpha;
#pragma unroll
        for (int j = 0; j < kNb; ++j) {
            const float pj = __builtin_amdgcn_exp2f(sc[j] - mb);
            l += pj;
            dn = fmaf(pj, dp[j], dn);
        }
        m = mb;
    });
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const float Dg = dn * inv;
    if (lane == 0) {
        p.lse2[g] = l > 0.f ? m + log2f(l) : INFINITY;  // +inf: every weight is 0
        p.Dq[g] = Dg;
    }

    // pass B: dQ with the exact weights
    float dq[E];
#pragma unroll
    for (int e = 0; e < E; ++e) dq[e] = 0.f;
    if (l > 0.f) {
        visit([&](const bool (&ok)[kNb], const uint4 (&kr)[kNb][CH], const uint4 (&vr)[kNb][CH]) {
#pragma unroll
            for (int j = 0; j < kNb; ++j) {
                const float sc = ok[j] ? row_score<T, D, G>(q, kr[j]) * p.scale_log2e : -INFINITY;
                const float dp = row_score<T, D, G>(go, vr[j]);
                const float ds = __builtin_amdgcn_exp2f(sc - m) * inv * (dp - Dg);  // 0 when !ok
                float kf[E];
                unpack_row<T, CH>(kr[j], kf);
#pragma unroll
                for (int e = 0; e < E; ++e) dq[e] = fmaf(ds, kf[e], dq[e]);
            }
        });
    }
#pragma unroll
    for (int cc = 0; cc < CH; ++cc) {
        float4* o = reinterpret_cast<float4*>(p.dQ + static_cast<size_t>(g) * D + (cc * G + lane) * kEpc);
#pragma unroll
        for (int i = 0; i < kEpc / 4; ++i)
            o[i] = make_float4(dq[cc * kEpc + 4 * i] * p.scale, dq[cc * kEpc + 4 * i + 1] * p.scale,
                               dq[cc * kEpc + 4 * i + 2] * p.scale, dq[cc * kEpc + 4 * i + 3] * p.scale);
    }
}

// One lane group per key j of slice s: sum over the entries (i, e) whose
// match e lies in the neighbourhood of j (so j is in window e of i), each
// query once (its first such window), causal pairs only.
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void bwd_key_kernel(BwdParams p)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;
    constexpr int kEpc = RW::kEpc;
    constexpr int kNb = CH >= 2 ? 4 : 8;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    const uint32_t kg = blk * RW::kQpb + threadIdx.x / G;  // global key id s * nkeys + j
    if (kg >= p.keys_total) return;
    uint32_t s, j;
    divmod(kg, p.div_keys, s, j);
    uint32_t ju, jv;
    divmod(j, p.div_wk, ju, jv);
    const size_t krow = static_cast<size_t>(s) * p.nkeys + j;
    uint4 kj[CH], vj[CH];
    load_row<T, D, G>(static_cast<const T*>(p.K), static_cast<uint32_t>(krow), lane, kj);
    load_row<T, D, G>(static_cast<const T*>(p.V), static_cast<uint32_t>(krow), lane, vj);

    float dk[E], dv[E];
#pragma unroll
    for (int e = 0; e < E; ++e) dk[e] = dv[e] = 0.f;
    const int r0 = max(static_cast<int>(ju) - p.b, 0), r1 = min(static_cast<int>(ju) + p.b, p.Hk - 1);
    const int c0 = max(static_cast<int>(jv) - p.b, 0), c1 = min(static_cast<int>(jv) + p.b, p.Wk - 1);
    const size_t sbase = static_cast<size_t>(s) * p.nkeys;
    for (int r = r0; r <= r1; ++r) {
        const int lo = p.offsets[sbase + static_cast<size_t>(r) * p.Wk + c0];
        const int hi = p.offsets[sbase + static_cast<size_t>(r) * p.Wk + c1 + 1];
        for (int x0 = lo; x0 < hi; x0 += kNb) {
            uint4 qr[kNb][CH], gr[kNb][CH];
            bool ok[kNb];
            uint32_t gq[kNb];
#pragma unroll
            for (int t = 0; t < kNb; ++t) {
                const int x = x0 + t;
                uint32_t e = 0, g = 0;
                ok[t] = x < hi;
                if (ok[t]) divmod(static_cast<uint32_t>(p.entries[x]), p.div_n, e, g);
                // the pair counts once: through the query's first window holding j
                for (int f = 0; f < static_cast<int>(e) && ok[t]; ++f) {
                    uint32_t fu, fv;
                    divmod(static_cast<uint32_t>(clamp_index(p.J[static_cast<size_t>(f) * p.n + g], p.nkeys)),
                           p.div_wk, fu, fv);
                    if (abs(static_cast<int>(fu) - static_cast<int>(ju)) <= p.b &&
                        abs(static_cast<int>(fv) - static_cast<int>(jv)) <= p.b)
                        ok[t] = false;
                }
                if (ok[t] && p.causal) {
                    uint32_t gs, grem;
                    divmod(g, p.div_plane, gs, grem);
                    ok[t] = j <= grem;
                }
                gq[t] = g;
                load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, qr[t]);
                load_row<T, D, G>(static_cast<const T*>(p.dO), g, lane, gr[t]);
            }
#pragma unroll
            for (int t = 0; t < kNb; ++t) {
                const float sc = row_score<T, D, G>(qr[t], kj) * p.scale_log2e;
                const float dp = row_score<T, D, G>(gr[t], vj);
                const float pj = ok[t] ? __builtin_amdgcn_exp2f(sc - p.lse2[gq[t]]) : 0.f;
                const float ds = pj * (dp - p.Dq[gq[t]]);
                float qf[E], gf[E];
                unpack_row<T, CH>(qr[t], qf);
                unpack_row<T, CH>(gr[t], gf);
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    dk[e] = fmaf(ds, qf[e], dk[e]);
                    dv[e] = fmaf(pj, gf[e], dv[e]);
                }
            }
        }
    }
#pragma unroll
    for (int cc = 0; cc < CH; ++cc) {
        float4* ok_ = reinterpret_cast<float4*>(p.dK + krow * D + (cc * G + lane) * kEpc);
        float4* ov = reinterpret_cast<float4*>(p.dV + krow * D + (cc * G + lane) * kEpc);
#pragma unroll
        for (int i = 0; i < kEpc / 4; ++i) {
            const int e0 = cc * kEpc + 4 * i;
            ok_[i] = make_float4(dk[e0] * p.scale, dk[e0 + 1] * p.scale, dk[e0 + 2] * p.scale, dk[e0 + 3] * p.scale);
            ov[i] = make_float4(dv[e0], dv[e0 + 1], dv[e0 + 2], dv[e0 + 3]);
        }
    }
}

// ---------------------------------------------------------------------------
// K5: self-normalised importance sampling (Section 4.2, Equations 11-17)
//
// Importance distribution of query i: with probability alpha a mode m of
// the kappa PatchMatch matches (uniformly) plus a centred binomial offset per
// axis (popcount of 2m Philox bits, minus m: a discrete Gaussian of variance
// m/2), clamped to the grid; otherwise a uniform key.  Sample t of query g
// uses the Philox block of counter (g, t, 0, kSnisStream).  Each sample is
// weighted by exp(a_ij) / r_i(j); the estimate is the weighted mean of the
// values, with the effective sample size and (optionally) the delta-method
// variance per channel.  Weights are kept in the base-2 domain relative to
// the running maximum, which leaves every ratio unchanged.
// ---------------------------------------------------------------------------
constexpr uint32_t kSnisStream = 0x534E4953u;
constexpr int kMaxRadius = 16;

struct SnisParams {
    const void* Q;
    const void* K;
    const void* V;
    const int32_t* modes;  // [kappa, n]
    void* out;
    float* ess;            // nullable [n]
    float* var;            // [n, D] (variance variant only)
    uint32_t n;
    int Hk, Wk;
    uint32_t nkeys;
    Div div_plane, div_wk;
    int kappa;
    int samples;
    int m;                 // binomial offsets use 2m bits per axis
    uint32_t alpha16;      // a mode is used iff the upper half of word 0 is below this
    float w_local;         // alpha / kappa
    float w_unif;          // (1 - alpha) / (Hk * Wk)
    float scale_log2e;
    uint32_t key0, key1;
    int causal;
};

// Probability that the clamped coordinate centre + offset lands on r, read
// from the offset's pmf and cdf tables (index offset + m).
__device__ __forceinline__ float axis_density(int r, int centre, int len, int m, const float* pmf, const float* cdf)
{
    if (len == 1) return 1.f;
    int x;  // the clamped edges hold the tail P(offset <= x)
    if (r == 0) {
        x = -centre;
    } else if (r == len - 1) {
        x = centre - (len - 1);
    } else {
        const int delta = r - centre;
        return (delta >= -m && delta <= m) ? pmf[delta + m] : 0.f;
    }
    return x < -m ? 0.f : (x >= m ? 1.f : cdf[x + m]);
}

// Sample t of query g: flat key index and log2 of its importance density.
__device__ __forceinline__ void snis_draw(const SnisParams& p, uint32_t g, uint32_t t, const int (&cu)[kMaxKappa],
                                          const int (&cv)[kMaxKappa], const float* pmf, const float* cdf,
                                          int32_t& j, float& lr2)
{
    const uint4 w = philox4x32_10(g, t, 0u, kSnisStream, p.key0, p.key1);
    int r, c;
    if ((w.x >> 16) < p.alpha16) {
        const uint32_t e = __umulhi(w.y, static_cast<uint32_t>(p.kappa));
        int u = cu[0], v = cv[0];
#pragma unroll
        for (int f = 1; f < kMaxKappa; ++f)
            if (static_cast<uint32_t>(f) == e) {
                u = cu[f];
                v = cv[f];
            }
        const uint32_t mask = p.m == kMaxRadius ? 0xFFFFFFFFu : ((1u << (2 * p.m)) - 1u);
        r = min(max(u + static_cast<int>(__popc(w.z & mask)) - p.m, 0), p.Hk - 1);
        c = min(max(v + static_cast<int>(__popc(w.w & mask)) - p.m, 0), p.Wk - 1);
    } else {
        r = static_cast<int>(__umulhi(w.z, static_cast<uint32_t>(p.Hk)));
        c = static_cast<int>(__umulhi(w.w, static_cast<uint32_t>(p.Wk)));
    }
    j = r * p.Wk + c;
    float local = 0.f;
#pragma unroll
    for (int e = 0; e < kMaxKappa; ++e)
        if (e < p.kappa)
            local += axis_density(r, cu[e], p.Hk, p.m, pmf, cdf) * axis_density(c, cv[e], p.Wk, p.m, pmf, cdf);
    lr2 = log2f(fmaf(p.w_local, local, p.w_unif));
}

template <typename T, int D, int G, bool VAR>
__global__ __launch_bounds__(kBlock) void snis_kernel(SnisParams p)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;
    constexpr int kNb = CH >= 2 ? 4 : 8;        // samples gathered per batch
    constexpr int kPer = (kNb + G - 1) / G;      // samples each lane draws per batch
    __shared__ float s_pmf[2 * kMaxRadius + 1], s_cdf[2 * kMaxRadius + 1];

    // offset tables from exact binomial coefficients C(2m, i) and their
    // prefix sums, scaled by 4^-m
    if (static_cast<int>(threadIdx.x) <= 2 * p.m) {
        const int i = threadIdx.x, n2 = 2 * p.m;
        uint64_t c = 1, acc = 1;
        for (int k = 1; k <= i; ++k) {
            c = c * static_cast<uint64_t>(n2 - k + 1) / static_cast<uint64_t>(k);
            acc += c;
        }
        s_pmf[i] = ldexpf(static_cast<float>(c), -n2);
        s_cdf[i] = ldexpf(static_cast<float>(acc), -n2);
    }
    __syncthreads();

    const int lane = threadIdx.x & (G - 1);
    const int gbase = (threadIdx.x & 63) - lane;
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    const uint32_t g = blk * RW::kQpb + threadIdx.x / G;
    if (g >= p.n) return;  // whole lane groups leave together

    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);
    const size_t slice = static_cast<size_t>(s) * p.nkeys * D;
    const T* Ks = static_cast<const T*>(p.K) + slice;
    const T* Vs = static_cast<const T*>(p.V) + slice;
    uint4 q[CH];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    int cu[kMaxKappa], cv[kMaxKappa];
#pragma unroll
    for (int e = 0; e < kMaxKappa; ++e) {
        uint32_t u = 0, v = 0;
        if (e < p.kappa)
            divmod(static_cast<uint32_t>(clamp_index(p.modes[static_cast<size_t>(e) * p.n + g], p.nkeys)), p.div_wk,
                   u, v);
        cu[e] = static_cast<int>(u);
        cv[e] = static_cast<int>(v);
    }

    // one batch: draws spread over the group's lanes, then every lane
    // gathers the batch's key and value rows and forms the base-2 log weights
    auto batch = [&](int t0, uint4 (&kr)[kNb][CH], uint4 (&vr)[kNb][CH], float (&lw)[kNb]) {
        int32_t mj[kPer];
        float ml[kPer];
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int sl = lane + i * G;
            mj[i] = 0;
            ml[i] = 0.f;
            if (sl < kNb && t0 + sl < p.samples) snis_draw(p, g, t0 + sl, cu, cv, s_pmf, s_cdf, mj[i], ml[i]);
        }
        int32_t j[kNb];
        float lr[kNb];
#pragma unroll
        for (int sl = 0; sl < kNb; ++sl) {
            j[sl] = __shfl(mj[sl / G], gbase + sl % G);
            lr[sl] = __shfl(ml[sl / G], gbase + sl % G);
            load_row<T, D, G>(Ks, j[sl], lane, kr[sl]);
            load_row<T, D, G>(Vs, j[sl], lane, vr[sl]);
        }
#pragma unroll
        for (int sl = 0; sl < kNb; ++sl) {
            const bool ok = t0 + sl < p.samples && !(p.causal && static_cast<uint32_t>(j[sl]) > rem);
            lw[sl] = ok ? row_score<T, D, G>(q, kr[sl]) * p.scale_log2e - lr[sl] : -INFINITY;
        }
    };

    float M = -INFINITY, S1 = 0.f, S2 = 0.f;
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;
    for (int t0 = 0; t0 < p.samples; t0 += kNb) {
        uint4 kr[kNb][CH], vr[kNb][CH];
        float lw[kNb];
        batch(t0, kr, vr, lw);
        float mb = M;
#pragma unroll
        for (int sl = 0; sl < kNb; ++sl) mb = fmaxf(mb, lw[sl]);
        if (mb == -INFINITY) continue;  // nothing usable yet
        const float alpha = __builtin_amdgcn_exp2f(M - mb);  // 0 on the first batch
        S1 *= alpha;
        S2 *= alpha * alpha;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] *= alpha;
#pragma unroll
        for (int sl = 0; sl < kNb; ++sl) {
            const float pj = __builtin_amdgcn_exp2f(lw[sl] - mb);  // exp2(-inf) = 0
            S1 += pj;
            S2 += pj * pj;
            accumulate_row<T, CH>(acc, pj, vr[sl]);
        }
        M = mb;
    }
    const float inv = S1 > 0.f ? 1.f / S1 : 0.f;  // no usable sample: zero row

    if constexpr (VAR) {
        // second pass over the same samples: sum_t (w_t / sum w)^2 (v_t - estimate)^2
        float mean[E], vacc[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            mean[e] = acc[e] * inv;
            vacc[e] = 0.f;
        }
        if (S1 > 0.f) {
            for (int t0 = 0; t0 < p.samples; t0 += kNb) {
                uint4 kr[kNb][CH], vr[kNb][CH];
                float lw[kNb];
                batch(t0, kr, vr, lw);
#pragma unroll
                for (int sl = 0; sl < kNb; ++sl) {
                    const float wn = __builtin_amdgcn_exp2f(lw[sl] - M) * inv;
                    const float wn2 = wn * wn;
                    float vals[E];
                    unpack_row<T, CH>(vr[sl], vals);
#pragma unroll
                    for (int e = 0; e < E; ++e) {
                        const float dlt = vals[e] - mean[e];
                        vacc[e] = fmaf(wn2 * dlt, dlt, vacc[e]);
                    }
                }
            }
        }
        constexpr int kEpc = RW::kEpc;
#pragma unroll
        for (int cc = 0; cc < CH; ++cc) {
            float4* o = reinterpret_cast<float4*>(p.var + static_cast<size_t>(g) * D + (cc * G + lane) * kEpc);
#pragma unroll
            for (int i = 0; i < kEpc / 4; ++i)
                o[i] = make_float4(vacc[cc * kEpc + 4 * i], vacc[cc * kEpc + 4 * i + 1], vacc[cc * kEpc + 4 * i + 2],
                                   vacc[cc * kEpc + 4 * i + 3]);
        }
    }
    store_row<T, D, G>(p.out, g, lane, acc, inv);
    if (lane == 0 && p.ess) p.ess[g] = S1 > 0.f ? S1 * S1 / S2 : 0.f;
}

// ---------------------------------------------------------------------------
// host-side launch helpers
// ---------------------------------------------------------------------------
// Launch with the dispatch stamping optional start/stop events (the kernel's
// parameter types fix the argument types).
template <typename T>
struct NoDeduce {
    using type = T;
};

template <typename... A>
hipError_t launch(void (*kernel)(A...), uint32_t blocks, hipStream_t st, hipEvent_t start, hipEvent_t stop,
                  typename NoDeduce<A>::type... args)
{
    if (start || stop)
        hipExtLaunchKernelGGL(kernel, dim3(blocks), dim3(kBlock), 0, st, start, stop, 0, args...);
    else
        hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kBlock), 0, st, args...);
    return hipGetLastError();
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
    const uint32_t blocks = (p.n + Row<T, D, G>::kQpb - 1) / Row<T, D, G>::kQpb;
    return launch(pm_init_kernel<T, D, G>, blocks, st, e0, e1, p);
}

#ifndef SCRAM_PM_QPG
#define SCRAM_PM_QPG 1
#endif
#ifndef SCRAM_PM_BATCH
#define SCRAM_PM_BATCH 4
#endif

template <typename T, int D, bool VALID>
hipError_t run_iter_v(const PmParams& p, uint32_t flags, uint32_t blocks, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kPm;
    constexpr int QPG = SCRAM_PM_QPG;
    constexpr int NB = SCRAM_PM_BATCH;
    const bool prop = !(flags & SCRAM_PM_NO_PROPAGATION);
    const bool rs = !(flags & SCRAM_PM_NO_RANDOM_SEARCH);
    if (prop && rs) return launch(pm_iter_kernel<T, D, G, QPG, NB, true, true, VALID>, blocks, st, e0, e1, p);
    if (prop) return launch(pm_iter_kernel<T, D, G, QPG, NB, true, false, VALID>, blocks, st, e0, e1, p);
    if (rs) return launch(pm_iter_kernel<T, D, G, QPG, NB, false, true, VALID>, blocks, st, e0, e1, p);
    return launch(pm_iter_kernel<T, D, G, QPG, NB, false, false, VALID>, blocks, st, e0, e1, p);
}

template <typename T, int D>
hipError_t run_iter(const PmParams& p, uint32_t flags, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kPm;
    constexpr int kQpb = Row<T, D, G>::kQpb * SCRAM_PM_QPG;
    const uint32_t blocks = (p.n + kQpb - 1) / kQpb;
    if (p.n_prev > 0 || p.causal) return run_iter_v<T, D, true>(p, flags, blocks, st, e0, e1);
    return run_iter_v<T, D, false>(p, flags, blocks, st, e0, e1);
}

template <typename T, int D, bool MULTI>
hipError_t run_attend_m(const AttParams& p, int window, uint32_t blocks, hipStream_t st, hipEvent_t e0,
                        hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kAttend;
    switch (window) {
        case 1: return launch(attend_window_kernel<T, D, G, 1, MULTI>, blocks, st, e0, e1, p);
        case 3: return launch(attend_window_kernel<T, D, G, 3, MULTI>, blocks, st, e0, e1, p);
        case 5: return launch(attend_window_kernel<T, D, G, 5, MULTI>, blocks, st, e0, e1, p);
        case 7: return launch(attend_window_kernel<T, D, G, 7, MULTI>, blocks, st, e0, e1, p);
        default: return launch(attend_kernel<T, D, G, MULTI>, blocks, st, e0, e1, p);
    }
}

template <typename T, int D>
hipError_t run_attend(const AttParams& p, int window, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kAttend;
    const uint32_t blocks = (p.n + Row<T, D, G>::kQpb - 1) / Row<T, D, G>::kQpb;
    if (p.kappa > 1 || p.causal) return run_attend_m<T, D, true>(p, window, blocks, st, e0, e1);
    return run_attend_m<T, D, false>(p, window, blocks, st, e0, e1);
}

template <typename T, int D>
hipError_t run_backward(const BwdParams& p, hipStream_t st, hipEvent_t* ev)
{
    constexpr int G = Lanes<T, D>::kAttend;
    const uint32_t qblocks = (p.n + Row<T, D, G>::kQpb - 1) / Row<T, D, G>::kQpb;
    const uint32_t kblocks = (p.keys_total + Row<T, D, G>::kQpb - 1) / Row<T, D, G>::kQpb;
    hipEvent_t q0 = ev ? ev[2] : nullptr, q1 = ev ? ev[3] : nullptr, k0 = ev ? ev[4] : nullptr,
               k1 = ev ? ev[5] : nullptr;
    hipError_t e = (p.kappa > 1 || p.causal) ? launch(bwd_query_kernel<T, D, G, true>, qblocks, st, q0, q1, p)
                                             : launch(bwd_query_kernel<T, D, G, false>, qblocks, st, q0, q1, p);
    if (e != hipSuccess) return e;
    return launch(bwd_key_kernel<T, D, G>, kblocks, st, k0, k1, p);
}

template <typename T, int D>
hipError_t run_snis(const SnisParams& p, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kAttend;
    const uint32_t blocks = (p.n + Row<T, D, G>::kQpb - 1) / Row<T, D, G>::kQpb;
    if (p.var) return launch(snis_kernel<T, D, G, true>, blocks, st, e0, e1, p);
    return launch(snis_kernel<T, D, G, false>, blocks, st, e0, e1, p);
}

// (dtype, d) -> instantiation
template <typename F>
hipError_t dispatch(int dtype, int d, F&& f)
{
    if (dtype == SCRAM_F32) {
        switch (d) {
            case 16: return f(float{}, std::integral_constant<int, 16>{});
            case 32: return f(float{}, std::integral_constant<int, 32>{});
            case 64: return f(float{}, std::integral_constant<int, 64>{});
            case 128: return f(float{}, std::integral_constant<int, 128>{});
        }
    } else if (dtype == SCRAM_BF16) {
        switch (d) {
            case 16: return f(uint16_t{}, std::integral_constant<int, 16>{});
            case 32: return f(uint16_t{}, std::integral_constant<int, 32>{});
            case 64: return f(uint16_t{}, std::integral_constant<int, 64>{});
            case 128: return f(uint16_t{}, std::integral_constant<int, 128>{});
        }
    }
    return hipErrorInvalidValue;
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
                          int32_t* Jn, float* sn, hipStream_t stream, hipEvent_t start, hipEvent_t stop)
{
    PmParams p = make_pm_params(Q, K, g, seed);
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

hipError_t launch_attend(int dtype, const void* Q, const void* K, const void* V, const int32_t* J, int kappa,
                         const Grid& g, int window, float scale, bool causal, void* out, hipStream_t stream,
                         hipEvent_t start, hipEvent_t stop)
{
    AttParams p{};
    p.Q = Q;
    p.K = K;
    p.V = V;
    p.J = J;
    p.out = out;
    p.n = static_cast<uint32_t>(g.S) * g.Hq * g.Wq;
    p.Hk = g.Hk;
    p.Wk = g.Wk;
    p.nkeys = static_cast<uint32_t>(g.Hk) * g.Wk;
    p.div_plane = make_div(static_cast<uint32_t>(g.Hq) * g.Wq);
    p.div_wk = make_div(g.Wk);
    p.b = window / 2;
    p.scale_log2e = scale * 1.4426950408889634f;
    p.kappa = kappa;
    p.causal = causal ? 1 : 0;
    return dispatch(dtype, g.d, [&](auto ty, auto d) {
        return run_attend<decltype(ty), decltype(d)::value>(p, window, stream, start, stop);
    });
}

size_t attend_backward_workspace_bytes(int S, int Hq, int Wq, int Hk, int Wk, int kappa)
{
    const size_t n = static_cast<size_t>(S) * Hq * Wq, N = static_cast<size_t>(S) * Hk * Wk;
    const size_t tiles = (N + kScanTile - 1) / kScanTile;
    auto r256 = [](size_t b) { return (b + 255) & ~static_cast<size_t>(255); };
    return r256(4 * N) + r256(4 * (N + 1)) + r256(4 * (tiles + 1)) + r256(4 * n * kappa) + 2 * r256(4 * n);
}

hipError_t launch_attend_backward(int dtype, const void* Q, const void* K, const void* V, const int32_t* J, int kappa,
                                  const Grid& g, int window, float scale, bool causal, const void* dO, float* dQ,
                                  float* dK, float* dV, void* workspace, hipStream_t stream, hipEvent_t* events)
{
    BwdParams p{};
    p.Q = Q;
    p.K = K;
    p.V = V;
    p.J = J;
    p.dO = dO;
    p.dQ = dQ;
    p.dK = dK;
    p.dV = dV;
    p.n = static_cast<uint32_t>(g.S) * g.Hq * g.Wq;
    p.Hq = g.Hq;
    p.Wq = g.Wq;
    p.Hk = g.Hk;
    p.Wk = g.Wk;
    p.nkeys = static_cast<uint32_t>(g.Hk) * g.Wk;
    p.keys_total = static_cast<uint32_t>(g.S) * p.nkeys;
    p.div_plane = make_div(static_cast<uint32_t>(g.Hq) * g.Wq);
    p.div_wk = make_div(g.Wk);
    p.div_n = make_div(p.n);
    p.div_keys = make_div(p.nkeys);
    p.b = window / 2;
    p.scale = scale;
    p.scale_log2e = scale * 1.4426950408889634f;
    p.kappa = kappa;
    p.causal = causal ? 1 : 0;

    // workspace: counts, offsets, tile sums, entries, log2 normalisers, D
    const size_t N = p.keys_total;
    const uint32_t tiles = static_cast<uint32_t>((N + kScanTile - 1) / kScanTile);
    auto r256 = [](size_t b) { return (b + 255) & ~static_cast<size_t>(255); };
    char* w = static_cast<char*>(workspace);
    int32_t* counts = reinterpret_cast<int32_t*>(w);
    w += r256(4 * N);
    int32_t* offsets = reinterpret_cast<int32_t*>(w);
    w += r256(4 * (N + 1));
    int32_t* sums = reinterpret_cast<int32_t*>(w);
    w += r256(4 * (static_cast<size_t>(tiles) + 1));
    int32_t* entries = reinterpret_cast<int32_t*>(w);
    w += r256(4 * static_cast<size_t>(p.n) * kappa);
    p.lse2 = reinterpret_cast<float*>(w);
    w += r256(4 * static_cast<size_t>(p.n));
    p.Dq = reinterpret_cast<float*>(w);
    p.offsets = offsets;
    p.entries = entries;

    auto grid_for = [](size_t items) {
        const size_t b = (items + kBlock - 1) / kBlock;
        return static_cast<uint32_t>(b < 1 ? 1 : (b > 4096 ? 4096 : b));
    };
    hipEvent_t e0 = events ? events[0] : nullptr, e1 = events ? events[1] : nullptr;
    const size_t entries_total = static_cast<size_t>(p.n) * kappa;
    hipError_t e;
    // inverse map: counting sort of the (query, match) entries by match key
    if ((e = launch(zero_i32_kernel, grid_for(N), stream, e0, nullptr, counts, N)) != hipSuccess) return e;
    if ((e = launch(bwd_count_kernel, grid_for(entries_total), stream, nullptr, nullptr, p, counts)) != hipSuccess)
        return e;
    if ((e = launch(scan_tiles_kernel, tiles, stream, nullptr, nullptr, static_cast<const int32_t*>(counts), offsets,
                    sums, N)) != hipSuccess)
        return e;
    if ((e = launch(scan_sums_kernel, 1u, stream, nullptr, nullptr, sums, tiles)) != hipSuccess) return e;
    if ((e = launch(scan_add_kernel, tiles, stream, nullptr, nullptr, offsets, static_cast<const int32_t*>(sums), N,
                    tiles)) != hipSuccess)
        return e;
    if ((e = launch(bwd_fill_kernel, grid_for(entries_total), stream, nullptr, e1, p, counts, entries)) != hipSuccess)
        return e;
    // gradients
    return dispatch(dtype, g.d, [&](auto ty, auto d) {
        return run_backward<decltype(ty), decltype(d)::value>(p, stream, events);
    });
}

hipError_t launch_snis(int dtype, const void* Q, const void* K, const void* V, const int32_t* modes, int kappa,
                       const Grid& g, const SnisSpec& spec, bool causal, void* out, float* ess, float* var,
                       hipStream_t stream, hipEvent_t start, hipEvent_t stop)
{
    SnisParams p{};
    p.Q = Q;
    p.K = K;
    p.V = V;
    p.modes = modes;
    p.out = out;
    p.ess = ess;
    p.var = var;
    p.n = static_cast<uint32_t>(g.S) * g.Hq * g.Wq;
    p.Hk = g.Hk;
    p.Wk = g.Wk;
    p.nkeys = static_cast<uint32_t>(g.Hk) * g.Wk;
    p.div_plane = make_div(static_cast<uint32_t>(g.Hq) * g.Wq);
    p.div_wk = make_div(g.Wk);
    p.kappa = kappa;
    p.samples = spec.samples;
    p.m = spec.radius;
    // the mixture weight at 1/65536 resolution, the same value in the draw and in r
    p.alpha16 = static_cast<uint32_t>(floor(static_cast<double>(spec.alpha) * 65536.0 + 0.5));
    const double a = p.alpha16 / 65536.0;
    p.w_local = static_cast<float>(a / kappa);
    p.w_unif = static_cast<float>((1.0 - a) / (static_cast<double>(g.Hk) * g.Wk));
    p.scale_log2e = spec.scale * 1.4426950408889634f;
    p.key0 = static_cast<uint32_t>(spec.seed & 0xFFFFFFFFu);
    p.key1 = static_cast<uint32_t>(spec.seed >> 32);
    p.causal = causal ? 1 : 0;
    return dispatch(dtype, g.d, [&](auto ty, auto d) {
        return run_snis<decltype(ty), decltype(d)::value>(p, stream, start, stop);
    });
}

}  // namespace scram
