// Device helpers shared by the HIP kernels of the SCRAM hot path for gfx950
// (MI355X):
//
//   scram_pm.hip       -- pm_init_kernel (random initial nearest-neighbour
//                         field, Algorithm 1's first loop, or the scores of a
//                         given field) and pm_iter_kernel (one synchronous
//                         (Jacobi) sweep of Algorithm 1: propagation from
//                         neighbours at jumps 8, 4, 2, 1 and random search at
//                         distances R, R/2, ..., 1)
//   scram_attend.hip   -- Algorithm 2 (Equations 8-9): online softmax over the
//                         (2b+1)^2 windows around the matches, fused with the
//                         gather of the values
//   scram_backward.hip -- gradients of the attend step (maps held fixed)
//   scram_snis.hip     -- self-normalised importance sampling around the
//                         matches (Section 4.2, Equations 11-17)
//
// Everything here lives in an unnamed namespace: each kernel file gets its
// own copy.
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

#pragma once

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
constexpr uint64_t kMaxBlocks = 0xFFFFFFFFull / kBlock;  // blocks of one dispatch (2^32 - 1 work-items)

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
// neighbouring keys -- share one L2.  A bijection for every nb.  Built with
// SCRAM_XCD_REMAP=0, blocks take their tiles in dispatch order instead.
#ifndef SCRAM_XCD_REMAP
#define SCRAM_XCD_REMAP 1
#endif
__device__ __forceinline__ uint32_t xcd_remap(uint32_t b, uint32_t nb)
{
    if (!SCRAM_XCD_REMAP) return b;
    const uint32_t x = b % kXcds, local = b / kXcds;
    const uint32_t q = nb / kXcds, r = nb % kXcds;
    const uint32_t start = x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q;
    return start + local;
}

// Block tiles.  The lane groups of a block cover a tile of `items` positions
// (a power of two; raster order inside the tile) of one slice's 2-D grid;
// blocks take the tiles of slice 0, then those of slice 1, ...  Within a
// slice the tiles go in raster order; on grids more than kBandMax tiles wide,
// in bands of kBandTiles tile columns instead (top to bottom, left to right
// within a band's tile row), so that the blocks in flight on an XCD cover a
// compact patch of the grid rather than part of one long tile row, and a
// tile's neighbours below are dispatched soon after it.  Neighbouring
// positions have nearby matches, so a squarish tile shares more of the rows
// its lane groups read in L1 than a row segment of the same size.  Grids
// narrower than the squarish tile get a flatter one, so that 1-D grids keep
// every lane group busy.
//
// The kernels that give an item the same result whatever else its tile holds
// (a lane group per query or key) take their tiles through make_tiling's
// skew, kLaneSkew: the tile's width is doubled (halved for a negative skew)
// that many times over the squarish one.  Every one of these is a build
// setting (0, 16 and 64 here); a build with other values -- other tile
// shapes and dispatch orders, same results -- is what the race checks of the
// sweep compare this one against.
#ifndef SCRAM_BAND_TILES
#define SCRAM_BAND_TILES 16
#endif
#ifndef SCRAM_BAND_MAX
#define SCRAM_BAND_MAX 64
#endif
#ifndef SCRAM_LANE_TILE_SKEW
#define SCRAM_LANE_TILE_SKEW 0
#endif
constexpr uint32_t kBandTiles = SCRAM_BAND_TILES;
constexpr uint32_t kBandMax = SCRAM_BAND_MAX;
constexpr int kLaneSkew = SCRAM_LANE_TILE_SKEW;

struct Tiling {
    uint32_t H, W, plane;  // one slice's grid
    uint32_t lw;           // log2 of the tile width
    uint32_t nw, bw;       // tiles per grid row, tile columns per band (nw: one band, raster order)
    Div div_slice;         // tiles per slice
    Div div_band, div_bw;  // tiles per band, bw
};

// Host: the tiling of one slice's H x W grid by blocks of `items` positions.
inline Tiling make_tiling(int H, int W, uint32_t items, int skew = 0)
{
    auto pow2_at_least = [](uint32_t v) {
        uint32_t p = 1;
        while (p < v) p <<= 1;
        return p;
    };
    uint32_t lw = 0;
    while ((1u << (2 * (lw + 1))) <= items) ++lw;  // squarish: width = sqrt(items) rounded down to a power of two
    for (; skew > 0 && (2u << lw) <= items; --skew) ++lw;
    for (; skew < 0 && lw > 0; ++skew) --lw;
    uint32_t tw = 1u << lw, th = items / tw;
    if (th > pow2_at_least(static_cast<uint32_t>(H))) {  // short grid: wider tiles
        th = pow2_at_least(static_cast<uint32_t>(H));
        tw = items / th;
    }
    if (tw > pow2_at_least(static_cast<uint32_t>(W))) {  // narrow grid: taller tiles
        tw = pow2_at_least(static_cast<uint32_t>(W));
        th = items / tw;
    }
    lw = 0;
    while ((1u << lw) < tw) ++lw;
    const uint32_t nw = (static_cast<uint32_t>(W) + tw - 1) / tw, nh = (static_cast<uint32_t>(H) + th - 1) / th;
    const uint32_t bw = nw > kBandMax ? kBandTiles : nw;
    return Tiling{static_cast<uint32_t>(H), static_cast<uint32_t>(W), static_cast<uint32_t>(H) * W, lw, nw, bw,
                  make_div(nw * nh), make_div(bw * nh), make_div(bw)};
}

inline uint64_t tiling_blocks(const Tiling& t, uint32_t slices) { return uint64_t(slices) * t.div_slice.d; }

// Tile row and column of the k-th tile of a slice, in the order above.
__device__ __forceinline__ void tile_coords(const Tiling& t, uint32_t k, uint32_t& tr, uint32_t& tc)
{
    uint32_t band, rem;
    divmod(k, t.div_band, band, rem);
    const uint32_t c0 = band * t.bw, wb = min(t.bw, t.nw - c0);  // the last band may be narrower
    if (wb == t.bw) {
        divmod(rem, t.div_bw, tr, tc);
    } else {
        tr = rem / wb;
        tc = rem - tr * wb;
    }
    tc += c0;
}

// Flat position g = s * H * W + x * W + y of item i (< kItems) of (remapped)
// block blk; false past the grid's right or bottom edge (g is then not
// meaningful).
template <uint32_t kItems>
__device__ __forceinline__ bool tile_item(const Tiling& t, uint32_t blk, uint32_t i, uint32_t& g)
{
    static_assert((kItems & (kItems - 1)) == 0, "tiles of a power-of-two size");
    uint32_t s, k, tr, tc;
    divmod(blk, t.div_slice, s, k);
    tile_coords(t, k, tr, tc);
    const uint32_t th = kItems >> t.lw;
    const uint32_t x = tr * th + (i >> t.lw), y = (tc << t.lw) + (i & ((1u << t.lw) - 1u));
    g = s * t.plane + x * t.W + y;
    return x < t.H && y < t.W;
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds of two
// 32x32->64 multiplies mixed with the other two words and the round key; the
// key advances by the two Weyl increments after every round.
__device__ __forceinline__ uint4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                               uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int i = 0; i < 10; ++i) {
        // each 64-bit product is one v_mad_u64_u32 (a multiply-high and a multiply-low would be two)
        const uint64_t a = static_cast<uint64_t>(0xD2511F53u) * c0;
        const uint64_t b = static_cast<uint64_t>(0xCD9E8D57u) * c2;
        const uint32_t n0 = static_cast<uint32_t>(b >> 32) ^ c1 ^ k0;
        const uint32_t n2 = static_cast<uint32_t>(a >> 32) ^ c3 ^ k1;
        c0 = n0;
        c1 = static_cast<uint32_t>(b);
        c2 = n2;
        c3 = static_cast<uint32_t>(a);
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

// Online softmax in the base-2 domain: the running reference m is raised
// (and the sums rescaled by 2^(m_old - m_new)) only when a score passes it by
// more than this, so weights 2^(s - m) stay below 2^kRescaleSlack and most
// window rows need no rescale; the ratio of the sums does not depend on m.
constexpr float kRescaleSlack = 8.f;

constexpr int kMaxKappa = 8;  // maps whose windows attend may unite

// ---------------------------------------------------------------------------
// value rows: accumulate, unpack, store
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

// Several windows and/or the causal mask: the centres of the kappa <= MK
// windows (MK a compile-time bound, so they live in registers) and the
// query's raster index.  skip(e, r, c): key (r, c) of window e is left out
// because an earlier window already holds it or it comes after the query.
template <int MK>
struct WindowSet {
    int kappa, b;
    bool causal;
    uint32_t local, Wk;
    int cu[MK], cv[MK];

    __device__ bool skip(int e, int r, int c) const
    {
        bool s = causal && static_cast<uint32_t>(r) * Wk + static_cast<uint32_t>(c) > local;
#pragma unroll
        for (int f = 0; f < MK; ++f)
            if (f < e) s = s || (abs(r - cu[f]) <= b && abs(c - cv[f]) <= b);
        return s;
    }

    // centre (u, v) of window e
    __device__ void centre(int e, uint32_t& u, uint32_t& v) const
    {
        u = static_cast<uint32_t>(cu[0]);
        v = static_cast<uint32_t>(cv[0]);
#pragma unroll
        for (int f = 1; f < MK; ++f)
            if (f == e) {
                u = static_cast<uint32_t>(cu[f]);
                v = static_cast<uint32_t>(cv[f]);
            }
    }
};

template <int MK, typename P>
__device__ __forceinline__ WindowSet<MK> make_window_set(const P& p, uint32_t g, uint32_t rem)
{
    WindowSet<MK> ws;
    ws.kappa = p.kappa;
    ws.b = p.b;
    ws.causal = p.causal != 0;
    ws.local = rem;
    ws.Wk = static_cast<uint32_t>(p.Wk);
#pragma unroll
    for (int e = 0; e < MK; ++e) {
        uint32_t u = 0, v = 0;
        if (e < p.kappa)
            divmod(static_cast<uint32_t>(clamp_index(p.J[static_cast<size_t>(e) * p.n + g], p.nkeys)), p.div_wk, u, v);
        ws.cu[e] = static_cast<int>(u);
        ws.cv[e] = static_cast<int>(v);
    }
    return ws;
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
hipError_t launch(void (*kernel)(A...), uint64_t blocks, hipStream_t st, hipEvent_t start, hipEvent_t stop,
                  typename NoDeduce<A>::type... args)
{
    // a dispatch holds at most 2^32 - 1 work-items; the front end rejects larger grids first
    if (blocks == 0 || blocks > kMaxBlocks) return hipErrorInvalidConfiguration;
    if (start || stop)
        hipExtLaunchKernelGGL(kernel, dim3(blocks), dim3(kBlock), 0, st, start, stop, 0, args...);
    else
        hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kBlock), 0, st, args...);
    return hipGetLastError();
}

// (dtype, d) -> instantiation; `none` for an unsupported pair
template <typename R, typename F>
R dispatch_value(int dtype, int d, R none, F&& f)
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
    return none;
}

template <typename F>
hipError_t dispatch(int dtype, int d, F&& f)
{
    return dispatch_value(dtype, d, hipErrorInvalidValue, static_cast<F&&>(f));
}

}  // namespace
}  // namespace scram
