// HIP kernels of the SCRAM hot path for gfx950 (MI355X).
//
//   pm_init_kernel   -- random initial nearest-neighbour field (Algorithm 1,
//                       first loop) or the scores of a given field
//   pm_iter_kernel   -- one synchronous (Jacobi) sweep of Algorithm 1:
//                       propagation from neighbours at jumps 8, 4, 2, 1 and
//                       random search at distances R, R/2, ..., 1
//   attend_kernel    -- Algorithm 2 at kappa = 1 (Equations 8-9): online
//                       softmax over the (2b+1)^2 window around the match,
//                       fused with the gather of the values
//
// Work decomposition.  Every kernel gives one query pixel to a "lane group"
// of G = row_bytes / 16 lanes of a 64-wide wavefront: each lane owns one
// 16-byte slice of the query row (4 fp32 or 8 bf16 channels) in registers, so
// gathering a candidate key row is one coalesced 16-byte load per lane (a
// 128-byte bf16 d=64 row is 8 lanes x 16 B) and the dot product is a per-lane
// fp32 FMA chain followed by a fixed butterfly across the group (DPP row
// permutes).  Every lane of the group ends with the bit-identical sum, so the
// argmax decisions are taken redundantly in registers with no extra traffic,
// and the same reduction order is used by the init and the sweep kernels: a
// score never depends on which kernel computed it.
//
// Candidate gathers are not a dense contraction, so there is no MFMA here;
// the sweeps are bound by the memory system (HBM / Infinity Cache / L2).
// Blocks are remapped so that consecutive query ranges land on the same XCD
// and share its L2.

#include <stdint.h>

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
// element / row helpers
// ---------------------------------------------------------------------------
template <typename T>
struct Elem;
template <>
struct Elem<float> {
    static constexpr int kPer16 = 4;
};
template <>
struct Elem<uint16_t> {  // bfloat16 storage
    static constexpr int kPer16 = 8;
};

template <typename T, int D>
struct Layout {
    static constexpr int kEpl = Elem<T>::kPer16;  // channels per lane
    static constexpr int kG = D / kEpl;           // lanes per query
    static constexpr int kQpb = kBlock / kG;      // queries per block
    static_assert(kG >= 2 && kG <= 32 && (kG & (kG - 1)) == 0, "lane group must be 2..32 lanes");
};

template <typename T>
__device__ __forceinline__ void unpack(const uint4& r, float* f);

template <>
__device__ __forceinline__ void unpack<float>(const uint4& r, float* f)
{
    f[0] = __uint_as_float(r.x);
    f[1] = __uint_as_float(r.y);
    f[2] = __uint_as_float(r.z);
    f[3] = __uint_as_float(r.w);
}

// bf16 -> fp32 is exact: the bf16 bits are the upper half of the fp32 bits.
template <>
__device__ __forceinline__ void unpack<uint16_t>(const uint4& r, float* f)
{
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(w[i] << 16);
        f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
}

// One lane's 16-byte slice of row `row` of a [rows, D] array.
template <typename T, int D>
__device__ __forceinline__ uint4 load_slice(const T* base, uint32_t row, int lane)
{
    return reinterpret_cast<const uint4*>(base + static_cast<size_t>(row) * D)[lane];
}

// Per-lane partial dot product in a fixed order.
template <typename T>
__device__ __forceinline__ float slice_dot(const float* q, const uint4& raw)
{
    constexpr int E = Elem<T>::kPer16;
    float k[E];
    unpack<T>(raw, k);
    float acc = q[0] * k[0];
#pragma unroll
    for (int e = 1; e < E; ++e) acc = fmaf(q[e], k[e], acc);
    return acc;
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
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
};

// ---------------------------------------------------------------------------
// K1: initial field and its scores
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(kBlock) void pm_init_kernel(PmParams p)
{
    using L = Layout<T, D>;
    const int lane = threadIdx.x & (L::kG - 1);
    const uint32_t g = blockIdx.x * L::kQpb + threadIdx.x / L::kG;
    if (g >= p.n) return;  // whole lane groups leave together
    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);

    int32_t idx;
    if (p.init) {
        idx = clamp_index(p.init[g], p.nkeys);
    } else {
        const uint4 w = philox4x32_10(g, 0u, 0u, 0u, p.key0, p.key1);
        const uint32_t u = __umulhi(w.x, static_cast<uint32_t>(p.Hk));
        const uint32_t v = __umulhi(w.y, static_cast<uint32_t>(p.Wk));
        idx = static_cast<int32_t>(u * p.Wk + v);
    }
    const T* Ks = static_cast<const T*>(p.K) + static_cast<size_t>(s) * p.nkeys * D;
    float q[L::kEpl];
    unpack<T>(load_slice<T, D>(static_cast<const T*>(p.Q), g, lane), q);
    const float sc = group_sum<L::kG>(slice_dot<T>(q, load_slice<T, D>(Ks, idx, lane)));
    if (lane == 0) {
        if (p.Jn) p.Jn[g] = idx;
        p.sn[g] = sc;
    }
}

// ---------------------------------------------------------------------------
// K2: one Jacobi sweep (propagation + random search), (Jp, sp) -> (Jn, sn)
// ---------------------------------------------------------------------------
template <typename T, int D, bool PROP, bool RS>
__global__ __launch_bounds__(kBlock) void pm_iter_kernel(PmParams p)
{
    using L = Layout<T, D>;
    constexpr int G = L::kG;
    const int lane = threadIdx.x & (G - 1);
    const int gbase = (threadIdx.x & 63) - lane;  // wave lane of the group's first lane
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    const uint32_t g = blk * L::kQpb + threadIdx.x / G;
    if (g >= p.n) return;  // whole lane groups leave together

    uint32_t s, rem, x, y;
    divmod(g, p.div_plane, s, rem);
    divmod(rem, p.div_wq, x, y);
    const T* Ks = static_cast<const T*>(p.K) + static_cast<size_t>(s) * p.nkeys * D;
    float q[L::kEpl];
    unpack<T>(load_slice<T, D>(static_cast<const T*>(p.Q), g, lane), q);
    int32_t cur = clamp_index(p.Jp[g], p.nkeys);
    float best = p.sp[g];

    if constexpr (PROP) {
        // Lane l of the group forms candidates l, l + G, ... of the 16
        // (jump index i/4 over 8,4,2,1; direction i%4 over row-1, row+1,
        // col-1, col+1): the neighbour's match shifted back by the offset.
        constexpr int kSlots = (16 + G - 1) / G;
        const int32_t* Jps = p.Jp + static_cast<size_t>(s) * p.plane_q;
        int32_t cand[kSlots];
#pragma unroll
        for (int m = 0; m < kSlots; ++m) {
            const int i = lane + m * G;
            int32_t c = -1;
            if (i < 16) {
                const int jump = 8 >> (i >> 2);
                const int dir = i & 3;
                const int ox = dir == 0 ? -jump : (dir == 1 ? jump : 0);
                const int oy = dir == 2 ? -jump : (dir == 3 ? jump : 0);
                const int nx = static_cast<int>(x) + ox, ny = static_cast<int>(y) + oy;
                if (nx >= 0 && nx < p.Hq && ny >= 0 && ny < p.Wq) {
                    const uint32_t nb = clamp_index(Jps[nx * p.Wq + ny], p.nkeys);
                    uint32_t nu, nv;
                    divmod(nb, p.div_wk, nu, nv);
                    const int r = static_cast<int>(nu) - ox, cc = static_cast<int>(nv) - oy;
                    if (r >= 0 && r < p.Hk && cc >= 0 && cc < p.Wk) c = r * p.Wk + cc;
                }
            }
            cand[m] = c;
        }
        // The 16 candidates do not depend on each other: gather them four at
        // a time with all loads in flight before the first dot product.  A
        // candidate equal to the incumbent cannot win and is not gathered.
        const int32_t cur0 = cur;
#pragma unroll
        for (int i0 = 0; i0 < 16; i0 += 4) {
            int32_t c[4];
            uint4 raw[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int i = i0 + j;
                c[j] = __shfl(cand[i / G], gbase + (i % G));
                if (c[j] >= 0 && c[j] != cur0) raw[j] = load_slice<T, D>(Ks, c[j], lane);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (c[j] >= 0 && c[j] != cur0) {
                    const float sc = group_sum<G>(slice_dot<T>(q, raw[j]));
                    if (better(sc, c[j], best, cur)) {
                        best = sc;
                        cur = c[j];
                    }
                }
            }
        }
    }

    if constexpr (RS) {
        uint32_t cu, cv;
        divmod(static_cast<uint32_t>(cur), p.div_wk, cu, cv);
        // Philox block m serves steps 2m and 2m+1.  The blocks do not depend
        // on the running best, so lane l of the group draws block b0 + l and
        // the steps fetch their words from it.
        const int nblk = (p.rs_steps + 1) >> 1;
        for (int b0 = 0; b0 < nblk; b0 += G) {
            uint4 w = make_uint4(0u, 0u, 0u, 0u);
            if (b0 + lane < nblk) w = philox4x32_10(g, p.t, static_cast<uint32_t>(b0 + lane), 0u, p.key0, p.key1);
            const int here = min(G, nblk - b0);
            for (int j = 0; j < here; ++j) {
                const uint32_t w0 = __shfl(w.x, gbase + j), w1 = __shfl(w.y, gbase + j);
                const uint32_t w2 = __shfl(w.z, gbase + j), w3 = __shfl(w.w, gbase + j);
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const int k = 2 * (b0 + j) + half;
                    if (k < p.rs_steps) {
                        const int dk = p.R >> k;
                        const uint32_t wr = half ? w2 : w0, wc = half ? w3 : w1;
                        const int lo_r = max(static_cast<int>(cu) - dk, 0);
                        const int hi_r = min(static_cast<int>(cu) + dk, p.Hk - 1);
                        const int lo_c = max(static_cast<int>(cv) - dk, 0);
                        const int hi_c = min(static_cast<int>(cv) + dk, p.Wk - 1);
                        const uint32_t r = lo_r + __umulhi(wr, static_cast<uint32_t>(hi_r - lo_r + 1));
                        const uint32_t c = lo_c + __umulhi(wc, static_cast<uint32_t>(hi_c - lo_c + 1));
                        const int32_t idx = static_cast<int32_t>(r * p.Wk + c);
                        if (idx != cur) {
                            const float sc = group_sum<G>(slice_dot<T>(q, load_slice<T, D>(Ks, idx, lane)));
                            if (better(sc, idx, best, cur)) {
                                best = sc;
                                cur = idx;
                                cu = r;
                                cv = c;
                            }
                        }
                    }
                }
            }
        }
    }

    if (lane == 0) {
        p.Jn[g] = cur;
        p.sn[g] = best;
    }
}

// ---------------------------------------------------------------------------
// K4: window softmax + value gather (online softmax, one window row of up to
// kNb keys per step; all key and value loads of a step issued together)
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(kBlock) void attend_kernel(AttParams p)
{
    using L = Layout<T, D>;
    constexpr int E = L::kEpl;
    constexpr int kNb = 8;
    const int lane = threadIdx.x & (L::kG - 1);
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    const uint32_t g = blk * L::kQpb + threadIdx.x / L::kG;
    if (g >= p.n) return;

    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);
    const size_t slice = static_cast<size_t>(s) * p.nkeys * D;
    const T* Ks = static_cast<const T*>(p.K) + slice;
    const T* Vs = static_cast<const T*>(p.V) + slice;
    float q[E];
    unpack<T>(load_slice<T, D>(static_cast<const T*>(p.Q), g, lane), q);
    uint32_t u, v;
    divmod(static_cast<uint32_t>(clamp_index(p.J[g], p.nkeys)), p.div_wk, u, v);
    const int r0 = max(static_cast<int>(u) - p.b, 0), r1 = min(static_cast<int>(u) + p.b, p.Hk - 1);
    const int c0 = max(static_cast<int>(v) - p.b, 0), c1 = min(static_cast<int>(v) + p.b, p.Wk - 1);

    float m = -INFINITY, l = 0.f;
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;

    for (int r = r0; r <= r1; ++r) {
        for (int cb = c0; cb <= c1; cb += kNb) {
            const int nk = min(kNb, c1 - cb + 1);
            const uint32_t row0 = static_cast<uint32_t>(r * p.Wk + cb);
            uint4 kr[kNb], vr[kNb];
#pragma unroll
            for (int j = 0; j < kNb; ++j) {
                if (j < nk) {
                    kr[j] = load_slice<T, D>(Ks, row0 + j, lane);
                    vr[j] = load_slice<T, D>(Vs, row0 + j, lane);
                }
            }
            float sc[kNb];
            float mb = m;
#pragma unroll
            for (int j = 0; j < kNb; ++j) {
                if (j < nk) {
                    sc[j] = group_sum<L::kG>(slice_dot<T>(q, kr[j])) * p.scale_log2e;
                    mb = fmaxf(mb, sc[j]);
                }
            }
            const float alpha = __builtin_amdgcn_exp2f(m - mb);
            l *= alpha;
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] *= alpha;
#pragma unroll
            for (int j = 0; j < kNb; ++j) {
                if (j < nk) {
                    const float pj = __builtin_amdgcn_exp2f(sc[j] - mb);
                    l += pj;
                    float vv[E];
                    unpack<T>(vr[j], vv);
#pragma unroll
                    for (int e = 0; e < E; ++e) acc[e] = fmaf(pj, vv[e], acc[e]);
                }
            }
            m = mb;
        }
    }

    const float inv = 1.f / l;
    uint4 o;
    if constexpr (E == 4) {
        o = make_uint4(__float_as_uint(acc[0] * inv), __float_as_uint(acc[1] * inv),
                       __float_as_uint(acc[2] * inv), __float_as_uint(acc[3] * inv));
    } else {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = f32_to_bf16_rne(acc[2 * i] * inv) | (f32_to_bf16_rne(acc[2 * i + 1] * inv) << 16);
        o = make_uint4(w[0], w[1], w[2], w[3]);
    }
    reinterpret_cast<uint4*>(static_cast<T*>(p.out) + static_cast<size_t>(g) * D)[lane] = o;
}

// ---------------------------------------------------------------------------
// host-side launch helpers
// ---------------------------------------------------------------------------
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
hipError_t run_init(const PmParams& p, hipStream_t st)
{
    using L = Layout<T, D>;
    const uint32_t blocks = (p.n + L::kQpb - 1) / L::kQpb;
    hipLaunchKernelGGL((pm_init_kernel<T, D>), dim3(blocks), dim3(kBlock), 0, st, p);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t run_iter(const PmParams& p, uint32_t flags, hipStream_t st)
{
    using L = Layout<T, D>;
    const uint32_t blocks = (p.n + L::kQpb - 1) / L::kQpb;
    const bool prop = !(flags & SCRAM_PM_NO_PROPAGATION);
    const bool rs = !(flags & SCRAM_PM_NO_RANDOM_SEARCH);
    if (prop && rs)
        hipLaunchKernelGGL((pm_iter_kernel<T, D, true, true>), dim3(blocks), dim3(kBlock), 0, st, p);
    else if (prop)
        hipLaunchKernelGGL((pm_iter_kernel<T, D, true, false>), dim3(blocks), dim3(kBlock), 0, st, p);
    else if (rs)
        hipLaunchKernelGGL((pm_iter_kernel<T, D, false, true>), dim3(blocks), dim3(kBlock), 0, st, p);
    else
        hipLaunchKernelGGL((pm_iter_kernel<T, D, false, false>), dim3(blocks), dim3(kBlock), 0, st, p);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t run_attend(const AttParams& p, hipStream_t st)
{
    using L = Layout<T, D>;
    const uint32_t blocks = (p.n + L::kQpb - 1) / L::kQpb;
    hipLaunchKernelGGL((attend_kernel<T, D>), dim3(blocks), dim3(kBlock), 0, st, p);
    return hipGetLastError();
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
                          const int32_t* init, int32_t* J, float* s, hipStream_t stream)
{
    PmParams p = make_pm_params(Q, K, g, seed);
    p.init = init;
    p.Jn = J;
    p.sn = s;
    return dispatch(dtype, g.d, [&](auto t, auto d) {
        return run_init<decltype(t), decltype(d)::value>(p, stream);
    });
}

hipError_t launch_pm_iter(int dtype, const void* Q, const void* K, const Grid& g, uint64_t seed,
                          uint32_t t, uint32_t flags, const int32_t* Jp, const float* sp, int32_t* Jn,
                          float* sn, hipStream_t stream)
{
    PmParams p = make_pm_params(Q, K, g, seed);
    p.t = t;
    p.Jp = Jp;
    p.sp = sp;
    p.Jn = Jn;
    p.sn = sn;
    return dispatch(dtype, g.d, [&](auto ty, auto d) {
        return run_iter<decltype(ty), decltype(d)::value>(p, flags, stream);
    });
}

hipError_t launch_attend(int dtype, const void* Q, const void* K, const void* V, const int32_t* J,
                         const Grid& g, int window, float scale, void* out, hipStream_t stream)
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
    return dispatch(dtype, g.d, [&](auto ty, auto d) {
        return run_attend<decltype(ty), decltype(d)::value>(p, stream);
    });
}

}  // namespace scram
