// Sparse window attention (Algorithm 2, Equations 8-9).

#include "scram_device.h"

namespace scram {
namespace {

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
    int Hq, Wq;
    Tiling tq;            // blocks -> tiles of the query grid (set per storage type and width)
};

// ---------------------------------------------------------------------------
// K4: window softmax + value gather
// ---------------------------------------------------------------------------

// Fixed window side W (odd), one window row per step: the W key rows and W
// value rows of a window row are gathered together (2W loads in flight),
// then the W scores (base-2 domain), one online-softmax rescale, and the
// value accumulation.  Keys outside the grid read a clamped (valid) row and
// get weight 0; window rows entirely outside the grid are skipped, and so,
// before any load, are rows whose every key an earlier window holds or the
// causal mask drops.
// MK = 0: one window, no mask; MK >= 1: up to MK windows and/or the causal mask.
template <typename T, int D, int G, int W, int MK>
__global__ __launch_bounds__(kBlock) void attend_window_kernel(AttParams p)
{
    constexpr bool MULTI = MK > 0;
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;  // channels per lane
    constexpr int B = W / 2;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    uint32_t g;
    if (!tile_item<RW::kQpb>(p.tq, blk, threadIdx.x / G, g)) return;

    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);
    const size_t slice = static_cast<size_t>(s) * p.nkeys * D;
    const T* Ks = static_cast<const T*>(p.K) + slice;
    const T* Vs = static_cast<const T*>(p.V) + slice;
    uint4 q[CH];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    WindowSet<(MK > 0 ? MK : 1)> wset;
    if constexpr (MULTI) wset = make_window_set<MK>(p, g, rem);
    const int nwin = MULTI ? p.kappa : 1;

    float m = -INFINITY, l = 0.f;
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;

    for (int e = 0; e < nwin; ++e) {
        uint32_t u, v;
        if constexpr (MULTI) {
            wset.centre(e, u, v);
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
            bool use[W];
            bool any = false;
#pragma unroll
            for (int c = 0; c < W; ++c) {
                use[c] = col_ok[c];
                if constexpr (MULTI) use[c] = use[c] && !wset.skip(e, r, cols[c]);
                any = any || use[c];
            }
            if constexpr (MULTI) {
                if (!any) continue;
            }
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
                sc[c] = use[c] ? row_score<T, D, G>(q, kr[c]) * p.scale_log2e : -INFINITY;
                mb = fmaxf(mb, sc[c]);
            }
            if (mb == -INFINITY) continue;  // nothing of this row is in the set
            if (mb > m + kRescaleSlack) {
                const float alpha = __builtin_amdgcn_exp2f(m - mb);  // 0 on the first row
                l *= alpha;
#pragma unroll
                for (int i = 0; i < E; ++i) acc[i] *= alpha;
                m = mb;
            }
#pragma unroll
            for (int c = 0; c < W; ++c) {
                const float pj = __builtin_amdgcn_exp2f(sc[c] - m);  // exp2(-inf) = 0
                l += pj;
                accumulate_row<T, CH>(acc, pj, vr[c]);
            }
        }
    }
    store_row<T, D, G>(p.out, g, lane, acc, l > 0.f ? 1.f / l : 0.f);  // an empty set gives a zero row
}

// Any window side: the clipped window is visited in row order, kNb keys at a
// time with their key and value loads in flight together; an online softmax
// keeps (running max m, running sum l, accumulator) in the base-2 domain.
template <typename T, int D, int G, int MK>
__global__ __launch_bounds__(kBlock) void attend_kernel(AttParams p)
{
    constexpr bool MULTI = MK > 0;
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;
    constexpr int kNb = CH >= 2 ? 4 : 8;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    uint32_t g;
    if (!tile_item<RW::kQpb>(p.tq, blk, threadIdx.x / G, g)) return;

    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);
    const size_t slice = static_cast<size_t>(s) * p.nkeys * D;
    const T* Ks = static_cast<const T*>(p.K) + slice;
    const T* Vs = static_cast<const T*>(p.V) + slice;
    uint4 q[CH];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    WindowSet<(MK > 0 ? MK : 1)> wset;
    if constexpr (MULTI) wset = make_window_set<MK>(p, g, rem);
    const int nsets = MULTI ? p.kappa : 1;

    float m = -INFINITY, l = 0.f;
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;

    for (int e = 0; e < nsets; ++e) {
        uint32_t u, v;
        if constexpr (MULTI) {
            wset.centre(e, u, v);
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
            if (mb > m + kRescaleSlack) {
                const float alpha = __builtin_amdgcn_exp2f(m - mb);
                l *= alpha;
#pragma unroll
                for (int i = 0; i < E; ++i) acc[i] *= alpha;
                m = mb;
            }
#pragma unroll
            for (int j = 0; j < kNb; ++j) {
                const float pj = __builtin_amdgcn_exp2f(sc[j] - m);
                l += pj;
                accumulate_row<T, CH>(acc, pj, vr[j]);
            }
        }
    }
    store_row<T, D, G>(p.out, g, lane, acc, l > 0.f ? 1.f / l : 0.f);  // an empty set gives a zero row
}

template <typename T, int D, int MK>
hipError_t run_attend_m(const AttParams& p, int window, uint64_t blocks, hipStream_t st, hipEvent_t e0,
                        hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kAttend;
    switch (window) {
        case 1: return launch(attend_window_kernel<T, D, G, 1, MK>, blocks, st, e0, e1, p);
        case 3: return launch(attend_window_kernel<T, D, G, 3, MK>, blocks, st, e0, e1, p);
        case 5: return launch(attend_window_kernel<T, D, G, 5, MK>, blocks, st, e0, e1, p);
        case 7: return launch(attend_window_kernel<T, D, G, 7, MK>, blocks, st, e0, e1, p);
        default: return launch(attend_kernel<T, D, G, MK>, blocks, st, e0, e1, p);
    }
}

template <typename T, int D>
hipError_t run_attend(const AttParams& p0, int window, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kAttend;
    AttParams p = p0;
    p.tq = make_tiling(p.Hq, p.Wq, Row<T, D, G>::kQpb);
    const uint64_t blocks = tiling_blocks(p.tq, p.n / p.tq.plane);
    // the smallest register budget that holds this call's window centres
    if (p.kappa == 1) {
        return p.causal ? run_attend_m<T, D, 1>(p, window, blocks, st, e0, e1)
                        : run_attend_m<T, D, 0>(p, window, blocks, st, e0, e1);
    }
    if (p.kappa == 2) return run_attend_m<T, D, 2>(p, window, blocks, st, e0, e1);
    if (p.kappa <= 4) return run_attend_m<T, D, 4>(p, window, blocks, st, e0, e1);
    return run_attend_m<T, D, kMaxKappa>(p, window, blocks, st, e0, e1);
}

}  // namespace

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
    p.Hq = g.Hq;
    p.Wq = g.Wq;
    p.b = window / 2;
    p.scale_log2e = scale * 1.4426950408889634f;
    p.kappa = kappa;
    p.causal = causal ? 1 : 0;
    return dispatch(dtype, g.d, [&](auto ty, auto d) {
        return run_attend<decltype(ty), decltype(d)::value>(p, window, stream, start, stop);
    });
}

uint64_t attend_max_blocks(int dtype, const Grid& g)
{
    return dispatch_value(dtype, g.d, uint64_t(0), [&](auto t, auto d) {
        using T = decltype(t);
        constexpr int D = decltype(d)::value;
        return tiling_blocks(make_tiling(g.Hq, g.Wq, Row<T, D, Lanes<T, D>::kAttend>::kQpb), g.S);
    });
}

}  // namespace scram
