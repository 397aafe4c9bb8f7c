// Sparse window attention (Algorithm 2, Equations 8-9).

#include "scram_tile.h"

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
    int rc;               // cluster radius of the tile kernel (Chebyshev, between match centres)
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

// ---------------------------------------------------------------------------
// K4 on the matrix cores (bf16 storage, windows of side 3, 5 or 7, up to 8
// maps, with or without the causal mask)
// ---------------------------------------------------------------------------
// A wave takes a 4 x 4 tile of queries (16 on an 8 x 8 block tile; 16
// consecutive items of narrower tiles).  Neighbouring queries' windows
// overlap -- the matches of a coherent region are a shifted copy of it -- so
// the wave reads each key and value row of the union of its 16 windows once
// instead of once per query: the queries' match centres are grouped into
// clusters (scram_tile.h: a query joins the cluster of the first unassigned
// query whose centre lies within Chebyshev distance rc), and each cluster's key box (its
// members' windows, clipped to the grid) is visited in blocks of 16 keys in
// raster order.  A block's rows are gathered a row per 4 consecutive lanes
// (whole 64-byte spans per load, as in the lane-group kernels), staged in the
// wave's LDS tile and read back in the operand layout of the products, while
// the next block's rows load.  Per block (lane (m, g4) = lane (l mod 16,
// l div 16)):
//   S^T = K_blk Q^T          keys x queries, 16x16x32 bf16 products over the
//                            channels; lane holds keys 4 g4 + i, query m
//   p = 2^(scale log2e s - m_ref) for the keys of the query's own window in
//                            its own cluster, 0 otherwise
//   O^T += V_blk^T P^T       channels x queries, 16x16x16 bf16 products over
//                            the block's 16 keys: the transposing LDS load
//                            hands each lane 4 consecutive staged value rows at
//                            one channel, the operand layout that matches P^T,
//                            and P enters as two bf16 parts (top 8 significant
//                            bits, then the top 8 of the rest), so its relative
//                            error is below 2^-16
// The softmax reference of a query starts at the score of its match (a key of
// its window) and is raised (and its sums rescaled) only when a score passes
// it by more than kRescaleSlack, as in the other kernels;
// every query is in exactly one cluster, and each key of its window is in
// that cluster's box exactly once, so the weights are those of the window.
// The other keys of the box enter with weight exactly 0, which leaves the
// sums unchanged for finite value rows (a non-finite value anywhere in the
// box would reach every query of the cluster through 0 * inf).
// Several maps (kappa <= MK windows per query, attention over their union):
// one pass per window e, each with the clusters and boxes of the wave's 16
// window-e centres, into the same online softmax state; a slot of pass e is
// left out when one of the query's windows 0 .. e-1 holds its key, so every
// key of the union enters once.  Up to four maps take a single pass over the
// clusters of all their centres instead, five to eight two such passes (the
// second holding back the keys of the first's windows): each
// window is kept in the box of its own centre's cluster, less the keys of
// the query's earlier windows (and of those after the query).
// (at most 96 VGPRs: five waves per SIMD hide more of the row loads than four; the causal mask's
// registers and those of up to 4 windows do not fit there without spills, so they take four, and
// up to 8 windows, or 4 with the causal mask, three)
template <int D, int W, bool CAUSAL, int MK>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(MK > 4 || (MK == 4 && CAUSAL) ? 3 : CAUSAL || MK > 1 ? 4 : 5))) void
attend_tile_kernel(AttParams p)
{
    constexpr int B = W / 2;
    constexpr int kDs = D / 32;        // 32-channel contraction steps of S^T
    constexpr int kOt = D / 16;        // 16-channel tiles of O^T
    constexpr int kRowB = 2 * D + 16;  // LDS row stride: the 16-byte pad spreads a column read over the banks
    constexpr int kPer = D / 32;       // 16-byte pieces per lane: a row (D / 8 pieces) is read by 4 consecutive lanes
    constexpr int kWaves = kBlock / 64;
    __shared__ __align__(16) unsigned char s_k[kWaves][16 * kRowB], s_v[kWaves][16 * kRowB];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m = lane & 15, g4 = lane >> 4;
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    const uint32_t item = tile_wave_item(p.tq, wave, m);  // this lane's query m
    uint32_t g, g0;
    const bool valid = tile_item<kBlock / 4>(p.tq, blk, item, g);
    tile_item<kBlock / 4>(p.tq, blk, 0, g0);  // item 0 of a tile is always inside the grid
    const uint32_t gq = valid ? g : g0;
    uint32_t s, rem;
    divmod(gq, p.div_plane, s, rem);
    // the slice's key and value rows: every item of a tile lies in one slice, and the caller keeps a
    // slice's rows below 4 GiB, so a row is a 32-bit byte offset from a wave-uniform base
    const size_t slice_bytes =
        static_cast<size_t>(__builtin_amdgcn_readfirstlane(s)) * p.nkeys * static_cast<size_t>(2 * D);
    const unsigned char* const Kb = static_cast<const unsigned char*>(p.K) + slice_bytes;
    const unsigned char* const Vb = static_cast<const unsigned char*>(p.V) + slice_bytes;
    const uint32_t centre = static_cast<uint32_t>(clamp_index(p.J[gq], p.nkeys));
    int u, v;
    {
        uint32_t uu, vv;
        divmod(centre, p.div_wk, uu, vv);
        u = static_cast<int>(uu);
        v = static_cast<int>(vv);
    }
    // B operand of S^T: query m, channels 32 ds + 8 g4 .. + 7; and the same channels of the match's key
    bf16x8_t qf[kDs];
    uint4 kc[kDs];
    const uint16_t* const qrow = static_cast<const uint16_t*>(p.Q) + static_cast<size_t>(gq) * D;
#pragma unroll
    for (int ds = 0; ds < kDs; ++ds) {
        qf[ds] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qrow + 32 * ds + 8 * g4));
        kc[ds] = *reinterpret_cast<const uint4*>(Kb + centre * (2u * D) + 64u * ds + 16u * g4);
    }

    // ---- clusters of the 16 match centres and their key boxes ----
    int qx = 0, qy = 0;  // causal: the query's position (queries and keys share the grid)
    if constexpr (CAUSAL) {
        uint32_t xx, yy;
        divmod(rem, p.div_wk, xx, yy);
        qx = static_cast<int>(xx);
        qy = static_cast<int>(yy);
    }
    // up to four windows: one pass over the clusters of all their centres instead of a pass per window;
    // five to eight: two such rounds, the second holding back the keys of the first round's windows
    // (lanes 16 e .. 16 e + 15 cluster window e's centres).  A query keeps the slots of window e in the
    // cluster of that window's centre, less the keys of its windows 0 .. e-1 (and with the causal mask
    // those after the query), so every key of the union enters once; coherent maps walk a third (two
    // windows) to a half (three) fewer blocks
    constexpr bool JOINT = MK == 2 || MK == 4 || MK == 8;
    constexpr int NJ = JOINT ? (MK < 4 ? MK : 4) : 1;  // windows clustered together: a round
    constexpr int NW = JOINT ? MK : 1;                 // windows in all (eight: two rounds of four)
    int ju[NW], jv[NW], jmine[NJ];  // window e's centre; the cluster that holds the round's window e
    int round = 0;
    TileClusters tc;
    // the clusters of round r's centres (windows NJ r .. NJ r + NJ - 1)
    auto joint_round = [&](int r) {
        if constexpr (JOINT) {
            const int ew = NJ * r + (g4 & (NJ - 1));  // the window whose centre this lane clusters
            int iu = u, iv = v;
#pragma unroll
            for (int e = 0; e < NW; ++e) iu = ew == e ? ju[e] : iu, iv = ew == e ? jv[e] : iv;
            tc = tile_clusters_joint<B, NJ>(valid && ew < p.kappa, iu, iv, lane, p.rc, p.Hk, p.Wk);
#pragma unroll
            for (int e = 0; e < NJ; ++e) jmine[e] = __shfl(tc.mine, m + 16 * e);
        }
    };
    if constexpr (JOINT) {
#pragma unroll
        for (int e = 0; e < NW; ++e) {
            ju[e] = u, jv[e] = v;  // window 0; a window past kappa repeats it and is not clustered
            if (e > 0 && e < p.kappa) {
                uint32_t uu, vv;
                divmod(static_cast<uint32_t>(clamp_index(p.J[static_cast<size_t>(e) * p.n + gq], p.nkeys)),
                       p.div_wk, uu, vv);
                ju[e] = static_cast<int>(uu), jv[e] = static_cast<int>(vv);
            }
        }
        joint_round(0);
    } else {
        tc = tile_clusters<B, CAUSAL>(valid, u, v, m, lane, p.rc, p.Hk, p.Wk, qx, qy);
    }
    if (tc.nclu == 0) return;  // no query of this wave lies inside the grid
    int nclu = tc.nclu, mine = tc.mine, wr0 = tc.wr0, wrn = tc.wrn;
    uint32_t wcols = tc.wcols;
    // several windows: the centres of windows 0 .. e-1 of query m, as rows relative to window e's first
    // row (dw) and columns (cv); their columns in the current box (xw; zero for f >= e and outside the
    // query's own cluster)
    constexpr int kOther = MK > 1 ? MK - 1 : 1;
    int cu[kOther], cv[kOther], dw[kOther];
    uint32_t xw[kOther];
#pragma unroll
    for (int f = 0; f < kOther; ++f) cu[f] = cv[f] = 0, dw[f] = 1 << 20, xw[f] = 0u;
    // joint pass, per cluster: window e's first row as a box row (jd), its rows less one, cut at the
    // box's last (jn), its columns in the box (jx); bit e of hm: the cluster holds window e's centre
    int jd[NW], jn[NW];
    uint32_t jx[NW], hm = 0u;
#pragma unroll
    for (int e = 0; e < NW; ++e) jd[e] = jn[e] = 0, jx[e] = 0u;
    int jqr = 0;        // causal: the query's row as a box row
    uint32_t jqc = 0u;  // and the box columns up to the query's

    const f32x4_t zero = f32x4_t{0.f, 0.f, 0.f, 0.f};
    f32x4_t acc[kOt];
#pragma unroll
    for (int o = 0; o < kOt; ++o) acc[o] = zero;
    // the softmax denominators: an all-ones row block times P^T sums P over the keys, for every query
    f32x4_t lacc = zero;
    const bf16x4_t ones = bf16x4_t{static_cast<__bf16>(1.f), static_cast<__bf16>(1.f), static_cast<__bf16>(1.f),
                                   static_cast<__bf16>(1.f)};
    const float sl2e = p.scale_log2e;  // > 0 (the caller routes other scales to the lane-group kernels)
    const float inv_sl2e = __builtin_amdgcn_rcpf(sl2e);
    // bit positions 0..3 as values the compiler cannot see, so that each mask below stays one
    // bit-field extract instead of a shift pair
    int bit_at[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) asm volatile("s_mov_b32 %0, %1" : "=s"(bit_at[i]) : "i"(i));
    // online softmax state of query m: reference mref (base-2 domain) and its negation as the exponent's
    // offset.  The reference starts at the score of the query's match, a key of its window, so that no
    // block has to set it; thr_q is the raw score above which a block may raise it (a little below the
    // exact test, which decides), and thr is thr_q while the wave is in query m's cluster, +inf in the
    // other clusters.
    float s_centre = 0.f;
#pragma unroll
    for (int ds = 0; ds < kDs; ++ds) {
        const uint4 qa = __builtin_bit_cast(uint4, qf[ds]);
        s_centre = dot2_bf16(qa.x, kc[ds].x, s_centre);
        s_centre = dot2_bf16(qa.y, kc[ds].y, s_centre);
        s_centre = dot2_bf16(qa.z, kc[ds].z, s_centre);
        s_centre = dot2_bf16(qa.w, kc[ds].w, s_centre);
    }
    s_centre += __shfl_xor(s_centre, 16);
    s_centre += __shfl_xor(s_centre, 32);
    float mref = s_centre * sl2e, nref = -mref;
    if (CAUSAL && centre > rem) {  // a match after the query is not in its set: no reference yet
        mref = -INFINITY;
        nref = 0.f;
    }
    float thr_q = (mref + (kRescaleSlack - 1.f)) * inv_sl2e, thr = INFINITY;

    // ---- the clusters' blocks of 16 keys, one at a time; the next block's rows load during this one's
    // products.  Block k of a cluster holds raster slots 16 k .. 16 k + 15 of its box; its 16 key rows and
    // 16 value rows are read a row per 4 consecutive lanes, staged in this wave's LDS tile and read back in
    // the products' operand layout.
    const int lslot = lane >> 2, lpiece = lane & 3;  // every lane: one key slot, 16-byte pieces lpiece (+ 4)
    static_assert(kPer == 1 || kPer == 2, "32 or 64 channels");
    unsigned char* const tk = s_k[wave];
    unsigned char* const tv = s_v[wave];
    // A operand of O^T for tile o, read with the transposing LDS load: in each 16-lane group the load
    // hands lane i element e of the 8 bytes that lane 4 e + i / 4 addresses, so lane (m, g4) addresses
    // value row 4 g4 + m / 4 at channels 4 (m mod 4) .. + 3 (+ 16 o) and receives rows 4 g4 .. + 3 at
    // channel 16 o + m
    const unsigned char* const tvt = tv + (4 * g4 + (m >> 2)) * kRowB + 8 * (m & 3);
    using Box = TileBox;
    auto box_of = [&](int cl) { return tile_box(tc, cl, p.Wk); };

    uint4 kr0, kr1, vr0, vr1;  // this lane's pieces of the rows in flight
    // a slot past the box's last row (weight 0) reads the box's last row, which the block holds anyway
    auto load = [&](uint32_t key, uint32_t klast) {
        const uint32_t off = min(key, klast) * (2u * D) + 16u * lpiece;
        kr0 = *reinterpret_cast<const uint4*>(Kb + off);
        vr0 = *reinterpret_cast<const uint4*>(Vb + off);
        if constexpr (kPer == 2) {
            kr1 = *reinterpret_cast<const uint4*>(Kb + off + 64);
            vr1 = *reinterpret_cast<const uint4*>(Vb + off + 64);
        }
    };
    auto stage = [&]() {
        const int off = lslot * kRowB + 16 * lpiece;
        *reinterpret_cast<uint4*>(tk + off) = kr0;
        *reinterpret_cast<uint4*>(tv + off) = vr0;
        if constexpr (kPer == 2) {
            *reinterpret_cast<uint4*>(tk + off + 64) = kr1;
            *reinterpret_cast<uint4*>(tv + off + 64) = vr1;
        }
    };
    // this lane's load slot: box column lc and key index lkey (past the box's last row the slots run on
    // into the rows below it, and their keys are clamped to the box's last)
    auto first_slot = [&](const Box& b, int& lc, uint32_t& lkey) {
        int lr;
        box_slot(lslot, b.bw, b.inv, lr, lc);
        lkey = static_cast<uint32_t>(b.r0 + lr) * static_cast<uint32_t>(p.Wk) + (b.c0 + lc);
    };
    auto step_slot = [](const Box& b, int& lc, uint32_t& lkey) {  // 16 slots on
        lc += b.r16;
        const bool carry = lc >= b.bw;
        lc -= carry ? b.bw : 0;
        lkey += carry ? b.kstep_wrap : b.kstep;
    };
    // one block: slot 16 k + 4 g4 of this lane's scores is box row wr0 + rr, column mcl; wc and wc2 are
    // the window's column bits of that row and of the next one (shifted past the row's end), zero outside
    // query m's own cluster
    auto compute = [&](const Box& bx, int rr, int mcl, uint32_t wc, uint32_t wc2, uint32_t wk, uint32_t wk2) {
        // S^T of this block: lane holds keys 4 g4 + i (slots 16 k + 4 g4 + i) for query m
        f32x4_t sc = zero;
#pragma unroll
        for (int ds = 0; ds < kDs; ++ds) {
            const bf16x8_t kf = __builtin_bit_cast(
                bf16x8_t, *reinterpret_cast<const uint4*>(tk + m * kRowB + 16 * (4 * ds + g4)));
            sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ds], sc, 0, 0, 0);
        }
        // which of the 4 slots lie in query m's window (bit i: slot 16 k + 4 g4 + i)
        uint32_t bits;
        if constexpr (JOINT) {
            // rr is the slot's box row: window e's slots when this cluster holds its centre, less those of
            // the query's earlier windows
            bits = 0u;
            uint32_t held = 0u;
#pragma unroll
            for (int e = 0; e < NW; ++e) {
                if (NW > NJ && e / NJ > round) break;  // the windows of later rounds come later
                const uint32_t w = tile_window_bits<false>(bx, rr - jd[e], mcl, jn[e], jx[e], jx[e] << bx.bw);
                bits |= ((hm >> e) & 1u) ? w & ~held : 0u;
                held |= w;
            }
            if constexpr (CAUSAL) bits &= tile_causal_bits(bx, rr, mcl, jqr, jqc);
        } else {
            bits = tile_window_bits<CAUSAL>(bx, rr, mcl, wrn, wc, wc2, tc.rcut, wk, wk2);
            if constexpr (MK > 1) bits &= ~tile_other_bits<kOther, B>(bx, rr, mcl, dw, xw);
        }
        // all ones for the slots of the window, zero elsewhere (one signed bit-field extract each)
        uint32_t keep[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            keep[i] = static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(bits), bit_at[i], 1));
        // the trigger looks at every slot of the block; the exact test at the window's slots only
        if (__ballot((sc[0] > thr) | (sc[1] > thr) | (sc[2] > thr) | (sc[3] > thr))) {
            // some query may pass its reference: the exact test decides
            float mx = -INFINITY;
#pragma unroll
            for (int i = 0; i < 4; ++i) mx = fmaxf(mx, keep[i] ? sc[i] : -INFINITY);
            mx *= sl2e;
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            if (mx > mref + kRescaleSlack) {
                const float alpha = __builtin_amdgcn_exp2f(mref - mx);
                lacc *= alpha;
#pragma unroll
                for (int o = 0; o < kOt; ++o) acc[o] *= alpha;
                mref = mx;
                nref = -mx;
                thr = (mx + (kRescaleSlack - 1.f)) * inv_sl2e;
                if constexpr (MK > 1) thr_q = thr;  // the query's later windows start from here
            }
        }
        uint32_t ph[4], pl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            // exponent of the window's slots; -inf (a weight of 0) elsewhere
            const uint32_t x = __float_as_uint(fmaf(sc[i], sl2e, nref));
            const float pk = __builtin_amdgcn_exp2f(__uint_as_float((x & keep[i]) | (0xFF800000u & ~keep[i])));
            ph[i] = __float_as_uint(pk) & 0xFFFF0000u;
            pl[i] = __float_as_uint(pk - __uint_as_float(ph[i]));
        }
        const bf16x4_t pth =
            __builtin_bit_cast(bf16x4_t, make_uint2(hi16_pair(ph[0], ph[1]), hi16_pair(ph[2], ph[3])));
        const bf16x4_t ptl =
            __builtin_bit_cast(bf16x4_t, make_uint2(hi16_pair(pl[0], pl[1]), hi16_pair(pl[2], pl[3])));
        lacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ones, pth, lacc, 0, 0, 0);
        lacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ones, ptl, lacc, 0, 0, 0);
#pragma unroll
        for (int o = 0; o < kOt; ++o) {
            const bf16x4_t vt = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                (__attribute__((address_space(3))) bf16x4_t*)(tvt + 32 * o));
            acc[o] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, pth, acc[o], 0, 0, 0);
            acc[o] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, ptl, acc[o], 0, 0, 0);
        }
    };

    // The blocks of a cluster are computed in a row; each block's rows load during the previous block's
    // products, the first block of the next cluster during the last block of this one.
    for (int e = 0;;) {
        Box bx = box_of(0);
        int lc;
        uint32_t lkey;
        first_slot(bx, lc, lkey);
        load(lkey, bx.klast);
        for (int c = 0;;) {
            int mr, mcl;
            box_slot(4 * g4, bx.bw, bx.inv, mr, mcl);
            int rr = mr - wr0;
            const bool here = c == mine;
            const uint32_t wc = here ? wcols : 0u;
            const uint32_t wc2 = here ? wcols << bx.bw : 0u;  // bw <= 27, and only bits below bw + 3 are read
            const uint32_t wk = CAUSAL && here ? tc.wcut : 0u;  // the query's own row (causal)
            const uint32_t wk2 = CAUSAL && here ? tc.wcut << bx.bw : 0u;
            bool in = here;
            if constexpr (JOINT) {
                rr = mr;
                hm = 0u;
#pragma unroll
                for (int e = 0; e < NW; ++e) {
                    if (NW > NJ && e / NJ > round) break;
                    jd[e] = ju[e] - B - bx.r0;
                    jn[e] = min(2 * B, bx.h - 1 - jd[e]);
                    // no columns for a window wholly below the box (its row count would be negative)
                    jx[e] = jn[e] >= 0 ? tile_col_bits(jv[e] - B - bx.c0, jv[e] + B - bx.c0, bx.bw) : 0u;
                    // this round's windows whose centre the cluster holds (earlier rounds' hold back keys)
                    hm |= (NW == NJ || e / NJ == round) && c == jmine[e % NJ] ? 1u << e : 0u;
                }
                in = hm != 0u;
                if constexpr (CAUSAL) {
                    jqr = qx - bx.r0;
                    const int qc = qy - bx.c0;
                    jqc = qc < 0 ? 0u : (qc >= bx.bw - 1 ? (1u << bx.bw) - 1u : (2u << qc) - 1u);
                }
            } else if constexpr (MK > 1) {
#pragma unroll
                for (int f = 0; f < kOther; ++f)
                    xw[f] = here && f < e ? tile_col_bits(cv[f] - B - bx.c0, cv[f] + B - bx.c0, bx.bw) : 0u;
            }
            thr = in ? thr_q : INFINITY;  // a query's cluster is visited once per window, its blocks in a row
            step_slot(bx, lc, lkey);
            for (int k = 1; k < bx.nb; ++k) {
                stage();
                load(lkey, bx.klast);
                step_slot(bx, lc, lkey);
                wave_lds_sync();
                compute(bx, rr, mcl, wc, wc2, wk, wk2);
                mcl += bx.r16;
                const bool carry = mcl >= bx.bw;
                mcl -= carry ? bx.bw : 0;
                rr += bx.q16 + (carry ? 1 : 0);
                wave_lds_sync();  // this block's LDS reads come before the next block's writes
            }
            stage();
            const bool more = c + 1 < nclu;
            Box nx = bx;
            if (more) {
                nx = box_of(c + 1);
                first_slot(nx, lc, lkey);
                load(lkey, nx.klast);
            }
            wave_lds_sync();
            compute(bx, rr, mcl, wc, wc2, wk, wk2);
            if (!more) break;
            bx = nx;
            ++c;
            wave_lds_sync();
        }
        if constexpr (MK == 1 || (JOINT && NW == NJ)) {
            break;
        } else if constexpr (JOINT) {
            // the next round: its centres' clusters; the earlier rounds' windows hold back their keys
            if (NJ * (round + 1) >= p.kappa) break;
            ++round;
            joint_round(round);
            nclu = tc.nclu, mine = tc.mine;
            wave_lds_sync();  // the last block's LDS reads come before the next round's writes
        } else {
            if (e + 1 >= p.kappa) break;
            // the next window: its centres' clusters and boxes; window e joins the earlier ones
#pragma unroll
            for (int f = 0; f < kOther; ++f)
                if (f == e) cu[f] = u, cv[f] = v;
            ++e;
            const uint32_t ce = static_cast<uint32_t>(clamp_index(p.J[static_cast<size_t>(e) * p.n + gq], p.nkeys));
            uint32_t uu, vv;
            divmod(ce, p.div_wk, uu, vv);
            u = static_cast<int>(uu);
            v = static_cast<int>(vv);
#pragma unroll
            for (int f = 0; f < kOther; ++f) dw[f] = f < e ? cu[f] - u : 1 << 20;
            tc = tile_clusters<B, CAUSAL>(valid, u, v, m, lane, p.rc, p.Hk, p.Wk, qx, qy);
            nclu = tc.nclu, mine = tc.mine, wr0 = tc.wr0, wrn = tc.wrn;
            wcols = tc.wcols;
            wave_lds_sync();  // the last block's LDS reads come before the next pass's writes
        }
    }
    if (!valid) return;
    const float lt = lacc[0];  // every row of the ones-block product holds query m's sum of weights
    const float inv = lt > 0.f ? __builtin_amdgcn_rcpf(lt) : 0.f;  // (1 ulp: far below the bf16 rounding)
    // lane holds channels 16 o + 4 g4 + i of query m; pairs rounded to bf16 (nearest even) together
    uint16_t* const orow = static_cast<uint16_t*>(p.out) + static_cast<size_t>(g) * D;
    auto bf2 = [](float a, float b) {
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
    };
#pragma unroll
    for (int o = 0; o < kOt; ++o) {
        const uint32_t w0 = bf2(acc[o][0] * inv, acc[o][1] * inv);
        const uint32_t w1 = bf2(acc[o][2] * inv, acc[o][3] * inv);
        *reinterpret_cast<uint2*>(orow + 16 * o + 4 * g4) = make_uint2(w0, w1);
    }
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

// The matrix-core kernel takes bf16 storage with 32 or 64 channels, windows
// of side 3, 5 or 7 (one per map, up to kMaxKappa maps; with or without the
// causal mask), a positive scale and slices of at most 4 GiB of key rows; the
// lane-group kernels take every other call.
#ifndef SCRAM_ATTEND_TILE
#define SCRAM_ATTEND_TILE 1
#endif
template <typename T, int D>
constexpr bool kTileKernel = SCRAM_ATTEND_TILE && std::is_same<T, uint16_t>::value && (D == 32 || D == 64);

template <typename T, int D>
hipError_t run_attend(const AttParams& p0, int window, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kAttend;
    AttParams p = p0;
    if constexpr (kTileKernel<T, D>) {
        if (p.kappa <= kMaxKappa && (window == 3 || window == 5 || window == 7) && p.scale_log2e > 0.f &&
            static_cast<uint64_t>(p.nkeys) * (2 * D) <= 0xFFFFFFFFull) {
            p.tq = make_tiling(p.Hq, p.Wq, kBlock / 4);
            // cluster radius: boxes at most 2 rc + window wide (27 for 7 x 7 windows), so a box's slots stay
            // below 1024 and its two-row column bit fields below 32 bits; 10 measured faster than 4-8 and 11
            p.rc = 10;
            const uint64_t tiles = tiling_blocks(p.tq, p.n / p.tq.plane);
            auto go = [&](auto w) {
                constexpr int Wn = decltype(w)::value;
                // the smallest bound on the windows per query that holds this call's
                auto with = [&](auto mk) {
                    constexpr int MK = decltype(mk)::value;
                    return p.causal ? launch(attend_tile_kernel<D, Wn, true, MK>, tiles, st, e0, e1, p)
                                    : launch(attend_tile_kernel<D, Wn, false, MK>, tiles, st, e0, e1, p);
                };
                return p.kappa == 1   ? with(std::integral_constant<int, 1>{})
                       : p.kappa == 2 ? with(std::integral_constant<int, 2>{})
                       : p.kappa <= 4 ? with(std::integral_constant<int, 4>{})
                                      : with(std::integral_constant<int, kMaxKappa>{});
            };
            return window == 3   ? go(std::integral_constant<int, 3>{})
                   : window == 5 ? go(std::integral_constant<int, 5>{})
                                 : go(std::integral_constant<int, 7>{});
        }
    }
    p.tq = make_tiling(p.Hq, p.Wq, Row<T, D, G>::kQpb, kLaneSkew);
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
        const uint64_t lanes = tiling_blocks(make_tiling(g.Hq, g.Wq, Row<T, D, Lanes<T, D>::kAttend>::kQpb, kLaneSkew), g.S);
        const uint64_t tiles = kTileKernel<T, D> ? tiling_blocks(make_tiling(g.Hq, g.Wq, kBlock / 4), g.S) : 0;
        return lanes > tiles ? lanes : tiles;
    });
}

}  // namespace scram
