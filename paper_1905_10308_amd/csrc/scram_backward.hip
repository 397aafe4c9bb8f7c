// Backward of the sparse window attention with the maps held fixed.

#include "scram_tile.h"

namespace scram {
namespace {

// ---------------------------------------------------------------------------
// K6: backward of the sparse attention, maps held fixed
//
// For query i with key set W_i (as in the forward), p_ij its softmax
// weights, dp_ij = dO_i . v_j and D_i = sum_j p_ij dp_ij:
//   dQ_i = scale sum_j p_ij (dp_ij - D_i) k_j
//   dK_j = scale sum_i p_ij (dp_ij - D_i) q_i,   dV_j = sum_i p_ij dO_i
// Query side (one lane group per query): one walk over W_i accumulates,
// online, the normaliser, D_i and the two sums dQ_i is made of, and stores
// log2 of the normaliser (with the max) and D_i for the key side.  Key side (one lane group
// per key): key j lies in W_i exactly when a match of i lies in the
// (2b+1)^2 neighbourhood of j, so the queries are found through the inverse
// map -- the (query, match) entries sorted by match key (a counting sort:
// the query kernel counts each match key's entries and records each entry's
// slot among them, a scan turns the counts into offsets, and the fill puts
// every entry at its key's offset plus its slot, without atomics).
// The keys of one neighbourhood row are consecutive, so their entries form
// one contiguous range; after the query kernel, q_i, dO_i and the query's
// statistics are copied into entry order, so the key kernel reads each
// range as contiguous rows.  No float atomics: every gradient row has one
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
    int32_t* counts;         // [S * nkeys] entries per match key (zeroed before the query kernel)
    int32_t* slots;          // [kappa * n] each entry's slot among its key's entries
    int32_t* heavy;          // [S * nkeys] keys left to bwd_heavy_kernel
    int32_t* n_heavy;        // their count
    void* qs;                // [kappa * n, D] q_i of each entry, in entry order
    void* gs;                // [kappa * n, D] dO_i of each entry, in entry order
    float2* st;              // [kappa * n] (log2 normaliser, D_i) of each entry
    uint32_t n;
    uint32_t keys_total;   // S * nkeys
    Tiling tq, tk;         // blocks -> tiles of the query grid (query kernel), the key grid (key kernel)
    int Hq, Wq, Hk, Wk;
    uint32_t nkeys;
    Div div_plane, div_wk, div_n, div_keys;
    int b;
    float scale;
    float scale_log2e;
    int kappa;
    int causal;
    int rc;                // cluster radius of the matrix-core query kernel
};

// a[0 .. count) = 0 and, when given, *word = 0
__global__ __launch_bounds__(kBlock) void zero_i32_kernel(int32_t* a, size_t count, int32_t* word)
{
    for (size_t i = static_cast<size_t>(blockIdx.x) * kBlock + threadIdx.x; i < count;
         i += static_cast<size_t>(gridDim.x) * kBlock)
        a[i] = 0;
    if (word != nullptr && blockIdx.x == 0 && threadIdx.x == 0) *word = 0;
}

// Exclusive scan of in[0 .. count) by one block, count <= kScanTile, into
// out (which may be in, in global or shared memory); returns the total to
// thread kBlock - 1.  wave_tot: kBlock / 64 ints of shared memory.
__device__ int32_t block_exclusive_scan(const int32_t* in, int32_t* out, size_t count, int32_t* wave_tot)
{
    const size_t base = static_cast<size_t>(threadIdx.x) * kScanItems;
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
    return before + run;
}

// Exclusive scan, step 1: each block scans a tile of kScanTile counts into
// out (tile-local prefixes; out may be in) and writes the tile's total to
// sums[tile].
__global__ __launch_bounds__(kBlock) void scan_tiles_kernel(const int32_t* in, int32_t* out, int32_t* sums,
                                                            size_t count)
{
    __shared__ int32_t wave_tot[kBlock / 64];
    const size_t base = static_cast<size_t>(blockIdx.x) * kScanTile;
    const int32_t tot = block_exclusive_scan(in + base, out + base, count - base < kScanTile ? count - base : kScanTile,
                                             wave_tot);
    if (threadIdx.x == kBlock - 1) sums[blockIdx.x] = tot;
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

// The inverse map from the scan: key k's entries start at
// offsets[k] = local[k] + pre[k / kScanTile] (local: tile-local exclusive
// prefixes of the counts, pre: exclusive prefixes of the tile totals, the
// grand total in pre[tiles]), and entry x goes to its key's start plus the
// slot the count recorded for it.  OWN_SCAN (tiles <= kScanTile): sums holds
// the raw tile totals and every block scans them into shared memory itself;
// otherwise scan_sums_kernel has turned sums into pre.
template <bool OWN_SCAN>
__global__ __launch_bounds__(kBlock) void bwd_fill_kernel(BwdParams p, const int32_t* local, const int32_t* sums,
                                                          uint32_t tiles, int32_t* offsets, int32_t* entries)
{
    __shared__ int32_t s_pre[OWN_SCAN ? kScanTile + 1 : 1];
    __shared__ int32_t wave_tot[kBlock / 64];
    const int32_t* pre = sums;
    if constexpr (OWN_SCAN) {
        const int32_t tot = block_exclusive_scan(sums, s_pre, tiles, wave_tot);
        if (threadIdx.x == kBlock - 1) s_pre[tiles] = tot;
        __syncthreads();
        pre = s_pre;
    }
    const size_t stride = static_cast<size_t>(gridDim.x) * kBlock;
    const size_t first = static_cast<size_t>(blockIdx.x) * kBlock + threadIdx.x;
    const size_t total = static_cast<size_t>(p.kappa) * p.n;
    for (size_t x = first; x < total; x += stride) {
        const uint32_t g = static_cast<uint32_t>(x % p.n);
        uint32_t s, rem;
        divmod(g, p.div_plane, s, rem);
        const size_t key = static_cast<size_t>(s) * p.nkeys + clamp_index(p.J[x], p.nkeys);
        entries[local[key] + pre[key / kScanTile] + p.slots[x]] = static_cast<int32_t>(x);
    }
    for (size_t k = first; k < p.keys_total; k += stride) offsets[k] = local[k] + pre[k / kScanTile];
    if (first == 0) offsets[p.keys_total] = pre[tiles];
}

// W > 0: window side W (odd), visited one window row at a time with its W
// key and W value rows loaded together (as the forward's window kernel);
// W = 0: any side, kNb keys at a time in row order.
template <typename T, int D, int G, bool MULTI, int W>
__global__ __launch_bounds__(kBlock) void bwd_query_kernel(BwdParams p)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;
    constexpr int kEpc = RW::kEpc;
    constexpr int kNb = CH >= 2 ? 2 : 4;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    uint32_t g;
    if (!tile_item<RW::kQpb>(p.tq, blk, threadIdx.x / G, g)) return;

    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);
    // the inverse map's count: one entry per match of this query, and its
    // slot among the entries of that match key
    if (lane == 0) {
        for (int e = 0; e < (MULTI ? p.kappa : 1); ++e) {
            const size_t x = static_cast<size_t>(e) * p.n + g;
            p.slots[x] = atomicAdd(p.counts + static_cast<size_t>(s) * p.nkeys + clamp_index(p.J[x], p.nkeys), 1);
        }
    }
    const size_t slice = static_cast<size_t>(s) * p.nkeys * D;
    const T* Ks = static_cast<const T*>(p.K) + slice;
    const T* Vs = static_cast<const T*>(p.V) + slice;
    uint4 q[CH], go[CH];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    load_row<T, D, G>(static_cast<const T*>(p.dO), g, lane, go);
    WindowSet<kMaxKappa> wset;
    if constexpr (MULTI) wset = make_window_set<kMaxKappa>(p, g, rem);
    const int nsets = MULTI ? p.kappa : 1;

    // visit(fn): every key of the set, kNb at a time with their key and
    // value rows loaded together; fn(ok[], kr, vr) per batch
    auto visit = [&](auto&& fn) {
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
            if constexpr (W > 0) {
                constexpr int B = W / 2;
                int cols[W];
                bool col_ok[W];
#pragma unroll
                for (int cc = 0; cc < W; ++cc) {
                    const int col = static_cast<int>(v) + cc - B;
                    col_ok[cc] = col >= 0 && col < p.Wk;
                    cols[cc] = min(max(col, 0), p.Wk - 1);
                }
                for (int a = 0; a < W; ++a) {
                    const int rr = static_cast<int>(u) + a - B;
                    if (rr < 0 || rr >= p.Hk) continue;
                    bool ok[W];
                    bool any = false;
#pragma unroll
                    for (int cc = 0; cc < W; ++cc) {
                        ok[cc] = col_ok[cc];
                        if constexpr (MULTI) ok[cc] = ok[cc] && !wset.skip(e, rr, cols[cc]);
                        any = any || ok[cc];
                    }
                    if (!any) continue;
                    uint4 kr[W][CH], vr[W][CH];
#pragma unroll
                    for (int cc = 0; cc < W; ++cc) {
                        load_row<T, D, G>(Ks, static_cast<uint32_t>(rr * p.Wk + cols[cc]), lane, kr[cc]);
                        load_row<T, D, G>(Vs, static_cast<uint32_t>(rr * p.Wk + cols[cc]), lane, vr[cc]);
                    }
                    fn(ok, kr, vr);
                }
                continue;
            }
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

    // One pass, online in the base-2 domain: running max m, normaliser l,
    // dn = sum e^(a - m) dp, and with k~ = k_j - k_ref the sums
    // A = sum e^(a - m) dp k~ and B = sum e^(a - m) k~.  Since the weights of
    // the set sum to one, dQ_i = scale (A - D_i B) / l for any fixed k_ref;
    // k_ref = the key at the first match keeps k~ small where neighbouring
    // keys are alike, so A - D_i B does not cancel, and a one-key set gives
    // exactly zero.
    float kref[E];
    {
        uint4 kr0[CH];
        load_row<T, D, G>(Ks, clamp_index(p.J[g], p.nkeys), lane, kr0);
        unpack_row<T, CH>(kr0, kref);
    }
    float m = -INFINITY, l = 0.f, dn = 0.f;
    float acc_a[E], acc_b[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc_a[e] = acc_b[e] = 0.f;
    visit([&](const auto& ok, const auto& kr, const auto& vr) {
        constexpr int kNb = std::extent<std::remove_reference_t<decltype(ok)>>::value;
        float sc[kNb], dp[kNb];
        float mb = m;
#pragma unroll
        for (int j = 0; j < kNb; ++j) {
            sc[j] = ok[j] ? row_score<T, D, G>(q, kr[j]) * p.scale_log2e : -INFINITY;
            dp[j] = row_score<T, D, G>(go, vr[j]);
            mb = fmaxf(mb, sc[j]);
        }
        if (mb == -INFINITY) return;
        if (mb > m + kRescaleSlack) {
            const float alpha = __builtin_amdgcn_exp2f(m - mb);
            l *= alpha;
            dn *= alpha;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                acc_a[e] *= alpha;
                acc_b[e] *= alpha;
            }
            m = mb;
        }
#pragma unroll
        for (int j = 0; j < kNb; ++j) {
            const float pj = __builtin_amdgcn_exp2f(sc[j] - m);  // 0 when !ok
            const float pd = pj * dp[j];
            l += pj;
            dn += pd;
            float kf[E];
            unpack_row<T, CH>(kr[j], kf);
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float kd = kf[e] - kref[e];
                acc_a[e] = fmaf(pd, kd, acc_a[e]);
                acc_b[e] = fmaf(pj, kd, acc_b[e]);
            }
        }
    });
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const float Dg = dn * inv;
    if (lane == 0) {
        p.lse2[g] = l > 0.f ? m + log2f(l) : INFINITY;  // +inf: every weight is 0
        p.Dq[g] = Dg;
    }
    float dq[E];
#pragma unroll
    for (int e = 0; e < E; ++e) dq[e] = (acc_a[e] - Dg * acc_b[e]) * inv;
#pragma unroll
    for (int cc = 0; cc < CH; ++cc) {
        float4* o = reinterpret_cast<float4*>(p.dQ + static_cast<size_t>(g) * D + (cc * G + lane) * kEpc);
#pragma unroll
        for (int i = 0; i < kEpc / 4; ++i)
            o[i] = make_float4(dq[cc * kEpc + 4 * i] * p.scale, dq[cc * kEpc + 4 * i + 1] * p.scale,
                               dq[cc * kEpc + 4 * i + 2] * p.scale, dq[cc * kEpc + 4 * i + 3] * p.scale);
    }
}

// Copy q_i, dO_i and (log2 normaliser, D_i) of every entry into entry order.
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void bwd_gather_kernel(BwdParams p)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    const int lane = threadIdx.x & (G - 1);
    const uint32_t x = blockIdx.x * RW::kQpb + threadIdx.x / G;
    if (x >= static_cast<uint32_t>(p.kappa) * p.n) return;
    uint32_t e, g;
    divmod(static_cast<uint32_t>(p.entries[x]), p.div_n, e, g);
    uint4 q[CH], go[CH];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    load_row<T, D, G>(static_cast<const T*>(p.dO), g, lane, go);
    uint4* qd = reinterpret_cast<uint4*>(static_cast<T*>(p.qs) + static_cast<size_t>(x) * D) + lane;
    uint4* gd = reinterpret_cast<uint4*>(static_cast<T*>(p.gs) + static_cast<size_t>(x) * D) + lane;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        qd[c * G] = q[c];
        gd[c * G] = go[c];
    }
    if (lane == 0) p.st[x] = make_float2(p.lse2[g], p.Dq[g]);
}

// Contributions of kNb entries (slots x[t], valid where ok[t]) to dK_j, dV_j
// (unscaled dK) for key j at (ju, jv): each query once -- through its first
// window holding j -- and, with the causal mask, only if j is not after it.
template <typename T, int D, int G, bool MULTI, int kNb>
__device__ __forceinline__ void key_batch(const BwdParams& p, const int (&x)[kNb], const bool (&valid)[kNb], uint32_t j,
                                          uint32_t ju, uint32_t jv, int lane, const uint4 (&kj)[Row<T, D, G>::kCh],
                                          const uint4 (&vj)[Row<T, D, G>::kCh], float* dk, float* dv)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;
    const T* qs = static_cast<const T*>(p.qs);
    const T* gs = static_cast<const T*>(p.gs);
    uint4 qr[kNb][CH], gr[kNb][CH];
    float2 st[kNb];
    int32_t code[kNb];
#pragma unroll
    for (int t = 0; t < kNb; ++t) {
        code[t] = p.entries[x[t]];
        st[t] = p.st[x[t]];
        load_row<T, D, G>(qs, static_cast<uint32_t>(x[t]), lane, qr[t]);
        load_row<T, D, G>(gs, static_cast<uint32_t>(x[t]), lane, gr[t]);
    }
#pragma unroll
    for (int t = 0; t < kNb; ++t) {
        bool ok = valid[t];
        if constexpr (MULTI) {
            uint32_t e, g;
            divmod(static_cast<uint32_t>(code[t]), p.div_n, e, g);
            for (int f = 0; f < static_cast<int>(e) && ok; ++f) {
                uint32_t fu, fv;
                divmod(static_cast<uint32_t>(clamp_index(p.J[static_cast<size_t>(f) * p.n + g], p.nkeys)), p.div_wk,
                       fu, fv);
                if (abs(static_cast<int>(fu) - static_cast<int>(ju)) <= p.b &&
                    abs(static_cast<int>(fv) - static_cast<int>(jv)) <= p.b)
                    ok = false;
            }
            if (ok && p.causal) {
                uint32_t gsl, grem;
                divmod(g, p.div_plane, gsl, grem);
                ok = j <= grem;
            }
        }
        const float sc = row_score<T, D, G>(qr[t], kj) * p.scale_log2e;
        const float dp = row_score<T, D, G>(gr[t], vj);
        const float pj = ok ? __builtin_amdgcn_exp2f(sc - st[t].x) : 0.f;
        const float ds = pj * (dp - st[t].y);
        float qf[E], gf[E];
        unpack_row<T, CH>(qr[t], qf);
        unpack_row<T, CH>(gr[t], gf);
#pragma unroll
        for (int e2 = 0; e2 < E; ++e2) {
            dk[e2] = fmaf(ds, qf[e2], dk[e2]);
            dv[e2] = fmaf(pj, gf[e2], dv[e2]);
        }
    }
}

// Keys whose neighbourhood holds more entries than this are handed to
// bwd_heavy_kernel (a team of lane groups per key) instead of one lane group.
#ifndef SCRAM_BWD_HEAVY_ENTRIES
#define SCRAM_BWD_HEAVY_ENTRIES 64
#endif
constexpr int kHeavyEntries = SCRAM_BWD_HEAVY_ENTRIES;
constexpr int kMaxRows = 8;
// Lane groups that share one heavy key (half a wave at four lanes per group).
#ifndef SCRAM_BWD_TEAM
#define SCRAM_BWD_TEAM 8
#endif  // neighbourhoods of up to this many rows are walked as one flat list

// The entry ranges of the neighbourhood rows r0..r1 of key j: row i covers
// entries [lo[i], lo[i] + pre[i+1] - pre[i]); pre[] is the running count.
struct Neighbourhood {
    int lo[kMaxRows];
    int pre[kMaxRows + 1];
    int total;
};

__device__ __forceinline__ Neighbourhood load_neighbourhood(const int32_t* off, int Wk, int r0, int r1, int c0, int c1)
{
    Neighbourhood nb;
    nb.pre[0] = 0;
#pragma unroll
    for (int i = 0; i < kMaxRows; ++i) {
        int lo = 0, len = 0;
        if (r0 + i <= r1) {
            lo = off[(r0 + i) * Wk + c0];
            len = off[(r0 + i) * Wk + c1 + 1] - lo;
        }
        nb.lo[i] = lo;
        nb.pre[i + 1] = nb.pre[i] + len;
    }
    nb.total = nb.pre[kMaxRows];
    return nb;
}

// Entry slot of flat position v (0 <= v < total): the last row with pre <= v.
__device__ __forceinline__ int flat_slot(const Neighbourhood& nb, int v)
{
    int x = nb.lo[0] + v;
#pragma unroll
    for (int i = 1; i < kMaxRows; ++i)
        if (v >= nb.pre[i]) x = nb.lo[i] + (v - nb.pre[i]);
    return x;
}

// Accumulate the entries of key j's neighbourhood taken by member `member`
// of a team of `team` lane groups (positions member, member + team, ...).
template <typename T, int D, int G, bool MULTI>
__device__ __forceinline__ void key_accumulate(const BwdParams& p, uint32_t j, uint32_t ju, uint32_t jv, int r0,
                                               int r1, int c0, int c1, const int32_t* off, int member, int team,
                                               int lane, const uint4 (&kj)[Row<T, D, G>::kCh],
                                               const uint4 (&vj)[Row<T, D, G>::kCh], float* dk, float* dv)
{
    constexpr int kNb = Row<T, D, G>::kCh >= 2 ? 2 : 4;
    if (r1 - r0 + 1 <= kMaxRows) {
        const Neighbourhood nb = load_neighbourhood(off, p.Wk, r0, r1, c0, c1);
        for (int v0 = member; v0 < nb.total; v0 += kNb * team) {
            int x[kNb];
            bool valid[kNb];
#pragma unroll
            for (int t = 0; t < kNb; ++t) {
                const int v = v0 + t * team;
                valid[t] = v < nb.total;
                x[t] = flat_slot(nb, min(v, nb.total - 1));  // in bounds; invalid slots get weight 0
            }
            key_batch<T, D, G, MULTI, kNb>(p, x, valid, j, ju, jv, lane, kj, vj, dk, dv);
        }
    } else {
        for (int r = r0; r <= r1; ++r) {
            const int lo = off[r * p.Wk + c0], hi = off[r * p.Wk + c1 + 1];
            for (int x0 = lo + member; x0 < hi; x0 += kNb * team) {
                int x[kNb];
                bool valid[kNb];
#pragma unroll
                for (int t = 0; t < kNb; ++t) {
                    valid[t] = x0 + t * team < hi;
                    x[t] = min(x0 + t * team, hi - 1);
                }
                key_batch<T, D, G, MULTI, kNb>(p, x, valid, j, ju, jv, lane, kj, vj, dk, dv);
            }
        }
    }
}

// dK_j (times scale) and dV_j from the lane's channels.
template <typename T, int D, int G>
__device__ __forceinline__ void store_key_grads(const BwdParams& p, uint32_t kg, int lane, const float* dk,
                                                const float* dv)
{
    constexpr int CH = Row<T, D, G>::kCh;
    constexpr int kEpc = Row<T, D, G>::kEpc;
#pragma unroll
    for (int cc = 0; cc < CH; ++cc) {
        float4* ok = reinterpret_cast<float4*>(p.dK + static_cast<size_t>(kg) * D + (cc * G + lane) * kEpc);
        float4* ov = reinterpret_cast<float4*>(p.dV + static_cast<size_t>(kg) * D + (cc * G + lane) * kEpc);
#pragma unroll
        for (int i = 0; i < kEpc / 4; ++i) {
            const int e0 = cc * kEpc + 4 * i;
            ok[i] = make_float4(dk[e0] * p.scale, dk[e0 + 1] * p.scale, dk[e0 + 2] * p.scale, dk[e0 + 3] * p.scale);
            ov[i] = make_float4(dv[e0], dv[e0 + 1], dv[e0 + 2], dv[e0 + 3]);
        }
    }
}

struct KeyPos {
    uint32_t s, j, ju, jv;
    int r0, r1, c0, c1;
};

__device__ __forceinline__ KeyPos key_pos(const BwdParams& p, uint32_t kg)
{
    KeyPos k;
    divmod(kg, p.div_keys, k.s, k.j);
    divmod(k.j, p.div_wk, k.ju, k.jv);
    k.r0 = max(static_cast<int>(k.ju) - p.b, 0);
    k.r1 = min(static_cast<int>(k.ju) + p.b, p.Hk - 1);
    k.c0 = max(static_cast<int>(k.jv) - p.b, 0);
    k.c1 = min(static_cast<int>(k.jv) + p.b, p.Wk - 1);
    return k;
}

// One lane group per key j: sum over the entries (i, e) whose match e lies
// in the neighbourhood of j (so j is in window e of i).  Keys with more than
// kHeavyEntries entries are appended to the heavy list instead.  The block
// ranks its tile's keys by entry count and hands them out in that order, so
// the keys of one wave carry similar work (a wave lasts as long as its
// busiest lane group).
template <typename T, int D, int G, bool MULTI>
__global__ __launch_bounds__(kBlock) void bwd_key_kernel(BwdParams p)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;
    constexpr int kKeys = RW::kQpb;  // keys of the block's tile
    __shared__ int32_t s_total[kKeys], s_key[kKeys], s_order[kKeys];
    const int lane = threadIdx.x & (G - 1);
    const int grp = threadIdx.x / G;
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    {
        // the tile's keys and their entry counts; -1: past the grid's edge or heavy
        uint32_t kg0;
        int total = -1;
        if (tile_item<RW::kQpb>(p.tk, blk, grp, kg0)) {
            const KeyPos k0 = key_pos(p, kg0);
            const int32_t* off0 = p.offsets + static_cast<size_t>(k0.s) * p.nkeys;
            total = 0;
            for (int r = k0.r0; r <= k0.r1; ++r) total += off0[r * p.Wk + k0.c1 + 1] - off0[r * p.Wk + k0.c0];
            if (total > kHeavyEntries) {
                if (lane == 0) p.heavy[atomicAdd(p.n_heavy, 1)] = static_cast<int32_t>(kg0);
                total = -1;
            }
        }
        if (lane == 0) {
            s_total[grp] = total;
            s_key[grp] = static_cast<int32_t>(kg0);
        }
    }
    __syncthreads();
    {
        // rank by entry count, most first (ties by position), so each wave takes keys of similar work
        const int mine = s_total[grp];
        int rank = 0;
        for (int i = 0; i < kKeys; ++i) {
            const int other = s_total[i];
            rank += (other > mine || (other == mine && i < grp)) ? 1 : 0;
        }
        if (lane == 0) s_order[rank] = grp;
    }
    __syncthreads();
    const int src = s_order[grp];
    if (s_total[src] < 0) return;
    const uint32_t kg = static_cast<uint32_t>(s_key[src]);  // global key id s * nkeys + j
    const KeyPos k = key_pos(p, kg);
    const int32_t* off = p.offsets + static_cast<size_t>(k.s) * p.nkeys;
    uint4 kj[CH], vj[CH];
    load_row<T, D, G>(static_cast<const T*>(p.K), kg, lane, kj);
    load_row<T, D, G>(static_cast<const T*>(p.V), kg, lane, vj);
    float dk[E], dv[E];
#pragma unroll
    for (int e = 0; e < E; ++e) dk[e] = dv[e] = 0.f;
    key_accumulate<T, D, G, MULTI>(p, k.j, k.ju, k.jv, k.r0, k.r1, k.c0, k.c1, off, 0, 1, lane, kj, vj, dk, dv);
    store_key_grads<T, D, G>(p, kg, lane, dk, dv);
}

// The heavy keys, one team of SCRAM_BWD_TEAM lane groups each (teams take
// keys w, w + total teams, ...): the team's lane groups stride over the
// key's entries and their partial sums are added across the team with xor
// shuffles.
template <typename T, int D, int G, bool MULTI>
__global__ __launch_bounds__(kBlock) void bwd_heavy_kernel(BwdParams p)
{
    using RW = Row<T, D, G>;
    constexpr int CH = RW::kCh;
    constexpr int E = CH * RW::kEpc;
    constexpr int kTeam = SCRAM_BWD_TEAM * G <= 64 ? SCRAM_BWD_TEAM : 64 / G;  // lane groups per key
    constexpr int kTeamLanes = kTeam * G;
    const int lane = threadIdx.x & (G - 1);
    const int member = (threadIdx.x & (kTeamLanes - 1)) / G;
    const int wave = blockIdx.x * (kBlock / kTeamLanes) + threadIdx.x / kTeamLanes;
    const int waves = gridDim.x * (kBlock / kTeamLanes);
    const int n_heavy = *p.n_heavy;
    for (int h = wave; h < n_heavy; h += waves) {
        const uint32_t kg = static_cast<uint32_t>(p.heavy[h]);
        const KeyPos k = key_pos(p, kg);
        const int32_t* off = p.offsets + static_cast<size_t>(k.s) * p.nkeys;
        uint4 kj[CH], vj[CH];
        load_row<T, D, G>(static_cast<const T*>(p.K), kg, lane, kj);
        load_row<T, D, G>(static_cast<const T*>(p.V), kg, lane, vj);
        float dk[E], dv[E];
#pragma unroll
        for (int e = 0; e < E; ++e) dk[e] = dv[e] = 0.f;
        key_accumulate<T, D, G, MULTI>(p, k.j, k.ju, k.jv, k.r0, k.r1, k.c0, k.c1, off, member, kTeam, lane, kj, vj,
                                       dk, dv);
#pragma unroll
        for (int m = G; m < kTeamLanes; m <<= 1)
#pragma unroll
            for (int e = 0; e < E; ++e) {
                dk[e] += __shfl_xor(dk[e], m);
                dv[e] += __shfl_xor(dv[e], m);
            }
        if (member == 0) store_key_grads<T, D, G>(p, kg, lane, dk, dv);
    }
}

// ---------------------------------------------------------------------------
// Key side on the matrix cores (bf16 storage).  Each wave takes a strip of 16
// keys of a 64-key tile (a 4 x 4 quarter of an 8 x 8 tile; items 16 w .. 16 w
// + 15 in raster order of flatter or taller tiles) and works alone, a block
// of its own: the number of entries
// per strip is very uneven, and a wave that finishes releases its LDS at once
// instead of holding it until the slowest strip of a shared block is done.  The
// queries whose key sets reach the strip are exactly the entries whose match
// lies in the strip's halo (the strip widened by b), one contiguous entry
// range per halo row.  Per chunk of 32 of those entries, staged in the wave's
// own LDS (q and dO rows, match, log2 normaliser, D), on the matrix cores
//   S^T = Q_E K_w^T,  dP^T = dO_E V_w^T                 (entries x keys),
// in registers P = window test ? 2^(S scale log2 e - lse2) : 0 and
// dS = P (dP - D), and again on the matrix cores
//   dV_w += P dO_E,   dK_w += dS Q_E                    (keys x channels).
// The output layout of the first products (lane l: key l mod 16 and four
// entries) is the operand layout of the second, so P and dS never leave
// registers (the entries' order along the contraction only has to agree
// between the two operands).  The channel-major operands dO_E, Q_E of the
// second products come from the staged rows through the transposing LDS load.
// P and dS enter as three bf16 parts that add up to the fp32 values exactly
// (products of bf16 parts are exact); all sums are fp32.
// ---------------------------------------------------------------------------
constexpr int kTileKeys = 64;                          // keys per block, 16 per wave
constexpr int kTileMaxB = 7;                           // windows up to 15 x 15
constexpr int kStripMaxRows = 16 + 2 * kTileMaxB;      // halo rows of the tallest strip (16 x 1)
constexpr int kStripCE = 32;                           // entries per chunk: one contraction step

template <int D>
struct KeyStrip {
    static constexpr int kRowB = 2 * D + 16;           // row stride in LDS, bytes (padded)
    static constexpr int kDs = D >= 32 ? D / 32 : 1;   // 32-channel steps of the first products
    static constexpr int kOt = D / 16;                 // 16-channel tiles of dK_w, dV_w
    static constexpr int kPieces = D / 8;              // 16-byte pieces per row
};

// The strip kernel's key-set tests: the window only, the window and the causal mask (one map), or
// several windows (and the causal mask if asked for).
enum StripMode { kStripPlain = 0, kStripCausal = 1, kStripMulti = 2 };

// waves per SIMD the strip kernel's registers are sized for
constexpr int strip_waves(int D) { return D > 64 ? 2 : 4; }

// x = hi + mid + lo exactly, each part a bf16 value held as an fp32 bit
// pattern with a zero low half: hi keeps the top 8 significant bits of x
// (truncation), x - hi is exact in fp32 and mid keeps its top 8, and the
// remaining lo has at most 8 significant bits (x has 24).
__device__ __forceinline__ void split3(float x, uint32_t& hi, uint32_t& mid, uint32_t& lo)
{
    hi = __float_as_uint(x) & 0xFFFF0000u;
    const float r1 = x - __uint_as_float(hi);
    mid = __float_as_uint(r1) & 0xFFFF0000u;
    lo = __float_as_uint(r1 - __uint_as_float(mid));
}

__device__ __forceinline__ bf16x8_t lds_frag(const unsigned char* p)
{
    return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(p));
}

constexpr int kStripWaves = kTileKeys / 16;  // strips of a tile, one one-wave block each

template <int D, int MODE>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(strip_waves(D)))) void
bwd_key_strip_kernel(BwdParams p)
{
    constexpr bool MULTI = MODE == kStripMulti;
    constexpr bool kQueryIndex = MODE != kStripPlain;  // entries carry their window and query's raster index
    using KS = KeyStrip<D>;
    constexpr int kCE = kStripCE;
    constexpr int kW = 1;  // waves per block
    // q rows of the chunk, then 64 bytes of skew, then its dO rows: lanes 2t and 2t + 1 stage row t of
    // each; with the skew the eight lanes of one 128-bit access (rows t .. t + 3 of both) use disjoint
    // halves of the 32 banks, without it the two rows of each pair share banks
    __shared__ __align__(16) unsigned char s_row[kW][2 * kCE * KS::kRowB + 64];
    __shared__ int4 s_meta[kW][kCE];        // match row, match column, lse2 bits, D bits
    // several windows: the strip's keys that one of the entry query's earlier windows holds (bit k: key
    // k); causal: the query's raster index
    __shared__ int32_t s_el[kW][kQueryIndex ? kCE : 1][2];
    __shared__ int32_t s_lo[kW][kStripMaxRows], s_pre[kW][kStripMaxRows + 1];

    const int lane = threadIdx.x & 63, wave = 0;
    const int m = lane & 15, g4 = lane >> 4;
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);

    // the tile (th x tw keys at x0, y0 of slice s) and this wave's strip in it
    uint32_t s, k, tr, tc;
    divmod(blk / kStripWaves, p.tk.div_slice, s, k);
    tile_coords(p.tk, k, tr, tc);
    const int tw = 1 << p.tk.lw, th = kTileKeys >> p.tk.lw;
    const int x0 = static_cast<int>(tr) * th, y0 = static_cast<int>(tc) * tw;
    const int w4 = static_cast<int>(blk % kStripWaves);
    // the strip: a 4 x 4 quarter of an 8 x 8 tile (its halo holds 11 % fewer match positions than that
    // of 2 rows of 8), else items 16 w4 .. 16 w4 + 15 of the tile in raster order; key i of the strip
    const bool quad = p.tk.lw == 3 && th == 8;
    const int it0 = 16 * w4;
    const int sr0 = quad ? x0 + 4 * (w4 >> 1) : x0 + (it0 >> p.tk.lw);
    const int sr1 = quad ? sr0 + 3 : x0 + ((it0 + 15) >> p.tk.lw);
    const int sc0 = quad ? y0 + 4 * (w4 & 1) : y0 + (it0 & (tw - 1));
    const int sc1 = quad ? sc0 + 3 : sc0 + min(tw, 16) - 1;
    auto strip_key = [&](int i, int& x, int& y) {
        x = quad ? sr0 + (i >> 2) : x0 + ((it0 + i) >> p.tk.lw);
        y = quad ? sc0 + (i & 3) : y0 + ((it0 + i) & (tw - 1));
    };
    // the strip is a rectangle: key i at row sr0 + i / sC, column sc0 + i mod sC.  Bits of the keys in
    // rows rlo .. rhi, columns clo .. chi (relative to the strip's first row and column)
    const int sC = sc1 - sc0 + 1, sR = 16 / sC;
    auto strip_bits = [&](int rlo, int rhi, int clo, int chi) {
        rlo = max(rlo, 0), rhi = min(rhi, sR - 1), clo = max(clo, 0), chi = min(chi, sC - 1);
        uint32_t bits = 0u;
        if (clo <= chi) {
            const uint32_t cb = ((2u << chi) - 1u) & ~((1u << clo) - 1u);
            for (int r = rlo; r <= rhi; ++r) bits |= cb << (sC * r);
        }
        return bits;
    };
    if (sr0 >= p.Hk || sc0 >= p.Wk) return;  // the strip lies past the grid's edge
    const int hr0 = max(sr0 - p.b, 0), hr1 = min(sr1 + p.b, p.Hk - 1);
    const int hc0 = max(sc0 - p.b, 0), hc1 = min(sc1 + p.b, p.Wk - 1);
    const int nrows = hr1 - hr0 + 1;  // at most kStripMaxRows
    const int32_t* off = p.offsets + static_cast<size_t>(s) * p.nkeys;
    int32_t* const lo_w = s_lo[wave];
    int32_t* const pre_w = s_pre[wave];
    int E;
    {
        // entry count of halo row `lane`, then an inclusive scan across the wave
        int cnt = 0;
        if (lane < nrows) {
            const int r = hr0 + lane;
            const int32_t lo = off[r * p.Wk + hc0];
            lo_w[lane] = lo;
            cnt = off[r * p.Wk + hc1 + 1] - lo;
        }
        int incl = cnt;
#pragma unroll
        for (int k2 = 1; k2 < 64; k2 <<= 1) {
            const int y = __shfl_up(incl, k2, 64);
            if (lane >= k2) incl += y;
        }
        if (lane < nrows) pre_w[lane + 1] = incl;
        if (lane == 0) pre_w[0] = 0;
        E = __shfl(incl, nrows - 1, 64);
    }
    wave_lds_sync();

    // this lane's key (column of the first products): key m of the strip
    int kx, ky;
    strip_key(m, kx, ky);
    const bool key_ok = kx < p.Hk && ky < p.Wk;
    const size_t kslice = static_cast<size_t>(s) * p.nkeys;
    const size_t krow = kslice + (key_ok ? static_cast<size_t>(kx) * p.Wk + ky : static_cast<size_t>(sr0) * p.Wk + sc0);
    bf16x8_t kf[KS::kDs], vf[KS::kDs];
#pragma unroll
    for (int ds = 0; ds < KS::kDs; ++ds) {
        const int d = 32 * ds + 8 * g4;
        uint4 kw = make_uint4(0u, 0u, 0u, 0u), vw = kw;
        if (d < D) {
            kw = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p.K) + krow * D + d);
            vw = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p.V) + krow * D + d);
        }
        kf[ds] = __builtin_bit_cast(bf16x8_t, kw);
        vf[ds] = __builtin_bit_cast(bf16x8_t, vw);
    }
    const uint32_t key_local = static_cast<uint32_t>(kx) * p.Wk + ky;  // raster index (causal test)

    f32x4_t dk[KS::kOt], dv[KS::kOt];
#pragma unroll
    for (int o = 0; o < KS::kOt; ++o) dk[o] = dv[o] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // staging: lane pair (2 t, 2 t + 1) finds entry slot t; the even lane brings its statistics
    const int t = lane >> 1, hf = lane & 1;
    const uint16_t* const Qb = static_cast<const uint16_t*>(p.Q);
    const uint16_t* const Gb = static_cast<const uint16_t*>(p.dO);
    auto slot_code = [&](int c0) {
        const int v = c0 + t;
        if (v >= E) return -1;
        int lo = 0, hi = nrows - 1;  // halo row holding flat position v: the last with pre <= v
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (pre_w[mid] <= v) lo = mid; else hi = mid - 1;
        }
        return static_cast<int>(p.entries[lo_w[lo] + (v - pre_w[lo])]);
    };
    unsigned char* const rows_q = s_row[wave];
    unsigned char* const rows_g = s_row[wave] + kCE * KS::kRowB + 64;
    // B operands of the second products, channel tile o: lane (n, g4) holds entries 4 g4 .. 4 g4 + 3 and
    // 16 + 4 g4 .. 16 + 4 g4 + 3 at channel 16 o + n.  The transposing LDS load hands lane (n, g4) rows
    // 4 g4 .. 4 g4 + 3 at channel 16 o + n when it addresses row 4 g4 + n / 4 at channels 4 (n mod 4) .. + 3
    // (+ 16 o); a second load 16 rows further gives the other four.
    const int tr_off = (4 * g4 + (m >> 2)) * KS::kRowB + 8 * (m & 3);
    auto tr_pair = [&](const unsigned char* a) {
        using lds_v4 = __attribute__((address_space(3))) bf16x4_t*;
        const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_v4)(a));
        const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_v4)(a + 16 * KS::kRowB));
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    };
    int code = slot_code(0);
    for (int c0 = 0; c0 < E; c0 += kCE) {
        {
            uint32_t qe = 0, qg = 0;
            if (code >= 0) divmod(static_cast<uint32_t>(code), p.div_n, qe, qg);
            int32_t match = -1;
            float lse = 0.f, dq = 0.f;
            if (hf == 0 && code >= 0) {
                match = p.J[code];
                lse = p.lse2[qg];
                dq = p.Dq[qg];
            }
            // the chunk's q and dO rows, kLR consecutive lanes per row (whole spans per load): lane l
            // brings pieces l mod kLR (+ kLR ...) of entry slots l / kLR + kRpi j; entry slot e's query
            // comes from lane 2 e (-1: past the entries, a zero row keeps the operands finite)
            constexpr int kLR = KS::kPieces < 8 ? KS::kPieces : 8;  // lanes per row
            constexpr int kRpi = 64 / kLR;                          // rows per load instruction
            constexpr int kRep = kCE / kRpi;                        // load instructions per row set
            constexpr int kPpl = KS::kPieces / kLR;                 // pieces per lane and row
            const int er = lane / kLR, ep = lane % kLR;
            const int my_q = code >= 0 ? static_cast<int>(qg) : -1;
            uint4 val[2][kRep][kPpl];
#pragma unroll
            for (int j = 0; j < kRep; ++j) {
                const int qj = __shfl(my_q, 2 * (er + kRpi * j), 64);
#pragma unroll
                for (int a = 0; a < 2; ++a) {
                    const uint16_t* const row = (a ? Gb : Qb) + static_cast<size_t>(max(qj, 0)) * D;
                    const uint4* src = reinterpret_cast<const uint4*>(row);
#pragma unroll
                    for (int k = 0; k < kPpl; ++k)
                        val[a][j][k] = qj >= 0 ? src[ep + kLR * k] : make_uint4(0u, 0u, 0u, 0u);
                }
            }
#pragma unroll
            for (int j = 0; j < kRep; ++j)
#pragma unroll
                for (int a = 0; a < 2; ++a)
#pragma unroll
                    for (int k = 0; k < kPpl; ++k)
                        *reinterpret_cast<uint4*>((a ? rows_g : rows_q) + (er + kRpi * j) * KS::kRowB +
                                                  (ep + kLR * k) * 16) = val[a][j][k];
            if (hf == 0) {
                int4 meta = make_int4(-(1 << 30), -(1 << 30), 0, 0);  // no key is near this match
                if constexpr (kQueryIndex) s_el[wave][t][0] = s_el[wave][t][1] = 0;
                if (code >= 0) {
                    uint32_t mu, mv;
                    divmod(static_cast<uint32_t>(clamp_index(match, p.nkeys)), p.div_wk, mu, mv);
                    meta = make_int4(static_cast<int>(mu), static_cast<int>(mv), __float_as_int(lse),
                                     __float_as_int(dq));
                    if constexpr (kQueryIndex) {
                        uint32_t sl, local;
                        divmod(qg, p.div_plane, sl, local);
                        s_el[wave][t][1] = static_cast<int32_t>(local);
                    }
                    if constexpr (MULTI) {
                        // the centres of the query's windows 0 .. e-1 (loaded together), then the strip's
                        // keys their (2 b + 1)^2 neighbourhoods hold
                        int32_t pc[kMaxKappa - 1];
#pragma unroll
                        for (int f = 0; f < kMaxKappa - 1; ++f)
                            pc[f] = f < static_cast<int>(qe) ? p.J[static_cast<size_t>(f) * p.n + qg] : 0;
                        uint32_t held = 0u;
#pragma unroll
                        for (int f = 0; f < kMaxKappa - 1; ++f) {
                            if (f < static_cast<int>(qe)) {
                                uint32_t fu, fv;
                                divmod(static_cast<uint32_t>(clamp_index(pc[f], p.nkeys)), p.div_wk, fu, fv);
                                const int ru = static_cast<int>(fu) - sr0, cv = static_cast<int>(fv) - sc0;
                                held |= strip_bits(ru - p.b, ru + p.b, cv - p.b, cv + p.b);
                            }
                        }
                        s_el[wave][t][0] = static_cast<int32_t>(held);
                    }
                }
                s_meta[wave][t] = meta;
            }
        }
        code = slot_code(c0 + kCE);  // the next chunk's entries load during the products
        wave_lds_sync();

        // S^T, dP^T for entries 16 et + (0..15) of the chunk against the strip's 16 keys
        f32x4_t sc[2], dp[2];
#pragma unroll
        for (int et = 0; et < 2; ++et) {
            sc[et] = dp[et] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            const int er = et * 16 + m;
#pragma unroll
            for (int ds = 0; ds < KS::kDs; ++ds) {
                const int d = 32 * ds + 8 * g4;
                bf16x8_t aq = __builtin_bit_cast(bf16x8_t, make_uint4(0u, 0u, 0u, 0u)), ag = aq;
                if (d < D) {
                    aq = lds_frag(rows_q + er * KS::kRowB + d * 2);
                    ag = lds_frag(rows_g + er * KS::kRowB + d * 2);
                }
                sc[et] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq, kf[ds], sc[et], 0, 0, 0);
                dp[et] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ag, vf[ds], dp[et], 0, 0, 0);
            }
        }
        // P and dS of (key m, entry 16 et + 4 g4 + r): operand slot 4 et + r of this lane, in three parts
        uint32_t ph[8], pm[8], pl[8], sh[8], sm[8], sl[8];
#pragma unroll
        for (int et = 0; et < 2; ++et) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int te = et * 16 + 4 * g4 + r;
                const int4 mt = s_meta[wave][te];
                bool ok = key_ok && abs(mt.x - kx) <= p.b && abs(mt.y - ky) <= p.b;
                if constexpr (MULTI) {
                    // not when an earlier window of the query holds this key (key m of the strip)
                    ok = ok && !((static_cast<uint32_t>(s_el[wave][te][0]) >> m) & 1u);
                    if (p.causal) ok = ok && key_local <= static_cast<uint32_t>(s_el[wave][te][1]);
                } else if constexpr (MODE == kStripCausal) {
                    ok = ok && key_local <= static_cast<uint32_t>(s_el[wave][te][1]);
                }
                const float pr = ok ? __builtin_amdgcn_exp2f(sc[et][r] * p.scale_log2e - __int_as_float(mt.z)) : 0.f;
                const float dsr = pr * (dp[et][r] - __int_as_float(mt.w));
                split3(pr, ph[4 * et + r], pm[4 * et + r], pl[4 * et + r]);
                split3(dsr, sh[4 * et + r], sm[4 * et + r], sl[4 * et + r]);
            }
        }
        auto operand = [](const uint32_t (&v)[8]) {
            return __builtin_bit_cast(bf16x8_t, make_uint4(hi16_pair(v[0], v[1]), hi16_pair(v[2], v[3]),
                                                           hi16_pair(v[4], v[5]), hi16_pair(v[6], v[7])));
        };
        const bf16x8_t aph = operand(ph), apm = operand(pm), apl = operand(pl);
        const bf16x8_t ash = operand(sh), asm_ = operand(sm), asl = operand(sl);
        // dV_w += P dO_E, dK_w += dS Q_E per 16-channel tile o
#pragma unroll
        for (int o = 0; o < KS::kOt; ++o) {
            const bf16x8_t bq = tr_pair(rows_q + tr_off + 32 * o), bg = tr_pair(rows_g + tr_off + 32 * o);
            dv[o] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aph, bg, dv[o], 0, 0, 0);
            dv[o] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(apm, bg, dv[o], 0, 0, 0);
            dv[o] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(apl, bg, dv[o], 0, 0, 0);
            dk[o] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ash, bq, dk[o], 0, 0, 0);
            dk[o] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(asm_, bq, dk[o], 0, 0, 0);
            dk[o] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(asl, bq, dk[o], 0, 0, 0);
        }
        wave_lds_sync();  // this chunk's LDS reads come before the next chunk's writes
    }

    // lane holds keys 4 g4 + r of the strip, channel 16 o + m
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        int ox, oy;
        strip_key(4 * g4 + r, ox, oy);
        if (ox >= p.Hk || oy >= p.Wk) continue;
        const size_t row = (kslice + static_cast<size_t>(ox) * p.Wk + oy) * D;
#pragma unroll
        for (int o = 0; o < KS::kOt; ++o) {
            p.dK[row + 16 * o + m] = dk[o][r] * p.scale;
            p.dV[row + 16 * o + m] = dv[o][r];
        }
    }
}

// ---------------------------------------------------------------------------
// Query side on the matrix cores (bf16 storage, d 32 or 64, windows 3/5/7,
// up to MK maps, with or without the causal mask; several maps as in the
// attend's matrix-core kernel: one pass over the joint clusters of up to four
// windows' centres, else a pass per window, with the keys of the query's
// earlier windows left out).  The wave's 16 queries, their clusters and key boxes are
// those of the attend's matrix-core kernel (scram_tile.h); the key and value
// rows of a box are read a block of 16 keys at a time, staged in LDS, and per
// block (lane (m, g4): keys 4 g4 + i, query m)
//   S^T = K_blk Q^T,  dP^T = V_blk dO^T          keys x queries, 16x16x32 bf16
//   p = 2^(s scale log2e - m_ref) on the query's window, 0 elsewhere; pd = p dp
//   B^T += K_blk^T P^T,  A^T += K_blk^T PD^T     channels x queries: K_blk^T by
//                                                the transposing LDS load
//   l += 1^T P^T,  dn += 1^T PD^T               all-ones blocks
// with P and PD as three bf16 parts each (they add up to the fp32 values
// exactly).  With D_i = dn / l and the match's key k_ref,
//   dQ_i = scale ((A - dn k_ref) - D_i (B - l k_ref)) / l
//        = scale sum_j p_ij (dp_ij - D_i)(k_j - k_ref) / l
// the sums of the lane-group kernel, formed from the same rounded weights on
// both sides, so the subtraction cancels no more than there.  Also writes the
// per-query statistics and the inverse map's count and slot of the query's
// match, as the lane-group kernel does.
template <int D, int W, bool CAUSAL, int MK>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(3))) void bwd_query_tile_kernel(BwdParams p)
{
    constexpr int B = W / 2;
    constexpr int kDs = D / 32;        // 32-channel contraction steps of S^T and dP^T
    constexpr int kOt = D / 16;        // 16-channel tiles of A^T, B^T
    constexpr int kRowB = 2 * D + 16;  // LDS row stride, bytes (padded)
    constexpr int kPer = D / 32;       // 16-byte pieces per lane: a row (D / 8 pieces) is read by 4 consecutive lanes
    constexpr int kWaves = kBlock / 64;
#ifndef SCRAM_BWD_TILE_PARTS
#define SCRAM_BWD_TILE_PARTS 3
#endif
    constexpr int kParts = SCRAM_BWD_TILE_PARTS;  // bf16 parts of each weight
    static_assert(kPer == 1 || kPer == 2, "32 or 64 channels");
    __shared__ __align__(16) unsigned char s_k[kWaves][16 * kRowB], s_v[kWaves][16 * kRowB];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m = lane & 15, g4 = lane >> 4;
    const uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
    uint32_t g, g0;
    const bool valid = tile_item<kBlock / 4>(p.tq, blk, tile_wave_item(p.tq, wave, m), g);
    tile_item<kBlock / 4>(p.tq, blk, 0, g0);  // item 0 of a tile is always inside the grid
    const uint32_t gq = valid ? g : g0;
    uint32_t s, rem;
    divmod(gq, p.div_plane, s, rem);
    // the slice's key and value rows as 32-bit byte offsets from a wave-uniform base (the caller keeps
    // a slice's rows below 4 GiB)
    const size_t slice_bytes =
        static_cast<size_t>(__builtin_amdgcn_readfirstlane(s)) * p.nkeys * static_cast<size_t>(2 * D);
    const unsigned char* const Kb = static_cast<const unsigned char*>(p.K) + slice_bytes;
    const unsigned char* const Vb = static_cast<const unsigned char*>(p.V) + slice_bytes;
    const uint32_t centre = static_cast<uint32_t>(clamp_index(p.J[gq], p.nkeys));
    // the inverse map's count: one entry per match of the query, and its slot among the entries of that
    // match key
    if (valid && g4 == 0) {
        p.slots[g] = atomicAdd(p.counts + static_cast<size_t>(s) * p.nkeys + centre, 1);
        if constexpr (MK > 1) {
            for (int e = 1; e < p.kappa; ++e) {
                const size_t x = static_cast<size_t>(e) * p.n + g;
                p.slots[x] = atomicAdd(p.counts + static_cast<size_t>(s) * p.nkeys + clamp_index(p.J[x], p.nkeys), 1);
            }
        }
    }
    int u, v;
    {
        uint32_t uu, vv;
        divmod(centre, p.div_wk, uu, vv);
        u = static_cast<int>(uu);
        v = static_cast<int>(vv);
    }
    // B operands of S^T and dP^T: query m, channels 32 ds + 8 g4 .. + 7 of q and dO; the same channels
    // of the match's key
    bf16x8_t qf[kDs], gf[kDs];
    uint4 kc[kDs];
    const uint16_t* const qrow = static_cast<const uint16_t*>(p.Q) + static_cast<size_t>(gq) * D;
    const uint16_t* const grow = static_cast<const uint16_t*>(p.dO) + static_cast<size_t>(gq) * D;
#pragma unroll
    for (int ds = 0; ds < kDs; ++ds) {
        qf[ds] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qrow + 32 * ds + 8 * g4));
        gf[ds] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(grow + 32 * ds + 8 * g4));
        kc[ds] = *reinterpret_cast<const uint4*>(Kb + centre * (2u * D) + 64u * ds + 16u * g4);
    }

    int qx = 0, qy = 0;  // causal: the query's position (queries and keys share the grid)
    if constexpr (CAUSAL) {
        uint32_t xx, yy;
        divmod(rem, p.div_wk, xx, yy);
        qx = static_cast<int>(xx);
        qy = static_cast<int>(yy);
    }
    // up to four windows: one pass over the clusters of all their centres, as in the attend's
    // matrix-core kernel (with four windows and the causal mask a few registers spill; the halved
    // block count still pays)
    constexpr bool JOINT = MK == 2 || MK == 4;
    constexpr int NJ = JOINT ? MK : 1;
    int ju[NJ], jv[NJ], jmine[NJ];  // window e's centre and the cluster that holds it (-1: no window e)
    TileClusters tc;
    if constexpr (JOINT) {
        const int ew = g4 & (NJ - 1);  // the window whose centre this lane clusters
        int iu = u, iv = v;
#pragma unroll
        for (int e = 0; e < NJ; ++e) {
            ju[e] = u, jv[e] = v;  // window 0; a window past kappa repeats it and is not clustered
            if (e > 0 && e < p.kappa) {
                uint32_t uu, vv;
                divmod(static_cast<uint32_t>(clamp_index(p.J[static_cast<size_t>(e) * p.n + gq], p.nkeys)),
                       p.div_wk, uu, vv);
                ju[e] = static_cast<int>(uu), jv[e] = static_cast<int>(vv);
            }
            iu = ew == e ? ju[e] : iu, iv = ew == e ? jv[e] : iv;
        }
        tc = tile_clusters_joint<B, NJ>(valid && ew < p.kappa, iu, iv, lane, p.rc, p.Hk, p.Wk);
#pragma unroll
        for (int e = 0; e < NJ; ++e) jmine[e] = __shfl(tc.mine, m + 16 * e);
    } else {
        tc = tile_clusters<B, CAUSAL>(valid, u, v, m, lane, p.rc, p.Hk, p.Wk, qx, qy);
    }
    if (tc.nclu == 0) return;  // no query of this wave lies inside the grid
    // several windows: windows 0 .. e-1 of query m as in the attend's matrix-core kernel
    constexpr int kOther = MK > 1 ? MK - 1 : 1;
    int cu[kOther], cv[kOther], dw[kOther];
    uint32_t xw[kOther];
#pragma unroll
    for (int f = 0; f < kOther; ++f) cu[f] = cv[f] = 0, dw[f] = 1 << 20, xw[f] = 0u;
    // joint pass, per cluster: window e's first row as a box row (jd), its rows less one, cut at the
    // box's last (jn), its columns in the box (jx); bit e of hm: the cluster holds window e's centre
    int jd[NJ], jn[NJ];
    uint32_t jx[NJ], hm = 0u;
#pragma unroll
    for (int e = 0; e < NJ; ++e) jd[e] = jn[e] = 0, jx[e] = 0u;
    int jqr = 0;        // causal: the query's row as a box row
    uint32_t jqc = 0u;  // and the box columns up to the query's

    const f32x4_t zero = f32x4_t{0.f, 0.f, 0.f, 0.f};
    f32x4_t acc_a[kOt], acc_b[kOt];
#pragma unroll
    for (int o = 0; o < kOt; ++o) acc_a[o] = acc_b[o] = zero;
    f32x4_t lacc = zero, dacc = zero;  // every row: sum of p, sum of p dp, of query m
    const bf16x4_t ones = bf16x4_t{static_cast<__bf16>(1.f), static_cast<__bf16>(1.f), static_cast<__bf16>(1.f),
                                   static_cast<__bf16>(1.f)};
    const float sl2e = p.scale_log2e;  // > 0 (the caller routes other scales to the lane-group kernels)
    const float inv_sl2e = __builtin_amdgcn_rcpf(sl2e);
    int bit_at[4];  // 0..3 as values the compiler cannot see: one bit-field extract per mask below
#pragma unroll
    for (int i = 0; i < 4; ++i) asm volatile("s_mov_b32 %0, %1" : "=s"(bit_at[i]) : "i"(i));
    // online softmax state of query m, starting at the score of its match (a key of its window), as in
    // the attend's matrix-core kernel; under the causal mask a match after the query is not in its set,
    // and the first kept key sets the reference.  (k_ref stays the match's key: any fixed vector gives
    // the same dQ, as sum_j p_ij (dp_ij - D_i) is zero.)
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
    if (CAUSAL && centre > rem) {
        mref = -INFINITY;
        nref = 0.f;
    }
    float thr_q = (mref + (kRescaleSlack - 1.f)) * inv_sl2e;
    float thr = INFINITY;

    const int lslot = lane >> 2, lpiece = lane & 3;  // every lane: one key slot, 16-byte pieces lpiece (+ 4)
    unsigned char* const tk = s_k[wave];
    unsigned char* const tv = s_v[wave];
    // A operand of A^T, B^T for tile o: lane (m, g4) addresses key row 4 g4 + m / 4 at channels
    // 4 (m mod 4) .. + 3 (+ 16 o) and the transposing load hands it rows 4 g4 .. + 3 at channel 16 o + m
    const unsigned char* const tkt = tk + (4 * g4 + (m >> 2)) * kRowB + 8 * (m & 3);
    const uint4 z4 = make_uint4(0u, 0u, 0u, 0u);
    uint4 kr0 = z4, kr1 = z4, vr0 = z4, vr1 = z4;  // this lane's pieces of the rows in flight
    auto load = [&](uint32_t key, uint32_t klast) {  // a slot past the box's last row reads its last row
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
    auto first_slot = [&](const TileBox& b, int& lc, uint32_t& lkey) {
        int lr;
        box_slot(lslot, b.bw, b.inv, lr, lc);
        lkey = static_cast<uint32_t>(b.r0 + lr) * static_cast<uint32_t>(p.Wk) + (b.c0 + lc);
    };
    auto step_slot = [](const TileBox& b, int& lc, uint32_t& lkey) {  // 16 slots on
        lc += b.r16;
        const bool carry = lc >= b.bw;
        lc -= carry ? b.bw : 0;
        lkey += carry ? b.kstep_wrap : b.kstep;
    };
    // the weights as bf16 parts: hi + mid + lo exactly (kParts 3), or hi + the top 8 bits of the rest
    auto pack3 = [](const uint32_t (&x)[4], bf16x4_t& h, bf16x4_t& md, bf16x4_t& lo) {
        uint32_t a[4], b[4], c[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (kParts == 3) {
                split3(__uint_as_float(x[i]), a[i], b[i], c[i]);
            } else {
                a[i] = x[i] & 0xFFFF0000u;
                b[i] = __float_as_uint(__uint_as_float(x[i]) - __uint_as_float(a[i]));
                c[i] = 0u;
            }
        }
        h = __builtin_bit_cast(bf16x4_t, make_uint2(hi16_pair(a[0], a[1]), hi16_pair(a[2], a[3])));
        md = __builtin_bit_cast(bf16x4_t, make_uint2(hi16_pair(b[0], b[1]), hi16_pair(b[2], b[3])));
        lo = __builtin_bit_cast(bf16x4_t, make_uint2(hi16_pair(c[0], c[1]), hi16_pair(c[2], c[3])));
    };
    auto compute = [&](const TileBox& bx, int rr, int mcl, uint32_t wc, uint32_t wc2, uint32_t wk, uint32_t wk2) {
        f32x4_t sc = zero, dp = zero;
#pragma unroll
        for (int ds = 0; ds < kDs; ++ds) {
            const bf16x8_t kf = __builtin_bit_cast(
                bf16x8_t, *reinterpret_cast<const uint4*>(tk + m * kRowB + 16 * (4 * ds + g4)));
            const bf16x8_t vf = __builtin_bit_cast(
                bf16x8_t, *reinterpret_cast<const uint4*>(tv + m * kRowB + 16 * (4 * ds + g4)));
            sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ds], sc, 0, 0, 0);
            dp = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, gf[ds], dp, 0, 0, 0);
        }
        uint32_t bits;
        if constexpr (JOINT) {
            // rr is the slot's box row: window e's slots when this cluster holds its centre, less those of
            // the query's earlier windows
            bits = 0u;
            uint32_t held = 0u;
#pragma unroll
            for (int e = 0; e < NJ; ++e) {
                const uint32_t w = tile_window_bits<false>(bx, rr - jd[e], mcl, jn[e], jx[e], jx[e] << bx.bw);
                bits |= ((hm >> e) & 1u) ? w & ~held : 0u;
                held |= w;
            }
            if constexpr (CAUSAL) bits &= tile_causal_bits(bx, rr, mcl, jqr, jqc);
        } else {
            bits = tile_window_bits<CAUSAL>(bx, rr, mcl, tc.wrn, wc, wc2, tc.rcut, wk, wk2);
            if constexpr (MK > 1) bits &= ~tile_other_bits<kOther, B>(bx, rr, mcl, dw, xw);
        }
        uint32_t keep[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            keep[i] = static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(bits), bit_at[i], 1));
        if (__ballot((sc[0] > thr) | (sc[1] > thr) | (sc[2] > thr) | (sc[3] > thr))) {
            float mx = -INFINITY;
#pragma unroll
            for (int i = 0; i < 4; ++i) mx = fmaxf(mx, keep[i] ? sc[i] : -INFINITY);
            mx *= sl2e;
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            if (mx > mref + kRescaleSlack) {
                const float alpha = __builtin_amdgcn_exp2f(mref - mx);
                lacc *= alpha;
                dacc *= alpha;
#pragma unroll
                for (int o = 0; o < kOt; ++o) {
                    acc_a[o] *= alpha;
                    acc_b[o] *= alpha;
                }
                mref = mx;
                nref = -mx;
                thr = (mx + (kRescaleSlack - 1.f)) * inv_sl2e;
                if constexpr (MK > 1) thr_q = thr;  // the query's later windows start from here
            }
        }
        uint32_t pw[4], pdw[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t x = __float_as_uint(fmaf(sc[i], sl2e, nref));
            const float pk = __builtin_amdgcn_exp2f(__uint_as_float((x & keep[i]) | (0xFF800000u & ~keep[i])));
            pw[i] = __float_as_uint(pk);
            pdw[i] = __float_as_uint(pk * dp[i]);
        }
        bf16x4_t ph, pm, pl, dh, dm, dl;
        pack3(pw, ph, pm, pl);
        pack3(pdw, dh, dm, dl);
        lacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ones, ph, lacc, 0, 0, 0);
        lacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ones, pm, lacc, 0, 0, 0);
        dacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ones, dh, dacc, 0, 0, 0);
        dacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ones, dm, dacc, 0, 0, 0);
        if constexpr (kParts == 3) {
            lacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ones, pl, lacc, 0, 0, 0);
            dacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ones, dl, dacc, 0, 0, 0);
        }
#pragma unroll
        for (int o = 0; o < kOt; ++o) {
            const bf16x4_t kt = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                (__attribute__((address_space(3))) bf16x4_t*)(tkt + 32 * o));
            acc_b[o] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(kt, ph, acc_b[o], 0, 0, 0);
            acc_b[o] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(kt, pm, acc_b[o], 0, 0, 0);
            acc_a[o] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(kt, dh, acc_a[o], 0, 0, 0);
            acc_a[o] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(kt, dm, acc_a[o], 0, 0, 0);
            if constexpr (kParts == 3) {
                acc_b[o] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(kt, pl, acc_b[o], 0, 0, 0);
                acc_a[o] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(kt, dl, acc_a[o], 0, 0, 0);
            }
        }
    };

    // the blocks of each cluster in a row; each block's rows load during the previous block's products
    for (int e = 0;;) {
        TileBox bx = tile_box(tc, 0, p.Wk);
        int lc;
        uint32_t lkey;
        first_slot(bx, lc, lkey);
        load(lkey, bx.klast);
        for (int c = 0;;) {
            int mr, mcl;
            box_slot(4 * g4, bx.bw, bx.inv, mr, mcl);
            int rr = mr - tc.wr0;
            const bool here = c == tc.mine;
            const uint32_t wc = here ? tc.wcols : 0u;
            const uint32_t wc2 = here ? tc.wcols << bx.bw : 0u;  // bw <= 27, and only bits below bw + 3 are read
            const uint32_t wk = CAUSAL && here ? tc.wcut : 0u;  // the query's own row (causal)
            const uint32_t wk2 = CAUSAL && here ? tc.wcut << bx.bw : 0u;
            bool in = here;
            if constexpr (JOINT) {
                rr = mr;
                hm = 0u;
#pragma unroll
                for (int e = 0; e < NJ; ++e) {
                    jd[e] = ju[e] - B - bx.r0;
                    jn[e] = min(2 * B, bx.h - 1 - jd[e]);
                    // no columns for a window wholly below the box (its row count would be negative)
                    jx[e] = jn[e] >= 0 ? tile_col_bits(jv[e] - B - bx.c0, jv[e] + B - bx.c0, bx.bw) : 0u;
                    hm |= c == jmine[e] ? 1u << e : 0u;
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
            const bool more = c + 1 < tc.nclu;
            TileBox nx = bx;
            if (more) {
                nx = tile_box(tc, c + 1, p.Wk);
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
        if constexpr (MK == 1 || JOINT) {
            break;
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
            wave_lds_sync();  // the last block's LDS reads come before the next pass's writes
        }
    }
    if (!valid) return;
    const float l = lacc[0], dn = dacc[0];
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const float Dg = dn * inv;
    if (g4 == 0) {
        p.lse2[g] = l > 0.f ? mref + log2f(l) : INFINITY;  // +inf: every weight is 0
        p.Dq[g] = Dg;
    }
    // lane holds channels 16 o + 4 g4 + i of query m
    const uint16_t* const krow = static_cast<const uint16_t*>(static_cast<const void*>(Kb + centre * (2u * D)));
    float* const dq = p.dQ + static_cast<size_t>(g) * D;
#pragma unroll
    for (int o = 0; o < kOt; ++o) {
        const uint2 kw = *reinterpret_cast<const uint2*>(krow + 16 * o + 4 * g4);
        const float kref[4] = {__uint_as_float(kw.x << 16), __uint_as_float(kw.x & 0xFFFF0000u),
                               __uint_as_float(kw.y << 16), __uint_as_float(kw.y & 0xFFFF0000u)};
        float r[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            r[i] = ((acc_a[o][i] - dn * kref[i]) - Dg * (acc_b[o][i] - l * kref[i])) * inv * p.scale;
        *reinterpret_cast<float4*>(dq + 16 * o + 4 * g4) = make_float4(r[0], r[1], r[2], r[3]);
    }
}

#ifndef SCRAM_BWD_QUERY_TILE
#define SCRAM_BWD_QUERY_TILE 1
#endif

// launch() for kernels whose blocks are one wave each
hipError_t launch_wave(void (*kernel)(BwdParams), uint64_t blocks, hipStream_t st, hipEvent_t start, hipEvent_t stop,
                       const BwdParams& p)
{
    if (blocks == 0 || blocks > 0xFFFFFFFFull / 64) return hipErrorInvalidConfiguration;
    if (start || stop)
        hipExtLaunchKernelGGL(kernel, dim3(blocks), dim3(64), 0, st, start, stop, 0, p);
    else
        hipLaunchKernelGGL(kernel, dim3(blocks), dim3(64), 0, st, p);
    return hipGetLastError();
}

// The query kernel, then the rest of the inverse map (inverse()), then the
// key side.
template <typename T, int D, typename Inverse>
hipError_t run_backward(const BwdParams& p0, hipStream_t st, hipEvent_t* ev, Inverse&& inverse)
{
    constexpr int G = Lanes<T, D>::kAttend;
    constexpr uint32_t kQpb = Row<T, D, G>::kQpb;
    BwdParams p = p0;
    p.tq = make_tiling(p.Hq, p.Wq, kQpb, kLaneSkew);
    p.tk = make_tiling(p.Hk, p.Wk, kQpb, kLaneSkew);
    const uint64_t qblocks = tiling_blocks(p.tq, p.n / p.tq.plane);
    const uint64_t gblocks = (static_cast<uint64_t>(p.kappa) * p.n + kQpb - 1) / kQpb;
    const uint64_t kblocks = tiling_blocks(p.tk, p.keys_total / p.nkeys);
    // the query-side interval opens with the clearing kernel launched before this
    hipEvent_t q1 = ev ? ev[3] : nullptr, k0 = ev ? ev[4] : nullptr, k1 = ev ? ev[5] : nullptr;
    const bool multi = p.kappa > 1 || p.causal;
    auto query = [&](auto w) {
        constexpr int W = decltype(w)::value;
        return multi ? launch(bwd_query_kernel<T, D, G, true, W>, qblocks, st, nullptr, q1, p)
                     : launch(bwd_query_kernel<T, D, G, false, W>, qblocks, st, nullptr, q1, p);
    };
    const int side = 2 * p.b + 1;
    // the matrix-core query kernel takes bf16 storage with 32 or 64 channels, up to 4 maps (with or
    // without the causal mask), windows 3, 5 or 7, a positive scale and slices of at most 4 GiB of key rows
    hipError_t e = hipSuccess;
    bool tile = false;
    if constexpr (SCRAM_BWD_QUERY_TILE && std::is_same<T, uint16_t>::value && (D == 32 || D == 64)) {
        if (p.kappa <= 4 && (side == 3 || side == 5 || side == 7) && p.scale_log2e > 0.f &&
            static_cast<uint64_t>(p.nkeys) * (2 * D) <= 0xFFFFFFFFull) {
            BwdParams pq = p;
            pq.tq = make_tiling(p.Hq, p.Wq, kBlock / 4);
            pq.rc = 10;  // as in the attend's matrix-core kernel
            const uint64_t tb = tiling_blocks(pq.tq, p.n / pq.tq.plane);
            auto go = [&](auto w) {
                constexpr int Wn = decltype(w)::value;
                auto with = [&](auto mk) {  // the smallest bound on the windows per query that holds this call's
                    constexpr int MK = decltype(mk)::value;
                    return p.causal ? launch(bwd_query_tile_kernel<D, Wn, true, MK>, tb, st, nullptr, q1, pq)
                                    : launch(bwd_query_tile_kernel<D, Wn, false, MK>, tb, st, nullptr, q1, pq);
                };
                return p.kappa == 1   ? with(std::integral_constant<int, 1>{})
                       : p.kappa == 2 ? with(std::integral_constant<int, 2>{})
                                      : with(std::integral_constant<int, 4>{});
            };
            e = side == 3   ? go(std::integral_constant<int, 3>{})
                : side == 5 ? go(std::integral_constant<int, 5>{})
                            : go(std::integral_constant<int, 7>{});
            tile = true;
        }
    }
    if (!tile)
        e = side == 1   ? query(std::integral_constant<int, 1>{})
            : side == 3 ? query(std::integral_constant<int, 3>{})
            : side == 5 ? query(std::integral_constant<int, 5>{})
            : side == 7 ? query(std::integral_constant<int, 7>{})
                        : query(std::integral_constant<int, 0>{});
    if (e != hipSuccess) return e;
    if ((e = inverse()) != hipSuccess) return e;
    if constexpr (std::is_same<T, uint16_t>::value) {
        // key side on the matrix cores; a one-key window (b = 0) stays on the lane-group kernels, whose dp
        // is the query kernel's own arithmetic, so that dS = p (dp - D) is exactly 0 there
        if (p.b >= 1 && p.b <= kTileMaxB) {
            BwdParams pt = p;
            pt.tk = make_tiling(p.Hk, p.Wk, kTileKeys);
            const uint64_t tblocks = kStripWaves * tiling_blocks(pt.tk, p.keys_total / p.nkeys);
            return p.kappa > 1 ? launch_wave(bwd_key_strip_kernel<D, kStripMulti>, tblocks, st, k0, k1, pt)
                   : p.causal  ? launch_wave(bwd_key_strip_kernel<D, kStripCausal>, tblocks, st, k0, k1, pt)
                               : launch_wave(bwd_key_strip_kernel<D, kStripPlain>, tblocks, st, k0, k1, pt);
        }
    }
    if ((e = launch(bwd_gather_kernel<T, D, G>, gblocks, st, k0, nullptr, p)) != hipSuccess) return e;
    e = multi ? launch(bwd_key_kernel<T, D, G, true>, kblocks, st, nullptr, nullptr, p)
              : launch(bwd_key_kernel<T, D, G, false>, kblocks, st, nullptr, nullptr, p);
    if (e != hipSuccess) return e;
    constexpr uint32_t kHeavyBlocks = 2048;  // loops over however many heavy keys there are
    return multi ? launch(bwd_heavy_kernel<T, D, G, true>, kHeavyBlocks, st, nullptr, k1, p)
                 : launch(bwd_heavy_kernel<T, D, G, false>, kHeavyBlocks, st, nullptr, k1, p);
}

}  // namespace

size_t attend_backward_workspace_bytes(int S, int Hq, int Wq, int Hk, int Wk, int d, int dtype, int kappa)
{
    const size_t n = static_cast<size_t>(S) * Hq * Wq, N = static_cast<size_t>(S) * Hk * Wk;
    const size_t tiles = (N + kScanTile - 1) / kScanTile;
    const size_t row = static_cast<size_t>(d) * (dtype == SCRAM_BF16 ? 2 : 4);
    auto r256 = [](size_t b) { return (b + 255) & ~static_cast<size_t>(255); };
    return r256(4 * N) + r256(4 * (N + 1)) + r256(4 * (tiles + 1)) + r256(4 * n * kappa) + 2 * r256(4 * n) +
           2 * r256(row * n * kappa) + r256(8 * n * kappa) + r256(4 * (N + 1)) + r256(4 * n * kappa);
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
    w += r256(4 * static_cast<size_t>(p.n));
    const size_t rows_bytes = static_cast<size_t>(g.d) * (dtype == SCRAM_BF16 ? 2 : 4) * p.n * kappa;
    p.qs = w;
    w += r256(rows_bytes);
    p.gs = w;
    w += r256(rows_bytes);
    p.st = reinterpret_cast<float2*>(w);
    w += r256(8 * static_cast<size_t>(p.n) * kappa);
    p.n_heavy = reinterpret_cast<int32_t*>(w);  // counter, then the list
    p.heavy = p.n_heavy + 1;
    w += r256(4 * (N + 1));
    p.slots = reinterpret_cast<int32_t*>(w);
    p.counts = counts;
    p.offsets = offsets;
    p.entries = entries;

    auto grid_for = [](size_t items) {
        const size_t b = (items + kBlock - 1) / kBlock;
        return static_cast<uint32_t>(b < 1 ? 1 : (b > 4096 ? 4096 : b));
    };
    hipEvent_t e0 = events ? events[0] : nullptr, e1 = events ? events[1] : nullptr;
    hipEvent_t q0 = events ? events[2] : nullptr;
    const size_t entries_total = static_cast<size_t>(p.n) * kappa;
    hipError_t e;
    // inverse map: a counting sort of the (query, match) entries by match key.
    // The counts (and the heavy-key counter) start at zero; the query kernel
    // counts; the scan and the fill follow it.
    if ((e = launch(zero_i32_kernel, grid_for(N), stream, q0, nullptr, counts, N, p.n_heavy)) != hipSuccess) return e;
    auto inverse = [&]() -> hipError_t {
        hipError_t r;
        if ((r = launch(scan_tiles_kernel, tiles, stream, e0, nullptr, static_cast<const int32_t*>(counts), counts,
                        sums, N)) != hipSuccess)
            return r;
        const uint32_t fill_blocks = grid_for(entries_total > N ? entries_total : N + 1);
        if (tiles <= static_cast<uint32_t>(kScanTile))
            return launch(bwd_fill_kernel<true>, fill_blocks, stream, nullptr, e1, p,
                          static_cast<const int32_t*>(counts), static_cast<const int32_t*>(sums), tiles, offsets,
                          entries);
        if ((r = launch(scan_sums_kernel, 1u, stream, nullptr, nullptr, sums, tiles)) != hipSuccess) return r;
        return launch(bwd_fill_kernel<false>, fill_blocks, stream, nullptr, e1, p,
                      static_cast<const int32_t*>(counts), static_cast<const int32_t*>(sums), tiles, offsets,
                      entries);
    };
    // gradients
    return dispatch(dtype, g.d, [&](auto ty, auto d) {
        return run_backward<decltype(ty), decltype(d)::value>(p, stream, events, inverse);
    });
}

uint64_t attend_backward_max_blocks(int dtype, const Grid& g, int kappa)
{
    return dispatch_value(dtype, g.d, uint64_t(0), [&](auto t, auto d) {
        using T = decltype(t);
        constexpr int D = decltype(d)::value;
        constexpr uint32_t kQpb = Row<T, D, Lanes<T, D>::kAttend>::kQpb;
        const uint64_t n = uint64_t(g.S) * g.Hq * g.Wq, keys = uint64_t(g.S) * g.Hk * g.Wk;
        uint64_t most = 4096;  // the grid-stride kernels of the inverse map
        auto keep = [&](uint64_t b) { most = b > most ? b : most; };
        keep(tiling_blocks(make_tiling(g.Hq, g.Wq, kQpb, kLaneSkew), g.S));    // query kernel
        keep((uint64_t(kappa) * n + kQpb - 1) / kQpb);              // entry-order copies
        keep(tiling_blocks(make_tiling(g.Hk, g.Wk, kQpb, kLaneSkew), g.S));    // key kernel
        keep(tiling_blocks(make_tiling(g.Hk, g.Wk, kTileKeys), g.S));  // key tiles on the matrix cores
        keep((keys + kScanTile - 1) / kScanTile);                   // scan tiles
        return most;
    });
}

}  // namespace scram
