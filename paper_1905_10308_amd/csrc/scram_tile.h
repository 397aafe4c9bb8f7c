// Matrix-core pieces shared by the attend (scram_attend.hip) and its backward
// (scram_backward.hip) for bf16 storage on gfx950.
//
// A wave takes 16 queries (a 4 x 4 quarter of an 8 x 8 block tile, or 16
// consecutive items of narrower tiles); lane l works on query m = l mod 16
// with lane group g4 = l div 16, so lanes 16.. repeat the queries of 0..15.
// Neighbouring queries' windows overlap, so the 16 match centres are grouped
// into clusters -- a query joins the cluster of the first unassigned query
// whose centre lies within Chebyshev distance rc -- and each cluster's key box
// (its members' windows, clipped to the grid) is visited in blocks of 16 keys
// in raster order.  Every query is in exactly one cluster and each key of its
// window is in that cluster's box exactly once.
//
// Everything here lives in an unnamed namespace, like scram_device.h.

#pragma once

#include <limits.h>

#include "scram_device.h"

namespace scram {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// bf16 pair (a in the low half, b in the high half) from the high halves of two fp32 patterns
__device__ __forceinline__ uint32_t hi16_pair(uint32_t a, uint32_t b)
{
    return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

template <int CTRL>
__device__ __forceinline__ int dpp_i(int x)
{
    return __builtin_amdgcn_mov_dpp(x, CTRL, 0xF, 0xF, true);
}

// min and max over the 16 lanes of a DPP row (every lane of the row gets both)
__device__ __forceinline__ void row_minmax(int& lo, int& hi)
{
    lo = min(lo, dpp_i<0xB1>(lo)), hi = max(hi, dpp_i<0xB1>(hi));
    lo = min(lo, dpp_i<0x4E>(lo)), hi = max(hi, dpp_i<0x4E>(hi));
    lo = min(lo, dpp_i<0x141>(lo)), hi = max(hi, dpp_i<0x141>(hi));
    lo = min(lo, dpp_i<0x140>(lo)), hi = max(hi, dpp_i<0x140>(hi));
}

// (row, column) of raster slot j of a box `bw` wide: exact for j < 1024 and
// bw <= 31 (the fraction of (j + 1/2) / bw stays 1/(2 bw) away from an
// integer, far more than the float error of the product)
__device__ __forceinline__ void box_slot(int j, int bw, float inv_bw, int& r, int& c)
{
    r = static_cast<int>((static_cast<float>(j) + 0.5f) * inv_bw);
    c = j - r * bw;
}

// LDS written by some lanes of a wave and then read by others: keep the
// compiler from moving accesses across this point (a wave's LDS instructions
// execute in order)
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The item of a block tile that lane (m, wave) works on: a 4 x 4 quarter of an
// 8 x 8 tile (lw == 3), else 16 consecutive items.
__device__ __forceinline__ uint32_t tile_wave_item(const Tiling& tq, int wave, int m)
{
    return tq.lw == 3 ? ((4u * (wave >> 1) + (m >> 2)) << 3) + 4u * (wave & 1) + (m & 3) : 16u * wave + m;
}

// A wave's clusters.  Cluster c's box (rows r0 .. r0 + h - 1, columns
// c0 .. c0 + bw - 1, nb blocks of 16 raster slots, a 16-slot step of q16 rows
// and r16 columns) is held by lane c of the t_ registers and read back with
// readlane; query m's window in its own cluster's box is rows wr0 .. wr0 + wrn
// with a bit per box column in wcols.  With the causal mask (keys after the
// query in raster order dropped; one grid for queries and keys) wrn and wcols
// cover the window's rows before the query's own row, and the query's row --
// window row rcut, if the window reaches it -- keeps the columns in wcut (up
// to the query's column); rcut is INT_MIN otherwise.
struct TileClusters {
    int t_r0, t_c0, t_bw, t_h, t_nb, t_q16, t_r16;
    float t_inv;
    int nclu, mine;
    int wr0, wrn, rcut;
    uint32_t wcols, wcut;
};

// Clusters of the 16 centres (u, v) of a wave (windows of half side B, key
// grid Hk x Wk, cluster radius rc); CAUSAL: the query sits at (qx, qy) of the
// same grid.  nclu == 0 when no query of the wave is valid.
template <int B, bool CAUSAL = false>
__device__ __forceinline__ TileClusters tile_clusters(bool valid, int u, int v, int m, int lane, int rc, int Hk,
                                                      int Wk, int qx = 0, int qy = 0)
{
    TileClusters tc;
    int t_r0 = 0, t_c0 = 0, t_bw = 1, t_h = 0;
    int nclu = 0, mine = -1;
    uint32_t todo = static_cast<uint32_t>(__ballot(valid)) & 0xFFFFu;  // bit m: query m (lanes 16.. repeat 0..15)
    while (todo) {
        const int a = __builtin_ctz(todo);
        const int ua = __builtin_amdgcn_readlane(u, a), va = __builtin_amdgcn_readlane(v, a);
        const bool mem = ((todo >> m) & 1u) && abs(u - ua) <= rc && abs(v - va) <= rc;
        todo &= ~(static_cast<uint32_t>(__ballot(mem)) & 0xFFFFu);
        mine = mem ? nclu : mine;
        int ulo = mem ? u : ua, uhi = ulo, vlo = mem ? v : va, vhi = vlo;
        row_minmax(ulo, uhi);
        row_minmax(vlo, vhi);
        const bool here = lane == nclu;
        t_r0 = here ? max(ulo - B, 0) : t_r0;
        t_c0 = here ? max(vlo - B, 0) : t_c0;
        t_h = here ? min(uhi + B, Hk - 1) - max(ulo - B, 0) + 1 : t_h;
        t_bw = here ? min(vhi + B, Wk - 1) - max(vlo - B, 0) + 1 : t_bw;
        ++nclu;
    }
    tc.t_r0 = t_r0, tc.t_c0 = t_c0, tc.t_bw = t_bw, tc.t_h = t_h, tc.nclu = nclu, tc.mine = mine;
    // the rest of each cluster's scalars, once for all clusters
    tc.t_inv = __builtin_amdgcn_rcpf(static_cast<float>(t_bw));
    tc.t_nb = (t_h * t_bw + 15) >> 4;
    box_slot(16, t_bw, tc.t_inv, tc.t_q16, tc.t_r16);
    tc.wr0 = 0, tc.wrn = -1, tc.wcols = 0, tc.rcut = INT_MIN, tc.wcut = 0;
    const int mc = max(mine, 0);
    const int r0 = __shfl(t_r0, mc), c0 = __shfl(t_c0, mc), bw = __shfl(t_bw, mc), h = __shfl(t_h, mc);
    if (mine >= 0) {
        tc.wr0 = u - B - r0;
        tc.wrn = min(u + B - r0, h - 1) - tc.wr0;
        const int lo = max(v - B - c0, 0), hi = min(v + B - c0, bw - 1);  // box columns, bw <= 31
        tc.wcols = ((2u << hi) - 1u) & ~((1u << lo) - 1u);
        if constexpr (CAUSAL) {
            const int cut = qx - r0 - tc.wr0;  // the query's row, as a window row
            if (cut >= 0 && cut <= tc.wrn) {
                const int qc = qy - c0;  // the query's column in the box
                tc.rcut = cut;
                tc.wcut = qc < 0 ? 0u : (qc >= 31 ? tc.wcols : tc.wcols & ((2u << qc) - 1u));
            }
            tc.wrn = min(tc.wrn, cut - 1);  // the rows before the query's
            if (tc.wrn < 0) tc.wcols = 0;   // none: no full row of the window counts
        }
    }
    return tc;
}

// Clusters of the centres of a wave's NJ (2 or 4) windows per query: lane i < 16 NJ holds centre i
// (window i / 16 of query i mod 16), the other lanes repeat them; valid is false for a centre that
// does not exist; mine is the cluster of the lane's centre.  Only the clusters' scalars are set (the
// caller places each window in its own box).
template <int B, int NJ>
__device__ __forceinline__ TileClusters tile_clusters_joint(bool valid, int u, int v, int lane, int rc, int Hk,
                                                            int Wk)
{
    static_assert(NJ == 2 || NJ == 4, "16 NJ centres in the lanes of a wave");
    constexpr uint64_t kItems = NJ == 4 ? ~0ull : 0xFFFFFFFFull;
    TileClusters tc;
    int t_r0 = 0, t_c0 = 0, t_bw = 1, t_h = 0;
    int nclu = 0, mine = -1;
    const int it = lane & (16 * NJ - 1);
    uint64_t todo = static_cast<uint64_t>(__ballot(valid)) & kItems;  // bit i: centre i
    while (todo) {
        const int a = __builtin_ctzll(todo);
        const int ua = __builtin_amdgcn_readlane(u, a), va = __builtin_amdgcn_readlane(v, a);
        const bool mem = ((todo >> it) & 1u) && abs(u - ua) <= rc && abs(v - va) <= rc;
        todo &= ~(static_cast<uint64_t>(__ballot(mem)) & kItems);
        mine = mem ? nclu : mine;
        int ulo = mem ? u : ua, uhi = ulo, vlo = mem ? v : va, vhi = vlo;
        row_minmax(ulo, uhi);
        row_minmax(vlo, vhi);
        // and across the 16-lane rows that hold the centres
        ulo = min(ulo, __shfl_xor(ulo, 16)), uhi = max(uhi, __shfl_xor(uhi, 16));
        vlo = min(vlo, __shfl_xor(vlo, 16)), vhi = max(vhi, __shfl_xor(vhi, 16));
        if constexpr (NJ == 4) {
            ulo = min(ulo, __shfl_xor(ulo, 32)), uhi = max(uhi, __shfl_xor(uhi, 32));
            vlo = min(vlo, __shfl_xor(vlo, 32)), vhi = max(vhi, __shfl_xor(vhi, 32));
        }
        const bool here = lane == nclu;
        t_r0 = here ? max(ulo - B, 0) : t_r0;
        t_c0 = here ? max(vlo - B, 0) : t_c0;
        t_h = here ? min(uhi + B, Hk - 1) - max(ulo - B, 0) + 1 : t_h;
        t_bw = here ? min(vhi + B, Wk - 1) - max(vlo - B, 0) + 1 : t_bw;
        ++nclu;
    }
    tc.t_r0 = t_r0, tc.t_c0 = t_c0, tc.t_bw = t_bw, tc.t_h = t_h, tc.nclu = nclu, tc.mine = mine;
    tc.t_inv = __builtin_amdgcn_rcpf(static_cast<float>(t_bw));
    tc.t_nb = (t_h * t_bw + 15) >> 4;
    box_slot(16, t_bw, tc.t_inv, tc.t_q16, tc.t_r16);
    tc.wr0 = 0, tc.wrn = -1, tc.wcols = 0, tc.rcut = INT_MIN, tc.wcut = 0;
    return tc;
}

// A cluster's scalars, read from the lanes that hold them.
struct TileBox {
    int r0, c0, bw, h, nb, q16, r16;
    float inv;
    uint32_t kstep, kstep_wrap;  // key index change of a 16-slot step, without and with a column carry
    uint32_t klast;              // key index of the box's last slot
};

__device__ __forceinline__ TileBox tile_box(const TileClusters& tc, int cl, int Wk)
{
    TileBox bx;
    bx.r0 = __builtin_amdgcn_readlane(tc.t_r0, cl);
    bx.c0 = __builtin_amdgcn_readlane(tc.t_c0, cl);
    bx.bw = __builtin_amdgcn_readlane(tc.t_bw, cl);
    bx.nb = __builtin_amdgcn_readlane(tc.t_nb, cl);
    bx.q16 = __builtin_amdgcn_readlane(tc.t_q16, cl);
    bx.r16 = __builtin_amdgcn_readlane(tc.t_r16, cl);
    bx.inv = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(tc.t_inv), cl));
    bx.kstep = static_cast<uint32_t>(bx.q16) * static_cast<uint32_t>(Wk) + bx.r16;
    bx.kstep_wrap = bx.kstep + Wk - bx.bw;
    bx.h = __builtin_amdgcn_readlane(tc.t_h, cl);
    bx.klast = static_cast<uint32_t>(bx.r0 + bx.h - 1) * static_cast<uint32_t>(Wk) + (bx.c0 + bx.bw - 1);
    return bx;
}

// Which of the 4 slots 16 k + 4 g4 + i of a block lie in query m's window (bit i), for the slot
// 16 k + 4 g4 at window row rr (box row wr0 + rr), column mcl; wc and wc2 are the window's column
// bits of that row and of the next one (shifted past the row's end), zero outside query m's own
// cluster; CAUSAL: wk and wk2 likewise for the query's own row, window row rcut.
template <bool CAUSAL = false>
__device__ __forceinline__ uint32_t tile_window_bits(const TileBox& bx, int rr, int mcl, int wrn, uint32_t wc,
                                                     uint32_t wc2, int rcut = 0, uint32_t wk = 0, uint32_t wk2 = 0)
{
    uint32_t bits = 0;
    if (bx.bw >= 3) {  // the 4 slots span at most two box rows: columns mcl .. mcl + 3 of row, next row
        const bool ok0 = static_cast<unsigned>(rr) <= static_cast<unsigned>(wrn);
        const bool ok1 = static_cast<unsigned>(rr + 1) <= static_cast<unsigned>(wrn);
        uint32_t w = (ok0 ? wc : 0u) | (ok1 ? wc2 : 0u);
        if constexpr (CAUSAL) w |= (rr == rcut ? wk : 0u) | (rr + 1 == rcut ? wk2 : 0u);
        bits = __builtin_amdgcn_ubfe(w, mcl, 4);
    } else {  // boxes one or two columns wide (grids that narrow): slot by slot
        int r = rr, cc = mcl;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            bool ok = static_cast<unsigned>(r) <= static_cast<unsigned>(wrn) && ((wc >> cc) & 1u);
            if constexpr (CAUSAL) ok = ok || (r == rcut && ((wk >> cc) & 1u));
            bits |= ok ? 1u << i : 0u;
            ++cc;
            const bool wrap = cc == bx.bw;
            cc = wrap ? 0 : cc;
            r += wrap ? 1 : 0;
        }
    }
    return bits;
}

// Which of the 4 slots of tile_window_bits lie at or before the query in raster order, for the slot
// 16 k + 4 g4 at box row rr, column mcl: the box rows before qr, and in row qr the box columns in qc.
__device__ __forceinline__ uint32_t tile_causal_bits(const TileBox& bx, int rr, int mcl, int qr, uint32_t qc)
{
    if (bx.bw >= 3) {  // the 4 slots span at most two box rows (bw <= 27: only bits below bw + 3 are read)
        const uint32_t full = (1u << bx.bw) - 1u;
        const uint32_t w0 = rr < qr ? full : (rr == qr ? qc : 0u);
        const uint32_t w1 = rr + 1 < qr ? full : (rr + 1 == qr ? qc : 0u);
        return __builtin_amdgcn_ubfe(w0 | (w1 << bx.bw), mcl, 4);
    }
    uint32_t bits = 0;
    int r = rr, cc = mcl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        bits |= r < qr || (r == qr && ((qc >> cc) & 1u)) ? 1u << i : 0u;
        ++cc;
        const bool wrap = cc == bx.bw;
        cc = wrap ? 0 : cc;
        r += wrap ? 1 : 0;
    }
    return bits;
}

// Box-column bits of the columns lo .. hi of a box `bw` wide (clipped to the box; zero when none is left).
__device__ __forceinline__ uint32_t tile_col_bits(int lo, int hi, int bw)
{
    lo = max(lo, 0), hi = min(hi, bw - 1);
    return lo <= hi ? ((2u << hi) - 1u) & ~((1u << lo) - 1u) : 0u;
}

// Which of the 4 slots of tile_window_bits lie in one of N other windows of side 2 B + 1: window f covers
// window rows d[f] .. d[f] + 2 B (rows of the window the slots are tested against) and the box columns
// in xw[f] (zero: no window).
template <int N, int B>
__device__ __forceinline__ uint32_t tile_other_bits(const TileBox& bx, int rr, int mcl, const int (&d)[N],
                                                    const uint32_t (&xw)[N])
{
    if (bx.bw >= 3) {
        uint32_t w = 0;
#pragma unroll
        for (int f = 0; f < N; ++f) {
            w |= static_cast<unsigned>(rr - d[f]) <= 2u * B ? xw[f] : 0u;
            w |= static_cast<unsigned>(rr + 1 - d[f]) <= 2u * B ? xw[f] << bx.bw : 0u;
        }
        return __builtin_amdgcn_ubfe(w, mcl, 4);
    }
    uint32_t bits = 0;
    int r = rr, cc = mcl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        bool in = false;
#pragma unroll
        for (int f = 0; f < N; ++f) in = in || (static_cast<unsigned>(r - d[f]) <= 2u * B && ((xw[f] >> cc) & 1u));
        bits |= in ? 1u << i : 0u;
        ++cc;
        const bool wrap = cc == bx.bw;
        cc = wrap ? 0 : cc;
        r += wrap ? 1 : 0;
    }
    return bits;
}

}  // namespace
}  // namespace scram
