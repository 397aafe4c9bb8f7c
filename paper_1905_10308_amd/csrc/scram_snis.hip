// Self-normalised importance sampling (Section 4.2, Equations 11-17).

#include "scram_device.h"

namespace scram {
namespace {

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
    int Hq, Wq;
    Tiling tq;             // blocks -> tiles of the query grid
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

// Sample t of query g: flat key index and log2 of its importance density
// (the query's kappa <= MK modes in cu, cv).
template <int MK>
__device__ __forceinline__ void snis_draw(const SnisParams& p, uint32_t g, uint32_t t, const int (&cu)[MK],
                                          const int (&cv)[MK], const float* pmf, const float* cdf, int32_t& j,
                                          float& lr2)
{
    const uint4 w = philox4x32_10(g, t, 0u, kSnisStream, p.key0, p.key1);
    int r, c;
    if ((w.x >> 16) < p.alpha16) {
        const uint32_t e = __umulhi(w.y, static_cast<uint32_t>(p.kappa));
        int u = cu[0], v = cv[0];
#pragma unroll
        for (int f = 1; f < MK; ++f)
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
    for (int e = 0; e < MK; ++e)
        if (e < p.kappa)
            local += axis_density(r, cu[e], p.Hk, p.m, pmf, cdf) * axis_density(c, cv[e], p.Wk, p.m, pmf, cdf);
    lr2 = log2f(fmaf(p.w_local, local, p.w_unif));
}

// Without the variance pass and with at most two modes the kernel fits 128
// VGPRs, i.e. four waves per SIMD; ask for that.  Otherwise the compiler's own
// allocation (three waves) stands.
template <bool VAR, int MK, bool KAHAN>
constexpr int snis_waves() { return !VAR && !KAHAN && MK <= 2 ? 4 : 1; }

// Compensated (Kahan) accumulation: s + x with the rounding error of each
// addition carried in c (the sum is s - c).  Sums of thousands of weights
// that repeat the same few values would otherwise round the same way at
// every addition and drift by up to T * 2^-24 relative.
__device__ __forceinline__ void kahan_add(float& s, float& c, float y_minus_c)
{
    const float t = s + y_minus_c;
    c = (t - s) - y_minus_c;
    s = t;
}

// Samples above which the sums are compensated (below, plain fp32 sums stay
// within a few hundred units of the last place).
constexpr int kKahanSamples = 256;

template <typename T, int D, int G, bool VAR, int MK, bool KAHAN>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(snis_waves<VAR, MK, KAHAN>())))
void snis_kernel(SnisParams p)
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
    uint32_t g;
    if (!tile_item<RW::kQpb>(p.tq, blk, threadIdx.x / G, g)) return;  // whole lane groups leave together

    uint32_t s, rem;
    divmod(g, p.div_plane, s, rem);
    const size_t slice = static_cast<size_t>(s) * p.nkeys * D;
    const T* Ks = static_cast<const T*>(p.K) + slice;
    const T* Vs = static_cast<const T*>(p.V) + slice;
    uint4 q[CH];
    load_row<T, D, G>(static_cast<const T*>(p.Q), g, lane, q);
    int cu[MK], cv[MK];
#pragma unroll
    for (int e = 0; e < MK; ++e) {
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
            if (sl < kNb && t0 + sl < p.samples) snis_draw<MK>(p, g, t0 + sl, cu, cv, s_pmf, s_cdf, mj[i], ml[i]);
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

    float M = -INFINITY, S1 = 0.f, S2 = 0.f, S1c = 0.f, S2c = 0.f;  // *c: Kahan compensations
    float acc[E], accc[KAHAN ? E : 1];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;
#pragma unroll
    for (int e = 0; e < (KAHAN ? E : 1); ++e) accc[e] = 0.f;
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
        if constexpr (KAHAN) {
            S1c *= alpha;
            S2c *= alpha * alpha;
#pragma unroll
            for (int e = 0; e < E; ++e) accc[e] *= alpha;
        }
#pragma unroll
        for (int sl = 0; sl < kNb; ++sl) {
            const float pj = __builtin_amdgcn_exp2f(lw[sl] - mb);  // exp2(-inf) = 0
            if constexpr (KAHAN) {
                kahan_add(S1, S1c, pj - S1c);
                kahan_add(S2, S2c, fmaf(pj, pj, -S2c));
                float vals[E];
                unpack_row<T, CH>(vr[sl], vals);
#pragma unroll
                for (int e = 0; e < E; ++e) kahan_add(acc[e], accc[e], fmaf(pj, vals[e], -accc[e]));
            } else {
                S1 += pj;
                S2 += pj * pj;
                accumulate_row<T, CH>(acc, pj, vr[sl]);
            }
        }
        M = mb;
    }
    if constexpr (KAHAN) {
        S1 -= S1c;
        S2 -= S2c;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] -= accc[e];
    }
    const float inv = S1 > 0.f ? 1.f / S1 : 0.f;  // no usable sample: zero row

    if constexpr (VAR) {
        // second pass over the same samples: sum_t (w_t / sum w)^2 (v_t - estimate)^2
        float mean[E], vacc[E], vaccc[KAHAN ? E : 1];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            mean[e] = acc[e] * inv;
            vacc[e] = 0.f;
        }
#pragma unroll
        for (int e = 0; e < (KAHAN ? E : 1); ++e) vaccc[e] = 0.f;
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
                        if constexpr (KAHAN)
                            kahan_add(vacc[e], vaccc[e], fmaf(wn2 * dlt, dlt, -vaccc[e]));
                        else
                            vacc[e] = fmaf(wn2 * dlt, dlt, vacc[e]);
                    }
                }
            }
            if constexpr (KAHAN) {
#pragma unroll
                for (int e = 0; e < E; ++e) vacc[e] -= vaccc[e];
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

template <typename T, int D>
hipError_t run_snis(const SnisParams& p0, hipStream_t st, hipEvent_t e0, hipEvent_t e1)
{
    constexpr int G = Lanes<T, D>::kAttend;
    SnisParams p = p0;
    p.tq = make_tiling(p.Hq, p.Wq, Row<T, D, G>::kQpb, kLaneSkew);
    const uint64_t blocks = tiling_blocks(p.tq, p.n / p.tq.plane);
    // the smallest register budget that holds the query's modes
    auto go = [&](auto mk) {
        constexpr int MK = decltype(mk)::value;
        if (p.samples > kKahanSamples) {
            if (p.var) return launch(snis_kernel<T, D, G, true, MK, true>, blocks, st, e0, e1, p);
            return launch(snis_kernel<T, D, G, false, MK, true>, blocks, st, e0, e1, p);
        }
        if (p.var) return launch(snis_kernel<T, D, G, true, MK, false>, blocks, st, e0, e1, p);
        return launch(snis_kernel<T, D, G, false, MK, false>, blocks, st, e0, e1, p);
    };
    if (p.kappa == 1) return go(std::integral_constant<int, 1>{});
    if (p.kappa == 2) return go(std::integral_constant<int, 2>{});
    if (p.kappa <= 4) return go(std::integral_constant<int, 4>{});
    return go(std::integral_constant<int, kMaxKappa>{});
}

}  // namespace

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
    p.Hq = g.Hq;
    p.Wq = g.Wq;
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

uint64_t snis_max_blocks(int dtype, const Grid& g)
{
    return dispatch_value(dtype, g.d, uint64_t(0), [&](auto t, auto d) {
        using T = decltype(t);
        constexpr int D = decltype(d)::value;
        return tiling_blocks(make_tiling(g.Hq, g.Wq, Row<T, D, Lanes<T, D>::kAttend>::kQpb, kLaneSkew), g.S);
    });
}

}  // namespace scram
