/*
 * scram_oracle.c -- plain fp64 CPU reference ("the oracle") for the SCRAM hot
 * path: PatchMatch argmax (Algorithm 1 at kappa = 1) followed by the sparse
 * window softmax / value gather (Algorithm 2, Equations 8-9).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The product path (the
 * HIP library under paper_1905_10308_amd/) never links, imports or calls it,
 * and this file shares no code, header, table or helper with that path.
 *
 * Written for a reader holding the paper.  Every floating-point quantity is
 * double; inputs are passed in as double (bf16 / fp32 data upcast exactly by
 * the caller).  Nothing here is blocked, fused or reordered beyond what the
 * algorithm states: one query at a time, candidates in the paper's order.
 * OpenMP (when enabled at build time) only splits the "parallel foreach" over
 * queries of one iteration; every read of an iteration comes from the map of
 * the previous iteration, so the thread count never changes a result.
 *
 * Readings of points the paper leaves open (each is also listed in the design
 * notes of the repository):
 *   - propagation (Alg. 1, propagation step): the candidate offered by the
 *     neighbour at p + jump*delta is that neighbour's match shifted back by
 *     jump*delta (coherent shift, Section 4.1 assumption (1));
 *   - the parallel foreach reads only the previous iteration's field (Jacobi);
 *   - out-of-grid neighbours and out-of-grid candidates are skipped; at
 *     kappa = 1 is_index_valid reduces to "inside the key grid";
 *   - "better" is a strict total order: higher score, then lower flat key
 *     index, so the visiting order of candidates never matters;
 *   - random search (Alg. 1, random search step): distances R, R/2, ... , 1
 *     with integer halving and R = max(Hk, Wk); a candidate is drawn
 *     uniformly from the square of half-side D around the running best,
 *     clipped to the key grid; the draw maps a 32-bit word w to
 *     lo + floor(w * (hi - lo + 1) / 2^32);
 *   - the random words come from Philox4x32-10 (Salmon, Moraes, Dror, Shaw,
 *     "Parallel random numbers: as easy as 1, 2, 3", SC 2011) with
 *     key = (seed mod 2^32, seed div 2^32).  Initialisation of query g uses
 *     counter (g, 0, 0, 0), words 0 and 1 for (u, v).  Iteration t >= 1,
 *     random-search step k uses counter (g, t, k div 2, 0), words
 *     2*(k mod 2) and 2*(k mod 2) + 1 for (row, column);
 *   - PatchMatch compares unscaled dot products q.k (the argmax does not
 *     depend on a positive scale); the attend step uses the caller's scale;
 *   - attend window keys outside the key grid are dropped and the softmax is
 *     normalised over the keys that remain (Alg. 2, Eq. 8).
 *
 * Several matches per query (kappa > 1, Section 4.2 and Algorithm 2's first
 * step): run c of PatchMatch receives the C = c maps of the previous runs and
 * is_index_valid rejects a key closer than L to any of them in Chebyshev
 * distance (max(|du|, |dv|) < L); L = 1 keeps only distinct keys (the
 * top-kappa-max variant), L > 1 keeps the matches apart (top-kappa-mode).  An
 * incumbent that is not valid counts as minus infinity, so the first valid
 * candidate replaces it.  Run c draws its random numbers with counter word 3
 * equal to c.  Algorithm 2 then attends over the union of the kappa windows,
 * every key once.
 *
 * Causal masking (Section 4.2.1), for a query grid equal to the key grid: a
 * key is valid for query i only if its raster index is at most i.  The
 * initial match is drawn uniformly from the valid keys, and the attend
 * window drops keys after the query.
 *
 * Backward of the sparse attention: the gradients with respect to Q, K and
 * V with the maps held fixed (the key sets are not differentiable).
 *
 * Self-normalised importance sampling (Section 4.2, Monte Carlo estimators,
 * Equations 11-17): the importance distribution mixes, with weight alpha, a
 * local density around each of the kappa PatchMatch modes and, with weight
 * 1 - alpha, the uniform distribution over the n = Hk * Wk keys.  Readings:
 *   - the local density is a discrete Gaussian written as a centred binomial
 *     per axis: offset = (number of ones among 2m fair bits) - m, so its
 *     pmf is C(2m, offset + m) / 4^m and its variance m / 2 (length-scale
 *     phi = sqrt(m / 2)); a row or column beyond the grid is clamped to the
 *     edge, which then holds the tail mass of that side;
 *   - alpha is used as round(alpha * 65536) / 65536;
 *   - sample t of query g uses the Philox block of counter
 *     (g, t, 0, 0x534E4953): word 0's upper 16 bits below round(alpha *
 *     65536) choose a mode (word 1, uniform over the kappa modes; words 2
 *     and 3 give the 2m row and 2m column bits, m <= 16), otherwise words
 *     2 and 3 draw a uniform row and column;
 *   - the variance estimate of Equation 15 uses the self-normalised weights
 *     w_t / sum_s w_s (with raw weights it would change with any constant
 *     factor in p^(u), which the estimator itself ignores).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_NO_PROPAGATION 1u
#define OR_NO_RANDOM_SEARCH 2u
#define OR_CAUSAL 4u

/* ------------------------------------------------------------------------ */
/* Philox4x32-10, from its published description: ten rounds; each round   */
/* multiplies words 0 and 2 by two fixed 32-bit constants, takes the high  */
/* and low halves of the 64-bit products and mixes them with words 1 and 3 */
/* and the round key; the key advances by two Weyl constants per round.    */
/* ------------------------------------------------------------------------ */
static const uint32_t PHILOX_MUL_A = 0xD2511F53u;
static const uint32_t PHILOX_MUL_B = 0xCD9E8D57u;
static const uint32_t PHILOX_WEYL_A = 0x9E3779B9u;
static const uint32_t PHILOX_WEYL_B = 0xBB67AE85u;

static void philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t x0 = ctr_in[0], x1 = ctr_in[1], x2 = ctr_in[2], x3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t pa = (uint64_t)PHILOX_MUL_A * (uint64_t)x0;
        uint64_t pb = (uint64_t)PHILOX_MUL_B * (uint64_t)x2;
        uint32_t pa_hi = (uint32_t)(pa >> 32), pa_lo = (uint32_t)pa;
        uint32_t pb_hi = (uint32_t)(pb >> 32), pb_lo = (uint32_t)pb;
        uint32_t y0 = pb_hi ^ x1 ^ k0;
        uint32_t y1 = pb_lo;
        uint32_t y2 = pa_hi ^ x3 ^ k1;
        uint32_t y3 = pa_lo;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
        k0 += PHILOX_WEYL_A;
        k1 += PHILOX_WEYL_B;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* Exposed so that a test can compare this generator with a library one. */
void oracle_philox4x32_10(const uint32_t* ctr, const uint32_t* key, uint32_t* out)
{
    philox4x32_10(ctr, key, out);
}

static void seed_key(uint64_t seed, uint32_t key[2])
{
    key[0] = (uint32_t)(seed & 0xffffffffu);
    key[1] = (uint32_t)(seed >> 32);
}

/* Uniform integer in [lo, hi] from one 32-bit word (multiply-high map). */
static int64_t pick_in_range(uint32_t w, int64_t lo, int64_t hi)
{
    uint64_t span = (uint64_t)(hi - lo + 1);
    return lo + (int64_t)(((uint64_t)w * span) >> 32);
}

/* ------------------------------------------------------------------------ */
/* Scores: Eq. 1 without the 1/sqrt(d_k) factor for PatchMatch.            */
/* ------------------------------------------------------------------------ */
static double dot(const double* a, const double* b, int d)
{
    double s = 0.0;
    for (int e = 0; e < d; ++e) s += a[e] * b[e];
    return s;
}

/* sum_e |a_e b_e|: the scale against which two dot products are "near". */
static double absdot(const double* a, const double* b, int d)
{
    double s = 0.0;
    for (int e = 0; e < d; ++e) s += fabs(a[e] * b[e]);
    return s;
}

/* higher score wins; equal scores go to the lower flat key index */
static int better(double sa, int64_t ia, double sb, int64_t ib)
{
    return sa > sb || (sa == sb && ia < ib);
}

typedef struct {
    const double* Q; /* [S, Hq, Wq, d] */
    const double* K; /* [S, Hk, Wk, d] */
    int64_t S, Hq, Wq, Hk, Wk;
    int d;
    uint32_t key[2];
    uint32_t flags;
    double tie_rel;
    const int32_t* prev; /* [n_prev, S, Hq, Wq] maps of previous runs, or NULL */
    int64_t n_prev;
    int64_t sep;         /* minimum Chebyshev distance to every previous match */
} pm_problem;

/* is_index_valid: key idx for query g (Algorithm 1, propagation and random search). */
static int index_valid(const pm_problem* P, int64_t g, int64_t idx)
{
    const int64_t plane = P->Hq * P->Wq;
    if ((P->flags & OR_CAUSAL) && idx > g % plane) return 0;
    const int64_t u = idx / P->Wk, v = idx % P->Wk;
    for (int64_t c = 0; c < P->n_prev; ++c) {
        const int64_t pj = P->prev[c * P->S * plane + g];
        const int64_t du = llabs(u - pj / P->Wk), dv = llabs(v - pj % P->Wk);
        const int64_t cheb = du > dv ? du : dv;
        if (cheb < P->sep) return 0;
    }
    return 1;
}

/* running state of one query inside one iteration */
typedef struct {
    const double* q;
    const double* Ks; /* key image of the query's slice */
    int64_t cur;      /* flat key index u*Wk + v */
    double best;      /* q . k_cur */
    double best_abs;  /* sum |q_e k_cur,e| */
    int tie;          /* a comparison of two different keys was within tie_rel */
    int64_t ncand;    /* candidates scored */
    /* optional trace of every scored candidate */
    int64_t* trace_idx;
    int32_t* trace_kind;
    double* trace_centre; /* for random-search entries: the window it was drawn from */
    int64_t trace_cap, trace_len;
} pm_state;

static void consider(const pm_problem* P, pm_state* st, int64_t g, int64_t r, int64_t c, int kind,
                     const int64_t window[4])
{
    int64_t idx = r * P->Wk + c;
    if (!index_valid(P, g, idx)) return;
    const double* k = st->Ks + idx * P->d;
    double sc = dot(st->q, k, P->d);
    st->ncand += 1;
    if (idx != st->cur && st->best != -INFINITY) {
        double a = absdot(st->q, k, P->d);
        double scale = a > st->best_abs ? a : st->best_abs;
        if (fabs(sc - st->best) <= P->tie_rel * scale) st->tie = 1;
    }
    if (st->trace_idx && st->trace_len < st->trace_cap) {
        int64_t n = st->trace_len++;
        st->trace_idx[n] = idx;
        st->trace_kind[n] = kind;
        for (int i = 0; i < 4; ++i) st->trace_centre[4 * n + i] = window ? (double)window[i] : -1.0;
    }
    if (better(sc, idx, st->best, st->cur)) {
        st->cur = idx;
        st->best = sc;
        st->best_abs = absdot(st->q, k, P->d);
    }
}

/*
 * One iteration of Algorithm 1 for query g: propagation from the neighbours
 * at distances 8, 4, 2, 1 in the four axis directions, then random search at
 * distances R, R/2, ..., 1 around the running best.  Reads J_prev / s_prev.
 */
static void pm_query_iteration(const pm_problem* P, int64_t g, int64_t t,
                               const int32_t* J_prev, const double* s_prev, pm_state* st)
{
    const int64_t plane = P->Hq * P->Wq;
    const int64_t s = g / plane;
    const int64_t x = (g % plane) / P->Wq;
    const int64_t y = g % P->Wq;
    st->q = P->Q + g * P->d;
    st->Ks = P->K + s * P->Hk * P->Wk * P->d;
    st->cur = J_prev[g];
    st->best = index_valid(P, g, st->cur) ? s_prev[g] : -INFINITY;
    st->best_abs = absdot(st->q, st->Ks + st->cur * P->d, P->d);

    if (!(P->flags & OR_NO_PROPAGATION)) {
        static const int jumps[4] = {8, 4, 2, 1};
        static const int dirs[4][2] = {{-1, 0}, {1, 0}, {0, -1}, {0, 1}};
        for (int jj = 0; jj < 4; ++jj) {
            for (int dd = 0; dd < 4; ++dd) {
                int64_t ox = (int64_t)jumps[jj] * dirs[dd][0];
                int64_t oy = (int64_t)jumps[jj] * dirs[dd][1];
                int64_t nx = x + ox, ny = y + oy;
                if (nx < 0 || nx >= P->Hq || ny < 0 || ny >= P->Wq) continue;
                int64_t nb = J_prev[s * plane + nx * P->Wq + ny];
                int64_t r = nb / P->Wk - ox;
                int64_t c = nb % P->Wk - oy;
                if (r < 0 || r >= P->Hk || c < 0 || c >= P->Wk) continue;
                consider(P, st, g, r, c, 1 + 4 * jj + dd, NULL);
            }
        }
    }

    if (!(P->flags & OR_NO_RANDOM_SEARCH)) {
        int64_t D = P->Hk > P->Wk ? P->Hk : P->Wk;
        for (int64_t k = 0;; ++k) {
            uint32_t ctr[4] = {(uint32_t)g, (uint32_t)t, (uint32_t)(k / 2), (uint32_t)P->n_prev};
            uint32_t w[4];
            philox4x32_10(ctr, P->key, w);
            uint32_t w_row = w[2 * (k % 2)], w_col = w[2 * (k % 2) + 1];
            int64_t u = st->cur / P->Wk, v = st->cur % P->Wk;
            int64_t lo_r = u - D < 0 ? 0 : u - D;
            int64_t hi_r = u + D > P->Hk - 1 ? P->Hk - 1 : u + D;
            int64_t lo_c = v - D < 0 ? 0 : v - D;
            int64_t hi_c = v + D > P->Wk - 1 ? P->Wk - 1 : v + D;
            int64_t window[4] = {lo_r, hi_r, lo_c, hi_c};
            int64_t r = pick_in_range(w_row, lo_r, hi_r);
            int64_t c = pick_in_range(w_col, lo_c, hi_c);
            consider(P, st, g, r, c, 100 + (int)k, window);
            if (D == 1) break;
            D /= 2;
        }
    }
}

static int check_dims(int64_t S, int64_t Hq, int64_t Wq, int64_t Hk, int64_t Wk, int d)
{
    if (S <= 0 || Hq <= 0 || Wq <= 0 || Hk <= 0 || Wk <= 0 || d <= 0) return -2;
    if (S * Hq * Wq >= ((int64_t)1 << 31) || Hk * Wk >= ((int64_t)1 << 31)) return -2;
    return 0;
}

/*
 * Random initialisation of the nearest-neighbour field (Alg. 1, first loop)
 * for run n_prev: counter (g, 0, 0, n_prev).  J0[g] = u*Wk + v with u uniform
 * in [0, Hk), v uniform in [0, Wk) (words 0, 1) -- or, with OR_CAUSAL, the
 * flat index uniform over the keys up to the query's own raster index
 * (word 0) -- and the fp64 score s0[g] = q_g . k_J0[g].
 */
int oracle_pm_init(const double* Q, const double* K, int64_t S, int64_t Hq, int64_t Wq,
                   int64_t Hk, int64_t Wk, int d, uint64_t seed, uint32_t flags, int64_t n_prev,
                   int32_t* J0, double* s0)
{
    if (check_dims(S, Hq, Wq, Hk, Wk, d) || n_prev < 0) return -2;
    if ((flags & OR_CAUSAL) && (Hq != Hk || Wq != Wk)) return -2;
    uint32_t key[2];
    seed_key(seed, key);
    const int64_t n = S * Hq * Wq, plane = Hq * Wq;
#pragma omp parallel for schedule(static)
    for (int64_t g = 0; g < n; ++g) {
        uint32_t ctr[4] = {(uint32_t)g, 0u, 0u, (uint32_t)n_prev};
        uint32_t w[4];
        philox4x32_10(ctr, key, w);
        int64_t idx;
        if (flags & OR_CAUSAL) {
            idx = pick_in_range(w[0], 0, g % plane);
        } else {
            int64_t u = pick_in_range(w[0], 0, Hk - 1);
            int64_t v = pick_in_range(w[1], 0, Wk - 1);
            idx = u * Wk + v;
        }
        J0[g] = (int32_t)idx;
        const double* Ks = K + (g / plane) * Hk * Wk * d;
        s0[g] = dot(Q + g * d, Ks + idx * d, d);
    }
    return 0;
}

/* fp64 score q_g . k_J[g] and its magnitude scale sum_e |q_e k_e| per query. */
int oracle_pm_scores(const double* Q, const double* K, int64_t S, int64_t Hq, int64_t Wq,
                     int64_t Hk, int64_t Wk, int d, const int32_t* J, double* score,
                     double* score_abs)
{
    if (check_dims(S, Hq, Wq, Hk, Wk, d)) return -2;
    const int64_t n = S * Hq * Wq, plane = Hq * Wq;
    for (int64_t g = 0; g < n; ++g)
        if (J[g] < 0 || J[g] >= Hk * Wk) return -2;
#pragma omp parallel for schedule(static)
    for (int64_t g = 0; g < n; ++g) {
        const double* k = K + (g / plane) * Hk * Wk * d + (int64_t)J[g] * d;
        score[g] = dot(Q + g * d, k, d);
        if (score_abs) score_abs[g] = absdot(Q + g * d, k, d);
    }
    return 0;
}

/*
 * One Jacobi iteration t (t >= 1) of run n_prev (with the maps of the n_prev
 * previous runs in prev) over the queries listed in query_ids (all
 * queries when query_ids is NULL).  Outputs are compact: entry i belongs to
 * query_ids[i] (or to query i).  tie_out[i] = 1 when some comparison made for
 * that query put two different keys within tie_rel * max(sum|q k|) of each
 * other.  *ncand_out receives the number of candidates scored.
 */
int oracle_pm_iteration(const double* Q, const double* K, int64_t S, int64_t Hq, int64_t Wq,
                        int64_t Hk, int64_t Wk, int d, uint64_t seed, int64_t t, uint32_t flags,
                        double tie_rel, const int32_t* prev, int64_t n_prev, int64_t sep,
                        const int32_t* J_prev, const double* s_prev,
                        const int64_t* query_ids, int64_t nq, int32_t* J_out, double* s_out,
                        uint8_t* tie_out, int64_t* ncand_out)
{
    if (check_dims(S, Hq, Wq, Hk, Wk, d) || t < 1 || n_prev < 0 || sep < 1) return -2;
    if ((flags & OR_CAUSAL) && (Hq != Hk || Wq != Wk)) return -2;
    if (n_prev > 0 && !prev) return -1;
    pm_problem P = {Q, K, S, Hq, Wq, Hk, Wk, d, {0, 0}, flags, tie_rel, prev, n_prev, sep};
    seed_key(seed, P.key);
    const int64_t n = S * Hq * Wq;
    const int64_t count = query_ids ? nq : n;
    for (int64_t g = 0; g < n; ++g)
        if (J_prev[g] < 0 || J_prev[g] >= Hk * Wk) return -2;
    if (query_ids)
        for (int64_t i = 0; i < nq; ++i)
            if (query_ids[i] < 0 || query_ids[i] >= n) return -2;
    int64_t total = 0;
#pragma omp parallel for schedule(static) reduction(+ : total)
    for (int64_t i = 0; i < count; ++i) {
        int64_t g = query_ids ? query_ids[i] : i;
        pm_state st;
        memset(&st, 0, sizeof st);
        pm_query_iteration(&P, g, t, J_prev, s_prev, &st);
        J_out[i] = (int32_t)st.cur;
        s_out[i] = st.best;
        if (tie_out) tie_out[i] = (uint8_t)st.tie;
        total += st.ncand;
    }
    if (ncand_out) *ncand_out = total;
    return 0;
}

/*
 * Trace of one query's iteration t: every scored (valid) candidate in order, its kind
 * (1 + 4*jump_index + direction_index for propagation, 100 + k for random
 * search step k) and, for random-search entries, the clipped window
 * (lo_r, hi_r, lo_c, hi_c) it was drawn from.  Returns the entry count.
 */
int64_t oracle_pm_trace(const double* Q, const double* K, int64_t S, int64_t Hq, int64_t Wq,
                        int64_t Hk, int64_t Wk, int d, uint64_t seed, int64_t t, uint32_t flags,
                        const int32_t* prev, int64_t n_prev, int64_t sep,
                        const int32_t* J_prev, const double* s_prev, int64_t g, int64_t cap,
                        int64_t* idx_out, int32_t* kind_out, double* window_out,
                        int32_t* final_out)
{
    if (check_dims(S, Hq, Wq, Hk, Wk, d) || t < 1 || g < 0 || g >= S * Hq * Wq) return -2;
    if (n_prev < 0 || sep < 1 || (n_prev > 0 && !prev)) return -2;
    if ((flags & OR_CAUSAL) && (Hq != Hk || Wq != Wk)) return -2;
    pm_problem P = {Q, K, S, Hq, Wq, Hk, Wk, d, {0, 0}, flags, 0.0, prev, n_prev, sep};
    seed_key(seed, P.key);
    pm_state st;
    memset(&st, 0, sizeof st);
    st.trace_idx = idx_out;
    st.trace_kind = kind_out;
    st.trace_centre = window_out;
    st.trace_cap = cap;
    pm_query_iteration(&P, g, t, J_prev, s_prev, &st);
    if (final_out) *final_out = (int32_t)st.cur;
    return st.trace_len;
}

/*
 * Whole PatchMatch run (Algorithm 1) number n_prev, given the maps of the
 * n_prev previous runs: random initialisation when init is NULL (else J_0 =
 * init and s_0 its fp64 scores), then iterations t0 .. t0 + iters - 1.
 * s_out holds minus infinity for a query whose final match is not valid.  ties_out (nullable) is [iters, n]: the tie flags of
 * each iteration.  ncand_out (nullable) receives the total candidates scored.
 */
int oracle_patchmatch(const double* Q, const double* K, int64_t S, int64_t Hq, int64_t Wq,
                      int64_t Hk, int64_t Wk, int d, int64_t iters, uint64_t seed,
                      const int32_t* init, int64_t t0, uint32_t flags, double tie_rel,
                      const int32_t* prev, int64_t n_prev, int64_t sep,
                      int32_t* J_out, double* s_out, uint8_t* ties_out, int64_t* ncand_out)
{
    if (check_dims(S, Hq, Wq, Hk, Wk, d) || iters < 0 || t0 < 1) return -2;
    const int64_t n = S * Hq * Wq;
    int32_t* Ja = (int32_t*)malloc(sizeof(int32_t) * n);
    int32_t* Jb = (int32_t*)malloc(sizeof(int32_t) * n);
    double* sa = (double*)malloc(sizeof(double) * n);
    double* sb = (double*)malloc(sizeof(double) * n);
    int rc = 0;
    int64_t total = 0;
    if (!Ja || !Jb || !sa || !sb) { rc = -6; goto done; }
    if (init) {
        memcpy(Ja, init, sizeof(int32_t) * n);
        rc = oracle_pm_scores(Q, K, S, Hq, Wq, Hk, Wk, d, Ja, sa, NULL);
    } else {
        rc = oracle_pm_init(Q, K, S, Hq, Wq, Hk, Wk, d, seed, flags, n_prev, Ja, sa);
    }
    if (rc) goto done;
    for (int64_t it = 0; it < iters; ++it) {
        int64_t nc = 0;
        rc = oracle_pm_iteration(Q, K, S, Hq, Wq, Hk, Wk, d, seed, t0 + it, flags, tie_rel, prev, n_prev,
                                 sep, Ja, sa, NULL, 0, Jb, sb, ties_out ? ties_out + it * n : NULL, &nc);
        if (rc) goto done;
        total += nc;
        int32_t* tj = Ja; Ja = Jb; Jb = tj;
        double* ts = sa; sa = sb; sb = ts;
    }
    memcpy(J_out, Ja, sizeof(int32_t) * n);
    if (s_out) memcpy(s_out, sa, sizeof(double) * n);
    if (ncand_out) *ncand_out = total;
done:
    free(Ja); free(Jb); free(sa); free(sb);
    return rc;
}

/* key (r, c) lies in the window of half-width b centred on flat key index centre */
static int in_window(int64_t r, int64_t c, int64_t centre, int64_t Wk, int64_t b)
{
    return llabs(r - centre / Wk) <= b && llabs(c - centre % Wk) <= b;
}

/*
 * The key set of query g in Algorithm 2: the union over the kappa matches
 * e of the windows {(u_e + a, v_e + c) : |a|, |c| <= b} (each key once, in
 * the order first met), intersected with the key grid and, with OR_CAUSAL,
 * with the keys up to the query.  keys must hold kappa * (2b+1)^2 entries.
 */
static int64_t window_keys(const int32_t* J, int64_t kappa, int64_t n, int64_t g, int64_t Hk, int64_t Wk, int64_t b,
                           int64_t last, int64_t* keys)
{
    int64_t nk = 0;
    for (int64_t e = 0; e < kappa; ++e) {
        const int64_t centre = J[e * n + g];
        const int64_t u = centre / Wk, v = centre % Wk;
        for (int64_t a = -b; a <= b; ++a)
            for (int64_t c = -b; c <= b; ++c) {
                int64_t r = u + a, col = v + c;
                if (r < 0 || r >= Hk || col < 0 || col >= Wk) continue;
                if (r * Wk + col > last) continue;
                int seen = 0; /* already in the window of an earlier match */
                for (int64_t f = 0; f < e && !seen; ++f) seen = in_window(r, col, J[f * n + g], Wk, b);
                if (!seen) keys[nk++] = r * Wk + col;
            }
    }
    return nk;
}

static int attend_args(const int32_t* J, int64_t kappa, int64_t S, int64_t Hq, int64_t Wq, int64_t Hk, int64_t Wk,
                       int d, int dv, int window, uint32_t flags)
{
    if (check_dims(S, Hq, Wq, Hk, Wk, d) || dv <= 0 || window < 1 || window % 2 == 0 || kappa < 1) return -2;
    if ((flags & OR_CAUSAL) && (Hq != Hk || Wq != Wk)) return -2;
    const int64_t n = S * Hq * Wq;
    for (int64_t g = 0; g < kappa * n; ++g)
        if (J[g] < 0 || J[g] >= Hk * Wk) return -2;
    return 0;
}

/*
 * Sparse non-local mean (Algorithm 2, Equations 8-9): for each listed query i
 * the key set above, scores a_j = scale * q_i . k_j and the output
 * sum_j softmax(a)_j v_j.  J is [kappa, S, Hq, Wq].  Two passes: the maximum
 * score first, then exp(a_j - max) weights.  An empty set (possible only with
 * OR_CAUSAL and a match after the query) gives a zero row.  out is compact
 * [count, dv].
 */
int oracle_sparse_attend(const double* Q, const double* K, const double* V, const int32_t* J,
                         int64_t kappa, int64_t S, int64_t Hq, int64_t Wq, int64_t Hk, int64_t Wk, int d,
                         int dv, int window, double scale, uint32_t flags, const int64_t* query_ids,
                         int64_t nq, double* out)
{
    if (attend_args(J, kappa, S, Hq, Wq, Hk, Wk, d, dv, window, flags)) return -2;
    const int64_t n = S * Hq * Wq, plane = Hq * Wq;
    const int64_t b = window / 2;
    const int64_t count = query_ids ? nq : n;
    if (query_ids)
        for (int64_t i = 0; i < nq; ++i)
            if (query_ids[i] < 0 || query_ids[i] >= n) return -2;
    const int64_t wr = window < Hk ? window : Hk, wc = window < Wk ? window : Wk;
    const int64_t cap = kappa * wr * wc; /* at most this many keys in one query's set */
    int rc = 0;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        int64_t g = query_ids ? query_ids[i] : i;
        int64_t s = g / plane;
        const int64_t last = (flags & OR_CAUSAL) ? g % plane : Hk * Wk - 1;
        const double* q = Q + g * d;
        const double* Ks = K + s * Hk * Wk * d;
        const double* Vs = V + s * Hk * Wk * dv;
        double* o = out + i * dv;
        int64_t* keys = (int64_t*)malloc(sizeof(int64_t) * cap);
        if (!keys) {
            rc = -6;
            continue;
        }
        /* 1. the key set: every window, clipped to the grid, each key once */
        const int64_t nk = window_keys(J, kappa, n, g, Hk, Wk, b, last, keys);
        /* 2. softmax over the set (two passes) and the weighted sum of values */
        double m = -INFINITY;
        for (int64_t j = 0; j < nk; ++j) {
            double sc = scale * dot(q, Ks + keys[j] * d, d);
            if (sc > m) m = sc;
        }
        double denom = 0.0;
        for (int e = 0; e < dv; ++e) o[e] = 0.0;
        for (int64_t j = 0; j < nk; ++j) {
            double w = exp(scale * dot(q, Ks + keys[j] * d, d) - m);
            denom += w;
            const double* vv = Vs + keys[j] * dv;
            for (int e = 0; e < dv; ++e) o[e] += w * vv[e];
        }
        for (int e = 0; e < dv; ++e) o[e] = nk > 0 ? o[e] / denom : 0.0; /* empty set: zero row */
        free(keys);
    }
    return rc;
}

/*
 * Gradients of the sparse attention output with the maps held fixed (the
 * key sets do not depend on Q, K, V).  With p_j the softmax weights of query
 * i over its key set, dp_j = dO_i . v_j and D_i = sum_j p_j dp_j
 * (= dO_i . o_i), the score gradient is ds_j = p_j (dp_j - D_i), and
 *   dQ_i += scale * sum_j ds_j k_j,   dK_j += scale * ds_j q_i,   dV_j += p_j dO_i.
 * Queries are visited in order (the scatter into dK, dV is sequential).
 * dQ [S,Hq,Wq,d], dK [S,Hk,Wk,d], dV [S,Hk,Wk,dv] are overwritten.
 */
int oracle_sparse_attend_backward(const double* Q, const double* K, const double* V, const int32_t* J, int64_t kappa,
                                  int64_t S, int64_t Hq, int64_t Wq, int64_t Hk, int64_t Wk, int d, int dv, int window,
                                  double scale, uint32_t flags, const double* dO, double* dQ, double* dK, double* dV)
{
    if (attend_args(J, kappa, S, Hq, Wq, Hk, Wk, d, dv, window, flags)) return -2;
    const int64_t n = S * Hq * Wq, plane = Hq * Wq, nkeys = Hk * Wk;
    const int64_t b = window / 2;
    const int64_t wr = window < Hk ? window : Hk, wc = window < Wk ? window : Wk;
    const int64_t cap = kappa * wr * wc;
    int64_t* keys = (int64_t*)malloc(sizeof(int64_t) * cap);
    double* p = (double*)malloc(sizeof(double) * cap);
    double* dp = (double*)malloc(sizeof(double) * cap);
    if (!keys || !p || !dp) {
        free(keys), free(p), free(dp);
        return -6;
    }
    memset(dQ, 0, sizeof(double) * n * d);
    memset(dK, 0, sizeof(double) * S * nkeys * d);
    memset(dV, 0, sizeof(double) * S * nkeys * dv);
    for (int64_t g = 0; g < n; ++g) {
        const int64_t s = g / plane;
        const int64_t last = (flags & OR_CAUSAL) ? g % plane : nkeys - 1;
        const double* q = Q + g * d;
        const double* go = dO + g * dv;
        const double* Ks = K + s * nkeys * d;
        const double* Vs = V + s * nkeys * dv;
        double* gK = dK + s * nkeys * d;
        double* gV = dV + s * nkeys * dv;
        const int64_t nk = window_keys(J, kappa, n, g, Hk, Wk, b, last, keys);
        if (nk == 0) continue;
        /* softmax weights over the set */
        double m = -INFINITY, l = 0.0;
        for (int64_t j = 0; j < nk; ++j) {
            p[j] = scale * dot(q, Ks + keys[j] * d, d);
            if (p[j] > m) m = p[j];
        }
        for (int64_t j = 0; j < nk; ++j) {
            p[j] = exp(p[j] - m);
            l += p[j];
        }
        double D = 0.0;
        for (int64_t j = 0; j < nk; ++j) {
            p[j] /= l;
            dp[j] = dot(go, Vs + keys[j] * dv, dv);
            D += p[j] * dp[j];
        }
        for (int64_t j = 0; j < nk; ++j) {
            const double ds = p[j] * (dp[j] - D);
            const double* k = Ks + keys[j] * d;
            for (int e = 0; e < d; ++e) {
                dQ[g * d + e] += scale * ds * k[e];
                gK[keys[j] * d + e] += scale * ds * q[e];
            }
            for (int e = 0; e < dv; ++e) gV[keys[j] * dv + e] += p[j] * go[e];
        }
    }
    free(keys), free(p), free(dp);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Self-normalised importance sampling (Section 4.2, Equations 11-17).      */
/* ------------------------------------------------------------------------ */
#define OR_SNIS_TAG 0x534E4953u

/* binomial coefficient C(n, k) for n <= 32, exact (integer arithmetic) */
static double choose(int n, int k)
{
    if (k < 0 || k > n) return 0.0;
    uint64_t c = 1;
    for (int i = 1; i <= k; ++i) c = c * (uint64_t)(n - k + i) / (uint64_t)i;
    return (double)c;
}

/* pmf of the centred binomial offset (2m fair bits, minus m) */
static double offset_pmf(int64_t delta, int m)
{
    if (delta < -m || delta > m) return 0.0;
    return choose(2 * m, (int)(delta + m)) / ldexp(1.0, 2 * m);
}

/* P(offset <= x) */
static double offset_cdf(int64_t x, int m)
{
    double acc = 0.0;
    for (int64_t delta = -m; delta <= x && delta <= m; ++delta) acc += offset_pmf(delta, m);
    return acc;
}

/* probability that the clamped coordinate centre + offset lands on r, 0 <= r < len */
static double axis_density(int64_t r, int64_t centre, int64_t len, int m)
{
    if (len == 1) return 1.0;
    if (r == 0) return offset_cdf(-centre, m);               /* every offset reaching row 0 or beyond */
    if (r == len - 1) return offset_cdf(centre - (len - 1), m); /* by symmetry, the far tail */
    return offset_pmf(r - centre, m);
}

static int alpha_q16(double alpha) { return (int)floor(alpha * 65536.0 + 0.5); }

static int popcount32(uint32_t x)
{
    int c = 0;
    for (; x; x &= x - 1) ++c;
    return c;
}

/* r_i(j) of Equation 17 for one query with modes[kappa] (flat key indices) */
static double snis_density(const int32_t* modes, int64_t kappa, int64_t Hk, int64_t Wk, int m, double alpha,
                           int64_t j)
{
    const double a = alpha_q16(alpha) / 65536.0;
    const int64_t r = j / Wk, c = j % Wk;
    double local = 0.0;
    for (int64_t e = 0; e < kappa; ++e)
        local += axis_density(r, modes[e] / Wk, Hk, m) * axis_density(c, modes[e] % Wk, Wk, m);
    return a / (double)kappa * local + (1.0 - a) / (double)(Hk * Wk);
}

/* sample t of query g drawn from r_i (Equation 12) */
static int64_t snis_draw(const int32_t* modes, int64_t kappa, int64_t Hk, int64_t Wk, int m, double alpha,
                         const uint32_t key[2], int64_t g, int64_t t)
{
    const uint32_t ctr[4] = {(uint32_t)g, (uint32_t)t, 0u, OR_SNIS_TAG};
    uint32_t w[4];
    philox4x32_10(ctr, key, w);
    int64_t r, c;
    if ((int)(w[0] >> 16) < alpha_q16(alpha)) {
        const int64_t e = pick_in_range(w[1], 0, kappa - 1);
        const uint32_t mask = m == 16 ? 0xFFFFFFFFu : ((1u << (2 * m)) - 1u);
        r = modes[e] / Wk + (popcount32(w[2] & mask) - m);
        c = modes[e] % Wk + (popcount32(w[3] & mask) - m);
        r = r < 0 ? 0 : (r > Hk - 1 ? Hk - 1 : r);
        c = c < 0 ? 0 : (c > Wk - 1 ? Wk - 1 : c);
    } else {
        r = pick_in_range(w[2], 0, Hk - 1);
        c = pick_in_range(w[3], 0, Wk - 1);
    }
    return r * Wk + c;
}

static int snis_args_ok(int64_t kappa, int radius, double alpha)
{
    return kappa >= 1 && radius >= 0 && radius <= 16 && alpha >= 0.0 && alpha <= 1.0;
}

/* r_i(j) for every key j of one query's modes (exposed for tests) */
int oracle_snis_density(const int32_t* modes, int64_t kappa, int64_t Hk, int64_t Wk, int radius, double alpha,
                        double* out)
{
    if (!snis_args_ok(kappa, radius, alpha) || Hk <= 0 || Wk <= 0) return -2;
    for (int64_t j = 0; j < Hk * Wk; ++j) out[j] = snis_density(modes, kappa, Hk, Wk, radius, alpha, j);
    return 0;
}

/* samples t = 0..T-1 of query g (exposed for tests) */
int oracle_snis_draws(const int32_t* modes, int64_t kappa, int64_t Hk, int64_t Wk, int radius, double alpha,
                      uint64_t seed, int64_t g, int64_t T, int64_t* out)
{
    if (!snis_args_ok(kappa, radius, alpha) || Hk <= 0 || Wk <= 0 || T < 0) return -2;
    uint32_t key[2];
    seed_key(seed, key);
    for (int64_t t = 0; t < T; ++t) out[t] = snis_draw(modes, kappa, Hk, Wk, radius, alpha, key, g, t);
    return 0;
}

/*
 * The SNIS estimate (Equations 11-17) for each listed query i: T samples
 * j_t ~ r_i, weights w_t = exp(a_ij_t) / r_i(j_t) with a = scale * q.k
 * (Equation 13; a key after the query under OR_CAUSAL has p^(u) = 0, so
 * weight 0), the estimate sum_t w_t v_j_t / sum_t w_t (Equation 14), the
 * effective sample size (sum w)^2 / sum w^2 (Equation 16) and the variance
 * sum_t (w_t / sum w)^2 (v_j_t - estimate)^2 per channel (Equation 15).
 * The weights are formed as exp(log w_t - max_s log w_s), which leaves every
 * ratio unchanged.  If every weight is 0 the row, its ESS and its variance
 * are 0.  modes is [kappa, S, Hq, Wq]; out and var are compact [count, dv],
 * ess is [count]; ess and var may be NULL.
 */
int oracle_snis(const double* Q, const double* K, const double* V, const int32_t* modes, int64_t kappa,
                int64_t S, int64_t Hq, int64_t Wq, int64_t Hk, int64_t Wk, int d, int dv, int64_t T,
                double alpha, int radius, double scale, uint64_t seed, uint32_t flags, const int64_t* query_ids,
                int64_t nq, double* out, double* ess, double* var)
{
    if (check_dims(S, Hq, Wq, Hk, Wk, d) || dv <= 0 || T < 1 || !snis_args_ok(kappa, radius, alpha)) return -2;
    if ((flags & OR_CAUSAL) && (Hq != Hk || Wq != Wk)) return -2;
    const int64_t n = S * Hq * Wq, plane = Hq * Wq;
    const int64_t count = query_ids ? nq : n;
    for (int64_t g = 0; g < kappa * n; ++g)
        if (modes[g] < 0 || modes[g] >= Hk * Wk) return -2;
    if (query_ids)
        for (int64_t i = 0; i < nq; ++i)
            if (query_ids[i] < 0 || query_ids[i] >= n) return -2;
    uint32_t key[2];
    seed_key(seed, key);
    int rc = 0;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        const int64_t g = query_ids ? query_ids[i] : i;
        const int64_t s = g / plane;
        const int64_t last = (flags & OR_CAUSAL) ? g % plane : Hk * Wk - 1;
        const double* q = Q + g * d;
        const double* Ks = K + s * Hk * Wk * d;
        const double* Vs = V + s * Hk * Wk * dv;
        int32_t* qm = (int32_t*)malloc(sizeof(int32_t) * kappa);
        int64_t* js = (int64_t*)malloc(sizeof(int64_t) * T);
        double* lw = (double*)malloc(sizeof(double) * T);
        if (!qm || !js || !lw) {
            free(qm), free(js), free(lw);
            rc = -6;
            continue;
        }
        for (int64_t e = 0; e < kappa; ++e) qm[e] = modes[e * n + g];
        /* samples and log weights */
        double mx = -INFINITY;
        for (int64_t t = 0; t < T; ++t) {
            js[t] = snis_draw(qm, kappa, Hk, Wk, radius, alpha, key, g, t);
            if (js[t] > last) {
                lw[t] = -INFINITY;
            } else {
                const double a = scale * dot(q, Ks + js[t] * d, d);
                lw[t] = a - log(snis_density(qm, kappa, Hk, Wk, radius, alpha, js[t]));
            }
            if (lw[t] > mx) mx = lw[t];
        }
        double* o = out + i * dv;
        double* vr = var ? var + i * dv : NULL;
        for (int e = 0; e < dv; ++e) {
            o[e] = 0.0;
            if (vr) vr[e] = 0.0;
        }
        double s1 = 0.0, s2 = 0.0;
        if (mx > -INFINITY) {
            for (int64_t t = 0; t < T; ++t) {
                const double w = exp(lw[t] - mx);
                s1 += w;
                s2 += w * w;
                const double* v = Vs + js[t] * dv;
                for (int e = 0; e < dv; ++e) o[e] += w * v[e];
            }
            for (int e = 0; e < dv; ++e) o[e] /= s1;
            if (vr) {
                for (int64_t t = 0; t < T; ++t) {
                    const double wn = exp(lw[t] - mx) / s1;
                    const double* v = Vs + js[t] * dv;
                    for (int e = 0; e < dv; ++e) vr[e] += wn * wn * (v[e] - o[e]) * (v[e] - o[e]);
                }
            }
        }
        if (ess) ess[i] = s2 > 0.0 ? s1 * s1 / s2 : 0.0;
        free(qm), free(js), free(lw);
    }
    return rc;
}

/* Threads the OpenMP runtime would use (1 when built without OpenMP). */
#ifdef _OPENMP
#include <omp.h>
int oracle_num_threads(void) { return omp_get_max_threads(); }
void oracle_set_num_threads(int n) { omp_set_num_threads(n); }
#else
int oracle_num_threads(void) { return 1; }
void oracle_set_num_threads(int n) { (void)n; }
#endif
