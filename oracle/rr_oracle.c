/*
 * RouteRelay reference oracle (arXiv 2609.07306).
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the plain, slow, obviously
 * correct CPU statement of what the route-maintenance path computes.  Only
 * the test-suite, the smoke check and the benchmark's CPU-baseline leg may
 * load it; the product path never calls it and shares no code with it.
 *
 * Plain single-threaded C99.  Every score is accumulated in binary64, in
 * index order.  A product of two binary32 inputs is exact in binary64, so a
 * score differs from the real dot product only by the binary64 rounding of
 * the running sum (relative 2^-53 per addition).
 *
 * What each part follows:
 *   - scores and full routing: Sec. 2.1, Eq. (1) S = Qc Kc^T and Eq. (2), a
 *     row-wise TopK over the key chunks;
 *   - the route ledger: Sec. 3.1, Eq. (4): per row, the selected set R, the
 *     near-miss sentinels (the m chunks ranked directly below the cut-off)
 *     and r uniformly drawn chunks from those left out, plus the layer the
 *     entry was built at; Sec. 4.1 stores routes [rows,k], sentinels
 *     [rows,m+r] and ages [rows];
 *   - rescoring and the trigger: Sec. 3.2, Eq. (5)-(8): A = R u C,
 *     alpha = min over R of the current scores, beta = max over C, the route
 *     is kept when alpha > beta + gamma, otherwise the row computes all of
 *     its scores, replaces its route and rebuilds its sentinels;
 *   - random sentinels are drawn without replacement from the pool left after
 *     removing R and the near-miss set (Sec. 3.4, the setting of Eq. (10)).
 *
 * Readings where the paper leaves a choice (each is also listed in the
 * design notes):
 *   - rank order: higher score first, equal scores broken by lower chunk id;
 *     -0 and +0 compare equal;
 *   - causal chunk mask: row i may select chunks j <= i only; a row with
 *     n_i <= k selects every valid chunk;
 *   - R and the near-miss part of C are stored sorted by ascending chunk id,
 *     padded with -1; the random part of C keeps its draw (slot) order;
 *   - trigger: a row is rerouted iff C is non-empty and beta + gamma >= alpha
 *     (the negation of the reuse test; equality reroutes);
 *   - random probes use the splitmix64 output function chained over
 *     (seed, layer, row, slot, attempt); a pool no larger than r is taken
 *     whole in ascending order; a pool of at most half the valid chunks is
 *     sampled by rank: slot s takes the y-th remaining pool id in ascending
 *     order with y = probe(attempt 0) mod (pool size - s); a larger pool by
 *     rejection: probes reduced modulo n_i, up to 64 attempts per slot
 *     rejecting ids outside the pool or already drawn, after which the slot
 *     takes the y-th remaining pool id with y = probe(attempt 64) mod
 *     (remaining pool size).  Both are uniform draws without replacement
 *     (Eq. (10)); rank sampling spares the small pools of early causal rows
 *     their long rejection runs;
 *   - mandatory sentinels (Sec. 3.1, item 3): the sink chunks j < n_sink
 *     and the recent chunks, the n_recent valid chunks at and below the
 *     row's own position (position i when n_q == n_k, else the last key
 *     chunk), minus any already in R or N, stored ascending after the random
 *     slots (n_sink + n_recent slots, -1 padded); the random pool leaves
 *     them out as well;
 *   - per-row guard margins (Eq. (8), gamma_i >= 0): gamma_rows[row] when
 *     given, else the scalar gamma;
 *   - hysteresis (Sec. 3.2): a minimum reuse horizon of min_reuse layers --
 *     a row (re)built at layer b is not rerouted at layers b+1 .. b+min_reuse
 *     (0: off); the paper's optional larger margin after a refresh is left to
 *     gamma_rows, which the caller may raise for such rows;
 *   - query-dependent budgets (Sec. 4.3-4.4): row i routes to its top k_i
 *     chunks (k_rows[row], 1 <= k_i <= k); the near-miss set is the next m;
 *     the route is stored in the ledger's k slots, -1 padded;
 *   - random sentinels persist until the row is next rebuilt;
 *   - score pairs: a (re)built row counts its n_i scores, a relay row counts
 *     |A| (valid candidate slots) plus n_i when it is rerouted;
 *   - age = layer - build layer for rows that keep their route.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t n_heads;    /* query heads H_q */
    int32_t n_kv_heads; /* key heads H_kv; query head h reads key head h / (H_q/H_kv) */
    int32_t n_q;        /* query chunks per head */
    int32_t n_k;        /* key chunks per head */
    int32_t d;          /* representation width */
    int32_t k;          /* route width */
    int32_t m;          /* near-miss sentinels */
    int32_t r;          /* random sentinels */
    int32_t causal;     /* 1: row i sees chunks j <= i */
    int32_t pad_;
    double gamma;       /* guard margin of the trigger */
    uint64_t seed;      /* random-probe seed */
    int32_t n_sink;     /* mandatory sentinels: the first n_sink chunks ... */
    int32_t n_recent;   /* ... and the n_recent most recent valid chunks */
    int32_t min_reuse;  /* a row (re)built at layer b keeps its route at layers b+1 .. b+min_reuse */
    int32_t pad2_;
    const double *gamma_rows; /* per-row guard margins gamma_i (NULL: gamma for every row) */
    const int32_t *k_rows;    /* per-row route widths 1 <= k_i <= k (NULL: k for every row) */
} orc_problem;

typedef struct {
    double s;
    int32_t id;
} orc_scored;

/* ---------------------------------------------------------------- hashing */

/* splitmix64 output function (Steele, Lea and Flood, OOPSLA 2014; Vigna's
 * public-domain reference): add the golden-ratio increment, then two
 * xor-shift-multiply rounds and a final xor-shift, all modulo 2^64. */
uint64_t orc_splitmix64(uint64_t z)
{
    z += 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* Counter hash of one random probe: the output function applied after
 * mixing in each coordinate in turn. */
uint64_t orc_probe_hash(uint64_t seed, uint64_t layer, uint64_t row, uint64_t slot,
                        uint64_t attempt)
{
    uint64_t h = orc_splitmix64(seed);
    h = orc_splitmix64(h ^ layer);
    h = orc_splitmix64(h ^ row);
    h = orc_splitmix64(h ^ slot);
    return orc_splitmix64(h ^ attempt);
}

/* ----------------------------------------------------------------- scores */

static double dot64(const float *a, const float *b, int d)
{
    double s = 0.0;
    for (int t = 0; t < d; ++t)
        s += (double)a[t] * (double)b[t];
    return s;
}

static double absdot64(const float *a, const float *b, int d)
{
    double s = 0.0;
    for (int t = 0; t < d; ++t)
        s += fabs((double)a[t] * (double)b[t]);
    return s;
}

static int cmp_rank(const void *x, const void *y)
{
    const orc_scored *a = (const orc_scored *)x;
    const orc_scored *b = (const orc_scored *)y;
    if (a->s > b->s) return -1;
    if (a->s < b->s) return 1;
    return (a->id < b->id) ? -1 : (a->id > b->id);
}

static int cmp_int(const void *x, const void *y)
{
    int32_t a = *(const int32_t *)x, b = *(const int32_t *)y;
    return (a < b) ? -1 : (a > b);
}

static int n_valid(const orc_problem *P, int i)
{
    if (!P->causal) return P->n_k;
    return (i + 1 < P->n_k) ? i + 1 : P->n_k;
}

static const float *q_row(const orc_problem *P, const float *Q, int64_t row)
{
    return Q + row * (int64_t)P->d;
}

static const float *k_row(const orc_problem *P, const float *K, int h, int j)
{
    int group = P->n_heads / P->n_kv_heads;
    int g = h / group;
    return K + ((int64_t)g * P->n_k + j) * (int64_t)P->d;
}

/* Scores of row (h, i) against every valid chunk, sorted by rank order. */
static int rank_row(const orc_problem *P, const float *Q, const float *K, int h, int i,
                    orc_scored *work)
{
    int ni = n_valid(P, i);
    const float *q = q_row(P, Q, (int64_t)h * P->n_q + i);
    for (int j = 0; j < ni; ++j) {
        work[j].s = dot64(q, k_row(P, K, h, j), P->d);
        work[j].id = j;
    }
    qsort(work, (size_t)ni, sizeof(orc_scored), cmp_rank);
    return ni;
}

/* The route width of a row: k_i when per-row budgets are given, else k. */
static int row_k(const orc_problem *P, int64_t row) { return P->k_rows ? P->k_rows[row] : P->k; }

/* Eq. (2) with the near-miss extension of Sec. 3.1: R = the first
 * min(ki, n_i) chunks in rank order, N = the next min(m, n_i - |R|); both
 * stored sorted by id and padded with -1 to widths kk and mm. */
static void split_route(const orc_scored *work, int ni, int kk, int ki, int mm, int32_t *R, int *nR,
                        int32_t *N, int *nN, double *R_scores)
{
    int a = ni < ki ? ni : ki;
    int b = (ni - a) < mm ? (ni - a) : mm;
    for (int t = 0; t < a; ++t) R[t] = work[t].id;
    qsort(R, (size_t)a, sizeof(int32_t), cmp_int);
    for (int t = a; t < kk; ++t) R[t] = -1;
    if (N) {
        for (int t = 0; t < b; ++t) N[t] = work[a + t].id;
        qsort(N, (size_t)b, sizeof(int32_t), cmp_int);
        for (int t = b; t < mm; ++t) N[t] = -1;
    }
    if (R_scores) {
        /* scores of R in the stored (id) order */
        for (int t = 0; t < kk; ++t) {
            R_scores[t] = NAN;
            for (int u = 0; u < a && R[t] >= 0; ++u)
                if (work[u].id == R[t]) R_scores[t] = work[u].s;
        }
    }
    *nR = a;
    if (nN) *nN = b;
}

/* ------------------------------------------------------- random sentinels */

/* Mandatory sentinels of row i (Sec. 3.1, item 3): the sink chunks
 * [0, n_sink) and the recent chunks [p - n_recent + 1, p], p the row's
 * position (i when n_q == n_k, else n_k - 1), both cut to the valid chunks,
 * without those already in R u N (marked in excl); written ascending to
 * out[0 .. n_sink + n_recent), -1 padded, and marked in excl.  Returns how
 * many were written. */
static int build_mandatory(const orc_problem *P, int i, int ni, unsigned char *excl, int32_t *out)
{
    int width = P->n_sink + P->n_recent, w = 0;
    int p = (P->n_q == P->n_k) ? i : P->n_k - 1;
    if (p > ni - 1) p = ni - 1;
    int lo = p - P->n_recent + 1;
    if (lo < 0) lo = 0;
    for (int j = 0; j < ni && w < width; ++j) {
        int sink = j < P->n_sink, recent = P->n_recent > 0 && j >= lo && j <= p;
        if ((sink || recent) && !excl[j]) {
            out[w++] = j;
            excl[j] = 1;
        }
    }
    for (int t = w; t < width; ++t) out[t] = -1;
    return w;
}

/* r probes drawn without replacement from the pool V_i minus (R u N u M).
 * excl is caller scratch of n_k bytes marking R, N and M; nM is |M|. */
static void draw_random(const orc_problem *P, int32_t layer, int64_t row, int ni,
                        int nR, int nN, int nM, int32_t *out, const unsigned char *excl_in,
                        unsigned char *excl)
{
    int r = P->r;
    if (excl != excl_in) memcpy(excl, excl_in, (size_t)P->n_k);
    int pool = ni - nR - nN - nM;
    if (pool <= r) {
        int w = 0;
        for (int j = 0; j < ni; ++j)
            if (!excl[j]) out[w++] = j;
        for (; w < r; ++w) out[w] = -1;
        return;
    }
    if (2 * pool <= ni) {
        /* rank sampling: the y-th remaining pool id, ascending */
        for (int s = 0; s < r; ++s) {
            uint64_t h = orc_probe_hash(P->seed, (uint64_t)layer, (uint64_t)row, (uint64_t)s, 0);
            int y = (int)(h % (uint64_t)(pool - s));
            int chosen = -1;
            for (int j = 0; j < ni; ++j) {
                if (excl[j]) continue;
                if (y == 0) { chosen = j; break; }
                --y;
            }
            excl[chosen] = 1;
            out[s] = chosen;
        }
        return;
    }
    for (int s = 0; s < r; ++s) {
        int chosen = -1;
        for (int t = 0; t < 64 && chosen < 0; ++t) {
            uint64_t h = orc_probe_hash(P->seed, (uint64_t)layer, (uint64_t)row, (uint64_t)s,
                                        (uint64_t)t);
            int x = (int)(h % (uint64_t)ni);
            if (!excl[x]) chosen = x;
        }
        if (chosen < 0) {
            int remaining = pool - s;
            uint64_t h = orc_probe_hash(P->seed, (uint64_t)layer, (uint64_t)row, (uint64_t)s, 64);
            int y = (int)(h % (uint64_t)remaining);
            for (int j = 0; j < ni; ++j) {
                if (excl[j]) continue;
                if (y == 0) { chosen = j; break; }
                --y;
            }
        }
        excl[chosen] = 1;
        out[s] = chosen;
    }
}

int orc_random_sentinels(const orc_problem *P, int32_t layer, int64_t row, int32_t ni,
                         const int32_t *R, int32_t nR, const int32_t *N, int32_t nN,
                         int32_t *out)
{
    unsigned char *excl = (unsigned char *)malloc((size_t)P->n_k);
    if (!excl) return -2;
    memset(excl, 0, (size_t)P->n_k);
    for (int t = 0; t < nR; ++t) excl[R[t]] = 1;
    for (int t = 0; t < nN; ++t) excl[N[t]] = 1;
    draw_random(P, layer, row, ni, nR, nN, 0, out, excl, excl);
    free(excl);
    return 0;
}

/* ------------------------------------------------------------ row sets */

static int64_t rows_total(const orc_problem *P)
{
    return (int64_t)P->n_heads * P->n_q;
}

#define FOR_ROWS(P, rows, n_rows, idx, row)                                   \
    for (int64_t idx = 0, row = 0;                                            \
         idx < ((rows) ? (n_rows) : rows_total(P)) &&                         \
         ((row = (rows) ? (rows)[idx] : idx), 1);                             \
         ++idx)

/* ----------------------------------------------------------- full routing */

/* Eq. (1)-(2): routes[row, 0..k) sorted by id, -1 padded.  route_scores (if
 * given) receives the binary64 scores in the same slots (NaN on padding).
 * pairs receives the number of scores evaluated (n_i per row). */
int orc_full_route(const orc_problem *P, const float *Q, const float *K, const int64_t *rows,
                   int64_t n_rows, int32_t *routes, double *route_scores, int64_t *pairs)
{
    orc_scored *work = (orc_scored *)malloc(sizeof(orc_scored) * (size_t)P->n_k);
    if (!work) return -2;
    int64_t total = 0;
    FOR_ROWS(P, rows, n_rows, idx, row) {
        int h = (int)(row / P->n_q), i = (int)(row % P->n_q);
        int ni = rank_row(P, Q, K, h, i, work);
        int nR;
        split_route(work, ni, P->k, row_k(P, row), 0, routes + row * P->k, &nR, NULL, NULL,
                    route_scores ? route_scores + row * P->k : NULL);
        total += ni;
    }
    if (pairs) *pairs = total;
    free(work);
    return 0;
}

/* Boundary scores used to classify near-ties: for each row the scores at
 * rank k_i, k_i+1, k_i+m and k_i+m+1 (1-based, k_i the row's route width;
 * NaN where the rank does not exist),
 * followed by sum_t |q_t k_t| of the same four chunks.  out is [rows, 8]. */
int orc_route_bounds(const orc_problem *P, const float *Q, const float *K, const int64_t *rows,
                     int64_t n_rows, double *out)
{
    orc_scored *work = (orc_scored *)malloc(sizeof(orc_scored) * (size_t)P->n_k);
    if (!work) return -2;
    FOR_ROWS(P, rows, n_rows, idx, row) {
        int h = (int)(row / P->n_q), i = (int)(row % P->n_q);
        int ni = rank_row(P, Q, K, h, i, work);
        const float *q = q_row(P, Q, row);
        int ki = row_k(P, row);
        int ranks[4] = {ki - 1, ki, ki + P->m - 1, ki + P->m};
        double *o = out + idx * 8;
        for (int u = 0; u < 4; ++u) {
            int rk = ranks[u];
            if (rk >= 0 && rk < ni) {
                o[u] = work[rk].s;
                o[4 + u] = absdot64(q, k_row(P, K, h, work[rk].id), P->d);
            } else {
                o[u] = NAN;
                o[4 + u] = NAN;
            }
        }
    }
    free(work);
    return 0;
}

/* ---------------------------------------------------------------- anchor */

static int sent_width(const orc_problem *P) { return P->m + P->r + P->n_sink + P->n_recent; }

static void rebuild_row(const orc_problem *P, int32_t layer, const float *Q, const float *K,
                        int64_t row, orc_scored *work, unsigned char *excl, int32_t *routes,
                        int32_t *sent, int32_t *build, int32_t *age, int *ni_out)
{
    int h = (int)(row / P->n_q), i = (int)(row % P->n_q);
    int c = sent_width(P);
    int ni = rank_row(P, Q, K, h, i, work);
    int nR, nN;
    int32_t *R = routes + row * P->k;
    int32_t *C = sent + row * c;
    split_route(work, ni, P->k, row_k(P, row), P->m, R, &nR, C, &nN, NULL);
    /* C = near-miss slots, random slots, then mandatory slots */
    memset(excl, 0, (size_t)P->n_k);
    for (int t = 0; t < nR; ++t) excl[R[t]] = 1;
    for (int t = 0; t < nN; ++t) excl[C[t]] = 1;
    int nM = build_mandatory(P, i, ni, excl, C + P->m + P->r);
    draw_random(P, layer, row, ni, nR, nN, nM, C + P->m, excl, excl);
    build[row] = layer;
    age[row] = 0;
    *ni_out = ni;
}

/* Anchor layer (Sec. 3.1): every row is fully routed and its ledger entry
 * (R, C, build layer) is rebuilt.  mask[row] = 1 for every row. */
int orc_anchor(const orc_problem *P, int32_t layer, const float *Q, const float *K,
               const int64_t *rows, int64_t n_rows, int32_t *routes, int32_t *sent,
               int32_t *build, int32_t *age, uint8_t *mask, int64_t *pairs)
{
    orc_scored *work = (orc_scored *)malloc(sizeof(orc_scored) * (size_t)P->n_k);
    unsigned char *excl = (unsigned char *)malloc((size_t)P->n_k);
    if (!work || !excl) { free(work); free(excl); return -2; }
    int64_t total = 0;
    FOR_ROWS(P, rows, n_rows, idx, row) {
        int ni;
        rebuild_row(P, layer, Q, K, row, work, excl, routes, sent, build, age, &ni);
        if (mask) mask[row] = 1;
        total += ni;
    }
    if (pairs) *pairs = total;
    free(work);
    free(excl);
    return 0;
}

/* ----------------------------------------------------------------- relay */

/* Intermediate layer (Sec. 3.2): each row rescores A = R u C at this layer,
 * keeps its route iff alpha > beta + gamma, otherwise refreshes.  alpha and
 * beta (and sum_t |q_t k_t| of the chunk attaining each) are returned per
 * row; beta is -inf when C has no valid slot.  row_pairs (if given) receives
 * each row's own score pairs (|A| plus n_i when rerouted); pairs their sum. */
int orc_relay(const orc_problem *P, int32_t layer, const float *Q, const float *K,
              const int64_t *rows, int64_t n_rows, int32_t *routes, int32_t *sent,
              int32_t *build, int32_t *age, uint8_t *mask, double *alpha, double *beta,
              double *alpha_abs, double *beta_abs, int64_t *pairs, int64_t *row_pairs)
{
    orc_scored *work = (orc_scored *)malloc(sizeof(orc_scored) * (size_t)P->n_k);
    unsigned char *excl = (unsigned char *)malloc((size_t)P->n_k);
    if (!work || !excl) { free(work); free(excl); return -2; }
    int c = sent_width(P);
    int64_t total = 0;
    FOR_ROWS(P, rows, n_rows, idx, row) {
        int h = (int)(row / P->n_q);
        const float *q = q_row(P, Q, row);
        int32_t *R = routes + row * P->k;
        int32_t *C = sent + row * c;
        double a = INFINITY, b = -INFINITY, a_abs = NAN, b_abs = NAN;
        int n_cand = 0, n_sent = 0;
        for (int t = 0; t < P->k; ++t) {
            if (R[t] < 0) continue;
            const float *kr = k_row(P, K, h, R[t]);
            double s = dot64(q, kr, P->d);
            ++n_cand;
            if (s < a) { a = s; a_abs = absdot64(q, kr, P->d); }
        }
        for (int t = 0; t < c; ++t) {
            if (C[t] < 0) continue;
            const float *kr = k_row(P, K, h, C[t]);
            double s = dot64(q, kr, P->d);
            ++n_cand;
            ++n_sent;
            if (s > b) { b = s; b_abs = absdot64(q, kr, P->d); }
        }
        int64_t own = n_cand;
        double g = P->gamma_rows ? P->gamma_rows[row] : P->gamma;
        int settled = P->min_reuse > 0 && layer - build[row] <= P->min_reuse;
        int reroute = (n_sent > 0) && !settled && (b + g >= a);
        if (alpha) alpha[row] = a;
        if (beta) beta[row] = b;
        if (alpha_abs) alpha_abs[row] = a_abs;
        if (beta_abs) beta_abs[row] = b_abs;
        if (reroute) {
            int ni;
            rebuild_row(P, layer, Q, K, row, work, excl, routes, sent, build, age, &ni);
            own += ni;
        } else {
            age[row] = layer - build[row];
        }
        total += own;
        if (row_pairs) row_pairs[row] = own;
        if (mask) mask[row] = (uint8_t)reroute;
    }
    if (pairs) *pairs = total;
    free(work);
    free(excl);
    return 0;
}
