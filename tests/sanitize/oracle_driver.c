/* Drives every entry point of the C oracle on small seeded problems, for a
 * build under AddressSanitizer and UndefinedBehaviorSanitizer: causal and
 * non-causal, GQA, k = n_k, m = r = 0, pools smaller than r, exact ties
 * (integer inputs) and the rank-sampling and rejection regimes of the
 * random-sentinel draw.  Exits non-zero on any failed call. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t n_heads, n_kv_heads, n_q, n_k, d, k, m, r, causal, pad_;
    double gamma;
    uint64_t seed;
    int32_t n_sink, n_recent, min_reuse, pad2_;
    const double *gamma_rows;
    const int32_t *k_rows;
} orc_problem;

uint64_t orc_splitmix64(uint64_t z);
int orc_random_sentinels(const orc_problem *P, int32_t layer, int64_t row, int32_t ni, const int32_t *R,
                         int32_t nR, const int32_t *N, int32_t nN, int32_t *out);
int orc_full_route(const orc_problem *P, const float *Q, const float *K, const int64_t *rows, int64_t n_rows,
                   int32_t *routes, double *route_scores, int64_t *pairs);
int orc_route_bounds(const orc_problem *P, const float *Q, const float *K, const int64_t *rows, int64_t n_rows,
                     double *out);
int orc_anchor(const orc_problem *P, int32_t layer, const float *Q, const float *K, const int64_t *rows,
               int64_t n_rows, int32_t *routes, int32_t *sent, int32_t *build, int32_t *age, uint8_t *mask,
               int64_t *pairs);
int orc_relay(const orc_problem *P, int32_t layer, const float *Q, const float *K, const int64_t *rows,
              int64_t n_rows, int32_t *routes, int32_t *sent, int32_t *build, int32_t *age, uint8_t *mask,
              double *alpha, double *beta, double *alpha_abs, double *beta_abs, int64_t *pairs,
              int64_t *row_pairs);

static uint64_t state = 12345;
static float draw(int integer)
{
    state = orc_splitmix64(state);
    if (integer) return (float)((int)(state % 5) - 2);
    return (float)((double)(state >> 11) / 9007199254740992.0 - 0.5);
}

static int run(int H, int Hkv, int n, int d, int k, int m, int r, int causal, int integer, double gamma,
               int n_sink, int n_recent, int min_reuse, int per_row_gamma)
{
    const int64_t rows = (int64_t)H * n;
    double *gr = malloc(sizeof(double) * (size_t)rows);
    for (int64_t t = 0; t < rows; ++t) gr[t] = (t % 3 == 0) ? INFINITY : (t % 3 == 1 ? 0.0 : 0.01);
    int32_t *kr = malloc(sizeof(int32_t) * (size_t)rows);
    for (int64_t t = 0; t < rows; ++t) kr[t] = 1 + (int32_t)(t % k);
    orc_problem P = {H, Hkv, n, n, d, k, m, r, causal, 0, gamma, 7, n_sink, n_recent, min_reuse, 0,
                     per_row_gamma ? gr : NULL, per_row_gamma ? kr : NULL};
    const int c = m + r + n_sink + n_recent;
    float *Q = malloc(sizeof(float) * (size_t)(rows * d));
    float *K = malloc(sizeof(float) * (size_t)((int64_t)Hkv * n * d));
    int32_t *routes = malloc(sizeof(int32_t) * (size_t)(rows * k));
    int32_t *sent = malloc(sizeof(int32_t) * (size_t)(rows * c + 1));
    int32_t *build = malloc(sizeof(int32_t) * (size_t)rows), *age = malloc(sizeof(int32_t) * (size_t)rows);
    uint8_t *mask = malloc((size_t)rows);
    double *rs = malloc(sizeof(double) * (size_t)(rows * k)), *bounds = malloc(sizeof(double) * (size_t)(rows * 8));
    double *al = malloc(sizeof(double) * (size_t)rows), *be = malloc(sizeof(double) * (size_t)rows);
    double *aa = malloc(sizeof(double) * (size_t)rows), *ba = malloc(sizeof(double) * (size_t)rows);
    int64_t *rp = malloc(sizeof(int64_t) * (size_t)rows);
    int64_t pairs = 0, sub[3] = {0, rows / 2, rows - 1};
    int bad = 0;
    for (int64_t t = 0; t < rows * d; ++t) Q[t] = draw(integer);
    for (int64_t t = 0; t < (int64_t)Hkv * n * d; ++t) K[t] = draw(integer);
    bad |= orc_full_route(&P, Q, K, NULL, 0, routes, rs, &pairs);
    bad |= orc_route_bounds(&P, Q, K, sub, 3, bounds);
    bad |= orc_anchor(&P, 0, Q, K, NULL, 0, routes, sent, build, age, mask, &pairs);
    for (int layer = 1; layer < 4; ++layer) {
        for (int64_t t = 0; t < rows * d; ++t) Q[t] += 0.5f * draw(integer);
        bad |= orc_relay(&P, layer, Q, K, NULL, 0, routes, sent, build, age, mask, al, be, aa, ba, &pairs, rp);
        bad |= orc_relay(&P, layer, Q, K, sub, 3, routes, sent, build, age, mask, al, be, aa, ba, &pairs, NULL);
    }
    {
        int32_t R[4] = {0, 1, 2, 3}, N[2] = {4, 5}, out[64];
        for (int ni = 6; ni <= n; ni += 7) {
            P.r = r < 64 ? r : 64;
            bad |= orc_random_sentinels(&P, 1, 3, ni, R, 4 < k ? 4 : k, N, 2, out);
        }
        P.r = r;
    }
    free(Q); free(K); free(routes); free(sent); free(build); free(age); free(mask); free(rs); free(bounds);
    free(al); free(be); free(aa); free(ba); free(rp); free(gr); free(kr);
    return bad;
}

int main(void)
{
    int bad = 0;
    bad |= run(1, 1, 40, 16, 5, 3, 4, 0, 0, 0.0, 0, 0, 0, 0);
    bad |= run(2, 1, 33, 8, 4, 2, 6, 1, 0, 0.0, 0, 0, 0, 0);      /* causal GQA, early rows with n_i < k */
    bad |= run(2, 2, 20, 8, 20, 0, 0, 0, 0, 0.0, 0, 0, 0, 0);     /* k = n_k, no sentinels */
    bad |= run(1, 1, 30, 8, 6, 6, 20, 0, 1, 0.0, 0, 0, 0, 0);     /* exact ties; pools below r */
    bad |= run(1, 1, 64, 8, 8, 4, 16, 1, 1, INFINITY, 0, 0, 0, 0); /* every row rerouted */
    bad |= run(1, 1, 64, 8, 8, 4, 16, 0, 0, -INFINITY, 0, 0, 0, 0);
    bad |= run(2, 1, 40, 8, 4, 3, 5, 1, 0, 0.0, 2, 3, 1, 1);      /* mandatory sentinels, hysteresis, per-row gamma */
    bad |= run(1, 1, 24, 8, 6, 4, 8, 0, 1, 0.0, 4, 4, 0, 1);      /* mandatory slots crowding a small pool */
    if (bad) { fprintf(stderr, "oracle call failed\n"); return 1; }
    printf("oracle driver ok\n");
    return 0;
}
