/* The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer: the
 * fit (plain, symmetric, refined) for every activation and bit width, and
 * forward, backward, pack and unpack, single- and multi-threaded, on random
 * inputs with special values, for every storage type and ragged sizes.
 * Built and run on the CPU by tests/test_host_sanitizers.py.  Exit status 0
 * when every call succeeded and the multi-threaded results equal the
 * single-threaded ones. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t kind, pad;
    double A, B, mu, sigma, p, sigma2;
} oracle_weight;

int oracle_fit(int act, int bits, const oracle_weight* w, int64_t n, int symmetric, float* s,
               float* v, double* loss, int64_t* cuts, double* dp_last, double* vd);
int oracle_fit_refined(int act, int bits, const oracle_weight* w, int64_t n, int symmetric,
                       int max_iter, float* s, float* v, double* sd, double* vd, double* loss,
                       double* loss_dp, int* iters);
int64_t oracle_packed_words(int64_t n, int bits);
void oracle_pack(const uint8_t* idx, int64_t n, int bits, uint32_t* words);
void oracle_unpack(const uint32_t* words, int64_t n, int bits, uint8_t* idx);
int oracle_fwd(int act, int dtype, int bits, int symmetric, const float* s, const void* x,
               void* y, uint32_t* codes, uint8_t* idx, int64_t n);
int oracle_bwd(int dtype, int bits, const float* v, const void* g, const uint32_t* codes,
               void* gin, int64_t n);
int oracle_fwd_mt(int act, int dtype, int bits, int symmetric, const float* s, const void* x,
                  void* y, uint32_t* codes, int64_t n, int threads);
int oracle_bwd_mt(int dtype, int bits, const float* v, const void* g, const uint32_t* codes,
                  void* gin, int64_t n, int threads);
void oracle_round_array(int dtype, const double* in, void* out, int64_t n);

static int failures = 0;
#define EXPECT(cond)                                                              \
    do {                                                                          \
        if (!(cond)) {                                                            \
            fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond);   \
            ++failures;                                                           \
        }                                                                         \
    } while (0)

static uint64_t rng_state = 88172645463325252ull;
static double uniform01(void)
{   /* xorshift64 */
    rng_state ^= rng_state << 13; rng_state ^= rng_state >> 7; rng_state ^= rng_state << 17;
    return (double)(rng_state >> 11) / 9007199254740992.0;
}

int main(void)
{
    oracle_weight wn = {1, 0, -10.0, 10.0, 0.0, 1.0, 0.0, 1.0};
    oracle_weight wu = {0, 0, -8.0, 8.0, 0.0, 1.0, 0.0, 1.0};
    for (int act = 0; act <= 6; ++act)
        for (int bits = 1; bits <= 4; ++bits) {
            float s[15], v[16];
            double loss, dp_last[16], vd[16];
            int64_t cuts[17];
            int rc = oracle_fit(act, bits, &wn, 300, 0, s, v, &loss, cuts, dp_last, vd);
            EXPECT(rc == 0 || rc == -2);
            rc = oracle_fit(act, bits, &wu, 300, act == 2 || act == 3, s, v, &loss, cuts, NULL, NULL);
            EXPECT(rc == 0 || rc == -2);
            double sd[15], vd2[16], loss_dp;
            int iters;
            rc = oracle_fit_refined(act, bits, &wu, 200, 0, 50, s, v, sd, vd2, &loss, &loss_dp, &iters);
            EXPECT(rc == 0 || rc == -2);
        }
    /* forward / backward / pack on random inputs */
    const int64_t sizes[] = {0, 1, 31, 33, 511, 513, 4097, 100003};
    for (int dt = 0; dt <= 2; ++dt)
        for (int bits = 1; bits <= 4; ++bits)
            for (size_t si = 0; si < sizeof sizes / sizeof sizes[0]; ++si) {
                const int64_t n = sizes[si];
                const size_t esz = dt == 0 ? 4 : 2;
                double* xd = malloc(sizeof(double) * (size_t)(n + 1));
                double* gd = malloc(sizeof(double) * (size_t)(n + 1));
                for (int64_t i = 0; i < n; ++i) {
                    xd[i] = (uniform01() - 0.5) * 40.0;
                    gd[i] = uniform01() - 0.5;
                }
                if (n > 8) { xd[0] = NAN; xd[1] = INFINITY; xd[2] = -INFINITY; xd[3] = -0.0; xd[4] = 1e-40; }
                void* x = malloc(esz * (size_t)(n + 1));
                void* g = malloc(esz * (size_t)(n + 1));
                void* y1 = malloc(esz * (size_t)(n + 1));
                void* y2 = malloc(esz * (size_t)(n + 1));
                void* gi1 = malloc(esz * (size_t)(n + 1));
                void* gi2 = malloc(esz * (size_t)(n + 1));
                const int64_t nw = oracle_packed_words(n, bits);
                uint32_t* c1 = calloc((size_t)(nw + 1), 4);
                uint32_t* c2 = calloc((size_t)(nw + 1), 4);
                uint8_t* idx = malloc((size_t)(n + 1));
                uint8_t* idx2 = malloc((size_t)(n + 1));
                oracle_round_array(dt, xd, x, n);
                oracle_round_array(dt, gd, g, n);
                float s[15], v[16];
                const int K = 1 << bits;
                for (int m = 0; m < K - 1; ++m) s[m] = (float)(-6.0 + 12.0 * (m + 1) / K);
                for (int m = 0; m < K; ++m) v[m] = (float)(0.1 * m - 0.3);
                EXPECT(oracle_fwd(1, dt, bits, 0, s, x, y1, c1, idx, n) == 0);
                EXPECT(oracle_fwd_mt(1, dt, bits, 0, s, x, y2, c2, n, 4) == 0);
                EXPECT(memcmp(y1, y2, esz * (size_t)n) == 0);
                EXPECT(memcmp(c1, c2, 4 * (size_t)nw) == 0);
                oracle_unpack(c1, n, bits, idx2);
                EXPECT(memcmp(idx, idx2, (size_t)n) == 0);
                oracle_pack(idx2, n, bits, c2);
                EXPECT(memcmp(c1, c2, 4 * (size_t)nw) == 0);
                EXPECT(oracle_bwd(dt, bits, v, g, c1, gi1, n) == 0);
                EXPECT(oracle_bwd_mt(dt, bits, v, g, c1, gi2, n, 4) == 0);
                EXPECT(memcmp(gi1, gi2, esz * (size_t)n) == 0);
                free(xd); free(gd); free(x); free(g); free(y1); free(y2); free(gi1); free(gi2);
                free(c1); free(c2); free(idx); free(idx2);
            }
    printf("oracle driver: %d failure(s)\n", failures);
    return failures == 0 ? 0 : 1;
}
