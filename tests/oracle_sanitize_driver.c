/* Drives every function of the CPU oracle (oracle/sbvr_oracle.c) on small
 * inputs, for a build with AddressSanitizer and UndefinedBehaviorSanitizer
 * (tests/test_oracle_sanitizers.py compiles the two files together and runs
 * this program).  Exit status 0 means every call returned and the few
 * invariants checked here held; the sanitizers abort on any memory or
 * undefined-behaviour error.  Test infrastructure only. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int n_ratio1, n_ratio2, n_scale, n_bias, normalise;
} oracle_params;

double oracle_fp16_to_double(uint16_t h);
uint16_t oracle_fp16_from_double(double v);
double oracle_quantile_linear(const double *data, int n, double q);
int oracle_candidate_count(const oracle_params *p);
void oracle_candidate_sets(const double *D, int n, int K, const oracle_params *p, double *r_out, double *s_out,
                           double *b_out);
int oracle_entry_coeffs(double r, double s, double b, int K, int normalise, uint16_t *coeff_out);
void oracle_subset_sums(const uint16_t *coeffs, int K, double *sums);
int oracle_nearest(const double *sums, int K, double x);
double oracle_entry_mse(const double *D, int n, const uint16_t *coeffs, int K);
double oracle_encode_group(const double *D, int n, int K, const oracle_params *p, uint16_t *coeff_out,
                           uint8_t *codes_out, int *entry_out);
int oracle_encode_matrix(int O, int I, int K, const float *W, const oracle_params *p, int nthreads,
                         uint32_t *planes, uint16_t *coeffs, double *mse_out);
void oracle_decompress(int O, int I, int K, const uint32_t *planes, const uint16_t *coeffs, double *out);
void oracle_gemv_dense(int O, int I, const double *W, const double *x, double *y);
int oracle_sbvr_gemv(int O, int I, int K, const uint32_t *planes, const uint16_t *coeffs, const uint16_t *x_fp16,
                     int B, const int *rows, int n_rows, int nthreads, double *y);
int oracle_act_quantize(int I, int l, const uint16_t *x, int32_t *q, float *s);
void oracle_act_planes(int n, int l, const int32_t *q, uint8_t *planes);
void oracle_act_decode(int I, int l, const uint8_t *planes, const float *s, double *x_hat);
double oracle_rtn_sym_mse(const double *D, int n, int bits);
double oracle_rtn_asym_mse(const double *D, int n, int bits);

static int failures = 0;
#define CHECK(c)                                                   \
    do {                                                           \
        if (!(c)) {                                                \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            ++failures;                                            \
        }                                                          \
    } while (0)

static double lcg_unit(uint64_t *st)
{
    *st = *st * 6364136223846793005ull + 1442695040888963407ull;
    return (double)(*st >> 11) * (1.0 / 9007199254740992.0);
}

int main(void)
{
    uint64_t st = 12345;
    /* binary16 round trip of every pattern that is not a NaN */
    for (uint32_t h = 0; h < 0x10000u; ++h) {
        if ((h & 0x7C00u) == 0x7C00u && (h & 0x3FFu))
            continue;
        CHECK(oracle_fp16_from_double(oracle_fp16_to_double((uint16_t)h)) == h);
    }
    double d8[8] = {-0.03, -0.02, -0.01, 0.0, 0.01, 0.02, 0.03, 0.04};
    CHECK(fabs(oracle_quantile_linear(d8, 8, 0.95) - 0.0365) < 1e-15);

    oracle_params p = {8, 8, 16, 4, 1};
    const int nc = oracle_candidate_count(&p);
    CHECK(nc == 1024);
    double R[16], S[16], B[4];
    oracle_candidate_sets(d8, 8, 4, &p, R, S, B);
    uint16_t c[8];
    CHECK(oracle_entry_coeffs(R[0], S[0], B[0], 4, 1, c) >= 0);
    double sums[256];
    oracle_subset_sums(c, 4, sums);
    CHECK(sums[0] == 0.0);
    int nn = oracle_nearest(sums, 4, 0.01);
    CHECK(nn >= 0 && nn < 16);
    CHECK(oracle_entry_mse(d8, 8, c, 4) >= 0.0);

    /* Algorithm 1 on Gaussian-like groups for K = 1..4, and a constant group */
    for (int K = 1; K <= 4; ++K) {
        double D[128];
        for (int j = 0; j < 128; ++j)
            D[j] = 0.02 * (lcg_unit(&st) + lcg_unit(&st) + lcg_unit(&st) - 1.5);
        uint16_t co[8];
        uint8_t codes[128];
        int entry = -2;
        double mse = oracle_encode_group(D, 128, K, &p, co, codes, &entry);
        CHECK(mse >= 0.0 && entry >= -1 && entry < nc);
        for (int j = 0; j < 128; ++j)
            CHECK(codes[j] < (1u << K));
    }
    {   /* an all-zero group: every scale candidate is 0, the degenerate case */
        double D[128] = {0};
        uint16_t co[8];
        uint8_t codes[128];
        int entry = 0;
        oracle_encode_group(D, 128, 4, &p, co, codes, &entry);
        CHECK(entry == -1);
    }

    /* whole-matrix encode, decompress, GEMV (all rows, some rows, B = 3),
     * several thread counts; ragged row count */
    const int O = 5, I = 384, K = 3, G = I / 128;
    float *W = malloc(sizeof(float) * O * I);
    for (int i = 0; i < O * I; ++i)
        W[i] = (float)(0.02 * (2.0 * lcg_unit(&st) - 1.0));
    uint32_t *planes = malloc(sizeof(uint32_t) * O * G * K * 4);
    uint16_t *coeffs = malloc(sizeof(uint16_t) * O * G * K);
    double *mse = malloc(sizeof(double) * O * G);
    for (int nt = 1; nt <= 3; nt += 2)
        CHECK(oracle_encode_matrix(O, I, K, W, &p, nt, planes, coeffs, mse) == nt);
    CHECK(oracle_encode_matrix(O, 100, K, W, &p, 1, planes, coeffs, mse) < 0);
    double *What = malloc(sizeof(double) * O * I);
    oracle_decompress(O, I, K, planes, coeffs, What);
    uint16_t x[3 * 384];
    double xd[3 * 384];
    for (int i = 0; i < 3 * I; ++i) {
        x[i] = oracle_fp16_from_double(2.0 * lcg_unit(&st) - 1.0);
        xd[i] = oracle_fp16_to_double(x[i]);
    }
    double yd[5], y[3 * 5], yr[3 * 2];
    oracle_gemv_dense(O, I, What, xd, yd);
    for (int nt = 1; nt <= 4; ++nt) {
        CHECK(oracle_sbvr_gemv(O, I, K, planes, coeffs, x, 3, NULL, O, nt, y) >= 1);
        for (int o = 0; o < O; ++o)
            CHECK(fabs(y[o] - yd[o]) <= 1e-12 * (fabs(yd[o]) + 1e-300) + 1e-18);
    }
    int rows[2] = {4, 0};
    CHECK(oracle_sbvr_gemv(O, I, K, planes, coeffs, x, 3, rows, 2, 2, yr) >= 1);
    CHECK(yr[0] == y[4] && yr[1] == y[0] && yr[2 + 0] == y[5 + 4]);
    CHECK(oracle_sbvr_gemv(O, I, K, planes, coeffs, x, 0, NULL, O, 1, y) < 0);

    /* online activation conversion (Sec. 4.3), including an all-zero group */
    int32_t q[384];
    float s[3];
    uint16_t xa[384];
    memcpy(xa, x, sizeof(xa));
    for (int j = 128; j < 256; ++j)
        xa[j] = 0;
    CHECK(oracle_act_quantize(I, 8, xa, q, s) == 0);
    CHECK(s[1] == 0.0f);
    uint8_t *ap = malloc((size_t)I * 8);
    oracle_act_planes(I, 8, q, ap);
    double xh[384];
    oracle_act_decode(I, 8, ap, s, xh);
    for (int j = 0; j < I; ++j)
        CHECK(fabs(xh[j] - (double)q[j] * (double)s[j / 128]) <= 1e-12);
    CHECK(oracle_act_quantize(100, 8, xa, q, s) < 0);

    CHECK(oracle_rtn_sym_mse(d8, 8, 4) >= 0.0);
    CHECK(oracle_rtn_asym_mse(d8, 8, 4) >= 0.0);

    free(W);
    free(planes);
    free(coeffs);
    free(mse);
    free(What);
    free(ap);
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("oracle sanitizer run: ok\n");
    return 0;
}
