/*
 * SBVR CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct CPU implementation of what the SBVR GEMV
 * path computes (Bang et al., "SBVR: Summation of BitVector Representation
 * for Efficient LLM Quantization").  Only the tests, the smoke check and the
 * CPU-baseline leg of the benchmark may load it.  It shares no code, header,
 * table or helper with the HIP library; the two only agree on the canonical
 * SBVR format, which each side writes out from the paper on its own:
 *
 *   planes  uint32 [O][G][K][4]  bit t of word w is element 32*w+t of group g
 *                                (LSB first); plane i pairs with coefficient i
 *   coeffs  uint16 [O][G][K]     IEEE binary16 bit patterns of c_{o,g,i}
 *   decoded weight  w_hat[o][128g+j] = sum_i c_{o,g,i} * bit_i(o,g,j)
 *
 * Arithmetic is IEEE binary64 throughout, compiled without contraction or
 * fast-math, so every result is reproducible bit for bit.
 *
 * Readings of the paper taken where it is silent or garbled (each one is a
 * documented reading, not a statement of the paper):
 *   R1  Eq. 4 scale: by default the geometric series is span-normalised,
 *       c_i = s * r^i / N(r) + b with N(r) = sum_i |r|^i, so that s is the
 *       width of the subset-sum point set (S spans data widths, Eqs. 8, 10).
 *       normalise = 0 gives the literal c_i = s * r^i + b.
 *   R2  R = R1 u R2: R1 built like S over (-1, -0.5], R2 built like B over
 *       [-2, -1); sizes n_ratio1, n_ratio2 (the paper's values are in an
 *       appendix that is not available).
 *   R3  q95 = linear-interpolation percentile of the signed group data.
 *   R4  Candidate coefficients are rounded to binary16 (RNE) before the
 *       subset sums are formed; sums and errors are binary64.
 *   R5  Nearest scans patterns p = sum_i bit_i 2^i in ascending order and
 *       keeps the first strict minimum of |x - sum_p|; Algorithm 1 keeps
 *       the first entry with a strictly smaller MSE.
 *   R6  Candidates with s <= 0 or a non-finite coefficient are skipped; if
 *       none is left the coefficients are (fp16(mean), 0, ..., 0).
 *   R7  Entries are visited r-outer, then s, then b (index order of Eq. 4).
 *   R11 Online activation conversion (Sec. 4.3, Eq. 12): the coefficients
 *       {-2^(l-1) s, s, 2s, ..., 2^(l-2) s} are the two's-complement weights
 *       of an l-bit integer code q; the per-vector scale "absmax / 2^l" as
 *       printed would leave half of [-absmax, absmax] outside that grid, so
 *       s = absmax / (2^(l-1) - 1).
 *   R12 Activation vectors are the 128-element groups of the inner dimension,
 *       the ones that meet a weight group in the inner product (Sec. 4.4).
 *   R13 The grid point is the conventional integer-grid rounding Sec. 4.3
 *       adopts (round to nearest, as the RTN of Sec. 3.1): t = x / s, q = t
 *       rounded to nearest even, within +-(2^(l-1) - 1); an all-zero vector
 *       has s = 0 and q = 0.  The paper names no precision for s and t; they
 *       are binary32, the default floating-point type of the PyTorch and
 *       CUDA implementation Sec. 5.1 describes (binary16 activations
 *       promoted to it), with correctly rounded division.
 *   R14 Encoder cache (Sec. 4.2, last paragraph and footnote), a separate
 *       entry point; the plain encoder searches every group.  Scope: one
 *       cache and one moving average per weight row, over its groups in
 *       index order (rows are independent).  The cache holds the coefficient
 *       sets (the evaluated (r, s, b) of Eq. 4) that the full search chose
 *       for the row's last `slots` searched groups, oldest replaced first;
 *       an R6 fallback adds nothing.  Before searching, every cached set is
 *       scored on the group with Algorithm 1's MSE; the smallest (the oldest
 *       set on ties) is used, with the bitvector assignment of Sec. 4.2, if
 *       it is strictly below the moving average of the quantization error,
 *       read as the mean MSE of all the row's earlier groups (cache hits
 *       included): binary64 sum in group order over their count.  The first
 *       group of a row always searches; slots = 0 is the plain encoder.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#define GROUP 128 /* weights per SBVR group along the inner-product dim (Sec. 4.1) */
#define KMAX 8

typedef struct {
    int n_ratio1;  /* |R1| */
    int n_ratio2;  /* |R2| */
    int n_scale;   /* N_scale (Eq. 6, 11) */
    int n_bias;    /* N_bias  (Eq. 7, 11) */
    int normalise; /* reading R1: 1 span-normalised, 0 literal Eq. 4 */
} oracle_params;

/* ------------------------------------------------------------------------ */
/* binary16 <-> binary64, written from the IEEE 754 definition.             */
/* ------------------------------------------------------------------------ */

double oracle_fp16_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int m = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)m, -24); /* subnormal: m * 2^-24 */
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(m + 1024), e - 25); /* 1.m * 2^(e-15) */
    return sign ? -v : v;
}

/* Round a binary64 value to the nearest binary16, ties to even. */
uint16_t oracle_fp16_from_double(double v)
{
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    double a = fabs(v);
    if (isnan(v))
        return 0x7e00;
    if (a == 0.0)
        return sign;
    /* Largest finite half is 65504; values at or above 65520 round to inf. */
    if (a >= 65520.0)
        return sign | 0x7c00;
    int e;
    frexp(a, &e); /* a = f * 2^e, f in [0.5, 1) -> unbiased exponent e-1 */
    int ue = e - 1;
    if (ue < -14) {
        /* subnormal range: quantum 2^-24 */
        double q = a * 16777216.0; /* a / 2^-24, exact (power of two) */
        double r = nearbyint(q);   /* default rounding mode: ties to even */
        uint32_t n = (uint32_t)r;  /* may reach 1024 = smallest normal */
        return sign | (uint16_t)n;
    }
    /* normal: significand with 10 fraction bits, quantum 2^(ue-10) */
    double q = ldexp(a, 10 - ue); /* in [1024, 2048) */
    double r = nearbyint(q);
    uint32_t n = (uint32_t)r;
    if (n == 2048) { /* rounded up to the next binade */
        n = 1024;
        ue += 1;
    }
    if (ue > 15)
        return sign | 0x7c00;
    return sign | (uint16_t)(((ue + 15) << 10) | (n - 1024));
}

/* ------------------------------------------------------------------------ */
/* Statistics used by the search-space formulas (Eqs. 8-11).                */
/* ------------------------------------------------------------------------ */

static int cmp_double(const void *a, const void *b)
{
    double x = *(const double *)a, y = *(const double *)b;
    return (x > y) - (x < y);
}

/* Linear-interpolation percentile (reading R3): position q*(n-1) in the
 * sorted data, interpolated between its two neighbours. */
double oracle_quantile_linear(const double *data, int n, double q)
{
    double *s = (double *)malloc(sizeof(double) * (size_t)n);
    memcpy(s, data, sizeof(double) * (size_t)n);
    qsort(s, (size_t)n, sizeof(double), cmp_double);
    double pos = q * (double)(n - 1);
    int lo = (int)floor(pos);
    if (lo >= n - 1) {
        double v = s[n - 1];
        free(s);
        return v;
    }
    double frac = pos - (double)lo;
    double v = s[lo] + frac * (s[lo + 1] - s[lo]);
    free(s);
    return v;
}

/* ------------------------------------------------------------------------ */
/* Search space (Sec. 4.2, Eqs. 4-11).                                      */
/* ------------------------------------------------------------------------ */

int oracle_candidate_count(const oracle_params *p)
{
    return (p->n_ratio1 + p->n_ratio2) * p->n_scale * p->n_bias;
}

/* Fill the candidate sets R, S and B for group data D (Eqs. 5-11).
 * r_out holds n_ratio1 + n_ratio2 values, s_out n_scale, b_out n_bias. */
void oracle_candidate_sets(const double *D, int n, int K, const oracle_params *p,
                           double *r_out, double *s_out, double *b_out)
{
    double mn = D[0], mx = D[0], sum = 0.0;
    for (int j = 0; j < n; ++j) {
        if (D[j] < mn) mn = D[j];
        if (D[j] > mx) mx = D[j];
        sum += D[j];
    }
    double avg = sum / (double)n;
    double q95 = oracle_quantile_linear(D, n, 0.95);

    /* Eq. 8 and Eq. 10: scale range; Eq. 11: granularity; Eq. 6: S. */
    double s_max = 1.1 * (mx - mn);
    double s_min = 2.0 * q95;
    double s_gran = (s_max - s_min) / (double)p->n_scale;
    for (int j = 0; j < p->n_scale; ++j)
        s_out[j] = s_min + (double)(j + 1) * s_gran;

    /* Eq. 9 and Eq. 10: bias range; Eq. 11: granularity; Eq. 7: B. */
    double b_max = 2.0 * fabs(avg) / (double)K;
    double b_min = -b_max;
    double b_gran = (b_max - b_min) / (double)p->n_bias;
    for (int k = 0; k < p->n_bias; ++k)
        b_out[k] = b_min + (double)k * b_gran;

    /* Eq. 5 with reading R2: R1 follows the S procedure over (-1, -0.5],
     * R2 follows the B procedure over [-2, -1). */
    double r1_gran = 0.5 / (double)p->n_ratio1;
    for (int i = 0; i < p->n_ratio1; ++i)
        r_out[i] = -1.0 + (double)(i + 1) * r1_gran;
    double r2_gran = 1.0 / (double)p->n_ratio2;
    for (int i = 0; i < p->n_ratio2; ++i)
        r_out[p->n_ratio1 + i] = -2.0 + (double)i * r2_gran;
}

/* Coefficient set of one search-space entry (Eq. 4 with readings R1, R4).
 * Returns 0 if a coefficient is not finite in binary16. */
int oracle_entry_coeffs(double r, double s, double b, int K, int normalise, uint16_t *coeff_out)
{
    double norm = 1.0;
    if (normalise) {
        double a = 1.0, t = 0.0;
        for (int i = 0; i < K; ++i) {
            t += fabs(a);
            a *= r;
        }
        norm = t;
    }
    double pw = 1.0; /* r^i by repeated multiplication */
    int ok = 1;
    for (int i = 0; i < K; ++i) {
        double c = (s * pw) / norm + b;
        uint16_t h = oracle_fp16_from_double(c);
        if ((h & 0x7c00) == 0x7c00)
            ok = 0;
        coeff_out[i] = h;
        pw *= r;
    }
    return ok;
}

/* AllSubsetSums (Algorithm 1, note 1; Sec. 4.1 worked example):
 * sums[p] = sum of the coefficients whose bit is set in p, in i order. */
void oracle_subset_sums(const uint16_t *coeffs, int K, double *sums)
{
    double c[KMAX];
    for (int i = 0; i < K; ++i)
        c[i] = oracle_fp16_to_double(coeffs[i]);
    for (int p = 0; p < (1 << K); ++p) {
        double t = 0.0;
        for (int i = 0; i < K; ++i)
            if ((p >> i) & 1)
                t += c[i];
        sums[p] = t;
    }
}

/* Nearest (Algorithm 1, note 2; reading R5): index of the closest sum. */
int oracle_nearest(const double *sums, int K, double x)
{
    int best = 0;
    double bd = fabs(x - sums[0]);
    for (int p = 1; p < (1 << K); ++p) {
        double d = fabs(x - sums[p]);
        if (d < bd) {
            bd = d;
            best = p;
        }
    }
    return best;
}

/* MSE of data D under a coefficient set (the inner loop of Algorithm 1). */
double oracle_entry_mse(const double *D, int n, const uint16_t *coeffs, int K)
{
    double sums[1 << KMAX];
    oracle_subset_sums(coeffs, K, sums);
    double err = 0.0;
    for (int j = 0; j < n; ++j) {
        int q = oracle_nearest(sums, K, D[j]);
        double d = D[j] - sums[q];
        err += d * d;
    }
    return err / (double)n;
}

/* SBVR Encoding (Algorithm 1) of one group, followed by the bitvector
 * assignment of Sec. 4.2: every element takes the pattern of its nearest
 * subset sum.  Writes K coefficients and n pattern codes; returns the MSE.
 * *entry_out receives the index of the chosen entry (-1: degenerate, R6). */
double oracle_encode_group(const double *D, int n, int K, const oracle_params *p,
                           uint16_t *coeff_out, uint8_t *codes_out, int *entry_out)
{
    int nr = p->n_ratio1 + p->n_ratio2;
    double *R = (double *)malloc(sizeof(double) * (size_t)nr);
    double *S = (double *)malloc(sizeof(double) * (size_t)p->n_scale);
    double *B = (double *)malloc(sizeof(double) * (size_t)p->n_bias);
    oracle_candidate_sets(D, n, K, p, R, S, B);

    double best_mse = INFINITY;
    int best_entry = -1;
    uint16_t best_c[KMAX], c[KMAX];
    int e = 0;
    for (int ir = 0; ir < nr; ++ir)
        for (int js = 0; js < p->n_scale; ++js)
            for (int kb = 0; kb < p->n_bias; ++kb, ++e) {
                if (!(S[js] > 0.0))
                    continue; /* R6 */
                if (!oracle_entry_coeffs(R[ir], S[js], B[kb], K, p->normalise, c))
                    continue; /* R6 */
                double mse = oracle_entry_mse(D, n, c, K);
                if (mse < best_mse) {
                    best_mse = mse;
                    best_entry = e;
                    memcpy(best_c, c, sizeof(uint16_t) * (size_t)K);
                }
            }
    if (best_entry < 0) { /* R6: no admissible entry */
        double sum = 0.0;
        for (int j = 0; j < n; ++j)
            sum += D[j];
        best_c[0] = oracle_fp16_from_double(sum / (double)n);
        for (int i = 1; i < K; ++i)
            best_c[i] = 0;
        best_mse = oracle_entry_mse(D, n, best_c, K);
    }
    double sums[1 << KMAX];
    oracle_subset_sums(best_c, K, sums);
    for (int j = 0; j < n; ++j)
        codes_out[j] = (uint8_t)oracle_nearest(sums, K, D[j]);
    memcpy(coeff_out, best_c, sizeof(uint16_t) * (size_t)K);
    if (entry_out)
        *entry_out = best_entry;
    free(R);
    free(S);
    free(B);
    return best_mse;
}

/* ------------------------------------------------------------------------ */
/* Whole-matrix encode: every (row, group) independently (Sec. 4.1/4.2).    */
/* ------------------------------------------------------------------------ */

typedef struct {
    int O, I, K;
    const float *W;
    const oracle_params *p;
    uint32_t *planes;
    uint16_t *coeffs;
    double *mse;
    long begin, end; /* flat (row, group) index range */
} encode_job;

static void *encode_worker(void *arg)
{
    encode_job *jb = (encode_job *)arg;
    int G = jb->I / GROUP, K = jb->K;
    double D[GROUP];
    uint8_t codes[GROUP];
    for (long t = jb->begin; t < jb->end; ++t) {
        long o = t / G, g = t % G;
        const float *src = jb->W + o * (long)jb->I + g * GROUP;
        for (int j = 0; j < GROUP; ++j)
            D[j] = (double)src[j];
        double mse = oracle_encode_group(D, GROUP, K, jb->p, jb->coeffs + t * K, codes, NULL);
        if (jb->mse)
            jb->mse[t] = mse;
        /* bitvector assignment: plane i gets bit i of each element's pattern */
        uint32_t *pl = jb->planes + t * (long)K * 4;
        memset(pl, 0, sizeof(uint32_t) * (size_t)K * 4);
        for (int j = 0; j < GROUP; ++j)
            for (int i = 0; i < K; ++i)
                if ((codes[j] >> i) & 1)
                    pl[i * 4 + j / 32] |= 1u << (j % 32);
    }
    return NULL;
}

static int resolve_threads(int nthreads)
{
    if (nthreads > 0)
        return nthreads;
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    return n > 0 ? (int)n : 1;
}

int oracle_encode_matrix(int O, int I, int K, const float *W, const oracle_params *p,
                         int nthreads, uint32_t *planes, uint16_t *coeffs, double *mse_out)
{
    if (O < 1 || I < GROUP || I % GROUP || K < 1 || K > KMAX)
        return -1;
    int nt = resolve_threads(nthreads);
    long total = (long)O * (I / GROUP);
    if (nt > total)
        nt = (int)total;
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nt);
    encode_job *jobs = (encode_job *)malloc(sizeof(encode_job) * (size_t)nt);
    for (int i = 0; i < nt; ++i) {
        encode_job j = {O, I, K, W, p, planes, coeffs, mse_out,
                        total * i / nt, total * (i + 1) / nt};
        jobs[i] = j;
        pthread_create(&th[i], NULL, encode_worker, &jobs[i]);
    }
    for (int i = 0; i < nt; ++i)
        pthread_join(th[i], NULL);
    free(th);
    free(jobs);
    return nt;
}

/* ------------------------------------------------------------------------ */
/* Encoder with the cache of Sec. 4.2 (last paragraph and its footnote;     */
/* reading R14): before the full search, the coefficient sets the search    */
/* chose for earlier groups are tried, and one is kept if its error is      */
/* below the moving average of the quantization error.                      */
/* ------------------------------------------------------------------------ */

#define ORACLE_CACHE_MAX 64

/* Bitvector assignment of Sec. 4.2 for a given coefficient set: every
 * element takes the pattern of its nearest subset sum (R5). */
static void assign_codes(const double *D, int n, const uint16_t *coeffs, int K, uint8_t *codes)
{
    double sums[1 << KMAX];
    oracle_subset_sums(coeffs, K, sums);
    for (int j = 0; j < n; ++j)
        codes[j] = (uint8_t)oracle_nearest(sums, K, D[j]);
}

static void store_group(const uint8_t *codes, const uint16_t *c, int K, uint32_t *pl, uint16_t *cf)
{
    memset(pl, 0, sizeof(uint32_t) * (size_t)K * 4);
    for (int j = 0; j < GROUP; ++j)
        for (int i = 0; i < K; ++i)
            if ((codes[j] >> i) & 1)
                pl[i * 4 + j / 32] |= 1u << (j % 32);
    memcpy(cf, c, sizeof(uint16_t) * (size_t)K);
}

/* One row's G groups in index order.  hit_out[g] = 1 where the group took a
 * cached set, 0 where it ran Algorithm 1. */
static void encode_row_cached(const float *Wrow, int I, int K, const oracle_params *p, int slots,
                              uint32_t *planes, uint16_t *coeffs, double *mse_out, uint8_t *hit_out)
{
    int G = I / GROUP;
    uint16_t cache[ORACLE_CACHE_MAX][KMAX];
    int n_cached = 0; /* sets held, at most slots */
    long n_ins = 0;   /* sets inserted so far; the next one replaces slot n_ins % slots */
    double mse_sum = 0.0;
    double D[GROUP];
    uint8_t codes[GROUP];
    for (int g = 0; g < G; ++g) {
        for (int j = 0; j < GROUP; ++j)
            D[j] = (double)Wrow[(long)g * GROUP + j];
        uint16_t c[KMAX];
        double mse = 0.0;
        int hit = 0;
        if (g > 0 && n_cached > 0) {
            double avg = mse_sum / (double)g; /* mean error of the row's earlier groups */
            double best = INFINITY;
            int best_slot = -1;
            for (int a = 0; a < n_cached; ++a) { /* oldest first: ties keep the older set */
                int slot = (int)((n_ins - n_cached + a) % slots);
                double m = oracle_entry_mse(D, GROUP, cache[slot], K);
                if (m < best) {
                    best = m;
                    best_slot = slot;
                }
            }
            if (best < avg) {
                hit = 1;
                mse = best;
                memcpy(c, cache[best_slot], sizeof(uint16_t) * (size_t)K);
                assign_codes(D, GROUP, c, K, codes);
            }
        }
        if (!hit) {
            int entry = -1;
            mse = oracle_encode_group(D, GROUP, K, p, c, codes, &entry);
            if (entry >= 0 && slots > 0) { /* R6 fallbacks are not entries: not cached */
                memcpy(cache[n_ins % slots], c, sizeof(uint16_t) * (size_t)K);
                ++n_ins;
                if (n_cached < slots)
                    ++n_cached;
            }
        }
        store_group(codes, c, K, planes + (long)g * K * 4, coeffs + (long)g * K);
        if (mse_out)
            mse_out[g] = mse;
        if (hit_out)
            hit_out[g] = (uint8_t)hit;
        mse_sum += mse;
    }
}

typedef struct {
    int I, K, slots;
    const float *W;
    const oracle_params *p;
    uint32_t *planes;
    uint16_t *coeffs;
    double *mse;
    uint8_t *hits;
    long begin, end; /* row range */
} cached_job;

static void *encode_cached_worker(void *arg)
{
    cached_job *jb = (cached_job *)arg;
    long G = jb->I / GROUP;
    for (long o = jb->begin; o < jb->end; ++o)
        encode_row_cached(jb->W + o * (long)jb->I, jb->I, jb->K, jb->p, jb->slots,
                          jb->planes + o * G * jb->K * 4, jb->coeffs + o * G * jb->K,
                          jb->mse ? jb->mse + o * G : NULL, jb->hits ? jb->hits + o * G : NULL);
    return NULL;
}

/* Whole matrix, rows in parallel (each row's groups in order).  slots = 0
 * gives the plain encoder's result.  Returns the thread count, -1 on a bad
 * shape or slot count. */
int oracle_encode_matrix_cached(int O, int I, int K, const float *W, const oracle_params *p, int slots,
                                int nthreads, uint32_t *planes, uint16_t *coeffs, double *mse_out,
                                uint8_t *hit_out)
{
    if (O < 1 || I < GROUP || I % GROUP || K < 1 || K > KMAX || slots < 0 || slots > ORACLE_CACHE_MAX)
        return -1;
    int nt = resolve_threads(nthreads);
    if (nt > O)
        nt = O;
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nt);
    cached_job *jobs = (cached_job *)malloc(sizeof(cached_job) * (size_t)nt);
    for (int i = 0; i < nt; ++i) {
        cached_job j = {I, K, slots, W, p, planes, coeffs, mse_out, hit_out,
                        (long)O * i / nt, (long)O * (i + 1) / nt};
        jobs[i] = j;
        pthread_create(&th[i], NULL, encode_cached_worker, &jobs[i]);
    }
    for (int i = 0; i < nt; ++i)
        pthread_join(th[i], NULL);
    free(th);
    free(jobs);
    return nt;
}

/* ------------------------------------------------------------------------ */
/* Decompression and the dense fp64 GEMV (the exact result the method       */
/* reaches without decompressing: y = W_hat x, Sec. 4.4).                    */
/* ------------------------------------------------------------------------ */

/* One decoded row: w_hat[128g+j] = sum_i c_{o,g,i} bit_i(o,g,j), exact in
 * binary64 (a sum of at most 8 binary16 values). */
static void decode_row(int o, int I, int K, const uint32_t *planes, const uint16_t *coeffs,
                       double *row)
{
    int G = I / GROUP;
    for (int g = 0; g < G; ++g) {
        const uint32_t *pl = planes + ((long)o * G + g) * K * 4;
        const uint16_t *cf = coeffs + ((long)o * G + g) * K;
        for (int j = 0; j < GROUP; ++j) {
            double w = 0.0;
            for (int i = 0; i < K; ++i)
                if ((pl[i * 4 + j / 32] >> (j % 32)) & 1u)
                    w += oracle_fp16_to_double(cf[i]);
            row[g * GROUP + j] = w;
        }
    }
}

void oracle_decompress(int O, int I, int K, const uint32_t *planes, const uint16_t *coeffs,
                       double *W_hat)
{
    for (int o = 0; o < O; ++o)
        decode_row(o, I, K, planes, coeffs, W_hat + (long)o * I);
}

/* Dense fp64 GEMV, sequential sum over the inner dimension. */
void oracle_gemv_dense(int O, int I, const double *W, const double *x, double *y)
{
    for (int o = 0; o < O; ++o) {
        double acc = 0.0;
        for (int j = 0; j < I; ++j)
            acc += W[(long)o * I + j] * x[j];
        y[o] = acc;
    }
}

typedef struct {
    int O, I, K, B;
    const uint32_t *planes;
    const uint16_t *coeffs;
    const double *x; /* [B][I] */
    const int *rows; /* row list (NULL: all rows) */
    double *y;       /* [B][n_rows] */
    int n_rows;
    int begin, end;
} gemv_job;

static void *gemv_worker(void *arg)
{
    gemv_job *jb = (gemv_job *)arg;
    double *row = (double *)malloc(sizeof(double) * (size_t)jb->I);
    for (int r = jb->begin; r < jb->end; ++r) {
        int o = jb->rows ? jb->rows[r] : r;
        decode_row(o, jb->I, jb->K, jb->planes, jb->coeffs, row);
        for (int b = 0; b < jb->B; ++b) {
            const double *xb = jb->x + (long)b * jb->I;
            double acc = 0.0;
            for (int j = 0; j < jb->I; ++j)
                acc += row[j] * xb[j];
            jb->y[(long)b * jb->n_rows + r] = acc;
        }
    }
    free(row);
    return NULL;
}

/* y[b][r] = sum_j w_hat[rows[r]][j] * x[b][j]: decompress each requested row
 * exactly and take the dense fp64 dot product with every activation vector.
 * x holds binary16 bit patterns [B][I]; rows may be NULL (all O rows).
 * Returns the number of threads used. */
int oracle_sbvr_gemv(int O, int I, int K, const uint32_t *planes, const uint16_t *coeffs,
                     const uint16_t *x_fp16, int B, const int *rows, int n_rows, int nthreads,
                     double *y)
{
    if (O < 1 || I < GROUP || I % GROUP || K < 1 || K > KMAX || B < 1)
        return -1;
    if (!rows)
        n_rows = O;
    double *x = (double *)malloc(sizeof(double) * (size_t)B * (size_t)I);
    for (long t = 0; t < (long)B * I; ++t)
        x[t] = oracle_fp16_to_double(x_fp16[t]);
    int nt = resolve_threads(nthreads);
    if (nt > n_rows)
        nt = n_rows;
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nt);
    gemv_job *jobs = (gemv_job *)malloc(sizeof(gemv_job) * (size_t)nt);
    for (int i = 0; i < nt; ++i) {
        gemv_job j = {O, I, K, B, planes, coeffs, x, rows, y, n_rows,
                      (int)((long)n_rows * i / nt), (int)((long)n_rows * (i + 1) / nt)};
        jobs[i] = j;
        pthread_create(&th[i], NULL, gemv_worker, &jobs[i]);
    }
    for (int i = 0; i < nt; ++i)
        pthread_join(th[i], NULL);
    free(th);
    free(jobs);
    free(x);
    return nt;
}

/* Same as oracle_sbvr_gemv with activations given as binary64 values. */
int oracle_sbvr_gemv_f64(int O, int I, int K, const uint32_t *planes, const uint16_t *coeffs,
                         const double *x, int B, const int *rows, int n_rows, int nthreads,
                         double *y)
{
    if (O < 1 || I < GROUP || I % GROUP || K < 1 || K > KMAX || B < 1)
        return -1;
    if (!rows)
        n_rows = O;
    int nt = resolve_threads(nthreads);
    if (nt > n_rows)
        nt = n_rows;
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nt);
    gemv_job *jobs = (gemv_job *)malloc(sizeof(gemv_job) * (size_t)nt);
    for (int i = 0; i < nt; ++i) {
        gemv_job j = {O, I, K, B, planes, coeffs, x, rows, y, n_rows,
                      (int)((long)n_rows * i / nt), (int)((long)n_rows * (i + 1) / nt)};
        jobs[i] = j;
        pthread_create(&th[i], NULL, gemv_worker, &jobs[i]);
    }
    for (int i = 0; i < nt; ++i)
        pthread_join(th[i], NULL);
    free(th);
    free(jobs);
    return nt;
}

/* ------------------------------------------------------------------------ */
/* Online activation conversion to SBVR-l (Sec. 4.3, Eq. 12; readings       */
/* R11-R13).                                                                 */
/* ------------------------------------------------------------------------ */

/* x: binary16 [I] (I a multiple of 128); q: codes [I]; s: scales [I / 128]. */
int oracle_act_quantize(int I, int l, const uint16_t *x, int32_t *q, float *s)
{
    if (I < GROUP || I % GROUP || l < 2 || l > 16)
        return -1;
    const int qmax = (1 << (l - 1)) - 1;
    for (int g = 0; g < I / GROUP; ++g) {
        float amax = 0.0f;
        for (int j = 0; j < GROUP; ++j) {
            const float v = (float)oracle_fp16_to_double(x[g * GROUP + j]);
            const float a = v < 0.0f ? -v : v;
            if (a > amax)
                amax = a;
        }
        const float sc = amax / (float)qmax;
        s[g] = sc;
        for (int j = 0; j < GROUP; ++j) {
            int code = 0;
            if (sc > 0.0f) {
                const float t = (float)oracle_fp16_to_double(x[g * GROUP + j]) / sc;
                code = (int)nearbyintf(t);
                if (code > qmax)
                    code = qmax;
                if (code < -qmax)
                    code = -qmax;
            }
            q[g * GROUP + j] = code;
        }
    }
    return 0;
}

/* Bitvectors of l-bit codes in Eq. 12's coefficient order: plane 0 carries
 * -2^(l-1) s, plane i >= 1 carries 2^(i-1) s.  planes: [n][l] of 0/1. */
void oracle_act_planes(int n, int l, const int32_t *q, uint8_t *planes)
{
    for (int e = 0; e < n; ++e) {
        const int neg = q[e] < 0;
        const int rest = q[e] + (neg ? (1 << (l - 1)) : 0);  /* in [0, 2^(l-1)) */
        planes[(long)e * l] = (uint8_t)neg;
        for (int i = 1; i < l; ++i)
            planes[(long)e * l + i] = (uint8_t)((rest >> (i - 1)) & 1);
    }
}

/* Decoded activations: x_hat = sum_i coefficient_i * bit_i with Eq. 12's
 * coefficients for the group's scale (binary64, exact). */
void oracle_act_decode(int I, int l, const uint8_t *planes, const float *s, double *x_hat)
{
    for (int e = 0; e < I; ++e) {
        const double sc = (double)s[e / GROUP];
        double v = planes[(long)e * l] ? -ldexp(sc, l - 1) : 0.0;
        for (int i = 1; i < l; ++i)
            if (planes[(long)e * l + i])
                v += ldexp(sc, i - 1);
        x_hat[e] = v;
    }
}

/* ------------------------------------------------------------------------ */
/* Round-to-nearest comparators (Sec. 3.1, Eqs. 2-3), diagnostics only.      */
/* ------------------------------------------------------------------------ */

/* Symmetric absmax RTN.  Eq. 2 as printed inverts the step; the reading
 * used here is delta = max|w| / (2^(b-1) - 1), q = clip(rne(w/delta)). */
double oracle_rtn_sym_mse(const double *D, int n, int bits)
{
    double amax = 0.0;
    for (int j = 0; j < n; ++j)
        if (fabs(D[j]) > amax)
            amax = fabs(D[j]);
    double qmax = (double)((1 << (bits - 1)) - 1);
    if (amax == 0.0)
        return 0.0;
    double delta = amax / qmax;
    double err = 0.0;
    for (int j = 0; j < n; ++j) {
        double q = nearbyint(D[j] / delta);
        if (q > qmax) q = qmax;
        if (q < -qmax) q = -qmax;
        double d = D[j] - q * delta;
        err += d * d;
    }
    return err / (double)n;
}

/* Asymmetric min-max RTN with 2^bits levels. */
double oracle_rtn_asym_mse(const double *D, int n, int bits)
{
    double mn = D[0], mx = D[0];
    for (int j = 0; j < n; ++j) {
        if (D[j] < mn) mn = D[j];
        if (D[j] > mx) mx = D[j];
    }
    double levels = (double)((1 << bits) - 1);
    if (mx == mn)
        return 0.0;
    double delta = (mx - mn) / levels;
    double err = 0.0;
    for (int j = 0; j < n; ++j) {
        double q = nearbyint((D[j] - mn) / delta);
        if (q > levels) q = levels;
        if (q < 0) q = 0;
        double d = D[j] - (mn + q * delta);
        err += d * d;
    }
    return err / (double)n;
}
