/*
 * sj_oracle.c -- reference (oracle) similarity join.  TEST INFRASTRUCTURE ONLY:
 * the tests, the package smoke check and the benchmark's CPU-baseline leg use
 * it to check and to time the GPU library; the library never calls it.
 *
 * It computes the plain definition of the similarity join of Ahle & Silvestri,
 * "Similarity Search with Tensor Core Units", Section 4: given point sets P and
 * Q in R^d, the set of pairs (x, y), x in P, y in Q, with D(x, y) <= r.  The
 * brute-force method of Section 4 (all pair distances through one product of
 * the n x d' matrices F_P and G_Q) returns exactly this set, so the oracle is
 * the definition written out with nested loops:
 *
 *   inner product (cosine on unit rows, Section 4 ip-distance examples):
 *       report (i, j)  iff  sum_k P[i][k] * Q[j][k]  >= s
 *   squared Euclidean distance (Section 4, squared L2 example):
 *       report (i, j)  iff  sum_k (P[i][k] - Q[j][k])^2  <= r2
 *
 * Readings taken where the paper is silent: both tests are inclusive; the L2
 * threshold applies to the squared distance; pairs are ordered index pairs
 * (duplicate rows are distinct points, a self-join includes (i, i)).
 *
 * Arithmetic: every stored element is decoded exactly to double (binary16,
 * bfloat16 and int8 are all subsets of binary64), scores are accumulated in
 * double in ascending k.  For integer-valued inputs whose partial sums stay
 * below 2^53 this is exact.
 *
 * Plain C, no intrinsics, no blocking; OpenMP only splits the independent rows
 * of P between threads.  Output pairs are in lexicographic (i, j) order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { OR_F16 = 1, OR_BF16 = 2, OR_I8 = 3 };
enum { OR_IP = 0, OR_L2 = 1 };

/* IEEE 754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.
 * Exponent field 0 holds zero and subnormals (fraction * 2^-24); 31 holds
 * infinities and NaNs; otherwise the value is (1024 + fraction) * 2^(e - 25). */
static double decode_f16(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25);
    return sign ? -v : v;
}

/* bfloat16: the upper 16 bits of an IEEE binary32: 1 sign bit, 8 exponent bits
 * (bias 127), 7 fraction bits.  Exponent field 0 holds zero and subnormals
 * (fraction * 2^-133); 255 holds infinities and NaNs; otherwise the value is
 * (128 + fraction) * 2^(e - 134). */
static double decode_bf16(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 7) & 0xff;
    int f = h & 0x7f;
    double v;
    if (e == 0)
        v = ldexp((double)f, -133);
    else if (e == 255)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(128 + f), e - 134);
    return sign ? -v : v;
}

static double elem(int dtype, const void *X, int64_t idx)
{
    switch (dtype) {
    case OR_F16:
        return decode_f16(((const uint16_t *)X)[idx]);
    case OR_BF16:
        return decode_bf16(((const uint16_t *)X)[idx]);
    case OR_I8:
        return (double)((const int8_t *)X)[idx];
    default:
        return NAN;
    }
}

/* Decode `count` stored elements into doubles. */
void or_decode(int dtype, const void *X, int64_t count, double *out)
{
    for (int64_t t = 0; t < count; ++t)
        out[t] = elem(dtype, X, t);
}

/* <P_i, Q_j> in double, ascending k. */
double or_score_ip(int dtype, const void *P, int64_t i, const void *Q, int64_t j, int64_t d)
{
    double s = 0.0;
    for (int64_t k = 0; k < d; ++k)
        s += elem(dtype, P, i * d + k) * elem(dtype, Q, j * d + k);
    return s;
}

/* ||P_i - Q_j||^2 in double, ascending k, from the coordinate differences. */
double or_score_l2(int dtype, const void *P, int64_t i, const void *Q, int64_t j, int64_t d)
{
    double s = 0.0;
    for (int64_t k = 0; k < d; ++k) {
        double t = elem(dtype, P, i * d + k) - elem(dtype, Q, j * d + k);
        s += t * t;
    }
    return s;
}

/* Does the pair belong to the join? */
static int matches(int metric, double score, double thr)
{
    return metric == OR_IP ? (score >= thr) : (score <= thr);
}

typedef struct {
    uint32_t *pairs;   /* matches of this row: j values */
    int64_t n, cap;
    uint32_t *band;    /* boundary-band j values */
    uint8_t *band_match;
    int64_t nb, capb;
} row_out;

static int push_u32(uint32_t **buf, int64_t *n, int64_t *cap, uint32_t v)
{
    if (*n == *cap) {
        int64_t nc = *cap ? 2 * *cap : 16;
        uint32_t *nb = (uint32_t *)realloc(*buf, (size_t)nc * sizeof(uint32_t));
        if (!nb)
            return -1;
        *buf = nb;
        *cap = nc;
    }
    (*buf)[(*n)++] = v;
    return 0;
}

/*
 * The join over the rows `rows[0..n_rows)` of P (all rows 0..n_p-1 when rows is
 * NULL) against every row of Q.
 *
 *   out_pairs: (i, j) uint32 pairs, lexicographic in (rows order, j); at most
 *              `cap` are written.
 *   band > 0 : pairs whose score lies within `band` of the threshold are also
 *              listed in band_pairs / band_match (match flag), at most band_cap.
 *   threads  : OpenMP threads (<= 0: the runtime default).
 *
 * Returns the total number of matches (which may exceed cap), -1 on bad
 * arguments, -2 when out of host memory.  *n_band receives the band size.
 */
int64_t or_join(int metric, int dtype, const void *P, int64_t n_p, const void *Q, int64_t n_q,
                int64_t d, double thr, const int64_t *rows, int64_t n_rows, double band,
                uint32_t *out_pairs, int64_t cap, uint32_t *band_pairs, uint8_t *band_match,
                int64_t band_cap, int64_t *n_band, int threads)
{
    if (n_p < 0 || n_q < 0 || d < 0 || (metric != OR_IP && metric != OR_L2))
        return -1;
    if (dtype != OR_F16 && dtype != OR_BF16 && dtype != OR_I8)
        return -1;
    if (!rows)
        n_rows = n_p;
    for (int64_t r = 0; rows && r < n_rows; ++r)
        if (rows[r] < 0 || rows[r] >= n_p)
            return -1;
    row_out *ro = (row_out *)calloc((size_t)(n_rows ? n_rows : 1), sizeof(row_out));
    if (!ro)
        return -2;
    int failed = 0;
#ifdef _OPENMP
    int nt = threads > 0 ? threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
#endif
    for (int64_t r = 0; r < n_rows; ++r) {
        int64_t i = rows ? rows[r] : r;
        row_out *o = &ro[r];
        for (int64_t j = 0; j < n_q; ++j) {
            double sc = metric == OR_IP ? or_score_ip(dtype, P, i, Q, j, d)
                                        : or_score_l2(dtype, P, i, Q, j, d);
            int m = matches(metric, sc, thr);
            if (m && push_u32(&o->pairs, &o->n, &o->cap, (uint32_t)j))
                failed = 1;
            if (band > 0.0 && fabs(sc - thr) <= band) {
                int64_t before = o->capb;
                if (push_u32(&o->band, &o->nb, &o->capb, (uint32_t)j)) {
                    failed = 1;
                } else {
                    if (o->capb != before) {
                        uint8_t *nm = (uint8_t *)realloc(o->band_match, (size_t)o->capb);
                        if (!nm) {
                            failed = 1;
                            continue;
                        }
                        o->band_match = nm;
                    }
                    o->band_match[o->nb - 1] = (uint8_t)m;
                }
            }
        }
    }
    int64_t total = 0, nb = 0;
    for (int64_t r = 0; r < n_rows; ++r) {
        int64_t i = rows ? rows[r] : r;
        for (int64_t t = 0; t < ro[r].n; ++t, ++total)
            if (total < cap) {
                out_pairs[2 * total] = (uint32_t)i;
                out_pairs[2 * total + 1] = ro[r].pairs[t];
            }
        for (int64_t t = 0; t < ro[r].nb; ++t, ++nb)
            if (nb < band_cap) {
                band_pairs[2 * nb] = (uint32_t)i;
                band_pairs[2 * nb + 1] = ro[r].band[t];
                band_match[nb] = ro[r].band_match[t];
            }
        free(ro[r].pairs);
        free(ro[r].band);
        free(ro[r].band_match);
    }
    free(ro);
    if (n_band)
        *n_band = nb;
    return failed ? -2 : total;
}

/* Number of matches of rows[0..n_rows) (all rows when NULL) against Q;
 * per_row (optional) receives the count of each listed row. */
int64_t or_count(int metric, int dtype, const void *P, int64_t n_p, const void *Q, int64_t n_q,
                 int64_t d, double thr, const int64_t *rows, int64_t n_rows, int64_t *per_row,
                 int threads)
{
    if (n_p < 0 || n_q < 0 || d < 0 || (metric != OR_IP && metric != OR_L2))
        return -1;
    if (dtype != OR_F16 && dtype != OR_BF16 && dtype != OR_I8)
        return -1;
    if (!rows)
        n_rows = n_p;
    for (int64_t r = 0; rows && r < n_rows; ++r)
        if (rows[r] < 0 || rows[r] >= n_p)
            return -1;
    int64_t total = 0;
#ifdef _OPENMP
    int nt = threads > 0 ? threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt) reduction(+ : total)
#endif
    for (int64_t r = 0; r < n_rows; ++r) {
        int64_t i = rows ? rows[r] : r;
        int64_t c = 0;
        for (int64_t j = 0; j < n_q; ++j) {
            double sc = metric == OR_IP ? or_score_ip(dtype, P, i, Q, j, d)
                                        : or_score_l2(dtype, P, i, Q, j, d);
            c += matches(metric, sc, thr);
        }
        if (per_row)
            per_row[r] = c;
        total += c;
    }
    return total;
}

/* Scores of the listed (i, j) pairs (metric's score, not the match flag).
 * OpenMP only splits the independent pairs between threads. */
void or_scores(int metric, int dtype, const void *P, const void *Q, int64_t d,
               const int64_t *pairs, int64_t n_pairs, double *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < n_pairs; ++t) {
        int64_t i = pairs[2 * t], j = pairs[2 * t + 1];
        out[t] = metric == OR_IP ? or_score_ip(dtype, P, i, Q, j, d)
                                 : or_score_l2(dtype, P, i, Q, j, d);
    }
}

/*
 * Section 4's ip-distance front ends, written from their definitions.
 *
 * Cosine similarity is the inner product of f(x) = g(x) = x / ||x||.
 * or_normalize writes every row of X (n x d, dtype) divided by its Euclidean
 * norm and rounded to the nearest value of the output type (binary16 for
 * out_dtype OR_F16, bfloat16 for OR_BF16), ties to even.  ||x|| is the square
 * root of the sum of the squares in double, ascending k (every square of a
 * decoded element is exact in double); each quotient is one double division.
 * A row whose norm is 0 is written as +0 throughout (its cosine with anything
 * is taken as 0).
 */

/* Round |v| (finite, >= 0) to a multiple of 2^scale_exp: the integer nearest
 * to |v| / 2^scale_exp, ties to the even integer. */
static double round_half_even_scaled(double a, int scale_exp)
{
    double q = ldexp(a, -scale_exp);   /* exact: a power-of-two scaling */
    double f = floor(q);
    double diff = q - f;              /* exact: q has few integer bits */
    if (diff > 0.5 || (diff == 0.5 && fmod(f, 2.0) != 0.0))
        f += 1.0;
    return f;
}

/* Nearest binary16 of v, ties to even: 11-bit significands, normal exponents
 * -14..15 (spacing 2^(e-10) in [2^e, 2^(e+1))), subnormal spacing 2^-24,
 * infinity above the largest finite value 65504. */
static uint16_t round_to_f16(double v)
{
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    double a = fabs(v);
    if (a == 0.0)
        return sign;
    int ex;
    frexp(a, &ex);
    int e = ex - 1;                   /* 2^e <= a < 2^(e+1) */
    if (e > 15)
        return sign | 0x7c00;
    if (e < -14) {                    /* subnormal range: spacing 2^-24 */
        double m = round_half_even_scaled(a, -24);   /* 0 .. 1024 */
        return sign | (uint16_t)m;    /* 1024 is the smallest normal, 0x0400 */
    }
    double m = round_half_even_scaled(a, e - 10);    /* 1024 .. 2048 */
    /* m = 2048 carries into the exponent; at e = 15 that is 0x7c00, infinity */
    uint32_t bits = ((uint32_t)(e + 15) << 10) + (uint32_t)m - 1024u;
    return sign | (uint16_t)bits;
}

/* Nearest bfloat16 of v, ties to even: 8-bit significands, normal exponents
 * -126..127 (spacing 2^(e-7)), subnormal spacing 2^-133. */
static uint16_t round_to_bf16(double v)
{
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    double a = fabs(v);
    if (a == 0.0)
        return sign;
    int ex;
    frexp(a, &ex);
    int e = ex - 1;
    if (e > 127)
        return sign | 0x7f80;
    if (e < -126) {
        double m = round_half_even_scaled(a, -133);  /* 0 .. 128 */
        return sign | (uint16_t)m;
    }
    double m = round_half_even_scaled(a, e - 7);     /* 128 .. 256 */
    /* m = 256 carries into the exponent; at e = 127 that is 0x7f80, infinity */
    uint32_t bits = ((uint32_t)(e + 127) << 7) + (uint32_t)m - 128u;
    return sign | (uint16_t)bits;
}

/* Exposed for the pins: the rounding of one double to binary16 / bfloat16. */
uint16_t or_round_f16(double v) { return round_to_f16(v); }
uint16_t or_round_bf16(double v) { return round_to_bf16(v); }

int or_normalize(int dtype, const void *X, int64_t n, int64_t d, int out_dtype, uint16_t *out)
{
    if (n < 0 || d < 0 || (dtype != OR_F16 && dtype != OR_BF16 && dtype != OR_I8) ||
        (out_dtype != OR_F16 && out_dtype != OR_BF16))
        return -1;
    for (int64_t i = 0; i < n; ++i) {
        double s = 0.0;
        for (int64_t k = 0; k < d; ++k) {
            double x = elem(dtype, X, i * d + k);
            s += x * x;
        }
        double norm = sqrt(s);
        for (int64_t k = 0; k < d; ++k) {
            if (norm == 0.0) {
                out[i * d + k] = 0;
                continue;
            }
            double y = elem(dtype, X, i * d + k) / norm;
            out[i * d + k] = out_dtype == OR_F16 ? round_to_f16(y) : round_to_bf16(y);
        }
    }
    return 0;
}

/*
 * Hamming distance (Section 4's example with f(x) = (x, 1 - x), g(y) = (1 - y, y)
 * on {0, 1}^d): the number of coordinates in which two bit rows differ.  A row
 * holds d bits, coordinate m in bit m % 8 of byte m / 8, ceil(d / 8) bytes per
 * row (bits past d are ignored).
 */
static int bit_at(const uint8_t *X, int64_t row, int64_t stride, int64_t m)
{
    return (X[row * stride + m / 8] >> (m % 8)) & 1;
}

int64_t or_hamming(const uint8_t *P, int64_t i, const uint8_t *Q, int64_t j, int64_t d)
{
    int64_t stride = (d + 7) / 8, h = 0;
    for (int64_t m = 0; m < d; ++m)
        h += bit_at(P, i, stride, m) != bit_at(Q, j, stride, m);
    return h;
}

/* All (i, j) with Hamming(P_i, Q_j) <= r, lexicographic; at most cap written;
 * returns the total, -1 on bad arguments, -2 out of memory. */
int64_t or_join_hamming(const uint8_t *P, int64_t n_p, const uint8_t *Q, int64_t n_q, int64_t d,
                        double r, uint32_t *out_pairs, int64_t cap, int threads)
{
    if (n_p < 0 || n_q < 0 || d < 0)
        return -1;
    row_out *ro = (row_out *)calloc((size_t)(n_p ? n_p : 1), sizeof(row_out));
    if (!ro)
        return -2;
    int failed = 0;
#ifdef _OPENMP
    int nt = threads > 0 ? threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
#endif
    for (int64_t i = 0; i < n_p; ++i)
        for (int64_t j = 0; j < n_q; ++j)
            if ((double)or_hamming(P, i, Q, j, d) <= r &&
                push_u32(&ro[i].pairs, &ro[i].n, &ro[i].cap, (uint32_t)j))
                failed = 1;
    int64_t total = 0;
    for (int64_t i = 0; i < n_p; ++i) {
        for (int64_t t = 0; t < ro[i].n; ++t, ++total)
            if (total < cap) {
                out_pairs[2 * total] = (uint32_t)i;
                out_pairs[2 * total + 1] = ro[i].pairs[t];
            }
        free(ro[i].pairs);
    }
    free(ro);
    return failed ? -2 : total;
}

/* Threads the OpenMP runtime would use by default (1 without OpenMP). */
int or_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * LSH-bucketed join (Section 4, the LSH method behind Theorem 3): points of
 * P and Q are hashed into buckets by L independent hash tables, each table's
 * hash being the concatenation of k functions from an LSH family, and a pair
 * is reported when its points share a bucket in at least one table and the
 * pair passes the exact distance test.  The oracle computes that set by its
 * definition: for every pair (i, j), the keys of every table are compared and
 * the exact test is applied; no bucketing, no sorting.
 *
 * The random draws of the LSH are inputs: A holds L*k rows of d int8 entries
 * (function f = t*k + u of table t is row f), B holds L*k int32 offsets, w is
 * the bucket width.  With the projection z_f(x) = sum_m A[f][m] * x_m, in
 * double and in ascending m (every product is exact, so this is the same
 * number for every evaluation in that order):
 *   w == 0 (random-hyperplane signs, for inner product / cosine):
 *       v_f(x) = 1 if z_f(x) >= 0 else 0
 *   w  > 0 (quantised projections, for squared Euclidean distance):
 *       v_f(x) = floor((z_f(x) + B[f]) / w)
 * The key of table t concatenates its k values, each reduced to its low
 * beta = floor(64 / k) bits (two's complement): key_t(x) = sum_u
 * (v_{tk+u}(x) mod 2^beta) * 2^(beta u); with k == 0 every key is 0 (one
 * bucket).  Keys are written table-major: keys[t * n + i].
 */
int or_lsh_keys(int dtype, const void *X, int64_t n, int64_t d, int64_t L, int64_t k,
                const int8_t *A, const int32_t *B, int32_t w, uint64_t *keys)
{
    if (n < 0 || d < 0 || L < 0 || k < 0 || k > 64 || w < 0)
        return -1;
    if (dtype != OR_F16 && dtype != OR_BF16 && dtype != OR_I8)
        return -1;
    const int beta = k > 0 ? (int)(64 / k) : 64;
    const uint64_t low = beta >= 64 ? ~(uint64_t)0 : (((uint64_t)1 << beta) - 1);
    /* OpenMP only splits the independent rows */
#ifdef _OPENMP
#pragma omp parallel for schedule(static)
#endif
    for (int64_t i = 0; i < n; ++i)
        for (int64_t t = 0; t < L; ++t) {
            uint64_t key = 0;
            for (int64_t u = 0; u < k; ++u) {
                const int64_t f = t * k + u;
                double z = 0.0;
                for (int64_t m = 0; m < d; ++m)
                    z += (double)A[f * d + m] * elem(dtype, X, i * d + m);
                int64_t v;
                if (w == 0)
                    v = z >= 0.0 ? 1 : 0;
                else
                    v = (int64_t)floor((z + (double)B[f]) / (double)w);
                key |= ((uint64_t)v & low) << (beta * u);
            }
            keys[t * n + i] = key;
        }
    return 0;
}

/*
 * The LSH-bucketed join: every (i, j) such that key_t(P_i) == key_t(Q_j) for
 * some table t and the pair passes the exact test of `metric` (as or_join).
 * Pairs are written in lexicographic (i, j) order, at most `cap`; returns the
 * total (which may exceed cap), -1 on bad arguments, -2 when out of memory.
 */
int64_t or_lsh_join(int metric, int dtype, const void *P, int64_t n_p, const void *Q,
                    int64_t n_q, int64_t d, double thr, int64_t L, int64_t k, const int8_t *A,
                    const int32_t *B, int32_t w, uint32_t *out_pairs, int64_t cap, int threads)
{
    if (n_p < 0 || n_q < 0 || d < 0 || L < 0 || (metric != OR_IP && metric != OR_L2))
        return -1;
    uint64_t *kp = (uint64_t *)malloc((size_t)(L * n_p + 1) * sizeof(uint64_t));
    uint64_t *kq = (uint64_t *)malloc((size_t)(L * n_q + 1) * sizeof(uint64_t));
    row_out *ro = (row_out *)calloc((size_t)(n_p ? n_p : 1), sizeof(row_out));
    int failed = !kp || !kq || !ro;
    if (!failed && (or_lsh_keys(dtype, P, n_p, d, L, k, A, B, w, kp) != 0 ||
                    or_lsh_keys(dtype, Q, n_q, d, L, k, A, B, w, kq) != 0)) {
        free(kp);
        free(kq);
        free(ro);
        return -1;
    }
    if (!failed) {
#ifdef _OPENMP
        int nt = threads > 0 ? threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
#endif
        for (int64_t i = 0; i < n_p; ++i)
            for (int64_t j = 0; j < n_q; ++j) {
                int collide = 0;
                for (int64_t t = 0; t < L && !collide; ++t)
                    collide = kp[t * n_p + i] == kq[t * n_q + j];
                if (!collide)
                    continue;
                double sc = metric == OR_IP ? or_score_ip(dtype, P, i, Q, j, d)
                                            : or_score_l2(dtype, P, i, Q, j, d);
                if (matches(metric, sc, thr) &&
                    push_u32(&ro[i].pairs, &ro[i].n, &ro[i].cap, (uint32_t)j))
                    failed = 1;
            }
    }
    int64_t total = 0;
    for (int64_t i = 0; ro && i < n_p; ++i) {
        for (int64_t t = 0; t < ro[i].n; ++t, ++total)
            if (total < cap) {
                out_pairs[2 * total] = (uint32_t)i;
                out_pairs[2 * total + 1] = ro[i].pairs[t];
            }
        free(ro[i].pairs);
    }
    free(ro);
    free(kp);
    free(kq);
    return failed ? -2 : total;
}
