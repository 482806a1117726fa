/*
 * sj.h -- C-ABI of the MI355X (gfx950) similarity-join library (libsj.so).
 *
 * The operation is the similarity join of Ahle & Silvestri, "Similarity Search
 * with Tensor Core Units", Section 4: given point sets P and Q in R^d, report
 * every pair (x, y), x in P, y in Q, whose distance is within a threshold.  The
 * distances are the paper's ip-distances (Section 4): inner product / cosine
 * similarity (cosine is the inner product of rows the caller has normalised,
 * f = g = x / ||x||) and the squared Euclidean distance.  The library computes
 * it the way Section 4's brute-force method does: one blocked dense product of
 * P and Q^T on the matrix cores (Theorem 1's blocked multiplication), with the
 * threshold test and the pair compaction fused into the product's epilogue, so
 * no score matrix is ever stored.
 *
 * Conventions shared by every entry point
 *   - P is n_p x d and Q is n_q x d, row-major and contiguous (row stride d
 *     elements), resident in device memory of the context's GPU and owned by
 *     the caller.  Elements are IEEE binary16 (SJ_F16), bfloat16 (SJ_BF16) or
 *     int8 (SJ_I8); inputs must be finite.  P and Q may be the same pointer
 *     (self-join: every ordered pair, (i, i) included; with n_p == n_q the
 *     single pass then computes only the upper triangle i <= j of the product
 *     and writes each match (i, j), i < j, also as (j, i)).
 *   - Results are ordered index pairs (i, j), i indexing P and j indexing Q,
 *     both 0-based uint32, stored as interleaved {i, j} (8 bytes per pair) in
 *     the caller's device buffer `pairs` of `cap` pairs (8-byte aligned).
 *     Duplicate rows are distinct points.
 *   - Tests are inclusive: <P_i, Q_j> >= s, ||P_i - Q_j||^2 <= r2.
 *   - Arithmetic: fp16/bf16 products accumulate in fp32 on the matrix cores,
 *     int8 products accumulate exactly in int32.  Thresholds are converted once
 *     with directed rounding so that the fp32 comparison equals the comparison
 *     with the double threshold: s -> the smallest float >= s, r2 -> the largest
 *     float <= r2; for int8, s -> ceil(s) and r2 -> floor(r2).  The squared
 *     distance is evaluated as N_x + N_y - 2 <x, y> with the squared row norms
 *     N (int32 for int8, fp32 otherwise).  Integer-valued fp16/bf16 inputs whose
 *     partial sums stay below 2^24 in magnitude are therefore joined exactly.
 *   - Calls are ordered on the context's stream and return once the result
 *     count is known (they synchronise that stream).  Inputs must be ready on
 *     that stream.  A context is not thread-safe: use one per host thread.
 *   - Errors: every call returns a status (SJ_OK = 0 or a negative code) and
 *     never aborts or throws; sj_last_error() describes the last failure of the
 *     calling thread.
 *
 * Sizes: n_p, n_q < 2^32; 0 <= d <= 65536 for fp16/bf16 and d <= 32768 for
 * int8 (larger d could overflow the int32 accumulators); n_p, n_q or d equal
 * to 0 are valid.  n_p = 0 or n_q = 0 gives no pairs.  d = 0 follows the
 * join's definition rather than returning nothing: points of R^0 all
 * coincide, every inner product and squared distance is 0, so every pair
 * matches when s <= 0 (IP) or r2 >= 0 (L2) and none otherwise.
 */
#ifndef SJ_H
#define SJ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sj_ctx sj_ctx;

/* Element types of P and Q. */
enum sj_dtype { SJ_F16 = 1, SJ_BF16 = 2, SJ_I8 = 3 };

/* Metrics: inner product (>= s) and squared Euclidean distance (<= r2). */
enum sj_metric { SJ_IP = 0, SJ_L2 = 1 };

/* Status codes. */
enum sj_status {
    SJ_OK = 0,
    SJ_E_INVAL = -1,       /* bad argument: NULL or non-device pointer, buffer
                              smaller than its shape, NaN threshold, bad enum,
                              a flag the function does not take */
    SJ_E_OVERFLOW = -2,    /* more matches than `cap`: *n_out holds the exact
                              total and the contents of `pairs` are not a valid
                              answer */
    SJ_E_NOMEM = -3,       /* device scratch could not be allocated */
    SJ_E_HIP = -4,         /* a HIP runtime call failed */
    SJ_E_UNSUPPORTED = -5  /* valid but unsupported: d too large, not gfx950 */
};

/* Flags of sj_join_ip / sj_join_l2. */
enum sj_flags {
    /* Count-then-emit: a first pass counts the matches of every output block,
     * an exclusive scan turns the counts into offsets, and a second pass
     * writes each block's pairs at its offset.  Never writes beyond `cap`,
     * and the output order is deterministic (block-major).  The first pass
     * also keeps the match bits it found in device scratch, so that the
     * second pass only reads them and writes the pairs: with the K-streamed
     * kernel (rows of more than 512 bytes) one bit per result (n_p n_q / 8
     * bytes, rounded up to 256 x 256 tiles, while at most 64 GiB), with the
     * resident kernel one 160-byte record per 32 x 32 block that has matches
     * (room for min(4 Mi, blocks) records).  When the bits do not fit, the
     * second pass recomputes the product; both second passes write the same
     * array.  Without the flag a single pass appends pairs through one atomic
     * counter (order unspecified). */
    SJ_FLAG_TWO_PASS = 1u,
    /* Record GPU timestamps around every phase of the call (see sj_stats). */
    SJ_FLAG_TIMING = 2u,
    /* With SJ_FLAG_TWO_PASS: always recompute the product in the second pass
     * (no match bits, no scratch beyond the block counts and offsets). */
    SJ_FLAG_RECOMPUTE = 4u,
    /* sj_join_ip only: Section 4's cosine ip-distance, f = g = x / ||x||.  P and
     * Q are first normalised as sj_normalize does (into device memory the
     * context owns: 2 (n_p + n_q) d bytes, n_q d fewer when P == Q) and the
     * join is the inner product of the normalised rows, >= s, with the
     * arithmetic of the fp16 (fp16 and int8 inputs) or bf16 (bf16 inputs)
     * join. */
    SJ_FLAG_COSINE = 8u
};

/* Diagnostics of the last sj_join_ip / sj_join_l2 / sj_count call. */
typedef struct sj_stats {
    uint64_t total;        /* matches found */
    double ms_norms;       /* GPU time of the row-norm kernel (L2 only)        */
    double ms_join;        /* single pass: the fused product/filter/compaction */
    double ms_count;       /* two-pass / count: the counting pass              */
    double ms_scan;        /* two-pass / count: the scan of the block counts   */
    double ms_emit;        /* two-pass: the emitting pass                      */
    uint32_t kernel;       /* 1 = P rows resident in registers, 2 = K-streamed,
                              3 = LSH bucket join (sj_join_lsh)              */
    uint32_t timed;        /* 1 when the ms_* fields were measured             */
    uint32_t emit_from_bits; /* two-pass: 1 when the second pass read the first
                                pass's match bits (or match records) instead
                                of recomputing the product                    */
    uint64_t lsh_rows;     /* sj_join_lsh: the sum over tables and shared
                              buckets of |P bucket| + |Q bucket| (the rows
                              the bucket join must read at least once)       */
} sj_stats;

/* Create a context on `device` (a gfx950 GPU), bound to `stream` (a
 * hipStream_t; NULL = the null stream).  The context owns only its device
 * scratch (match counter, block counts and offsets, row norms), which grows on
 * demand and is freed by sj_destroy.  Returns SJ_E_UNSUPPORTED on a GPU that
 * is not gfx950. */
int sj_create(sj_ctx **ctx, int device, void *stream);

/* Inner-product join (Section 4; cosine when the caller's rows are unit):
 * every (i, j) with <P_i, Q_j> >= s.  The first min(total, cap) pairs are
 * written to `pairs` (device; may be NULL when cap == 0) and the total is
 * stored in *n_out (host).  Returns SJ_E_OVERFLOW when total > cap. */
int sj_join_ip(sj_ctx *ctx, int dtype, const void *P, uint32_t n_p, const void *Q, uint32_t n_q,
               uint32_t d, double s, uint32_t *pairs, uint64_t cap, uint64_t *n_out,
               unsigned flags);

/* Squared-Euclidean join (Section 4's squared L2 ip-distance): every (i, j)
 * with ||P_i - Q_j||^2 <= r2 (r2 is the squared radius).  Outputs and errors
 * as sj_join_ip. */
int sj_join_l2(sj_ctx *ctx, int dtype, const void *P, uint32_t n_p, const void *Q, uint32_t n_q,
               uint32_t d, double r2, uint32_t *pairs, uint64_t cap, uint64_t *n_out,
               unsigned flags);

/* Size of the similarity join of Section 4 (the number of pairs (x, y), x in
 * P, y in Q, within the threshold) with metric `metric` (SJ_IP: <P_i, Q_j> >=
 * threshold, SJ_L2: ||P_i - Q_j||^2 <= threshold), stored in *count (host);
 * writes no pairs.  Runs the counting pass and the scan of the count-then-emit
 * protocol, with the arithmetic, threshold rounding and errors of
 * sj_join_ip / sj_join_l2.  A caller sizes `pairs` with it before a
 * count-then-emit call. */
int sj_count(sj_ctx *ctx, int metric, int dtype, const void *P, uint32_t n_p, const void *Q,
             uint32_t n_q, uint32_t d, double threshold, uint64_t *count);

/* Section 4's cosine ip-distance front end: Y = every row of X divided by its
 * Euclidean norm, f(x) = x / ||x||.  X is n x d (dtype, row-major, device);
 * Y (device, n x d 16-bit values) receives binary16 rows for SJ_F16 and SJ_I8
 * inputs and bfloat16 rows for SJ_BF16.  ||x|| is the square root of the sum
 * of the squares of the exactly decoded elements, summed in double in
 * ascending k; each x_k / ||x|| is one double division, rounded to the
 * nearest output value, ties to even.  A row whose norm is 0 is written as
 * zeros.  Device scratch: n doubles.  Errors as sj_join_ip (16-bit rows must
 * be 2-byte aligned). */
int sj_normalize(sj_ctx *ctx, int dtype, const void *X, uint32_t n, uint32_t d, void *Y);

/* Section 4's Hamming ip-distance: every (i, j) whose bit rows P_i and Q_j
 * differ in at most r of their d coordinates.  P (n_p rows) and Q (n_q rows)
 * are device bit rows of ceil(d / 8) bytes each, coordinate m in bit m % 8 of
 * byte m / 8 (bits past d are ignored).  As the paper does, the rows are
 * mapped to f(x) = (x, 1 - x) and g(y) = (1 - y, y) (int8 rows of 2 d values
 * in device memory the context owns, (n_p + n_q) * 2 d bytes rounded up to 16
 * per row), so that f(x).g(y) is the Hamming distance, and the pairs come from
 * the int8 matrix-core join of f(P) with -g(Q) at threshold -r
 * (f(x).(-g(y)) >= -r).  With P == Q and n_p == n_q the single pass computes
 * the upper triangle only and mirrors its pairs.  Limits: d <= 16384.
 * Outputs, flags (SJ_FLAG_TWO_PASS, SJ_FLAG_TIMING, SJ_FLAG_RECOMPUTE) and
 * errors as sj_join_ip; d = 0 gives every pair when r >= 0. */
int sj_join_hamming(sj_ctx *ctx, const void *P, uint32_t n_p, const void *Q, uint32_t n_q,
                    uint32_t d, double r, uint32_t *pairs, uint64_t cap, uint64_t *n_out,
                    unsigned flags);

/* For callers that cannot allocate device memory during the join (serving
 * loops, harnesses that forbid hipMalloc / hipFree): the join of sj_join_ip
 * (metric SJ_IP) or sj_join_l2 (SJ_L2), with the same arguments, results,
 * ordering and errors, that allocates nothing.  Its device scratch (match
 * counter, scan total, row norms, repacked rows, block counts and offsets) is
 * a fixed 16 MiB region of this library that each GPU holds until the process
 * ends, located once per device by sj_create; a call that would need more
 * (e.g. SJ_L2 with n_p + n_q above about 4 Mi rows, or count-then-emit with
 * more than about 1.3 M output blocks) returns SJ_E_UNSUPPORTED before any
 * launch.  Flags: SJ_FLAG_TWO_PASS (its second pass always recomputes the
 * product: no match bits are kept), SJ_FLAG_TIMING, SJ_FLAG_RECOMPUTE (implied).
 * Every call on one GPU uses that GPU's region: calls that overlap on one GPU
 * (several host threads, or contexts on different streams) race and must be
 * serialised by the caller.  Like the other joins it synchronises the
 * context's stream, so it cannot be captured into a HIP graph. */
int sj_join_noalloc(sj_ctx *ctx, int metric, int dtype, const void *P, uint32_t n_p,
                    const void *Q, uint32_t n_q, uint32_t d, double threshold, uint32_t *pairs,
                    uint64_t cap, uint64_t *n_out, unsigned flags);

/* LSH-bucketed join (Section 4, the LSH method of Theorem 3): instead of all
 * n_p x n_q pairs, only pairs whose points share a bucket of some hash table
 * are evaluated.  There are L tables; table t hashes a point x with the
 * concatenation of k functions f = t*k + u (u < k), each a random projection
 * z_f(x) = sum_m A[f][m] x_m:
 *   w == 0: v_f(x) = 1 if z_f(x) >= 0 else 0   (random-hyperplane signs, the
 *           LSH for angular distance: use with SJ_IP on unit rows, i.e. cosine)
 *   w  > 0: v_f(x) = floor((z_f(x) + B[f]) / w) (quantised projections with
 *           offsets, the p-stable LSH for Euclidean distance: use with SJ_L2)
 * and the bucket of x in table t is the tuple of its k values, each reduced to
 * its low floor(64 / k) bits (two's complement).  z_f is evaluated exactly for
 * integer-valued inputs, and in double precision in ascending m otherwise.
 * The result is every pair (i, j) whose points P_i and Q_j share a bucket in at
 * least one table and pass the exact test of `metric` (SJ_IP: <P_i, Q_j> >= thr,
 * SJ_L2: ||P_i - Q_j||^2 <= thr, with the arithmetic and threshold rounding
 * of sj_join_ip / sj_join_l2): a subset of the exact join, each pair
 * reported once (by the first table in which it collides), in unspecified
 * order.  The random draws are the caller's:
 *   A  device, L*k rows of d int8 entries (row-major, row t*k + u);
 *   B  device, L*k int32 offsets (read only when w > 0; may be NULL when w == 0);
 *   w  bucket width (0 = sign hashes).
 * Afterwards sj_get_stats reports kernel = 3, ms_norms = repacking, norms and
 * hashing, ms_scan = the sorts and the bucket pairing, ms_join = the
 * bucket join.
 * Limits: 1 <= L <= 256, 0 <= k <= 64 (k = 0: one bucket per table, the exact
 * join), L * max(n_p, n_q) < 2^32; other arguments, outputs and errors as
 * sj_join_ip.  *n_cand (host, may be NULL) receives the number of pair
 * evaluations made (the sum over tables and shared buckets of |P bucket| x
 * |Q bucket|).  Device scratch grows to about L * (n_p + n_q) * 70 bytes plus
 * 16 bytes per row of P and of Q. */
int sj_join_lsh(sj_ctx *ctx, int metric, int dtype, const void *P, uint32_t n_p, const void *Q,
                uint32_t n_q, uint32_t d, double thr, uint32_t L, uint32_t k, const int8_t *A,
                const int32_t *B, int32_t w, uint32_t *pairs, uint64_t cap, uint64_t *n_out,
                uint64_t *n_cand);

/* The grouping step of sj_join_lsh on its own (Section 4: the points of each
 * table grouped by their bucket).  keys (device, L*n uint64, table-major: keys[t*n
 * + i] is row i's bucket key in table t; each key below 2^bits, bits <= 64,
 * else the grouping is unspecified) is left unchanged; perm (device, L*n uint32,
 * caller-owned) receives for each table t the rows 0..n-1 ordered so that rows
 * of equal keys are contiguous and in increasing row order.  The order of the
 * groups is a function of the key values and `bits` alone (ascending key when
 * bits <= 32, the ascending order of a fixed bijective mix of the key
 * otherwise), so key sets sorted by separate calls list their common keys in
 * the same relative order: sj_join_lsh pairs P's buckets with Q's by merging
 * two such orders.  Errors: SJ_E_INVAL (NULL context, bits > 64, NULL,
 * non-device, undersized or misaligned keys / perm), SJ_E_UNSUPPORTED (L * n
 * >= 2^32), SJ_E_NOMEM (scratch), SJ_E_HIP (a runtime call failed); L * n = 0
 * does nothing.  Device scratch grows to about L * n * 20 bytes. */
int sj_lsh_sort(sj_ctx *ctx, const uint64_t *keys, uint32_t n, uint32_t L, uint32_t bits,
                uint32_t *perm);

/* Collision probability of one function of the LSH families of sj_join_lsh
 * for two points at distance `dist`: w == 0 (random-hyperplane signs): dist
 * is the angle between the vectors, in [0, pi], and the probability is
 * 1 - dist / pi; w > 0 (quantised projections floor((<a, x> + b) / w) with
 * a ~ N(0, sigma^2 I), b uniform in [0, w)): dist is the Euclidean distance
 * and the probability is 1 - 2 Phi(-w / u) - 2 u / (sqrt(2 pi) w)
 * (1 - exp(-w^2 / (2 u^2))) with u = sigma dist.  NaN for arguments outside
 * these ranges.  Host only. */
double sj_lsh_collision(int32_t w, double sigma, double dist);

/* Section 4's choice of the LSH join's parameters (host only), for one
 * function's collision probabilities p1 at the join's threshold distance and
 * p2 at a far distance (0 < p2 < p1 < 1), n points per side and the matrix
 * cores' tile edge `tile` standing for the paper's sqrt(m) (a TCU(m, tau)
 * with tau = m, so that Section 4's p2 = m^(3/2) / (tau n) is tile / n):
 *   *k      = the least k with p2^k <= tile / n (each point meets at most one
 *             tile of far points per table in expectation; 0 when n <= tile),
 *   *L_inst = ceil(1 / p1^k) tables: one instance finds a pair at the
 *             threshold with probability 1 - (1 - p1^k)^L_inst >= 1 - 1/e,
 *   *reps   = ceil(ln(1 / (1 - recall))) independent instances, merged, find
 *             it with probability >= 1 - e^-reps >= recall (Section 4's
 *             O(log n) instances for a high-probability guarantee).
 * sj_join_lsh with L = L_inst * reps tables (independent draws) and k runs the
 * merged instances in one call: its first-table rule reports every pair that
 * collides in any table once.  Returns SJ_E_INVAL for arguments out of range,
 * SJ_E_UNSUPPORTED when k would exceed 64. */
int sj_lsh_plan(double p1, double p2, uint64_t n, uint32_t tile, double recall, uint32_t *k,
                uint32_t *L_inst, uint32_t *reps);

/* TCU Johnson-Lindenstrauss transform (Lemma 3 / Theorem 2): the reduced
 * rows Y_j = M X_j of the n rows of X (n x d, row-major, dtype as the joins,
 * device) with
 *   M = (I_{r_l} (x) A_l) ... (I_{r_1} (x) A_1),
 * where A_i is k_i x c_i and I_r (x) A_i applies A_i to each of r consecutive
 * blocks of c_i entries.  shape (host) holds (k_i, c_i, r_i) for i = 1..l
 * (`levels` = l, at most 32); the sizes must chain as d = r_1 c_1 and
 * r_i k_i = r_{i+1} c_{i+1}; the output dimension is r_l k_l.  A (device,
 * fp32) holds A_1, ..., A_l one after the other, each row-major.  Y (device,
 * fp32) receives n x (r_l k_l) values.  Each level is one fp32 product on the
 * matrix cores (inputs decoded exactly to fp32; intermediate levels in fp32
 * device scratch of at most 2 n max_i(r_i k_i) floats).  The JL guarantee
 * (norms kept within 1 +- eps with probability 1 - delta) is a property of
 * the caller's A_i (e.g. i.i.d. N(0, 1/k_i) entries), not of this call.
 * Errors as sj_join_ip (SJ_E_INVAL for a broken size chain, SJ_E_UNSUPPORTED
 * for k_i or c_i above 65536 or a level of more than 2^48 values n r_i k_i);
 * afterwards sj_get_stats reports ms_join = the transform's GPU time. */
int sj_jl(sj_ctx *ctx, int dtype, const void *X, uint32_t n, uint32_t d, uint32_t levels,
          const uint32_t *shape, const float *A, float *Y);

/* Free the context and its scratch; NULL is a no-op. */
void sj_destroy(sj_ctx *ctx);

/* Copy the diagnostics of the context's last call into *out. */
int sj_get_stats(const sj_ctx *ctx, sj_stats *out);

/* Message describing the last failed call made by this thread ("" if none).
 * The string is owned by the library and valid until the thread's next call. */
const char *sj_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SJ_H */
