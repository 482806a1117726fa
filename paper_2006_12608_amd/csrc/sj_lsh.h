// sj_lsh.h -- interface between the LSH-bucketed join's host code (sj_lsh_api.cpp)
// and its gfx950 kernels (sj_lsh.hip).  Not part of the public C-ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sjl {

// Rows of one operand as the kernels read them: n rows of row_bytes bytes
// (a multiple of 16, 16-byte aligned, zero beyond the d stored elements).
struct Rows {
    const uint8_t *X;
    uint32_t n, row_bytes;
};

// Bucket keys of every row in every table, table-major: keys[t * n + i].
// Sign hashes (w == 0) are stored compressed, bit u = v_{t k + u}; quantised
// hashes (w > 0) as the concatenation of their values' low floor(64 / k) bits.
// Either way two rows share a bucket of table t exactly when their keys are
// equal.  key_bits(k, w) is the number of low bits a key can occupy.
// The projection entries come widened by launch_widen (widened_bytes(...)
// bytes: int32 for int8 rows, double otherwise; each row padded with zeros
// to a whole number of 16-byte chunks of the input rows).
uint32_t key_bits(uint32_t k, int32_t w);
size_t widened_bytes(int dtype, uint32_t L, uint32_t k, uint32_t d);
hipError_t launch_widen(int dtype, const int8_t *A, uint32_t n_fn, uint32_t d, void *out,
                        hipStream_t s);
hipError_t launch_keys(int dtype, const Rows &r, uint32_t d, uint32_t L, uint32_t k,
                       const void *Aw, const int32_t *B, int32_t w,
                       uint64_t *keys, hipStream_t s);

// The same keys with the projections on the matrix cores (rows of at most
// 512 bytes, L k <= 512, k >= 2 for quantised hashes:
// keys_fast_applies): decisions the fp32 sums make certain are kept, the
// other (row, table) keys are recomputed exactly.  `ws` is workspace of
// keys_fast_bytes(n_max, L, k, row_bytes) bytes whose first part (the fp16 /
// bf16 projection rows and their norms) is filled when `widen` is set and
// reused otherwise; `nfix` a zeroed device counter per call; Aw as launch_keys.
bool keys_fast_applies(int dtype, uint32_t row_bytes, uint32_t L, uint32_t k, int32_t w);
size_t keys_fast_bytes(uint32_t n_max, uint32_t L, uint32_t k, uint32_t row_bytes);
hipError_t launch_keys_fast(int dtype, const Rows &r, uint32_t d, uint32_t L, uint32_t k,
                            const int8_t *A, const void *Aw, const int32_t *B, int32_t w, uint64_t *keys, void *ws, bool widen,
                            unsigned long long *nfix, hipStream_t s);

// Sorts each table's keys with the row indices as values (n rows per table):
// sorted[t * n + p], perm[t * n + p] = the p-th smallest key of table t and its
// row, rows of equal keys in increasing order (a stable radix sort over the
// keys' low `bits` bits, tables as segments; sj_sort.hip).  `temp` must hold
// sort_temp_bytes(n, L) bytes; `keys` is not modified.
size_t sort_temp_bytes(uint32_t n, uint32_t L);
hipError_t sort_tables(const uint64_t *keys, uint64_t *sorted, uint32_t *perm, uint32_t n,
                       uint32_t L, uint32_t bits, void *temp, hipStream_t s);

// Tile edge of the bucket join (rows of P and of Q per workgroup tile).
constexpr uint32_t TILE = 128;
// Low bits of the packed bucket-pair counter that hold the running tile count.
constexpr int TILE_BITS = 38;

// Bucket pairs: for every table and every key present in both P and Q, one
// record (t, first sorted position in P, P rows, first sorted position in Q)
// plus its Q rows and its first tile within its table.  Table t keeps its
// records in its own region [t tcap, (t + 1) tcap) and its own counters (a
// cache line each, CSTRIDE words apart, so the tables' atomics do not
// contend): counters[t CSTRIDE] = records << TILE_BITS | tiles (one packed
// atomic numbers the records, so first tiles increase with the record), and
// counters[t CSTRIDE + 1] = pair evaluations.
constexpr int CSTRIDE = 16;
struct BucketPairs {
    uint4 *head;          // {t, p0, np, q0}
    uint32_t *nq;
    unsigned long long *tile0;
    unsigned long long *counters;   // L * CSTRIDE words
    uint32_t tcap;        // records per table region
};

hipError_t launch_bucket_pairs(const uint64_t *sorted_p, uint32_t n_p, const uint64_t *sorted_q,
                               uint32_t n_q, uint32_t L, const BucketPairs &bp, hipStream_t s);

struct JoinArgs {
    Rows P, Q;
    uint32_t L;
    const uint32_t *perm_p, *perm_q;      // L x n sorted-position -> row
    const uint64_t *keys_p, *keys_q;      // L x n row -> key (first-table rule)
    const uint4 *head;
    const uint32_t *nq;
    const unsigned long long *tile0;
    uint32_t tcap;                        // records per table region
    uint64_t n_tiles;
    uint64_t tbase[65];                   // first tile of each table (tbase[L] = n_tiles)
    uint32_t nrec[64];                    // records of each table
    float thr_f;                          // as sjk::JoinArgs
    int32_t thr_i;
    const void *norm_p, *norm_q;
    uint32_t *pairs;
    uint64_t cap;
    unsigned long long *counter;
};

hipError_t launch_join(int dtype, int metric, const JoinArgs &g, int num_cus, hipStream_t s);

}  // namespace sjl
