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
// sorted[t * n + p], perm[t * n + p] = the p-th smallest sort key of table t
// and its row, rows of equal keys in increasing order, where the sort key is
// the key itself when `bits` <= 32 and a fixed bijective mix of it otherwise
// (sj_sort.hip): equal sort keys are exactly equal keys, and every operand is
// sorted in the same order.  `temp` must hold sort_temp_bytes(n, L) bytes;
// `keys` is not modified.
size_t sort_temp_bytes(uint32_t n, uint32_t L);
hipError_t sort_tables(const uint64_t *keys, uint64_t *sorted, uint32_t *perm, uint32_t n,
                       uint32_t L, uint32_t bits, void *temp, hipStream_t s);

// Tile edge of the bucket join (rows of P and of Q per workgroup tile).
constexpr uint32_t TILE = 128;

// The buckets P and Q share, as records in key order within each table,
// tables in order: record r is table t[r] and pq[r] = {p0, np, q0, nq}: P's
// sorted positions [p0, p0 + np) and Q's [q0, q0 + nq) of that table
// (positions within the table's segment).
struct Records {
    uint32_t *t;
    uint4 *pq;
};

// Per row a 16-byte fingerprint of its keys in the first min(L, 16) tables
// (byte t: 8 bits of a multiplicative hash of keys[t n + row]), for the
// bucket join's first-table rule.
hipError_t launch_fingerprints(const uint64_t *keys, uint32_t n, uint32_t L, uint4 *fp,
                               hipStream_t s);

// Marks, for every table t and sorted position p of P that starts a bucket
// whose key Q also has, flag[t n_p + p] = 1 (else 0) with the bucket's sizes
// and Q's first position in f_np / f_q0 / f_nq at that index; writes the
// bucket pairs' pair evaluations (sum of np nq) to n_cand[0] and their rows
// (sum of np + nq) to n_cand[7].  ws: bucket_find_ws_bytes(n_p, L) bytes.
inline size_t bucket_find_ws_bytes(uint32_t n_p, uint32_t L)
{
    return (size_t)((n_p + 255) / 256) * L * 24;
}
hipError_t launch_bucket_find(const uint64_t *sorted_p, uint32_t n_p, const uint64_t *sorted_q,
                              uint32_t n_q, uint32_t L, void *ws, uint32_t *flag, uint32_t *f_np,
                              uint32_t *f_q0, uint32_t *f_nq, unsigned long long *n_cand,
                              hipStream_t s);
// Writes the marked positions as records (rec_off: exclusive scan of flag).
hipError_t launch_bucket_write(uint32_t n_p, uint32_t L, const uint32_t *flag,
                               const uint32_t *f_np, const uint32_t *f_q0, const uint32_t *f_nq,
                               const unsigned long long *rec_off, const Records &rec,
                               hipStream_t s);

// Tiles.  The records are cut into chunks of PACK_CHUNK; within a chunk,
// consecutive records that each fit one tile (np, nq <= TILE) are packed
// greedily into groups of at most TILE P rows and TILE Q rows, one tile per
// group, and every other record is tiled alone by ceil(np / TILE) x
// ceil(nq / TILE) tiles.  A descriptor is (first record, number of records:
// 0 for a record tiled alone, with the record's table and rows copied into
// it, else the group's size) and its first tile.
// count pass (write = false): per chunk the number of descriptors and of
// tiles (chunk_desc, chunk_tiles; *overflow set when a chunk's tiles do not
// fit 32 bits); write pass: the descriptors at desc_off[chunk] with tiles
// numbered from tile_off[chunk].
constexpr uint32_t PACK_CHUNK = 256;
struct Descs {
    uint4 *head;                  // {first record, count, table (count 0), 0}
    uint4 *pq;                    // count 0: the record's {p0, np, q0, nq}
    unsigned long long *tile;     // first tile
};
hipError_t launch_pack(const Records &rec, uint32_t n_rec, bool write, uint32_t *chunk_desc,
                       uint32_t *chunk_tiles, const unsigned long long *desc_off,
                       const unsigned long long *tile_off, const Descs &desc,
                       unsigned long long *overflow, hipStream_t s);

// Row records (rows of rb <= REC_ROW bytes): per row one 128-byte line
// holding the row zero-padded to a multiple of 32 bytes (the k-steps' reads),
// then fingerprint bytes of its keys in the first min(L, F) tables, F = 112 -
// that length (byte 16 rec_fp_chunk(rb) + t for table t, as in
// launch_fingerprints; zero past L), and its squared norm (bytes 112..115:
// int32 for int8 rows, float otherwise; zero for inner products, norm null),
// so that the bucket join gathers each row with one request.
constexpr uint32_t REC_ROW = 96, REC_BYTES = 128;
__host__ __device__ constexpr uint32_t rec_fp_chunk(uint32_t rb) { return (rb + 31) / 32 * 2; }
hipError_t launch_rowrec(const Rows &r, const void *norm, const uint64_t *keys, uint32_t L,
                         uint8_t *out, hipStream_t s);

struct JoinArgs {
    Rows P, Q;
    const uint8_t *rec_p, *rec_q;         // row records, or null (rows, norms, fp)
    uint32_t L;
    const uint32_t *perm_p, *perm_q;      // L x n sorted-position -> row
    const uint64_t *keys_p, *keys_q;      // L x n row -> key (first-table rule)
    const uint4 *fp_p, *fp_q;             // per row: launch_fingerprints
    Records rec;
    Descs desc;
    uint32_t n_desc;
    uint64_t n_tiles;
    float thr_f;                          // as sjk::JoinArgs
    int32_t thr_i;
    const void *norm_p, *norm_q;
    uint32_t *pairs;
    uint64_t cap;
    unsigned long long *counter;
};

hipError_t launch_join(int dtype, int metric, const JoinArgs &g, int num_cus, hipStream_t s);

}  // namespace sjl
