// sj_internal.h -- interface between the host API (sj_api.cpp) and the gfx950
// kernels (sj_kernels_*.hip).  Not part of the public C-ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sjk {

enum { DT_F16 = 1, DT_BF16 = 2, DT_I8 = 3 };
enum { MET_IP = 0, MET_L2 = 1 };

// What the fused epilogue does with the matches it finds.
enum Mode {
    MODE_SINGLE = 0,  // append through one atomic counter per wave (single pass)
    MODE_COUNT = 1,   // count the matches of every output block, write no pairs
    MODE_EMIT = 2,    // write each block's matches at its precomputed offset
    MODE_MASK = 3,    // count as MODE_COUNT and keep every result's match bit
                      // (K-streamed kernel only), for an emit pass that reads
                      // the bits instead of recomputing the product
    MODE_RECORD = 4,  // count as MODE_COUNT and append one MatchRecord per
                      // 32x32 block with matches to the workgroup's own list
                      // (resident kernel only), for an emit pass that reads
                      // the records instead of recomputing
    MODE_TRI = 5      // single pass of a self-join (Q is P) over the upper
                      // triangle only: tiles below the diagonal are skipped,
                      // each match (i, j) with i < j is written as (i, j) and
                      // (j, i), and (i, i) once
};

// The matches of one 32x32 block of results, as found by the first pass of
// count-then-emit (MODE_RECORD): the block's output block, the number of that
// output block's matches that precede this block's, the block's first row and
// column, and 64 lane masks in the MFMA accumulator layout (bit r of lane l's
// mask is row i0 + 8 (r / 4) + 4 (l / 32) + r % 4, column j0 + l % 32).
struct MatchRecord {
    uint64_t blk;
    uint32_t pos, i0, j0, pad[3];
    uint16_t mask[64];
};
static_assert(sizeof(MatchRecord) == 160, "record layout");

// Kernel families.
enum Family {
    FAM_RESIDENT = 1,  // P rows held in VGPRs for the whole of d; Q tiles streamed via LDS
    FAM_STREAMED = 2   // both operands streamed through LDS in K chunks (large d)
};

// Tile geometry of the K-streamed kernel, shared by its planner and by the
// pass that emits pairs from its match bits: workgroup tiles of ST_BM rows of
// P by ST_BN rows of Q, ST_NW waves, each owning ST_SA x ST_SB blocks of 32x32
// results (rows 32 ST_SA wave_row + ..., columns 32 ST_SB wave_col + ...; the
// waves of a workgroup form a (ST_NW / 2) x 2 grid).  One output block per
// wave and tile.
constexpr int ST_BM = 256, ST_BN = 256, ST_NW = 8, ST_SA = 2, ST_SB = 4;
static_assert(ST_BM == 32 * ST_SA * (ST_NW / 2) && ST_BN == 32 * ST_SB * 2, "wave grid");
// Match bits of one output block: ST_SA * ST_SB blocks of 32x32 results as
// 16-bit lane masks in the MFMA accumulator layout (bit r of lane l's mask is
// row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32 of the block), stored
// lane-major: lane l's masks of blocks s = column block * ST_SA + row block
// are the 16 contiguous bytes [16 l, 16 l + 16) (mask s in bytes 2 s, 2 s + 1).
constexpr uint32_t ST_MASK_WORDS = ST_SA * ST_SB * 64;
static_assert(ST_SA * ST_SB == 8, "one 16-byte access per lane");

struct JoinArgs {
    const uint8_t *P;            // n_p rows of row_bytes bytes
    const uint8_t *Q;            // n_q rows of row_bytes bytes
    uint32_t n_p, n_q;
    uint32_t row_bytes;          // bytes per row: a multiple of 16, rows 16-byte aligned
    float thr_f;                 // fp16/bf16: IP s32 (acc >= thr_f); L2 r2_32
    int32_t thr_i;               // int8: IP ceil(s) (acc >= thr_i); L2 floor(r2)
    const void *norm_p;          // L2: squared norms of P rows (int32 for int8, float otherwise)
    const void *norm_q;          // L2: squared norms of Q rows
    uint32_t *pairs;             // cap x {i, j}
    uint64_t cap;
    unsigned long long *counter; // MODE_SINGLE: running match count
    uint32_t *block_counts;      // MODE_COUNT: one count per output block
    const unsigned long long *block_offsets;  // MODE_EMIT: exclusive prefix of block_counts
    uint16_t *masks;             // MODE_MASK: ST_MASK_WORDS per output block
    MatchRecord *records;        // MODE_RECORD: rec_cap records per workgroup, by workgroup
    uint32_t rec_cap;
    uint32_t *rec_counts;        // MODE_RECORD: records found per workgroup (may pass rec_cap)
    unsigned long long *rec_max; // MODE_RECORD: largest of rec_counts (atomic max)
    uint32_t qsplit;             // FAM_RESIDENT: Q ranges per P block
};

// A launch decided by plan_join; the count and emit passes of one call use the
// same plan so that their output blocks coincide.
struct Plan {
    int family;
    int variant;                 // index into the family's instantiation table
    uint32_t grid, block;
    uint32_t qsplit;
    uint64_t n_blocks;           // number of output blocks (entries of block_counts)
    uint64_t wg_blocks32;        // FAM_RESIDENT: most 32x32 result blocks of one workgroup
};

// Chooses the kernel for (dtype, metric, shape) on a GPU with `num_cus` CUs.
// Returns false when the shape is unsupported.
bool plan_join(int dtype, int metric, uint32_t n_p, uint32_t n_q, uint32_t row_bytes,
               int num_cus, Plan *plan);

hipError_t launch_join(const Plan &plan, int dtype, int metric, int mode, const JoinArgs &args,
                       hipStream_t stream);

// Second pass of count-then-emit for the K-streamed kernel after a MODE_MASK
// first pass: every output block's pairs from its match bits, written at its
// offset in the same order as a MODE_EMIT pass (reads g.masks, g.block_counts,
// g.block_offsets; writes g.pairs below g.cap).
hipError_t launch_emit_masks(const Plan &plan, const JoinArgs &g, hipStream_t stream);

// Second pass of count-then-emit after a MODE_RECORD first pass of the
// resident kernel (n_wg workgroups, none with more than rec_cap records): the
// pairs of every record, each written at its output block's offset plus its
// position, in the order of a MODE_EMIT pass.
hipError_t launch_emit_records(const JoinArgs &g, uint32_t n_wg, hipStream_t stream);

// Squared row norms: out[i] = sum_k X[i][k]^2 (int32 for int8, fp32 otherwise).
// Rows as in JoinArgs (16-byte aligned, row_bytes a multiple of 16).
hipError_t launch_norms(int dtype, const uint8_t *X, uint32_t n, uint32_t row_bytes, void *out,
                        hipStream_t stream);

// Copies n rows of src_bytes bytes (any alignment) into rows of dst_bytes
// bytes (dst_bytes >= src_bytes, a multiple of 16), zero-filling the tail.
hipError_t launch_repack(const uint8_t *src, uint32_t n, uint32_t src_bytes, uint8_t *dst,
                         uint32_t dst_bytes, hipStream_t stream);

// Section 4's cosine front end: Y (n x d, 16-bit) = every row of X (n x d of
// dtype, row-major) divided by its Euclidean norm (double, ascending k) and
// rounded to the nearest binary16 (fp16 and int8 inputs) or bfloat16 (bf16
// inputs), ties to even; zero rows give zeros.  `norm` is n doubles of scratch.
hipError_t launch_normalize(int dtype, const void *X, uint32_t n, uint32_t d, double *norm,
                            void *Y, hipStream_t stream);

// Section 4's Hamming front end: bit rows (ceil(d / 8) bytes, coordinate m in
// bit m % 8 of byte m / 8) to int8 rows of out_bytes bytes (a multiple of 16,
// at least 2 d): side 0 writes f(x) = (x, 1 - x), side 1 writes -g(y) =
// (y - 1, -y), zero past 2 d; <f(x), -g(y)> = -Hamming(x, y).
hipError_t launch_unpack_hamming(const uint8_t *bits, uint32_t n, uint32_t d, uint32_t out_bytes,
                                 int side, uint8_t *out, hipStream_t stream);

// Zeroes n 64-bit words on `stream` (one small kernel, no memset node).
hipError_t launch_zero_u64(unsigned long long *p, uint32_t n, hipStream_t stream);

// Exclusive scan of n uint32 counts into n uint64 offsets; *total receives the
// sum.  `partials` needs scan_partials_size(n) elements of scratch.
uint64_t scan_partials_size(uint64_t n);
hipError_t launch_scan(const uint32_t *counts, uint64_t n, unsigned long long *offsets,
                       unsigned long long *partials, unsigned long long *total,
                       hipStream_t stream);

// Per-dtype launchers (one translation unit per element type).
hipError_t launch_join_f16(const Plan &, int metric, int mode, const JoinArgs &, hipStream_t);
hipError_t launch_join_bf16(const Plan &, int metric, int mode, const JoinArgs &, hipStream_t);
hipError_t launch_join_i8(const Plan &, int metric, int mode, const JoinArgs &, hipStream_t);
// Workgroups of a resident-kernel variant that one CU holds at once.
int resident_occupancy_f16(int metric, int variant);
int resident_occupancy_bf16(int metric, int variant);
int resident_occupancy_i8(int metric, int variant);

}  // namespace sjk
