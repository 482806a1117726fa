// sj_aux.hip -- kernel planning and dispatch, the squared-row-norm kernel, the
// exclusive scan of the count-then-emit protocol and its emit pass from match
// bits (gfx950).
#include "sj_internal.h"

#include <type_traits>

namespace sjk {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// ------------------------------------------------------------------ planning
// Resident-P limits: 32-byte k-steps of the largest variant (16 for 2-byte
// elements, 8 for int8, i.e. d <= 256 either way); workgroup of 8 waves over
// 32 * WMB rows each (WMB = 4 for int8 rows of at most 64 bytes, else 2); Q
// tiles of 256 rows for rows of at most 64 bytes, 128 up to 256 bytes and 64
// for the longest rows.  Must agree with sj_join_kernels.h.
static const int kResKS16[4] = {2, 4, 8, 16};
static const int kResKS8[4] = {1, 2, 4, 8};
static const uint32_t kResNW = 8;
static uint32_t res_bn(int ks) { return ks <= 2 ? 256 : ks <= 8 ? 128 : 64; }
static const uint32_t kStBM = ST_BM, kStBN = ST_BN, kStG = 8, kStNW = ST_NW;

bool plan_join(int dtype, int metric, uint32_t n_p, uint32_t n_q, uint32_t row_bytes, int num_cus,
               Plan *plan)
{
    const uint32_t ks_needed = row_bytes == 0 ? 1u : (row_bytes + 31) / 32;
    const int *tab = dtype == DT_I8 ? kResKS8 : kResKS16;
    int variant = -1;
    for (int v = 0; v < 4; ++v)
        if ((uint32_t)tab[v] >= ks_needed) {
            variant = v;
            break;
        }
    if (variant >= 0) {
        const int ks = tab[variant];
        const uint32_t wmb = (dtype == DT_I8 && ks <= 2) ? 4 : 2;
        const uint32_t bm = kResNW * 32 * wmb;
        const uint64_t n_pb = (n_p + (uint64_t)bm - 1) / bm;
        const uint64_t bn = res_bn(ks);
        const uint64_t n_qt = (n_q + bn - 1) / bn;
        // Enough workgroups to fill every CU twice (with exactly one round,
        // one late workgroup start stretches the whole kernel); splits of Q
        // are powers of two so that, with workgroups dealt round-robin to the
        // 8 XCDs, each XCD's workgroups sweep the same Q range (shared in that
        // XCD's L2).
        const int occ = dtype == DT_I8    ? resident_occupancy_i8(metric, variant)
                        : dtype == DT_F16 ? resident_occupancy_f16(metric, variant)
                                          : resident_occupancy_bf16(metric, variant);
        uint64_t qsplit = 1;
        while (n_pb * qsplit < 2ull * (uint64_t)occ * (uint64_t)num_cus && qsplit * 2 <= n_qt &&
               qsplit < 64)
            qsplit *= 2;
        plan->family = FAM_RESIDENT;
        plan->variant = variant;
        plan->qsplit = (uint32_t)qsplit;
        plan->block = kResNW * 64;
        const uint64_t grid = n_pb * qsplit;
        if (grid > 0x7fffffffull)
            return false;
        plan->grid = (uint32_t)grid;
        plan->n_blocks = n_pb * kResNW * n_qt;
        // a workgroup sweeps at most ceil(n_qt / qsplit) tiles of bm x bn results
        plan->wg_blocks32 = ((n_qt + qsplit - 1) / qsplit) * (bm / 32) * (bn / 32);
        return true;
    }
    const uint64_t n_pt = (n_p + (uint64_t)kStBM - 1) / kStBM;
    const uint64_t n_qt = (n_q + (uint64_t)kStBN - 1) / kStBN;
    const uint64_t groups = ((n_pt + kStG - 1) / kStG) * ((n_qt + kStG - 1) / kStG);
    const uint64_t grid = groups * kStG * kStG;
    if (grid > 0x7fffffffull)
        return false;
    plan->family = FAM_STREAMED;
    plan->variant = 0;
    plan->qsplit = 1;
    plan->block = kStNW * 64;
    plan->grid = (uint32_t)grid;
    plan->n_blocks = n_pt * n_qt * kStNW;
    plan->wg_blocks32 = 0;
    return true;
}

hipError_t launch_join(const Plan &plan, int dtype, int metric, int mode, const JoinArgs &args,
                       hipStream_t stream)
{
    switch (dtype) {
    case DT_F16: return launch_join_f16(plan, metric, mode, args, stream);
    case DT_BF16: return launch_join_bf16(plan, metric, mode, args, stream);
    case DT_I8: return launch_join_i8(plan, metric, mode, args, stream);
    }
    return hipErrorInvalidValue;
}

// ----------------------------------------------------------------- row norms
// One team of TEAM lanes per row; each lane sums the squares of its 16-byte
// chunks, the team reduces with cross-lane shuffles.  int8 sums are exact in
// int32; fp16/bf16 sums are accumulated in fp32.
template <int DT, int TEAM>
__global__ void __launch_bounds__(256) row_norms(const uint8_t *X, uint32_t n, uint32_t row_bytes,
                                                 void *out)
{
    const uint64_t gt = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    const uint64_t row = gt / TEAM;
    const uint32_t sub = (uint32_t)(gt % TEAM);
    typedef typename std::conditional<DT == DT_I8, int, float>::type V;
    V acc = V(0);
    if (row < n) {
        const uint8_t *p = X + (size_t)row * row_bytes;
        for (uint32_t off = 16 * sub; off < row_bytes; off += 16 * TEAM) {
            const i32x4 v = *(const i32x4 *)(p + off);
            if constexpr (DT == DT_I8) {
#pragma unroll
                for (int w = 0; w < 4; ++w)
#pragma unroll
                    for (int b = 0; b < 4; ++b) {
                        const int x = (int)(int8_t)((uint32_t)v[w] >> (8 * b));
                        acc += x * x;
                    }
            } else if constexpr (DT == DT_F16) {
                const f16x8 h = __builtin_bit_cast(f16x8, v);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float x = (float)h[e];
                    acc = __builtin_fmaf(x, x, acc);
                }
            } else {
                const bf16x8 h = __builtin_bit_cast(bf16x8, v);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float x = (float)h[e];
                    acc = __builtin_fmaf(x, x, acc);
                }
            }
        }
    }
#pragma unroll
    for (int m = TEAM / 2; m > 0; m >>= 1)
        acc += __shfl_xor(acc, m, TEAM);
    if (row < n && sub == 0)
        ((V *)out)[row] = acc;
}

template <int DT>
static hipError_t norms_dt(const uint8_t *X, uint32_t n, uint32_t row_bytes, void *out,
                           hipStream_t st)
{
    if (row_bytes <= 128) {
        const uint64_t threads = (uint64_t)n * 4;
        hipLaunchKernelGGL((row_norms<DT, 4>), dim3((uint32_t)((threads + 255) / 256)), dim3(256), 0,
                           st, X, n, row_bytes, out);
    } else {
        const uint64_t threads = (uint64_t)n * 32;
        hipLaunchKernelGGL((row_norms<DT, 32>), dim3((uint32_t)((threads + 255) / 256)), dim3(256),
                           0, st, X, n, row_bytes, out);
    }
    return hipGetLastError();
}

hipError_t launch_norms(int dtype, const uint8_t *X, uint32_t n, uint32_t row_bytes, void *out,
                        hipStream_t stream)
{
    if (n == 0)
        return hipSuccess;
    switch (dtype) {
    case DT_F16: return norms_dt<DT_F16>(X, n, row_bytes, out, stream);
    case DT_BF16: return norms_dt<DT_BF16>(X, n, row_bytes, out, stream);
    case DT_I8: return norms_dt<DT_I8>(X, n, row_bytes, out, stream);
    }
    return hipErrorInvalidValue;
}

// ------------------------------------------------------------------- repack
// One thread per 4-byte word of the destination, gathered byte by byte (only
// inputs whose rows are not 16-byte aligned take this path).
__global__ void __launch_bounds__(256) repack_rows(const uint8_t *src, uint32_t n,
                                                   uint32_t src_bytes, uint8_t *dst,
                                                   uint32_t dst_bytes)
{
    const uint64_t words = (uint64_t)n * (dst_bytes / 4);
    for (uint64_t w = (uint64_t)blockIdx.x * 256 + threadIdx.x; w < words;
         w += (uint64_t)gridDim.x * 256) {
        const uint64_t row = w / (dst_bytes / 4);
        const uint32_t col = (uint32_t)(w % (dst_bytes / 4)) * 4;
        uint32_t v = 0;
#pragma unroll
        for (uint32_t b = 0; b < 4; ++b)
            if (col + b < src_bytes)
                v |= (uint32_t)src[row * src_bytes + col + b] << (8 * b);
        *(uint32_t *)(dst + row * dst_bytes + col) = v;
    }
}

hipError_t launch_repack(const uint8_t *src, uint32_t n, uint32_t src_bytes, uint8_t *dst,
                         uint32_t dst_bytes, hipStream_t stream)
{
    if (n == 0)
        return hipSuccess;
    const uint64_t words = (uint64_t)n * (dst_bytes / 4);
    const uint64_t blocks = (words + 255) / 256;
    const uint32_t grid = (uint32_t)(blocks < 65536 ? blocks : 65536);
    hipLaunchKernelGGL(repack_rows, dim3(grid), dim3(256), 0, stream, src, n, src_bytes, dst,
                       dst_bytes);
    return hipGetLastError();
}

// --------------------------------------------------------------------- fill
// Zeroes n 64-bit words (counters that must start at zero), with a kernel
// rather than a memset node.
__global__ void __launch_bounds__(64) zero_u64(unsigned long long *p, uint32_t n)
{
    for (uint32_t k = threadIdx.x; k < n; k += 64)
        p[k] = 0ull;
}

hipError_t launch_zero_u64(unsigned long long *p, uint32_t n, hipStream_t stream)
{
    hipLaunchKernelGGL(zero_u64, dim3(1), dim3(64), 0, stream, p, n);
    return hipGetLastError();
}

// ---------------------------------------------------------------------- scan
// Exclusive scan of uint32 block counts into uint64 offsets, in three kernels:
// per-chunk sums, a scan of the chunk sums by one workgroup (which also writes
// the total), and a rescan of every chunk from its offset.
static const uint32_t kScanT = 256, kScanE = 16, kScanChunk = kScanT * kScanE;

uint64_t scan_partials_size(uint64_t n) { return (n + kScanChunk - 1) / kScanChunk + 1; }

__device__ __forceinline__ unsigned long long wave_incl_scan(unsigned long long v, int lane)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const unsigned long long u = __shfl_up(v, o, 64);
        if (lane >= o)
            v += u;
    }
    return v;
}

// Exclusive scan over the 256 threads of a workgroup; returns the workgroup sum.
__device__ __forceinline__ unsigned long long block_excl_scan(unsigned long long v,
                                                              unsigned long long &excl)
{
    __shared__ unsigned long long s_w[kScanT / 64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const unsigned long long inc = wave_incl_scan(v, lane);
    if (lane == 63)
        s_w[w] = inc;
    __syncthreads();
    unsigned long long before = 0, total = 0;
#pragma unroll
    for (int k = 0; k < (int)(kScanT / 64); ++k) {
        if (k < w)
            before += s_w[k];
        total += s_w[k];
    }
    excl = before + inc - v;
    __syncthreads();
    return total;
}

__global__ void __launch_bounds__(256) scan_reduce(const uint32_t *c, uint64_t n,
                                                   unsigned long long *partials)
{
    const uint64_t base = (uint64_t)blockIdx.x * kScanChunk + (uint64_t)threadIdx.x * kScanE;
    unsigned long long s = 0;
#pragma unroll
    for (uint32_t e = 0; e < kScanE; ++e)
        if (base + e < n)
            s += c[base + e];
    unsigned long long excl;
    const unsigned long long tot = block_excl_scan(s, excl);
    if (threadIdx.x == 0)
        partials[blockIdx.x] = tot;
}

__global__ void __launch_bounds__(256) scan_top(unsigned long long *partials, uint64_t np,
                                                unsigned long long *total)
{
    unsigned long long carry = 0;
    for (uint64_t b = 0; b < np; b += kScanT) {
        const uint64_t k = b + threadIdx.x;
        const unsigned long long v = k < np ? partials[k] : 0ull;
        unsigned long long excl;
        const unsigned long long tot = block_excl_scan(v, excl);
        if (k < np)
            partials[k] = carry + excl;
        carry += tot;
    }
    if (threadIdx.x == 0)
        *total = carry;
}

__global__ void __launch_bounds__(256) scan_apply(const uint32_t *c, uint64_t n,
                                                  const unsigned long long *partials,
                                                  unsigned long long *offsets)
{
    const uint64_t base = (uint64_t)blockIdx.x * kScanChunk + (uint64_t)threadIdx.x * kScanE;
    uint32_t v[kScanE];
    unsigned long long s = 0;
#pragma unroll
    for (uint32_t e = 0; e < kScanE; ++e) {
        v[e] = base + e < n ? c[base + e] : 0u;
        s += v[e];
    }
    unsigned long long excl;
    block_excl_scan(s, excl);
    unsigned long long run = partials[blockIdx.x] + excl;
#pragma unroll
    for (uint32_t e = 0; e < kScanE; ++e)
        if (base + e < n) {
            offsets[base + e] = run;
            run += v[e];
        }
}

hipError_t launch_scan(const uint32_t *counts, uint64_t n, unsigned long long *offsets,
                       unsigned long long *partials, unsigned long long *total, hipStream_t stream)
{
    const uint64_t np = (n + kScanChunk - 1) / kScanChunk;
    if (np > 0x7fffffffull)
        return hipErrorInvalidValue;
    if (np)
        hipLaunchKernelGGL(scan_reduce, dim3((uint32_t)np), dim3(kScanT), 0, stream, counts, n,
                           partials);
    hipLaunchKernelGGL(scan_top, dim3(1), dim3(kScanT), 0, stream, partials, np, total);
    if (np)
        hipLaunchKernelGGL(scan_apply, dim3((uint32_t)np), dim3(kScanT), 0, stream, counts, n,
                           partials, offsets);
    return hipGetLastError();
}

// ------------------------------------------------ emit from the match bits
// Second pass of count-then-emit after a MODE_MASK first pass of the
// K-streamed kernel: each wave takes kEmitBlocks consecutive output blocks,
// loads their counts, offsets and match bits at once (one 16-byte load per
// lane per block), and writes every block's pairs from its offset in the
// order of the emit pass that recomputes the product (column block, row block,
// lanes by their exclusive prefix of the per-lane counts, register order
// within a lane), so both second passes produce the same array.  Bound by HBM:
// 1/8 byte read per result and 8 bytes written per match.
// 16 blocks (two tiles) per wave: on the 131072 x 1024 clustered workload
// 1.59 ms, against 1.77-1.81 ms for 2, 4, 8, 12 or 32 blocks.
static const uint32_t kEmitBlocks = 16;

// Inclusive prefix sum over the 64 lanes of a wave: Hillis-Steele steps inside
// each row of 16 lanes (DPP row shifts by 1, 2, 4, 8; lanes shifted in from
// outside the row contribute 0), then the totals of rows 0 and 2 into rows 1
// and 3 (row broadcast of lane 15) and the total of lanes 0-31 into rows 2 and
// 3 (row broadcast of lane 31).  Sums of packed 16-bit fields stay separate
// while every field's total stays below 2^16.
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t x)
{
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);
    return x;
}

__global__ void __launch_bounds__(256) emit_masks(JoinArgs g, uint64_t n_blocks)
{
    static_assert(ST_SA == 2 && ST_SB == 4, "one 32-bit word per column block");
    typedef __attribute__((address_space(1))) const i32x4 gmask;
    typedef __attribute__((address_space(1))) uint64_t gpair;
    const int lane = threadIdx.x & 63;
    // wave-uniform block index (scalar registers, scalar arithmetic below)
    const uint32_t wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint64_t blk0 = ((uint64_t)blockIdx.x * 4 + wv) * kEmitBlocks;
    if (blk0 >= n_blocks)   // uniform per wave
        return;
    uint32_t cnt[kEmitBlocks];
    uint64_t off[kEmitBlocks];
    i32x4 mw[kEmitBlocks];
#pragma unroll
    for (uint32_t k = 0; k < kEmitBlocks; ++k) {
        const bool in = blk0 + k < n_blocks;
        cnt[k] = in ? g.block_counts[blk0 + k] : 0u;
        off[k] = in ? g.block_offsets[blk0 + k] : 0ull;
        mw[k] = in ? *((gmask *)g.masks + ((blk0 + k) * 64 + lane)) : i32x4{0, 0, 0, 0};
    }
    const uint32_t n_qt = (g.n_q + ST_BN - 1) / ST_BN;
    const uint32_t half = (uint32_t)lane >> 5, c32 = (uint32_t)lane & 31;
    gpair *out = (gpair *)g.pairs;
#pragma unroll
    for (uint32_t k = 0; k < kEmitBlocks; ++k) {
        if (cnt[k] == 0)
            continue;
        const uint64_t blk = blk0 + k;
        // the match bits exist only for at most 2^26 blocks (64 GiB), so the
        // tile index fits 32 bits
        const uint32_t tile = (uint32_t)(blk / ST_NW);
        const uint32_t wave = (uint32_t)(blk % ST_NW);
        const uint32_t pt = tile / n_qt, qt = tile % n_qt;
        const uint32_t wr = wave >> 1, wc = wave & 1;
        const uint32_t i0 = pt * ST_BM + 32 * ST_SA * wr + 4 * half;
        // Word b of the record holds column block b: its 32x32 row block 0 in
        // the low 16 bits, row block 1 in the high 16 bits.  The lanes' match
        // counts of both halves, packed, are scanned over the wave at once.
        uint32_t w[ST_SB], incl[ST_SB];
#pragma unroll
        for (int b = 0; b < ST_SB; ++b) {
            w[b] = (uint32_t)mw[k][b];
            const uint32_t c = (uint32_t)__builtin_popcount(w[b] & 0xffffu) |
                               ((uint32_t)__builtin_popcount(w[b] >> 16) << 16);
            incl[b] = wave_incl_scan_u32(c);
        }
        // block-relative start of each (column block, row block) segment
        uint32_t seg = 0;
#pragma unroll
        for (int b = 0; b < ST_SB; ++b) {
            const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)incl[b], 63);
            const uint32_t c = (uint32_t)__builtin_popcount(w[b] & 0xffffu) |
                               ((uint32_t)__builtin_popcount(w[b] >> 16) << 16);
            const uint32_t excl = incl[b] - c;
            uint64_t slot0 = off[k] + seg + (excl & 0xffffu);
            seg += tot & 0xffffu;
            uint64_t slot1 = off[k] + seg + (excl >> 16);
            seg += tot >> 16;
            const uint32_t j = qt * ST_BN + 32 * ST_SB * wc + 32 * b + c32;
            // bit r: row block r / 16, register r % 16, i.e. row
            // i0 + 32 (r / 16) + 8 ((r % 16) / 4) + r % 4 = i0 + 2 (r & 28) + (r & 3)
            uint32_t mm = w[b];
            while (mm != 0) {
                const uint32_t r = (uint32_t)__builtin_ctz(mm);
                mm &= mm - 1;
                const bool hi = r >= 16;
                const uint64_t slot = hi ? slot1 : slot0;
                slot1 += hi ? 1u : 0u;
                slot0 += hi ? 0u : 1u;
                if (slot < g.cap)
                    out[slot] = (uint64_t)(i0 + 2 * (r & 28) + (r & 3)) | ((uint64_t)j << 32);
            }
        }
    }
}

// Second pass of count-then-emit after a MODE_RECORD first pass of the
// resident kernel: workgroup w handles the records of first-pass workgroup w,
// one wave per record, and writes each record's pairs at its output block's
// offset plus the record's position, lanes by their exclusive prefix of the
// per-lane counts, register order within a lane (the order of a MODE_EMIT
// pass).
__global__ void __launch_bounds__(256) emit_records(JoinArgs g)
{
    typedef __attribute__((address_space(1))) const MatchRecord grec;
    typedef __attribute__((address_space(1))) const uint16_t gmask16;
    typedef __attribute__((address_space(1))) uint64_t gpair;
    const int lane = threadIdx.x & 63;
    const uint32_t wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t n = min(g.rec_counts[blockIdx.x], g.rec_cap);
    grec *list = (grec *)g.records + (uint64_t)blockIdx.x * g.rec_cap;
    gpair *out = (gpair *)g.pairs;
    const uint32_t half = (uint32_t)lane >> 5, c32 = (uint32_t)lane & 31;
    for (uint32_t k = wv; k < n; k += 4) {
        grec *rec = list + k;
        const uint64_t blk = rec->blk;
        const uint32_t pos = rec->pos, i0 = rec->i0, j0 = rec->j0;
        uint32_t m = ((gmask16 *)rec->mask)[lane];
        const uint32_t cnt = (uint32_t)__builtin_popcount(m);
        const uint32_t excl = wave_incl_scan_u32(cnt) - cnt;
        uint64_t slot = g.block_offsets[blk] + pos + excl;
        const uint32_t ib = i0 + 4 * half, j = j0 + c32;
        while (m != 0) {
            const uint32_t r = (uint32_t)__builtin_ctz(m);
            m &= m - 1;
            if (slot < g.cap)
                out[slot] = (uint64_t)(ib + 8 * (r >> 2) + (r & 3)) | ((uint64_t)j << 32);
            ++slot;
        }
    }
}

hipError_t launch_emit_records(const JoinArgs &g, uint32_t n_wg, hipStream_t stream)
{
    if (n_wg)
        hipLaunchKernelGGL(emit_records, dim3(n_wg), dim3(256), 0, stream, g);
    return hipGetLastError();
}

hipError_t launch_emit_masks(const Plan &plan, const JoinArgs &g, hipStream_t stream)
{
    if (plan.family != FAM_STREAMED)
        return hipErrorInvalidValue;
    const uint64_t per_wg = 4ull * kEmitBlocks;
    const uint64_t grid = (plan.n_blocks + per_wg - 1) / per_wg;
    if (grid > 0x7fffffffull)
        return hipErrorInvalidValue;
    if (grid)
        hipLaunchKernelGGL(emit_masks, dim3((uint32_t)grid), dim3(256), 0, stream, g,
                           plan.n_blocks);
    return hipGetLastError();
}

}  // namespace sjk
