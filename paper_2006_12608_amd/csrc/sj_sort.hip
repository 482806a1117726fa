// sj_sort.hip -- the sort of the LSH-bucketed join (Section 4: the points of a
// table are grouped by bucket): every table's n keys sorted with their rows,
// on gfx950.
//
// Only the grouping of equal keys matters, so a table's keys are sorted in
// the order of a bijective mix of them, m(key), when they use more than 32
// bits: 32-bit sort keys (the key itself, or the top half of m(key)) are
// sorted with their rows, the full m(key) of every sorted position is then
// gathered through the permutation, and the rare runs whose top halves are
// equal but whose m differ are put in the order of m by a local sort.  The
// outputs are the sorted m(key) (or keys) and their rows; equal outputs are
// exactly equal keys, and P and Q are sorted in one order.
//
// The 32-bit sort is a stable least-significant-digit radix sort over 8-bit
// digits, run on all L tables at once: each table is a segment of n entries,
// each segment is cut into blocks of SORT_TILE entries, and every pass is
//   sort_hist:    per (segment, digit, block) counts of the pass's digit;
//   exclusive scan of the counts laid out [segment][digit][block] (segment s
//                 then starts at s n, since every segment holds n entries):
//                 each (segment, digit, block)'s first output position;
//   sort_scatter: each block ranks its entries stably by digit (wave ballots
//                 find the lanes that share a digit; a per-wave running count
//                 per digit continues the rank across the wave's rounds), puts
//                 them in digit order in LDS and writes each digit's run to its
//                 position, so a block's stores are contiguous runs.
// Bound by HBM: each pass reads the sort keys twice and the rows once and
// writes both (20 bytes per entry).
#include "sj_internal.h"
#include "sj_lsh.h"

namespace sjl {

constexpr int SORT_T = 256;                    // threads per block (4 waves)
constexpr int SORT_IPT = 8;                    // entries per thread
constexpr int SORT_TILE = SORT_T * SORT_IPT;   // entries per block
constexpr int SORT_BITS = 8;                   // digit width
constexpr int SORT_BINS = 1 << SORT_BITS;
static_assert(SORT_BINS == SORT_T, "one thread per digit in the block-wide steps");

// Counts of the digit (key >> shift) & mask in block `blk` of segment `seg`.
__global__ void __launch_bounds__(SORT_T) sort_hist(const uint32_t *keys, uint32_t n, uint32_t bps,
                                                    uint32_t shift, uint32_t mask, uint32_t *hist)
{
    __shared__ uint32_t cnt[SORT_T / 64][SORT_BINS];
    const uint32_t b = blockIdx.x, seg = b / bps, blk = b - seg * bps;
    const int tid = threadIdx.x, wave = tid >> 6;
    for (int i = tid; i < (SORT_T / 64) * SORT_BINS; i += SORT_T)
        (&cnt[0][0])[i] = 0u;
    __syncthreads();
    const uint64_t base = (uint64_t)seg * n;
    const uint32_t lo = blk * SORT_TILE, hi = min(lo + (uint32_t)SORT_TILE, n);
    // all of this thread's keys are loaded before the first count
    uint32_t dg[SORT_IPT];
#pragma unroll
    for (int r = 0; r < SORT_IPT; ++r) {
        const uint32_t i = lo + r * SORT_T + tid;
        dg[r] = i < hi ? (keys[base + i] >> shift) & mask : 0xffffffffu;
    }
#pragma unroll
    for (int r = 0; r < SORT_IPT; ++r)
        if (dg[r] != 0xffffffffu)
            atomicAdd(&cnt[wave][dg[r]], 1u);
    __syncthreads();
    uint32_t c = 0;
#pragma unroll
    for (int w = 0; w < SORT_T / 64; ++w)
        c += cnt[w][tid];
    hist[((uint64_t)seg * SORT_BINS + tid) * bps + blk] = c;
}

__device__ __forceinline__ uint32_t lanes_below_mask(uint64_t m)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Exclusive prefix over the block's SORT_T threads of v (one value each).
__device__ __forceinline__ uint32_t block_excl_prefix(uint32_t v, uint32_t *s_w)
{
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    uint32_t inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t u = __shfl_up(inc, o, 64);
        if (lane >= o)
            inc += u;
    }
    if (lane == 63)
        s_w[wave] = inc;
    __syncthreads();
    uint32_t before = 0;
#pragma unroll
    for (int w = 0; w < SORT_T / 64; ++w)
        before += w < wave ? s_w[w] : 0u;
    return before + inc - v;
}

// One pass: entries of kin / vin (vin null: the row index, i.e. the entry's
// position in its segment) to kout / vout in stable order of their digit.
// Wave w of a block owns the block's entries [PER_WAVE w, PER_WAVE (w + 1)) and takes
// them 64 at a time in order, so a digit's rank within the block is (its
// count in earlier waves) + (its count in this wave's earlier rounds) + (the
// lanes below with the same digit).
__global__ void __launch_bounds__(SORT_T) sort_scatter(const uint32_t *kin, const uint32_t *vin,
                                                       uint32_t *kout, uint32_t *vout, uint32_t n,
                                                       uint32_t bps, uint32_t shift,
                                                       uint32_t nbits,
                                                       const unsigned long long *offs)
{
    __shared__ uint32_t s_k[SORT_TILE];
    __shared__ uint32_t s_v[SORT_TILE];
    __shared__ uint32_t s_run[SORT_T / 64][SORT_BINS];
    __shared__ uint32_t s_start[SORT_BINS];
    __shared__ unsigned long long s_off[SORT_BINS];
    __shared__ uint32_t s_w[SORT_T / 64];
    const uint32_t b = blockIdx.x, seg = b / bps, blk = b - seg * bps;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t mask = (1u << nbits) - 1u;
    const uint32_t lo = blk * SORT_TILE;
    const uint32_t cnt = min((uint32_t)SORT_TILE, n - lo);
    const uint64_t base = (uint64_t)seg * n + lo;
    for (int i = tid; i < (SORT_T / 64) * SORT_BINS; i += SORT_T)
        (&s_run[0][0])[i] = 0u;
    __syncthreads();

    constexpr int PER_WAVE = SORT_TILE / (SORT_T / 64);
    uint32_t key[SORT_IPT];
    uint32_t val[SORT_IPT], rank[SORT_IPT];
#pragma unroll
    for (int r = 0; r < SORT_IPT; ++r) {
        const uint32_t li = wave * PER_WAVE + r * 64 + lane;
        const bool valid = li < cnt;
        key[r] = valid ? kin[base + li] : 0u;
        val[r] = valid ? (vin ? vin[base + li] : lo + li) : 0u;
    }
#pragma unroll
    for (int r = 0; r < SORT_IPT; ++r) {
        const uint32_t li = wave * PER_WAVE + r * 64 + lane;
        const bool valid = li < cnt;
        const uint32_t dg = (key[r] >> shift) & mask;
        uint64_t peers = __ballot(valid);
        for (uint32_t bit = 0; bit < nbits; ++bit) {
            const bool set = (dg >> bit) & 1u;
            const uint64_t bal = __ballot(set);
            peers &= set ? bal : ~bal;
        }
        const uint32_t below = lanes_below_mask(peers);
        const uint32_t before = s_run[wave][dg];
        rank[r] = before + below;
        // the group's first lane moves the wave's running count past it
        if (valid && below == 0)
            s_run[wave][dg] = before + (uint32_t)__popcll(peers);
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    }
    __syncthreads();
    // digit `tid`: each wave's base (count in earlier waves), the digit's first
    // local position and its first output position
    {
        uint32_t run = 0;
#pragma unroll
        for (int w = 0; w < SORT_T / 64; ++w) {
            const uint32_t c = s_run[w][tid];
            s_run[w][tid] = run;
            run += c;
        }
        s_start[tid] = block_excl_prefix(run, s_w);
        s_off[tid] = offs[((uint64_t)seg * SORT_BINS + tid) * bps + blk];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < SORT_IPT; ++r) {
        const uint32_t li = wave * PER_WAVE + r * 64 + lane;
        if (li < cnt) {
            const uint32_t dg = (key[r] >> shift) & mask;
            const uint32_t pos = s_start[dg] + s_run[wave][dg] + rank[r];
            if (pos < (uint32_t)SORT_TILE) {   // always: the ranks are a permutation
                s_k[pos] = key[r];
                s_v[pos] = val[r];
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SORT_IPT; ++j) {
        const uint32_t p = j * SORT_T + tid;
        if (p < cnt) {
            const uint32_t k = s_k[p];
            const uint32_t dg = (k >> shift) & mask;
            const unsigned long long at = s_off[dg] + (p - s_start[dg]);
            if (at < (unsigned long long)n * gridDim.x / bps) {   // within L n
                kout[at] = k;
                vout[at] = s_v[p];
            }
        }
    }
}

// A bijection of 64-bit keys (a multiplication by an odd constant, then an
// xor of the high half into the low half, both invertible).
__device__ __forceinline__ uint64_t mix_key(uint64_t k)
{
    k *= 0x9E3779B97F4A7C15ull;
    return k ^ (k >> 32);
}

// The 32-bit sort keys: the key itself (keys of at most 32 bits) or the top
// half of its mix.
__global__ void __launch_bounds__(256) sort_key_kernel(const uint64_t *keys, uint64_t total,
                                                       int wide, uint32_t *sk)
{
    const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < total)
        sk[i] = wide ? (uint32_t)(mix_key(keys[i]) >> 32) : (uint32_t)keys[i];
}

// The sorted outputs through the permutation: the key (or its mix) of the
// row at every sorted position; with wide keys also clears the run marks.
__global__ void __launch_bounds__(256) gather_key_kernel(const uint64_t *keys, uint32_t n,
                                                         uint64_t total, int wide,
                                                         const uint32_t *perm, uint64_t *sorted,
                                                         uint32_t *mark)
{
    const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total)
        return;
    const uint64_t seg = i / n;
    const uint64_t k = keys[seg * n + perm[i]];
    sorted[i] = wide ? mix_key(k) : k;
    if (wide)
        mark[i] = 0;
}

// Wide keys, after the gather: a break is a position whose mixed key differs
// from its predecessor's within a run of equal top halves.  The run's first
// break walks back to the run's first position and marks it.  Only `sk` and
// `sorted` are read, and nothing else writes them here.
__global__ void __launch_bounds__(256) break_kernel(const uint32_t *sk, const uint64_t *sorted,
                                                    uint32_t n, uint64_t total, uint32_t *mark)
{
    const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total)
        return;
    const uint64_t s0 = i / n * n;
    if (i == s0 || sk[i - 1] != sk[i] || sorted[i - 1] == sorted[i])
        return;
    uint64_t a = i - 1;
    while (a > s0 && sk[a - 1] == sk[i]) {
        if (sorted[a - 1] != sorted[a])
            return;   // an earlier break marks the run
        --a;
    }
    mark[a] = 1;
}

// Sorts every marked run by the mixed key, stably (insertion sort).  Two
// distinct keys share a top half with probability 2^-32, so D distinct keys in
// a table give about D^2 / 2^33 marked runs (about 100 at D = 10^6), each
// joining the rows of two buckets; the cost of a run is its number of
// inversions, at most the product of the two buckets' sizes.  Runs are
// disjoint and each has one first position, so no two threads write the same
// entries.
__global__ void __launch_bounds__(256) fixup_kernel(const uint32_t *sk, const uint32_t *mark,
                                                    uint32_t n, uint64_t total, uint64_t *sorted,
                                                    uint32_t *perm)
{
    const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= total || !mark[i])
        return;
    const uint64_t end = (i / n + 1) * n;
    uint64_t e = i + 1;
    while (e < end && sk[e] == sk[i])
        ++e;
    for (uint64_t a = i + 1; a < e; ++a) {
        const uint64_t k = sorted[a];
        const uint32_t v = perm[a];
        uint64_t b = a;
        while (b > i && sorted[b - 1] > k) {
            sorted[b] = sorted[b - 1];
            perm[b] = perm[b - 1];
            --b;
        }
        sorted[b] = k;
        perm[b] = v;
    }
}

// Blocks per segment, and the counts' length (segments x digits x blocks).
static uint32_t blocks_per_segment(uint32_t n) { return (n + SORT_TILE - 1) / SORT_TILE; }

size_t sort_temp_bytes(uint32_t n, uint32_t L)
{
    const uint64_t total = (uint64_t)n * L;
    const uint64_t counts = (uint64_t)L * SORT_BINS * blocks_per_segment(n);
    auto up = [](uint64_t x) { return (x + 255) & ~(uint64_t)255; };
    return 2 * up(total * 4) + up(total * 4) + up(counts * 4) + up(counts * 8) +
           up(sjk::scan_partials_size(counts) * 8) + 256;
}

hipError_t sort_tables(const uint64_t *keys, uint64_t *sorted, uint32_t *perm, uint32_t n,
                       uint32_t L, uint32_t bits, void *temp, hipStream_t s)
{
    if (n == 0 || L == 0)
        return hipSuccess;
    const uint64_t total = (uint64_t)n * L;
    const uint32_t bps = blocks_per_segment(n);
    const uint64_t counts = (uint64_t)L * SORT_BINS * bps;
    auto up = [](uint64_t x) { return (x + 255) & ~(uint64_t)255; };
    uint8_t *t = (uint8_t *)temp;
    uint32_t *ska = (uint32_t *)t;                             // sort keys, two buffers
    uint32_t *skb = (uint32_t *)(t + up(total * 4));
    uint32_t *tv = (uint32_t *)(t + 2 * up(total * 4));        // rows, second buffer
    uint32_t *hist = (uint32_t *)(t + 3 * up(total * 4));
    unsigned long long *offs = (unsigned long long *)((uint8_t *)hist + up(counts * 4));
    unsigned long long *part = (unsigned long long *)((uint8_t *)offs + up(counts * 8));
    unsigned long long *tot =
        (unsigned long long *)((uint8_t *)part + up(sjk::scan_partials_size(counts) * 8));
    const bool wide = bits > 32;
    const uint32_t sbits = wide ? 32u : bits;
    const dim3 g1((uint32_t)((total + 255) / 256));
    hipLaunchKernelGGL(sort_key_kernel, g1, dim3(256), 0, s, keys, total, wide ? 1 : 0, ska);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    // at least one pass (with no key bits it is a stable copy that also
    // writes the rows); the last pass leaves the rows in `perm`
    const uint32_t passes = sbits == 0 ? 1u : (sbits + SORT_BITS - 1) / SORT_BITS;
    const uint32_t grid = L * bps;
    const uint32_t *kin = ska;
    const uint32_t *vin = nullptr;
    for (uint32_t pass = 0; pass < passes; ++pass) {
        const uint32_t shift = pass * SORT_BITS;
        const uint32_t nbits = sbits == 0 ? 0u : min((uint32_t)SORT_BITS, sbits - shift);
        const bool to_out = ((passes - 1 - pass) & 1u) == 0;
        uint32_t *kout = kin == ska ? skb : ska;
        uint32_t *vout = to_out ? perm : tv;
        hipLaunchKernelGGL(sort_hist, dim3(grid), dim3(SORT_T), 0, s, kin, n, bps, shift,
                           (1u << nbits) - 1u, hist);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        if ((e = sjk::launch_scan(hist, counts, offs, part, tot, s)) != hipSuccess)
            return e;
        hipLaunchKernelGGL(sort_scatter, dim3(grid), dim3(SORT_T), 0, s, kin, vin, kout, vout, n,
                           bps, shift, nbits, offs);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        kin = kout;
        vin = vout;
    }
    // the rows' second buffer is free after the last pass: the run marks
    hipLaunchKernelGGL(gather_key_kernel, g1, dim3(256), 0, s, keys, n, total, wide ? 1 : 0, perm,
                       sorted, tv);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    if (wide) {
        hipLaunchKernelGGL(break_kernel, g1, dim3(256), 0, s, kin, sorted, n, total, tv);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        hipLaunchKernelGGL(fixup_kernel, g1, dim3(256), 0, s, kin, tv, n, total, sorted, perm);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace sjl
