// sj_join_kernels.h -- the fused similarity-join kernels for gfx950 (CDNA4).
//
// The join of Ahle & Silvestri, "Similarity Search with Tensor Core Units",
// Section 4 (brute force): all pair scores come from one blocked dense product
// P.Q^T (Theorem 1's blocked multiplication), here on 32x32 MFMA tiles
// (v_mfma_f32_32x32x16_{f16,bf16}, v_mfma_i32_32x32x32_i8).  Each output tile
// lives only in registers: the epilogue applies the threshold test (Section 4's
// D(x, y) <= r, inclusive) and compacts the matching (i, j) pairs with
// wavefront ballots and one atomic (or one precomputed offset) per wavefront.
//
// Data layout: P and Q are row-major, K-contiguous.  Both MFMA operands take,
// per lane, 16 contiguous bytes of one row: lane l supplies row (l % 32) and
// bytes [32*ks + 16*(l / 32), +16) of the row for k-step ks.  A row of d
// elements is therefore processed as ceil(d * esize / 32) k-steps of 32 bytes,
// zero-padded at the end (zero padding leaves inner products and squared
// distances unchanged).  The 32x32 result holds, in lane l and accumulator
// register r, the entry (row 8*(r/4) + 4*(l/32) + r%4, column l%32).
#pragma once

#include "sj_internal.h"

#include <type_traits>

namespace sjk {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

template <int DT>
struct Mma;

template <>
struct Mma<DT_F16> {
    typedef f32x16 acc_t;
    typedef float val_t;
    static __device__ __forceinline__ acc_t mma(i32x4 a, i32x4 b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    }
};

template <>
struct Mma<DT_BF16> {
    typedef f32x16 acc_t;
    typedef float val_t;
    static __device__ __forceinline__ acc_t mma(i32x4 a, i32x4 b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
};

template <>
struct Mma<DT_I8> {
    typedef i32x16 acc_t;
    typedef int val_t;
    static __device__ __forceinline__ acc_t mma(i32x4 a, i32x4 b, acc_t c)
    {
        return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
    }
};

__device__ __forceinline__ float vmax(float a, float b) { return __builtin_fmaxf(a, b); }
__device__ __forceinline__ int vmax(int a, int b) { return a > b ? a : b; }
__device__ __forceinline__ float vmin(float a, float b) { return __builtin_fminf(a, b); }
__device__ __forceinline__ int vmin(int a, int b) { return a < b ? a : b; }

template <typename V>
__device__ __forceinline__ V big_val();
template <>
__device__ __forceinline__ float big_val<float>() { return __builtin_inff(); }
template <>
__device__ __forceinline__ int big_val<int>() { return 0x3fffffff; }

// 16 bytes at byte `off` of row `row`, zero past the row or past n_rows.
// Rows are 16-byte aligned and row_bytes is a multiple of 16 (the host repacks
// inputs that are not), so a chunk is either wholly inside a row or outside.
__device__ __forceinline__ i32x4 load_chunk(const uint8_t *base, uint32_t row, uint32_t n_rows,
                                            uint32_t row_bytes, uint32_t off)
{
    i32x4 v = {0, 0, 0, 0};
    if (row < n_rows && off < row_bytes)
        v = *(const i32x4 *)(base + (size_t)row * row_bytes + off);
    return v;
}

__device__ __forceinline__ uint64_t first_lane_u64(uint64_t v)
{
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// One 16-byte buffer load per lane straight into LDS: lane l's bytes land at
// lds + 16 l (lds is wave-uniform).  The descriptor covers [base, base + n_bytes);
// offsets at or past n_bytes read zeros.
__device__ __forceinline__ void buffer_load_lds16(const uint8_t *base, uint32_t n_bytes,
                                                  uint32_t voff, uint8_t *lds,
                                                  uint32_t soff = 0)
{
#if defined(__HIP_DEVICE_COMPILE__)
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void *)base, 0, n_bytes, 0x00020000);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void *)lds,
                                             16, voff, soff, 0, 0);
#endif
}

// Explicit address spaces for the pair stores: through a generic pointer the
// compiler may emit flat stores, which count on the LDS counter out of order
// and so force full waits on every LDS read in the loop that follows.
// A pair travels as one 64-bit word: i in the low half, j in the high half
// (the (i, j) uint32 layout of the output buffer).
typedef __attribute__((address_space(1))) uint64_t global_pair;
typedef __attribute__((address_space(3))) uint64_t lds_pair;

__device__ __forceinline__ global_pair *pair_slot(const JoinArgs &g, uint64_t k)
{
    return (global_pair *)g.pairs + k;
}

__device__ __forceinline__ uint64_t pack_pair(uint32_t i, uint32_t j)
{
    return (uint64_t)i | ((uint64_t)j << 32);
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// LDS tile layout: a row of CPR 16-byte chunks is stored with a stride of
// CPR + 1 chunks.  The LDS has 64 banks of 4 bytes, so a 128-bit access serves
// 16 lanes per cycle; a B-fragment read has 16 consecutive rows fetch the same
// chunk c, and their bank groups ((CPR + 1) r + c) mod 16 are all distinct for
// every CPR used here (2, 4, 8, 16, 32 and the streamed kernel's 8).

// Exact test of one pair.  IP: acc >= thr.  L2: 2 acc >= (N_x + N_y) - r2,
// i.e. N_x + N_y - 2 <x,y> <= r2 with the fp32 additions rounded in this order
// (monotone in N_x, which the per-lane bound below relies on).
template <int DT, int MET>
__device__ __forceinline__ bool pair_matches(typename Mma<DT>::val_t acc,
                                             typename Mma<DT>::val_t nx,
                                             typename Mma<DT>::val_t ny, const JoinArgs &g)
{
    if constexpr (MET == MET_IP) {
        if constexpr (DT == DT_I8)
            return acc >= g.thr_i;
        else
            return acc >= g.thr_f;
    } else {
        if constexpr (DT == DT_I8)
            return 2 * acc >= nx + ny - g.thr_i;
        else
            return 2.0f * acc >= (nx + ny) - g.thr_f;
    }
}

// Epilogue of one wave over a (32*WMB) x 32 block of results, in two parts.
// Accumulator acc[a] register r of lane l holds the pair
//   (i, j) = (ibase + 32 a + 8 (r / 4) + r % 4,  j)  with ibase = prow0 + 4 (l / 32).
//
// lane_may_match: a necessary condition per lane, from one max over the lane's
// 16 * WMB results.  IP: max acc >= thr.  L2: 2 max acc >= (nmin + N_y) - r2,
// where nmin is the smallest squared norm among the lane's rows; `nb` carries
// nmin - r2 for int8 (exact integers) and nmin itself for fp32, whose bound
// keeps the rounding order of the exact test: since fl(fl(N_x + N_y) - r2) is
// monotone in N_x, a lane whose bound fails holds no match.  Columns past n_q
// are not excluded here (the exact test does that).
template <int DT, int MET>
__device__ __forceinline__ bool lane_bound(typename Mma<DT>::val_t m, typename Mma<DT>::val_t nb,
                                           typename Mma<DT>::val_t ny, const JoinArgs &g)
{
    typedef typename Mma<DT>::val_t V;
    if constexpr (MET == MET_IP)
        return pair_matches<DT, MET>(m, V(0), V(0), g);
    else if constexpr (DT == DT_I8)
        return 2 * m >= nb + ny;
    else
        return 2.0f * m >= (nb + ny) - g.thr_f;
}

// Running max over the flattened results v = 16 a + r, v in [LO, HI), of
// acc[WMB]; LO == 0 starts the chain.
template <int LO, int HI, int WMB, typename ACC, typename V>
__device__ __forceinline__ void fold_max(const ACC (&acc)[WMB], V &m)
{
    if constexpr (LO < HI) {
        if constexpr (LO == 0)
            m = acc[0][0];
        else
            m = vmax(m, acc[LO / 16][LO % 16]);
        fold_max<LO + 1, HI, WMB>(acc, m);
    }
}

// Running maxima over the results v = 16 a + r, v in [LO, HI), of acc[WMB].
// With at most two blocks one chain per block (mb[a], so the exact path can
// skip a block whose own bound fails); with more, one chain in mb[0] (fewer
// VALU instructions; the exact path then re-derives the block bounds).
template <int WMB>
constexpr bool per_block_max()
{
    return WMB <= 2;
}

template <int LO, int HI, int WMB, typename ACC, typename V>
__device__ __forceinline__ void fold_max_blk(const ACC (&acc)[WMB], V (&mb)[WMB])
{
    if constexpr (LO < HI) {
        constexpr int c = per_block_max<WMB>() ? LO / 16 : 0;
        constexpr bool first = per_block_max<WMB>() ? LO % 16 == 0 : LO == 0;
        if constexpr (first)
            mb[c] = acc[LO / 16][LO % 16];
        else
            mb[c] = vmax(mb[c], acc[LO / 16][LO % 16]);
        fold_max_blk<LO + 1, HI, WMB>(acc, mb);
    }
}

template <int WMB, typename V>
__device__ __forceinline__ V max_of(const V (&mb)[WMB])
{
    V m = mb[0];
    if constexpr (per_block_max<WMB>()) {
#pragma unroll
        for (int a = 1; a < WMB; ++a)
            m = vmax(m, mb[a]);
    }
    return m;
}

template <int DT, int MET, int WMB>
__device__ __forceinline__ bool lane_may_match(const typename Mma<DT>::acc_t (&acc)[WMB],
                                               typename Mma<DT>::val_t nb,
                                               typename Mma<DT>::val_t ny, const JoinArgs &g)
{
    typename Mma<DT>::val_t m;
    fold_max<0, 16 * WMB, WMB>(acc, m);
    return lane_bound<DT, MET>(m, nb, ny, g);
}

// The per-lane constant of the L2 bound (see lane_may_match).
template <int DT, int MET>
__device__ __forceinline__ typename Mma<DT>::val_t bound_base(typename Mma<DT>::val_t nmin,
                                                              const JoinArgs &g)
{
    if constexpr (MET == MET_L2 && DT == DT_I8)
        return nmin - g.thr_i;
    else
        return nmin;
}

// Per-wave output staging: a wave appends its matches to its own LDS buffer
// and moves them to the global pair buffer in bulk, with coalesced stores.
// Single-pass mode reserves the global slots with one atomicAdd per flush;
// the emit pass (when a kernel stages there) writes them in order from the
// output block's offset (`dst`).
struct WaveOut {
    lds_pair *buf;   // this wave's LDS buffer of `cap` pairs
    uint32_t cap;
    uint32_t fill;   // wave-uniform
    uint64_t dst;    // emit pass: next global slot of this wave's block
    uint64_t blk;    // MODE_RECORD: output block of the blocks being tested
    __attribute__((address_space(3))) uint32_t *nrec;   // MODE_RECORD: workgroup's record count
};

// Modes whose first pass only counts (no pairs written).
template <int MODE>
constexpr bool counting_mode()
{
    return MODE == MODE_COUNT || MODE == MODE_RECORD;
}

// Single-pass modes: pairs staged per wave, slots reserved by atomics.
template <int MODE>
constexpr bool single_mode()
{
    return MODE == MODE_SINGLE || MODE == MODE_TRI;
}

// MODE_RECORD: append the block's MatchRecord to the workgroup's list (an LDS
// counter, so no global atomics in the product loop; records past rec_cap are
// counted, not written, and the host then recomputes instead of reading them).
__device__ __forceinline__ void append_record(uint32_t m, uint32_t ib, uint32_t j, int lane,
                                              uint64_t pos, const JoinArgs &g, const WaveOut &wo)
{
    typedef __attribute__((address_space(1))) uint16_t global_u16;
    typedef __attribute__((address_space(1))) MatchRecord global_rec;
    uint32_t k = 0;
    if (lane == 0)
        k = __hip_atomic_fetch_add(wo.nrec, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    k = __builtin_amdgcn_readfirstlane(k);
    if (k >= g.rec_cap)
        return;
    global_rec *rec = (global_rec *)g.records + ((uint64_t)blockIdx.x * g.rec_cap + k);
    ((global_u16 *)rec->mask)[lane] = (uint16_t)m;
    const uint32_t i0 = __builtin_amdgcn_readfirstlane(ib);
    const uint32_t j0 = __builtin_amdgcn_readfirstlane(j);
    if (lane == 0) {
        rec->blk = wo.blk;
        rec->pos = (uint32_t)pos;
        rec->i0 = i0;
        rec->j0 = j0;
    }
}

template <int MODE>
__device__ __forceinline__ void flush_wave_out(WaveOut &wo, int lane, const JoinArgs &g)
{
    if (wo.fill == 0)
        return;
    uint64_t base;
    if constexpr (MODE == MODE_EMIT) {
        base = wo.dst;
        wo.dst += wo.fill;
    } else {
        unsigned long long b = 0;
        if (lane == 0)
            b = atomicAdd(g.counter, (unsigned long long)wo.fill);
        base = first_lane_u64(b);
    }
    for (uint32_t k = lane; k < wo.fill; k += 64)
        if (base + k < g.cap)
            *pair_slot(g, base + k) = wo.buf[k];
    wo.fill = 0;
}

// Final flush of every wave's staging buffer with one atomicAdd per workgroup
// (all waves must call it; it contains barriers).
template <int NW>
__device__ __forceinline__ void flush_workgroup_out(WaveOut &wo, int wave, int lane,
                                                    const JoinArgs &g)
{
    __shared__ uint32_t s_fill[NW];
    __shared__ unsigned long long s_base;
    if (lane == 0)
        s_fill[wave] = wo.fill;
    __syncthreads();
    if (wave == 0) {
        uint32_t tot = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w)
            tot += s_fill[w];
        if (lane == 0)
            s_base = tot ? atomicAdd(g.counter, (unsigned long long)tot) : 0ull;
    }
    __syncthreads();
    uint64_t base = s_base;
    for (int w = 0; w < wave; ++w)
        base += s_fill[w];
    for (uint32_t k = lane; k < wo.fill; k += 64)
        if (base + k < g.cap)
            *pair_slot(g, base + k) = wo.buf[k];
    wo.fill = 0;
}

// Exact test of every result of one 32x32 block (accumulator `acc`, rows
// ib + 8 (r / 4) + r % 4 of this lane, column j): bit r of the returned mask is
// set iff that result is a match and its row and column exist.  L2 row norms
// come from `nrow` (LDS: this lane's rows of the block).
template <int DT, int MET, bool TRI = false>
__device__ __forceinline__ uint32_t block_mask(const typename Mma<DT>::acc_t &acc, uint32_t ib,
                                               uint32_t j, typename Mma<DT>::val_t ny,
                                               const typename Mma<DT>::val_t *nrow,
                                               const JoinArgs &g)
{
    typedef typename Mma<DT>::val_t V;
    uint32_t m = 0;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        bool ok;
        if constexpr (MET == MET_L2)
            ok = pair_matches<DT, MET>(acc[r], nrow[8 * (r >> 2) + (r & 3)], ny, g);
        else
            ok = pair_matches<DT, MET>(acc[r], V(0), V(0), g);
        m |= ok ? (1u << r) : 0u;
    }
    // rows past n_p and columns past n_q (lane 0 holds the block's first row
    // and column; the test is uniform)
    const uint32_t ib0 = __builtin_amdgcn_readfirstlane(ib);
    const uint32_t j0 = __builtin_amdgcn_readfirstlane(j);
    if ((uint64_t)ib0 + 32 > g.n_p || (uint64_t)j0 + 32 > g.n_q) {
        uint32_t valid = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r)
            valid |= ib + 8 * (r >> 2) + (r & 3) < g.n_p ? (1u << r) : 0u;
        m &= j < g.n_q ? valid : 0u;
    }
    if constexpr (TRI) {
        // self-join, upper triangle: only rows i <= j (a block whose last row
        // is at most its first column needs no test)
        if (ib0 + 31 > j0) {
            uint32_t up = 0;
#pragma unroll
            for (int r = 0; r < 16; ++r)
                up |= ib + 8 * (r >> 2) + (r & 3) <= j ? (1u << r) : 0u;
            m &= up;
        }
    }
    return m;
}

// Single-pass staging of the pairs selected by per-lane masks m (bit r:
// accumulator register r): the wave's total and each lane's prefix come from
// five ballots over the lanes' counts, and every lane writes pair(r) for its
// set bits in register order at its prefix in the wave's LDS buffer (flushed
// first when the block would not fit).
template <int MODE, typename F>
__device__ __forceinline__ void stage_pairs(uint32_t m, int lane, const JoinArgs &g, WaveOut &wo,
                                            F &&pair)
{
    const uint32_t cnt = (uint32_t)__builtin_popcount(m);
    uint32_t tot = 0, pre = 0;
#pragma unroll
    for (int b = 0; b < 5; ++b) {
        const uint64_t bits = __ballot((cnt >> b) & 1);
        tot += (uint32_t)__popcll(bits) << b;
        pre += lanes_below(bits) << b;
    }
    if (tot == 0)
        return;
    if (wo.fill + tot > wo.cap)
        flush_wave_out<MODE>(wo, lane, g);
    uint32_t pos = wo.fill + pre;
    wo.fill += tot;
    while (m != 0) {
        const int r = __builtin_ctz(m);
        m &= m - 1;
        wo.buf[pos++] = pair(r);
    }
}

// exact_block: the block's match mask (block_mask); per-lane counts give the
// wave's total and each lane's exclusive prefix (five ballots over the
// count's bits), and every lane writes its own matches at its prefix, in
// register order.  MODE_SINGLE appends to the wave's LDS staging buffer (which
// holds a whole block), MODE_EMIT writes at the output block's running offset
// (or stages, when the kernel provides a staging buffer), MODE_COUNT only
// counts.  The code is kept short on purpose: it is inlined at every sub-tile
// and runs rarely, and a long exact path costs instruction-cache misses when
// it does run.
template <int DT, int MET, int MODE>
__device__ __forceinline__ void exact_block(const typename Mma<DT>::acc_t &acc, uint32_t ib,
                                            uint32_t j, int lane, typename Mma<DT>::val_t ny,
                                            const typename Mma<DT>::val_t *nrow,
                                            const JoinArgs &g, uint64_t &blk_run, WaveOut &wo)
{
    // Opaque to the optimiser: keeps the per-result row indices from being
    // hoisted into (and occupying registers of) the caller's main loop.
    asm volatile("" : "+v"(ib));
    uint32_t m = block_mask<DT, MET, MODE == MODE_TRI>(acc, ib, j, ny, nrow, g);
    if constexpr (MODE == MODE_TRI) {
        // the mirror images (j, i) of the matches off the diagonal, staged
        // like the block's own pairs
        uint32_t off = m;
        const uint32_t ib0 = __builtin_amdgcn_readfirstlane(ib);
        const uint32_t j0 = __builtin_amdgcn_readfirstlane(j);
        if (ib0 + 31 > j0) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                off &= ib + 8 * (r >> 2) + (r & 3) == j ? ~(1u << r) : ~0u;
        }
        stage_pairs<MODE>(off, lane, g, wo, [&](int r) {
            return pack_pair(j, ib + 8 * (r >> 2) + (r & 3));
        });
    }
    const uint32_t cnt = (uint32_t)__builtin_popcount(m);
    uint32_t tot = 0, pre = 0;
#pragma unroll
    for (int b = 0; b < 5; ++b) {
        const uint64_t bits = __ballot((cnt >> b) & 1);
        tot += (uint32_t)__popcll(bits) << b;
        pre += lanes_below(bits) << b;
    }
    if constexpr (counting_mode<MODE>()) {
        if constexpr (MODE == MODE_RECORD) {
            if (tot != 0)
                append_record(m, ib, j, lane, blk_run, g, wo);
        }
        blk_run += tot;
        return;
    }
    if (tot == 0)
        return;
    auto write_all = [&](auto &&dst, uint64_t base) {
        uint64_t pos = base + pre;
        while (m != 0) {
            const int r = __builtin_ctz(m);
            m &= m - 1;
            dst(pos++, pack_pair(ib + 8 * (r >> 2) + (r & 3), j));
        }
    };
    if (single_mode<MODE>() || wo.cap > 1) {
        // staged: the buffer holds at least one whole block
        if (wo.fill + tot > wo.cap)
            flush_wave_out<MODE>(wo, lane, g);
        const uint32_t base = wo.fill;
        wo.fill += tot;
        write_all([&](uint64_t k, uint64_t v) { wo.buf[k] = v; }, base);
    } else {
        const uint64_t base = blk_run;
        blk_run += tot;
        write_all(
            [&](uint64_t slot, uint64_t v) {
                if (slot < g.cap)
                    *pair_slot(g, slot) = v;
            },
            base);
    }
}

// All WMB blocks of a wave's sub-tile whose own bound holds for some lane.
template <int DT, int MET, int MODE, int WMB>
__device__ __forceinline__ void exact_blocks(const typename Mma<DT>::acc_t (&acc)[WMB],
                                             const typename Mma<DT>::val_t (&mb)[WMB],
                                             uint32_t ibase, uint32_t j, int lane,
                                             typename Mma<DT>::val_t nb,
                                             typename Mma<DT>::val_t ny,
                                             const typename Mma<DT>::val_t *nrows,
                                             const JoinArgs &g, uint64_t &blk_run, WaveOut &wo)
{
#pragma unroll
    for (int a = 0; a < WMB; ++a) {
        bool may;
        if constexpr (per_block_max<WMB>()) {
            may = lane_bound<DT, MET>(mb[a], nb, ny, g);
        } else {
            typename Mma<DT>::acc_t one[1] = {acc[a]};
            may = lane_may_match<DT, MET, 1>(one, nb, ny, g);
        }
        if (__ballot(may) != 0)
            exact_block<DT, MET, MODE>(acc[a], ibase + 32 * a, j, lane, ny, nrows + 32 * a, g,
                                       blk_run, wo);
    }
}

// Squared norms of a wave's 32 * WMB rows into LDS (rows past n_p get a large
// placeholder and are excluded by the exact test); returns the smallest norm
// among this lane's rows.
template <int DT, int WMB>
__device__ __forceinline__ typename Mma<DT>::val_t stage_row_norms(uint32_t prow0, int lane,
                                                                   typename Mma<DT>::val_t *s_n,
                                                                   const JoinArgs &g)
{
    typedef typename Mma<DT>::val_t V;
    const V *np = (const V *)g.norm_p;
#pragma unroll
    for (int k = 0; k < WMB / 2; ++k) {
        const uint32_t i = prow0 + 64 * k + lane;
        s_n[64 * k + lane] = i < g.n_p ? np[i] : big_val<V>();
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int half = lane >> 5;
    V nmin = big_val<V>();
#pragma unroll
    for (int a = 0; a < WMB; ++a)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            nmin = vmin(nmin, s_n[32 * a + 4 * half + 8 * (r >> 2) + (r & 3)]);
    return nmin;
}

// Compile-time loop: f(std::integral_constant<int, I>) for I = B .. E-1 (a
// guaranteed full unroll, unlike #pragma unroll on a large body).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f)
{
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// ---------------------------------------------------------------------------
// Family 1: P rows resident in registers.
//
// A workgroup of NW waves owns BM = NW * 32 * WMB consecutive rows of P; each
// wave keeps its 32*WMB rows, all KS k-steps, as MFMA A-fragments in VGPRs for
// the whole kernel.  The workgroup sweeps its range of Q in tiles of BN rows,
// double-buffered in LDS (rows padded by one chunk); the next tile's direct
// global-to-LDS loads are issued before the current tile's MFMAs.  A tile is
// one stream of k-steps over its 32-row sub-tiles (see the tile loop): the
// B-fragment reads run a few steps ahead of the MFMAs, and with two
// accumulator sets the epilogue bound of sub-tile s - 1 is folded in while
// the MFMAs of sub-tile s run.  Output block (count/emit passes) = one wave's
// rows x one Q tile; block index = (global wave row-block) * n_qtiles + tile.
template <int DT, int MET, int MODE, int KS, int WMB, int NW, int BN>
__global__ void __launch_bounds__(NW * 64) join_resident(JoinArgs g)
{
    typedef Mma<DT> M;
    typedef typename M::acc_t acc_t;
    typedef typename M::val_t V;
    constexpr int CPR = KS * 2;             // 16-byte chunks per row
    constexpr int LS = (CPR + 1) * 16;      // padded LDS row stride in bytes
    constexpr int TCH = BN * (CPR + 1);     // LDS positions per Q tile
    constexpr int SUBS = BN / 32;
    constexpr int BM = NW * 32 * WMB;
    constexpr bool NEED_NORMS = (MET == MET_L2);
    // Sub-tile pipeline (two accumulator sets); at 16 k-steps only the inner
    // product fits a second set in 256 VGPRs (the L2 epilogue needs more).
    constexpr bool PIPE = KS <= 8 || MET == MET_IP;

    // Two distinct LDS buffers (not one array indexed at run time): the tile
    // loop is unrolled by two so every access names its buffer statically, which
    // lets the compiler see that the direct loads into one buffer never alias
    // the reads of the other (and not wait for them).
    __shared__ __attribute__((aligned(16))) uint8_t s_q0[BN * LS];
    __shared__ __attribute__((aligned(16))) uint8_t s_q1[BN * LS];
    __shared__ V s_nq0[NEED_NORMS ? BN : 1];
    __shared__ V s_nq1[NEED_NORMS ? BN : 1];
    __shared__ V s_np[NEED_NORMS ? NW : 1][NEED_NORMS ? 32 * WMB : 1];
    constexpr int OUT_CAP = single_mode<MODE>() ? 1024 : 1;   // a whole 32x32 block
    __shared__ uint64_t s_out[NW][OUT_CAP];
    __shared__ uint32_t s_nrec;   // MODE_RECORD: records of this workgroup

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, c32 = lane & 31;
    const uint32_t qsplit = g.qsplit;
    const uint32_t n_qt = (g.n_q + BN - 1) / BN;
    WaveOut wo{(lds_pair *)s_out[wave], (uint32_t)OUT_CAP, 0u, 0ull, 0ull,
               (__attribute__((address_space(3))) uint32_t *)&s_nrec};
    // A workgroup sweeps a range of Q tiles for one block of P rows.  In the
    // self-join triangle (tiles whose columns all lie below a block's first
    // row hold no pair (i, j) with i <= j) blocks pb and n_pb - 1 - pb are
    // paired and the workgroup takes its share of the two blocks' tiles, one
    // block after the other (a segment each), so every workgroup sweeps
    // about as many tiles.
    auto segment = [&](int seg) __attribute__((always_inline)) {
        uint32_t pb, t0, t1;
        if constexpr (MODE == MODE_TRI) {
            // Workgroups are dealt to the 8 XCDs in turn; numbered XCD-major,
            // the ones on one XCD take neighbouring block pairs, whose sweeps
            // meet the same Q tiles within a few dozen tiles of each other
            // and so share that XCD's L2.
            const uint32_t G = gridDim.x;
            const uint32_t bid = G % 8 == 0 ? (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8
                                            : blockIdx.x;
            const uint32_t n_pb = (g.n_p + BM - 1) / BM;
            const uint32_t pp = bid / qsplit, qs = bid - pp * qsplit;
            const uint32_t pa = pp, pz = n_pb - 1 - pp;
            const uint32_t la = n_qt - min(pa * BM / BN, n_qt);
            const uint32_t lz = pz != pa ? n_qt - min(pz * BM / BN, n_qt) : 0u;
            const uint64_t tot = (uint64_t)la + lz;
            const uint32_t s0 = (uint32_t)((uint64_t)qs * tot / qsplit);
            const uint32_t s1 = (uint32_t)((uint64_t)(qs + 1) * tot / qsplit);
            if (seg == 0) {
                pb = pa;
                t0 = min(s0, la);
                t1 = min(s1, la);
            } else {
                pb = pz;
                t0 = max(s0, la) - la;
                t1 = max(s1, la) - la;
            }
            const uint32_t t_lo = min(pb * BM / BN, n_qt);
            t0 += t_lo;
            t1 += t_lo;
            if (t0 >= t1)
                return;   // uniform: the workgroup's share holds no tile of this block
        } else {
            (void)seg;
            pb = blockIdx.x / qsplit;
            const uint32_t qs = blockIdx.x - pb * qsplit;
            t0 = (uint32_t)((uint64_t)qs * n_qt / qsplit);
            t1 = (uint32_t)((uint64_t)(qs + 1) * n_qt / qsplit);
        }
        const uint32_t prow0 = pb * BM + wave * 32 * WMB;
        const uint32_t ibase = prow0 + 4 * half;

        i32x4 A[WMB][KS];
    #pragma unroll
        for (int a = 0; a < WMB; ++a)
    #pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                A[a][ks] = load_chunk(g.P, prow0 + 32 * a + c32, g.n_p, g.row_bytes,
                                      32 * ks + 16 * half);

        V nmin = big_val<V>();
        const V *nrows = nullptr;
        if constexpr (NEED_NORMS) {
            nmin = stage_row_norms<DT, WMB>(prow0, lane, s_np[wave], g);
            nrows = &s_np[wave][4 * half];
        }
        const V nb = bound_base<DT, MET>(nmin, g);
        // Drain the resident-row loads here: otherwise the wait inserted for their
        // first use inside the tile loop also waits for the next tile's prefetch.
        __builtin_amdgcn_s_waitcnt(0);

        // Q tiles go straight from global memory into LDS (no staging registers)
        // with buffer loads: each wave instruction fills 64 consecutive 16-byte
        // LDS positions; the lane at position p loads chunk p % (CPR + 1) of tile
        // row p / (CPR + 1) (the pad position reloads chunk 0).  The tile's buffer
        // descriptor ends at row n_q, so rows past it read zeros (their columns
        // are never reported); chunks past row_bytes read the row's last chunk
        // (they meet the zero padding of the resident rows).  (A global_load_lds
        // would do the same, but the compiler then treats every LDS read of the
        // loop as unordered and drains them all at each use.)
        constexpr int NCALL = (TCH + 64 * NW - 1) / (64 * NW);   // direct loads per wave
        const int wv = __builtin_amdgcn_readfirstlane(wave);
        uint32_t loff[NCALL];   // this lane's byte offset in the tile, per load
    #pragma unroll
        for (int kk = 0; kk < NCALL; ++kk) {
            const int pos = 64 * (kk * NW + wv) + lane;
            const int cp = pos % (CPR + 1);
            const uint32_t row = min(pos / (CPR + 1), BN - 1);
            loff[kk] = row * g.row_bytes + min((uint32_t)(16 * (cp == CPR ? 0 : cp)), g.row_bytes - 16);
        }
        // waves whose last load would start past the tile skip it (uniform)
        const bool last_call = TCH % (64 * NW) == 0 || 64 * ((NCALL - 1) * NW + wv) < TCH;
        auto stage_issue = [&](uint32_t t, uint8_t *dst) {
            const uint32_t rows = min(g.n_q - t * BN, (uint32_t)BN);
            const uint8_t *base = g.Q + (size_t)t * BN * g.row_bytes;
    #pragma unroll
            for (int kk = 0; kk < NCALL; ++kk) {
                if (kk == NCALL - 1 && !last_call)
                    break;
                buffer_load_lds16(base, rows * g.row_bytes, loff[kk], dst + 1024 * (kk * NW + wv));
            }
        };
        auto norm_load = [&](uint32_t t, V &stn) {
            if constexpr (NEED_NORMS) {
                if (tid < BN) {
                    const uint32_t jq = t * BN + tid;
                    stn = jq < g.n_q ? ((const V *)g.norm_q)[jq] : big_val<V>();
                }
            }
        };
        auto norm_store = [&](V *dst, V stn) {
            if constexpr (NEED_NORMS) {
                if (tid < BN)
                    dst[tid] = stn;
            }
        };
        if (t0 < t1) {
            V stn = V(0);
            stage_issue(t0, s_q0);
            norm_load(t0, stn);
            norm_store(s_nq0, stn);
        }
        if constexpr (MODE == MODE_RECORD) {
            if (tid == 0)
                s_nrec = 0;
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();

        const uint64_t wave_row_block = (uint64_t)pb * NW + wave;
        // Bound of one wave sub-tile from its running max, then the exact path if
        // any lane may match.
        auto check = [&](const acc_t(&a)[WMB], const V(&mb)[WMB], uint32_t jp, V nyp,
                         uint64_t &run) __attribute__((always_inline)) {
            const bool may = lane_bound<DT, MET>(max_of<WMB>(mb), nb, nyp, g);
            if (__builtin_expect(__ballot(may) != 0, 0))
                exact_blocks<DT, MET, MODE, WMB>(a, mb, ibase, jp, lane, nb, nyp, nrows, g, run, wo);
        };

        // A tile is a stream of SUBS * KS k-steps (sub-tile s = step / KS).  Each
        // step issues the LDS read of the B-fragment LOOK steps ahead (a ring of
        // LOOK + 1 fragments, continued across sub-tiles) and the WMB MFMAs of its
        // own fragment; with two accumulator sets it also folds 16 WMB / KS results
        // of the previous sub-tile into that sub-tile's running max, so the
        // epilogue's VALU work runs beside the matrix cores.  Scheduling barriers
        // between steps keep this order (left alone, the compiler drains every
        // read right before its MFMAs).
        constexpr int NSTEP = SUBS * KS;
        constexpr int LOOK = KS >= 16 ? 2 : 3;
        constexpr int RING = LOOK + 1;
        constexpr int NVAL = 16 * WMB;
        constexpr int NACC = PIPE ? 2 : 1;
        acc_t acc[NACC][WMB];
    #pragma unroll
        for (int c = 0; c < NACC; ++c)
    #pragma unroll
            for (int a = 0; a < WMB; ++a)
                acc[c][a] = acc_t{};
        // Previous sub-tile of the pipeline when it belongs to the previous tile.
        bool have_prev = false;
        uint32_t j_prev = 0;
        V ny_prev = V(0);
        uint64_t blk_prev = 0, run_prev = 0;

        auto tile = [&](uint32_t t, const uint8_t *cur, uint8_t *nxt, const V *ncur, V *nnxt)
                        __attribute__((always_inline)) {
            const bool more = t + 1 < t1;
            V stn = V(0);
            if (more) {
                stage_issue(t + 1, nxt);
                norm_load(t + 1, stn);
            }
            const uint64_t blk = wave_row_block * n_qt + t;
            uint64_t blk_run = 0;
            if constexpr (MODE == MODE_EMIT)
                blk_run = g.block_offsets[blk];

            // this lane's B-fragment of step q: row 32 (q / KS) + c32, chunk
            // 2 (q % KS) + half
            const uint8_t *bq = cur + c32 * LS + 16 * half;
            i32x4 ring[RING];
            static_for<0, (LOOK < NSTEP ? LOOK : NSTEP)>([&](auto Q) __attribute__((always_inline)) {
                constexpr int q = decltype(Q)::value;
                ring[q] = *(const i32x4 *)(bq + (q / KS) * 32 * LS + (q % KS) * 32);
            });
            V ny_sub[SUBS];
            static_for<0, SUBS>([&](auto S) __attribute__((always_inline)) {
                constexpr int s = decltype(S)::value;
                constexpr int ci = PIPE ? (s & 1) : 0, pi = PIPE ? (ci ^ 1) : 0;
                ny_sub[s] = V(0);
                if constexpr (NEED_NORMS)
                    ny_sub[s] = ncur[32 * s + c32];
                V mb[WMB];
    #pragma unroll
                for (int a = 0; a < WMB; ++a)
                    mb[a] = V(0);
                static_for<0, KS>([&](auto K) __attribute__((always_inline)) {
                    constexpr int ks = decltype(K)::value, q = s * KS + ks;
                    if constexpr (q + LOOK < NSTEP) {
                        constexpr int qn = q + LOOK;
                        ring[qn % RING] =
                            *(const i32x4 *)(bq + (qn / KS) * 32 * LS + (qn % KS) * 32);
                    }
    #pragma unroll
                    for (int a = 0; a < WMB; ++a)
                        acc[ci][a] = M::mma(A[a][ks], ring[q % RING], ks == 0 ? acc_t{} : acc[ci][a]);
                    if constexpr (PIPE)
                        fold_max_blk<ks * NVAL / KS, (ks + 1) * NVAL / KS, WMB>(acc[pi], mb);
                    __builtin_amdgcn_sched_barrier(0);
                });
                if constexpr (PIPE) {
                    if constexpr (s == 0) {
                        if (have_prev) {
                            wo.blk = blk_prev;
                            check(acc[pi], mb, j_prev, ny_prev, run_prev);
                            if constexpr (counting_mode<MODE>()) {
                                if (lane == 0)
                                    g.block_counts[blk_prev] = (uint32_t)run_prev;
                            }
                        }
                    } else {
                        wo.blk = blk;
                        check(acc[pi], mb, t * BN + 32 * (s - 1) + c32, ny_sub[s - 1], blk_run);
                    }
                } else {
                    fold_max_blk<0, NVAL, WMB>(acc[0], mb);
                    wo.blk = blk;
                    check(acc[0], mb, t * BN + 32 * s + c32, ny_sub[s], blk_run);
                }
            });
            if constexpr (PIPE) {
                j_prev = t * BN + 32 * (SUBS - 1) + c32;
                ny_prev = ny_sub[SUBS - 1];
                blk_prev = blk;
                run_prev = blk_run;
                have_prev = true;
            } else if constexpr (counting_mode<MODE>()) {
                if (lane == 0)
                    g.block_counts[blk] = (uint32_t)blk_run;
            }
            if (more)
                norm_store(nnxt, stn);
            __builtin_amdgcn_s_waitcnt(0);   // this wave's direct loads of tile t+1 landed
            __syncthreads();
        };
        for (uint32_t t = t0; t < t1; t += 2) {
            tile(t, s_q0, s_q1, s_nq0, s_nq1);
            if (t + 1 < t1)
                tile(t + 1, s_q1, s_q0, s_nq1, s_nq0);
        }
        if constexpr (PIPE) {
            if (have_prev) {
                V mb[WMB];
                fold_max_blk<0, NVAL, WMB>(acc[NACC - 1], mb);
                wo.blk = blk_prev;
                check(acc[NACC - 1], mb, j_prev, ny_prev, run_prev);
                if constexpr (counting_mode<MODE>()) {
                    if (lane == 0)
                        g.block_counts[blk_prev] = (uint32_t)run_prev;
                }
            }
        }
    };
    if constexpr (MODE == MODE_TRI) {
#pragma nounroll
        for (int seg = 0; seg < 2; ++seg)
            segment(seg);
    } else {
        segment(0);
    }
    if constexpr (single_mode<MODE>())
        flush_workgroup_out<NW>(wo, wave, lane, g);
    if constexpr (MODE == MODE_RECORD) {
        __syncthreads();
        if (tid == 0) {
            const uint32_t n = s_nrec;
            g.rec_counts[blockIdx.x] = n;
            atomicMax(g.rec_max, (unsigned long long)n);
        }
    }
}

// ---------------------------------------------------------------------------
// Family 2: both operands streamed through LDS in chunks of KC bytes of d
// (for rows too long to keep in registers).
//
// A workgroup of 8 waves (two per SIMD) computes a 256 x 256 output tile; wave
// (wr, wc), wr < 4, wc < 2, owns rows [64 wr, +64) (two A-blocks) and columns
// [128 wc, +128) (four B-blocks), so a k-step reads 2 A- and 4 B-fragments
// from LDS for 8 MFMAs.  P and Q chunks are double-buffered in LDS (one
// workgroup per CU).  Tiles are visited in groups of 8 P tiles x 8 Q tiles so
// that concurrently running workgroups share their operand rows in L2.
// Output block = one wave's 64 x 128 region; index = tile * 8 + wave.
constexpr int ST_KC = 128;   // K chunk bytes (tile geometry in sj_internal.h)

template <int DT, int MET, int MODE>
__global__ void __launch_bounds__(ST_NW * 64) join_streamed(JoinArgs g)
{
    typedef Mma<DT> M;
    typedef typename M::acc_t acc_t;
    typedef typename M::val_t V;
    constexpr int CPR = ST_KC / 16;                   // 8 chunks per row per K chunk
    constexpr int LS = (CPR + 1) * 16;                // padded row stride
    constexpr int ROWS = ST_BM + ST_BN;               // P rows, then Q rows
    constexpr int NPOS = ROWS * (CPR + 1);            // LDS positions per stage
    constexpr int NT = ST_NW * 64;                    // threads
    constexpr int NLD = NPOS / NT;                    // direct loads per thread
    constexpr int P_LOADS = ST_BM * (CPR + 1) / 64;   // wave loads below this fill P rows
    constexpr int KSC = ST_KC / 32;                   // k-steps per chunk
    constexpr int SA = ST_SA, SB = ST_SB;             // A- and B-blocks per wave
    constexpr bool NEED_NORMS = (MET == MET_L2);
    static_assert(NPOS % NT == 0 && (ST_BM * (CPR + 1)) % 64 == 0, "load layout");

    // two stages as distinct arrays (see join_resident)
    __shared__ __attribute__((aligned(16))) uint8_t s_op0[ROWS * LS];
    __shared__ __attribute__((aligned(16))) uint8_t s_op1[ROWS * LS];
    __shared__ V s_np[NEED_NORMS ? ST_NW : 1][NEED_NORMS ? 32 * SA : 1];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, c32 = lane & 31;
    const int wr = wave >> 1, wc = wave & 1;

    // tile order: groups of 8 x 8 tiles, row-major inside a group
    const uint32_t n_pt = (g.n_p + ST_BM - 1) / ST_BM, n_qt = (g.n_q + ST_BN - 1) / ST_BN;
    const uint32_t tile = blockIdx.x;
    constexpr uint32_t G = 8;
    const uint32_t groups_q = (n_qt + G - 1) / G;
    const uint32_t grp = tile / (G * G), in = tile % (G * G);
    const uint32_t gp = grp / groups_q, gq = grp % groups_q;
    const uint32_t hp = min(G, n_pt - gp * G), hq = min(G, n_qt - gq * G);
    // groups at the ragged edges are smaller; their tiles are numbered densely
    if (in >= hp * hq)
        return;
    const uint32_t pt = gp * G + in / hq, qt = gq * G + in % hq;
    // self-join triangle: a tile wholly below the diagonal holds no pair i <= j
    if (MODE == MODE_TRI && pt > qt)
        return;
    const uint32_t p0 = pt * ST_BM, q0 = qt * ST_BN;
    const uint32_t n_chunks = (g.row_bytes + ST_KC - 1) / ST_KC;

    // Direct loads: wave instruction k = wave + ST_NW i fills LDS positions
    // [64 k, 64 k + 64); position p holds chunk p % (CPR + 1) (the pad position
    // repeats chunk 0) of tile row p / (CPR + 1).  Per-lane offsets within the
    // P or Q descriptor (rows past n_p / n_q read zeros), plus the chunk's byte
    // offset kc * KC.
    const uint32_t bytes_p = min(g.n_p - p0, (uint32_t)ST_BM) * g.row_bytes;
    const uint32_t bytes_q = min(g.n_q - q0, (uint32_t)ST_BN) * g.row_bytes;
    const uint8_t *base_p = g.P + (size_t)p0 * g.row_bytes;
    const uint8_t *base_q = g.Q + (size_t)q0 * g.row_bytes;
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    uint32_t voff[NLD], vcol[NLD];
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
        const int pos = 64 * (wv + ST_NW * i) + lane;
        const int r = pos / (CPR + 1), cp = pos % (CPR + 1);
        vcol[i] = 16 * (cp == CPR ? 0 : cp);
        voff[i] = (uint32_t)(r < ST_BM ? r : r - ST_BM) * g.row_bytes + vcol[i];
    }
    auto stage_issue = [&](uint32_t kc, uint8_t *dst) {
        const uint32_t kb = kc * ST_KC;
        if (kb + ST_KC <= g.row_bytes) {                 // uniform
#pragma unroll
            for (int i = 0; i < NLD; ++i) {
                const int k = wv + ST_NW * i;
                const bool is_p = k < P_LOADS;
                buffer_load_lds16(is_p ? base_p : base_q, is_p ? bytes_p : bytes_q, voff[i],
                                  dst + 1024 * k, kb);
            }
        } else {
            // the last chunk of a row that is not a multiple of KC: columns
            // past the row read zeros (offset at the descriptor's end)
#pragma unroll
            for (int i = 0; i < NLD; ++i) {
                const int k = wv + ST_NW * i;
                const bool is_p = k < P_LOADS;
                const uint32_t nbytes = is_p ? bytes_p : bytes_q;
                const uint32_t vo = kb + vcol[i] >= g.row_bytes ? nbytes : voff[i] + kb;
                buffer_load_lds16(is_p ? base_p : base_q, nbytes, vo, dst + 1024 * k);
            }
        }
    };

    acc_t acc[SA][SB];
#pragma unroll
    for (int a = 0; a < SA; ++a)
#pragma unroll
        for (int s = 0; s < SB; ++s)
            acc[a][s] = acc_t{};

    // One K chunk: KSC k-steps, each reading SA A- and SB B-fragments (a ring
    // of LOOK + 1 steps, LOOK steps ahead) and issuing SA * SB MFMAs.
    constexpr int LOOK = 2, RING = LOOK + 1;
    auto chunk = [&](uint32_t kc, const uint8_t *cur, uint8_t *nxt)
                     __attribute__((always_inline)) {
        if (kc + 1 < n_chunks)
            stage_issue(kc + 1, nxt);
        const uint8_t *pa = cur + (32 * SA * wr + c32) * LS + 16 * half;
        const uint8_t *pb = cur + (ST_BM + 32 * SB * wc + c32) * LS + 16 * half;
        i32x4 ring[RING][SA + SB];
        auto fetch = [&](i32x4(&f)[SA + SB], int ks) __attribute__((always_inline)) {
#pragma unroll
            for (int a = 0; a < SA; ++a)
                f[a] = *(const i32x4 *)(pa + 32 * a * LS + 32 * ks);
#pragma unroll
            for (int b = 0; b < SB; ++b)
                f[SA + b] = *(const i32x4 *)(pb + 32 * b * LS + 32 * ks);
        };
        static_for<0, LOOK>([&](auto Q) __attribute__((always_inline)) {
            fetch(ring[decltype(Q)::value], decltype(Q)::value);
        });
        static_for<0, KSC>([&](auto K) __attribute__((always_inline)) {
            constexpr int ks = decltype(K)::value;
            if constexpr (ks + LOOK < KSC)
                fetch(ring[(ks + LOOK) % RING], ks + LOOK);
            const i32x4(&f)[SA + SB] = ring[ks % RING];
#pragma unroll
            for (int a = 0; a < SA; ++a)
#pragma unroll
                for (int b = 0; b < SB; ++b)
                    acc[a][b] = M::mma(f[a], f[SA + b], acc[a][b]);
            __builtin_amdgcn_sched_barrier(0);
        });
        __builtin_amdgcn_s_waitcnt(0);   // this wave's loads of chunk kc + 1 landed
        __syncthreads();
    };

    stage_issue(0, s_op0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (uint32_t kc = 0; kc < n_chunks; kc += 2) {
        chunk(kc, s_op0, s_op1);
        if (kc + 1 < n_chunks)
            chunk(kc + 1, s_op1, s_op0);
    }

    const uint32_t prow0 = p0 + 32 * SA * wr;
    const uint32_t ibase = prow0 + 4 * half;
    V nmin = big_val<V>();
    const V *nrows = nullptr;
    if constexpr (NEED_NORMS) {
        nmin = stage_row_norms<DT, SA>(prow0, lane, s_np[wave], g);
        nrows = &s_np[wave][4 * half];
    }
    const V nb = bound_base<DT, MET>(nmin, g);
    // After the last chunk's barrier the operand stages are free: each wave
    // stages its matches in an eighth of them (2304 pairs), for the single
    // pass and the emit pass alike.
    constexpr uint32_t STAGE_BYTES = 2 * ROWS * LS / ST_NW;
    static_assert(STAGE_BYTES / 8 >= 1024, "a whole 32x32 block must fit the staging buffer");
    uint8_t *stage_mem = (wave < ST_NW / 2 ? s_op0 : s_op1) + (wave % (ST_NW / 2)) * STAGE_BYTES;
    WaveOut wo{(lds_pair *)stage_mem, STAGE_BYTES / 8, 0u, 0ull};
    const uint64_t blk = (uint64_t)(pt * n_qt + qt) * ST_NW + wave;
    uint64_t blk_run = 0;
    if constexpr (MODE == MODE_MASK) {
        // Every block is tested exactly and its match bits are kept for the
        // emit pass (one 16-byte store per lane); the output block's count is
        // the wave's sum of the lanes' popcounts (at most 16 SA SB < 2^8).
        typedef __attribute__((address_space(1))) i32x4 global_i32x4;
        uint32_t mw[SA * SB / 2] = {};
        uint32_t lane_cnt = 0;
#pragma unroll
        for (int b = 0; b < SB; ++b) {
            const uint32_t j = q0 + 32 * SB * wc + 32 * b + c32;
            V ny = V(0);
            if constexpr (NEED_NORMS)
                ny = j < g.n_q ? ((const V *)g.norm_q)[j] : big_val<V>();
#pragma unroll
            for (int a = 0; a < SA; ++a) {
                const uint32_t m =
                    block_mask<DT, MET>(acc[a][b], ibase + 32 * a, j, ny, nrows + 32 * a, g);
                const int sb = b * SA + a;
                mw[sb / 2] |= m << (16 * (sb % 2));
                lane_cnt += (uint32_t)__builtin_popcount(m);
            }
        }
        static_assert(SA * SB == 8 && 16 * SA * SB < 256, "mask record and count bits");
        *((global_i32x4 *)g.masks + (blk * 64 + lane)) =
            i32x4{(int)mw[0], (int)mw[1], (int)mw[2], (int)mw[3]};
        uint32_t tot = 0;
#pragma unroll
        for (int bit = 0; bit < 8; ++bit)
            tot += (uint32_t)__popcll(__ballot((lane_cnt >> bit) & 1)) << bit;
        if (lane == 0)
            g.block_counts[blk] = tot;
        return;
    }
    if constexpr (MODE == MODE_EMIT)
        wo.dst = g.block_offsets[blk];
#pragma unroll
    for (int b = 0; b < SB; ++b) {
        const uint32_t j = q0 + 32 * SB * wc + 32 * b + c32;
        V ny = V(0);
        if constexpr (NEED_NORMS)
            ny = j < g.n_q ? ((const V *)g.norm_q)[j] : big_val<V>();
        acc_t blk_acc[SA];
#pragma unroll
        for (int a = 0; a < SA; ++a)
            blk_acc[a] = acc[a][b];
        V mb[SA];
        fold_max_blk<0, 16 * SA, SA>(blk_acc, mb);
        const bool may = lane_bound<DT, MET>(max_of<SA>(mb), nb, ny, g);
        if (__ballot(may) != 0)
            exact_blocks<DT, MET, MODE, SA>(blk_acc, mb, ibase, j, lane, nb, ny, nrows, g,
                                            blk_run, wo);
    }
    if constexpr (single_mode<MODE>())
        flush_workgroup_out<ST_NW>(wo, wave, lane, g);
    if constexpr (MODE == MODE_EMIT)
        flush_wave_out<MODE>(wo, lane, g);
    if constexpr (MODE == MODE_COUNT) {
        if (lane == 0)
            g.block_counts[blk] = (uint32_t)blk_run;
    }
}

// ---------------------------------------------------------------------------
// Instantiation tables.  Resident variants by k-steps (KS * 32 bytes of row):
// index 0..3 -> KS = 1, 2, 4, 8 for int8 and 2, 4, 8, 16 for fp16/bf16.
template <int DT>
struct ResidentCfg;
template <>
struct ResidentCfg<DT_F16> {
    static constexpr int KS[4] = {2, 4, 8, 16};
};
template <>
struct ResidentCfg<DT_BF16> {
    static constexpr int KS[4] = {2, 4, 8, 16};
};
template <>
struct ResidentCfg<DT_I8> {
    static constexpr int KS[4] = {1, 2, 4, 8};
};

// Eight waves (two per SIMD) per workgroup: one tile load from L2 feeds 256
// or 512 rows of P, and each Q tile is staged once per CU.
constexpr int RES_NW = 8;
// 32-row A-blocks per wave: two, which with the two accumulator sets of the
// sub-tile pipeline keeps every variant within 256 VGPRs; four for int8 rows
// of at most 64 bytes, whose A-fragments are small (each B-fragment read from
// LDS then feeds four MFMAs, and a workgroup covers 512 rows of P).
template <int DT, int KS>
constexpr int res_wmb()
{
    return DT == DT_I8 && KS <= 2 ? 4 : 2;
}
// Q tile rows: 256 for rows of at most 64 bytes (a short tile would spend a
// large share of its time in the barrier and the next tile's loads), else 128
// (four sub-tiles per barrier) unless the rows are so long that two
// double-buffered tiles per CU would not fit in LDS.
template <int KS>
constexpr int res_bn()
{
    return KS <= 2 ? 256 : KS <= 8 ? 128 : 64;
}

template <int DT, int MET, int MODE, int V>
hipError_t launch_resident_v(const Plan &p, const JoinArgs &g, hipStream_t st)
{
    constexpr int KS = ResidentCfg<DT>::KS[V];
    constexpr int WMB = res_wmb<DT, KS>();
    constexpr int BN = res_bn<KS>();
    // the self-join triangle pairs the blocks of P rows (see join_resident)
    const uint32_t grid =
        MODE == MODE_TRI ? (p.grid / p.qsplit + 1) / 2 * p.qsplit : p.grid;
    hipLaunchKernelGGL((join_resident<DT, MET, MODE, KS, WMB, RES_NW, BN>), dim3(grid),
                       dim3(RES_NW * 64), 0, st, g);
    return hipGetLastError();
}

// Workgroups of a resident variant that fit on one CU (registers and LDS).
template <int DT, int MET, int V>
int resident_occupancy_v()
{
    constexpr int KS = ResidentCfg<DT>::KS[V];
    constexpr int WMB = res_wmb<DT, KS>();
    constexpr int BN = res_bn<KS>();
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, reinterpret_cast<const void *>(&join_resident<DT, MET, MODE_SINGLE, KS, WMB, RES_NW, BN>),
            RES_NW * 64, 0) != hipSuccess)
        n = 1;
    return n < 1 ? 1 : n;
}

template <int DT>
int resident_occupancy_dtype(int metric, int variant)
{
    static int cache[2][4];   // written with the same value by any racing caller
    int &c = cache[metric == MET_L2][variant & 3];
    if (c == 0) {
        const bool l2 = metric == MET_L2;
        switch (variant) {
        case 0: c = l2 ? resident_occupancy_v<DT, MET_L2, 0>() : resident_occupancy_v<DT, MET_IP, 0>(); break;
        case 1: c = l2 ? resident_occupancy_v<DT, MET_L2, 1>() : resident_occupancy_v<DT, MET_IP, 1>(); break;
        case 2: c = l2 ? resident_occupancy_v<DT, MET_L2, 2>() : resident_occupancy_v<DT, MET_IP, 2>(); break;
        default: c = l2 ? resident_occupancy_v<DT, MET_L2, 3>() : resident_occupancy_v<DT, MET_IP, 3>(); break;
        }
    }
    return c;
}

template <int DT, int MET, int MODE>
hipError_t launch_mode(const Plan &p, const JoinArgs &g, hipStream_t st)
{
    if (p.family == FAM_STREAMED) {
        hipLaunchKernelGGL((join_streamed<DT, MET, MODE>), dim3(p.grid), dim3(ST_NW * 64), 0, st,
                           g);
        return hipGetLastError();
    }
    switch (p.variant) {
    case 0: return launch_resident_v<DT, MET, MODE, 0>(p, g, st);
    case 1: return launch_resident_v<DT, MET, MODE, 1>(p, g, st);
    case 2: return launch_resident_v<DT, MET, MODE, 2>(p, g, st);
    case 3: return launch_resident_v<DT, MET, MODE, 3>(p, g, st);
    default: return hipErrorInvalidValue;
    }
}

template <int DT>
hipError_t launch_dtype(const Plan &p, int metric, int mode, const JoinArgs &g, hipStream_t st)
{
    if (mode == MODE_RECORD) {
        // resident kernel only
        if (p.family != FAM_RESIDENT || (metric != MET_IP && metric != MET_L2))
            return hipErrorInvalidValue;
        const bool l2 = metric == MET_L2;
        switch (p.variant) {
        case 0: return l2 ? launch_resident_v<DT, MET_L2, MODE_RECORD, 0>(p, g, st)
                          : launch_resident_v<DT, MET_IP, MODE_RECORD, 0>(p, g, st);
        case 1: return l2 ? launch_resident_v<DT, MET_L2, MODE_RECORD, 1>(p, g, st)
                          : launch_resident_v<DT, MET_IP, MODE_RECORD, 1>(p, g, st);
        case 2: return l2 ? launch_resident_v<DT, MET_L2, MODE_RECORD, 2>(p, g, st)
                          : launch_resident_v<DT, MET_IP, MODE_RECORD, 2>(p, g, st);
        case 3: return l2 ? launch_resident_v<DT, MET_L2, MODE_RECORD, 3>(p, g, st)
                          : launch_resident_v<DT, MET_IP, MODE_RECORD, 3>(p, g, st);
        default: return hipErrorInvalidValue;
        }
    }
    if (mode == MODE_TRI) {
        if (metric != MET_IP && metric != MET_L2)
            return hipErrorInvalidValue;
        const bool l2 = metric == MET_L2;
        if (p.family == FAM_STREAMED) {
            if (l2)
                hipLaunchKernelGGL((join_streamed<DT, MET_L2, MODE_TRI>), dim3(p.grid),
                                   dim3(ST_NW * 64), 0, st, g);
            else
                hipLaunchKernelGGL((join_streamed<DT, MET_IP, MODE_TRI>), dim3(p.grid),
                                   dim3(ST_NW * 64), 0, st, g);
            return hipGetLastError();
        }
        switch (p.variant) {
        case 0: return l2 ? launch_resident_v<DT, MET_L2, MODE_TRI, 0>(p, g, st)
                          : launch_resident_v<DT, MET_IP, MODE_TRI, 0>(p, g, st);
        case 1: return l2 ? launch_resident_v<DT, MET_L2, MODE_TRI, 1>(p, g, st)
                          : launch_resident_v<DT, MET_IP, MODE_TRI, 1>(p, g, st);
        case 2: return l2 ? launch_resident_v<DT, MET_L2, MODE_TRI, 2>(p, g, st)
                          : launch_resident_v<DT, MET_IP, MODE_TRI, 2>(p, g, st);
        case 3: return l2 ? launch_resident_v<DT, MET_L2, MODE_TRI, 3>(p, g, st)
                          : launch_resident_v<DT, MET_IP, MODE_TRI, 3>(p, g, st);
        default: return hipErrorInvalidValue;
        }
    }
    if (mode == MODE_MASK) {
        // K-streamed kernel only
        if (p.family != FAM_STREAMED || (metric != MET_IP && metric != MET_L2))
            return hipErrorInvalidValue;
        if (metric == MET_IP)
            hipLaunchKernelGGL((join_streamed<DT, MET_IP, MODE_MASK>), dim3(p.grid),
                               dim3(ST_NW * 64), 0, st, g);
        else
            hipLaunchKernelGGL((join_streamed<DT, MET_L2, MODE_MASK>), dim3(p.grid),
                               dim3(ST_NW * 64), 0, st, g);
        return hipGetLastError();
    }
    if (metric == MET_IP) {
        switch (mode) {
        case MODE_SINGLE: return launch_mode<DT, MET_IP, MODE_SINGLE>(p, g, st);
        case MODE_COUNT: return launch_mode<DT, MET_IP, MODE_COUNT>(p, g, st);
        case MODE_EMIT: return launch_mode<DT, MET_IP, MODE_EMIT>(p, g, st);
        }
    } else if (metric == MET_L2) {
        switch (mode) {
        case MODE_SINGLE: return launch_mode<DT, MET_L2, MODE_SINGLE>(p, g, st);
        case MODE_COUNT: return launch_mode<DT, MET_L2, MODE_COUNT>(p, g, st);
        case MODE_EMIT: return launch_mode<DT, MET_L2, MODE_EMIT>(p, g, st);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace sjk
