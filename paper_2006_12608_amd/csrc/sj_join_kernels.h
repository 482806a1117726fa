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

// 16 bytes at byte `off` of row `row`, zero outside the row or past n_rows.
// `aligned` (uniform): row_bytes % 16 == 0 and the base is 16-byte aligned, so a
// chunk is either wholly inside the row or wholly outside it.
__device__ __forceinline__ i32x4 load_chunk(const uint8_t *base, uint32_t row, uint32_t n_rows,
                                            uint32_t row_bytes, uint32_t off, bool aligned)
{
    i32x4 v = {0, 0, 0, 0};
    if (row < n_rows && off < row_bytes) {
        const uint8_t *p = base + (size_t)row * row_bytes + off;
        if (aligned) {
            v = *(const i32x4 *)p;
        } else {
            uint32_t w[4] = {0, 0, 0, 0};
            const uint32_t lim = row_bytes - off;
#pragma unroll
            for (int b = 0; b < 16; ++b)
                if ((uint32_t)b < lim)
                    w[b >> 2] |= (uint32_t)p[b] << (8 * (b & 3));
            v = i32x4{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
        }
    }
    return v;
}

__device__ __forceinline__ uint64_t first_lane_u64(uint64_t v)
{
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

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

// Epilogue of one wave over a (32*WMB) x 32 block of results:
// accumulators acc[a] hold rows prow0 + 32a + (8(r/4) + 4 half + r%4), column j.
//  1. Cheap necessary condition per lane (one max over all its results against
//     a per-lane bound); a wave whose lanes all fail is done.
//  2. Otherwise every result is tested exactly; ballots give each wave's match
//     count; MODE_SINGLE reserves space with one atomicAdd per wave, MODE_EMIT
//     takes the block's running offset; matches are stored so that each store
//     instruction writes consecutive slots.
template <int DT, int MET, int MODE, int WMB>
__device__ __forceinline__ void epilogue(const typename Mma<DT>::acc_t (&acc)[WMB], uint32_t prow0,
                                         uint32_t j, int half, int lane,
                                         typename Mma<DT>::val_t nmin,
                                         typename Mma<DT>::val_t ny, const JoinArgs &g,
                                         uint64_t &blk_run)
{
    typedef typename Mma<DT>::val_t V;
    V m = acc[0][0];
#pragma unroll
    for (int a = 0; a < WMB; ++a)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            if (a | r)
                m = vmax(m, acc[a][r]);
    bool pass;
    if constexpr (MET == MET_IP) {
        pass = pair_matches<DT, MET>(m, V(0), V(0), g);
    } else {
        pass = pair_matches<DT, MET>(m, nmin, ny, g);
    }
    pass = pass && (j < g.n_q);
    if (__ballot(pass) == 0)
        return;

    const V *np = (const V *)g.norm_p;
    uint32_t tot = 0;
#pragma unroll
    for (int a = 0; a < WMB; ++a)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint32_t i = prow0 + 32 * a + 8 * (r >> 2) + 4 * half + (r & 3);
            bool p = false;
            if (i < g.n_p && j < g.n_q) {
                V nx = V(0);
                if constexpr (MET == MET_L2)
                    nx = np[i];
                p = pair_matches<DT, MET>(acc[a][r], nx, ny, g);
            }
            tot += (uint32_t)__popcll(__ballot(p));
        }
    if constexpr (MODE == MODE_COUNT) {
        blk_run += tot;
        return;
    }
    if (tot == 0)
        return;
    uint64_t base;
    if constexpr (MODE == MODE_SINGLE) {
        unsigned long long b = 0;
        if (lane == 0)
            b = atomicAdd(g.counter, (unsigned long long)tot);
        base = first_lane_u64(b);
    } else {
        base = blk_run;
        blk_run += tot;
    }
#pragma unroll
    for (int a = 0; a < WMB; ++a)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint32_t i = prow0 + 32 * a + 8 * (r >> 2) + 4 * half + (r & 3);
            bool p = false;
            if (i < g.n_p && j < g.n_q) {
                V nx = V(0);
                if constexpr (MET == MET_L2)
                    nx = np[i];
                p = pair_matches<DT, MET>(acc[a][r], nx, ny, g);
            }
            const uint64_t mk = __ballot(p);
            if (p) {
                const uint64_t slot = base + lanes_below(mk);
                if (slot < g.cap)
                    *(uint2 *)(g.pairs + 2 * slot) = make_uint2(i, j);
            }
            base += (uint64_t)__popcll(mk);
        }
}

// ---------------------------------------------------------------------------
// Family 1: P rows resident in registers.
//
// A workgroup of NW waves owns BM = NW * 32 * WMB consecutive rows of P; each
// wave keeps its 32*WMB rows, all KS k-steps, as MFMA A-fragments in VGPRs for
// the whole kernel.  The workgroup sweeps its range of Q in tiles of BN rows,
// double-buffered in LDS (row stride padded by 16 bytes so that the 32 rows a
// B-fragment read touches fall in different banks).  Per tile and per 32-row
// sub-tile each wave issues KS * WMB MFMAs and runs the epilogue.
// Output block (for the count/emit passes) = one wave's rows x one Q tile;
// block index = (global wave row-block) * n_qtiles + tile.
template <int DT, int MET, int MODE, int KS, int WMB, int NW, int BN>
__global__ void __launch_bounds__(NW * 64) join_resident(JoinArgs g, uint32_t aligned)
{
    typedef Mma<DT> M;
    typedef typename M::acc_t acc_t;
    typedef typename M::val_t V;
    constexpr int LS = KS * 32 + 16;        // LDS row stride in bytes
    constexpr int NT = NW * 64;
    constexpr int CPR = KS * 2;             // 16-byte chunks per row
    constexpr int TCH = BN * CPR;           // chunks per Q tile
    constexpr int CPT = (TCH + NT - 1) / NT;
    constexpr int SUBS = BN / 32;
    constexpr int BM = NW * 32 * WMB;
    constexpr bool NEED_NORMS = (MET == MET_L2);

    __shared__ __attribute__((aligned(16))) uint8_t s_q[2][BN * LS];
    __shared__ V s_nq[NEED_NORMS ? 2 : 1][NEED_NORMS ? BN : 1];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, c32 = lane & 31;
    const bool al = aligned != 0;
    const uint32_t qsplit = g.qsplit;
    const uint32_t pb = blockIdx.x / qsplit, qs = blockIdx.x - pb * qsplit;
    const uint32_t n_qt = (g.n_q + BN - 1) / BN;
    const uint32_t t0 = (uint32_t)((uint64_t)qs * n_qt / qsplit);
    const uint32_t t1 = (uint32_t)((uint64_t)(qs + 1) * n_qt / qsplit);
    const uint32_t prow0 = pb * BM + wave * 32 * WMB;

    i32x4 A[WMB][KS];
#pragma unroll
    for (int a = 0; a < WMB; ++a)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            A[a][ks] = load_chunk(g.P, prow0 + 32 * a + c32, g.n_p, g.row_bytes,
                                  32 * ks + 16 * half, al);

    V nmin = big_val<V>();
    if constexpr (NEED_NORMS) {
        const V *np = (const V *)g.norm_p;
#pragma unroll
        for (int a = 0; a < WMB; ++a)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const uint32_t i = prow0 + 32 * a + 8 * (r >> 2) + 4 * half + (r & 3);
                if (i < g.n_p)
                    nmin = vmin(nmin, np[i]);
            }
    }

    auto stage_load = [&](uint32_t t, i32x4(&st)[CPT], V &stn) {
#pragma unroll
        for (int k = 0; k < CPT; ++k) {
            const int c = tid + k * NT;
            if (TCH % NT == 0 || c < TCH)
                st[k] = load_chunk(g.Q, t * BN + c / CPR, g.n_q, g.row_bytes, 16 * (c % CPR), al);
        }
        if constexpr (NEED_NORMS) {
            if (tid < BN) {
                const uint32_t jq = t * BN + tid;
                stn = jq < g.n_q ? ((const V *)g.norm_q)[jq] : big_val<V>();
            }
        }
    };
    auto stage_store = [&](int buf, const i32x4(&st)[CPT], V stn) {
#pragma unroll
        for (int k = 0; k < CPT; ++k) {
            const int c = tid + k * NT;
            if (TCH % NT == 0 || c < TCH)
                *(i32x4 *)&s_q[buf][(c / CPR) * LS + 16 * (c % CPR)] = st[k];
        }
        if constexpr (NEED_NORMS) {
            if (tid < BN)
                s_nq[buf][tid] = stn;
        }
    };

    if (t0 < t1) {
        i32x4 st[CPT];
        V stn = V(0);
        stage_load(t0, st, stn);
        stage_store(0, st, stn);
    }
    __syncthreads();

    const uint64_t wave_row_block = (uint64_t)pb * NW + wave;
    for (uint32_t t = t0; t < t1; ++t) {
        const int buf = (t - t0) & 1;
        const bool more = t + 1 < t1;
        i32x4 st[CPT];
        V stn = V(0);
        if (more)
            stage_load(t + 1, st, stn);

        const uint64_t blk = wave_row_block * n_qt + t;
        uint64_t blk_run = 0;
        if constexpr (MODE == MODE_EMIT)
            blk_run = g.block_offsets[blk];

#pragma unroll
        for (int s = 0; s < SUBS; ++s) {
            acc_t acc[WMB];
#pragma unroll
            for (int a = 0; a < WMB; ++a)
                acc[a] = acc_t{};
            const uint8_t *bp = &s_q[buf][(32 * s + c32) * LS + 16 * half];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const i32x4 b = *(const i32x4 *)(bp + 32 * ks);
#pragma unroll
                for (int a = 0; a < WMB; ++a)
                    acc[a] = M::mma(A[a][ks], b, acc[a]);
            }
            V ny = V(0);
            if constexpr (NEED_NORMS)
                ny = s_nq[buf][32 * s + c32];
            epilogue<DT, MET, MODE, WMB>(acc, prow0, t * BN + 32 * s + c32, half, lane, nmin, ny,
                                         g, blk_run);
        }
        if constexpr (MODE == MODE_COUNT) {
            if (lane == 0)
                g.block_counts[blk] = (uint32_t)blk_run;
        }
        if (more)
            stage_store(buf ^ 1, st, stn);
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Family 2: both operands streamed through LDS in chunks of KC bytes of d
// (for rows too long to keep in registers).
//
// A workgroup of 4 waves computes a 128 x 128 output tile; wave (wr, wc) owns
// rows [64 wr, +64) (two A-blocks) and columns [64 wc, +64) (two sub-tiles), so
// it holds four 32x32 accumulators.  P and Q chunks are double-buffered in LDS.
// Tiles are visited in groups of 8 P tiles x 8 Q tiles so that concurrently
// running workgroups share their operand rows in L2.
// Output block = one wave's 64 x 64 region; index = tile * 4 + wave.
constexpr int ST_BM = 128, ST_BN = 128, ST_KC = 128;

template <int DT, int MET, int MODE>
__global__ void __launch_bounds__(256) join_streamed(JoinArgs g, uint32_t aligned)
{
    typedef Mma<DT> M;
    typedef typename M::acc_t acc_t;
    typedef typename M::val_t V;
    constexpr int LS = ST_KC + 16;
    constexpr int CPR = ST_KC / 16;                   // 8 chunks per row per K chunk
    constexpr int TCH = (ST_BM + ST_BN) * CPR;        // 2048 chunks
    constexpr int CPT = TCH / 256;                    // 8 per thread
    constexpr int KSC = ST_KC / 32;                   // 4 k-steps per chunk
    constexpr bool NEED_NORMS = (MET == MET_L2);

    __shared__ __attribute__((aligned(16))) uint8_t s_op[2][(ST_BM + ST_BN) * LS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, c32 = lane & 31;
    const int wr = wave >> 1, wc = wave & 1;
    const bool al = aligned != 0;

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
    const uint32_t p0 = pt * ST_BM, q0 = qt * ST_BN;
    const uint32_t n_chunks = (g.row_bytes + ST_KC - 1) / ST_KC;

    auto stage_load = [&](uint32_t kc, i32x4(&st)[CPT]) {
#pragma unroll
        for (int k = 0; k < CPT; ++k) {
            const int c = tid + k * 256;
            const int r = c / CPR, cc = c % CPR;
            const uint32_t off = kc * ST_KC + 16 * cc;
            st[k] = r < ST_BM ? load_chunk(g.P, p0 + r, g.n_p, g.row_bytes, off, al)
                              : load_chunk(g.Q, q0 + r - ST_BM, g.n_q, g.row_bytes, off, al);
        }
    };
    auto stage_store = [&](int buf, const i32x4(&st)[CPT]) {
#pragma unroll
        for (int k = 0; k < CPT; ++k) {
            const int c = tid + k * 256;
            *(i32x4 *)&s_op[buf][(c / CPR) * LS + 16 * (c % CPR)] = st[k];
        }
    };

    acc_t acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int s = 0; s < 2; ++s)
            acc[a][s] = acc_t{};

    {
        i32x4 st[CPT];
        stage_load(0, st);
        stage_store(0, st);
    }
    __syncthreads();
    for (uint32_t kc = 0; kc < n_chunks; ++kc) {
        const int buf = kc & 1;
        const bool more = kc + 1 < n_chunks;
        i32x4 st[CPT];
        if (more)
            stage_load(kc + 1, st);
        const uint8_t *pa = &s_op[buf][(64 * wr + c32) * LS + 16 * half];
        const uint8_t *pbq = &s_op[buf][(ST_BM + 64 * wc + c32) * LS + 16 * half];
#pragma unroll
        for (int ks = 0; ks < KSC; ++ks) {
            i32x4 fa[2], fb[2];
#pragma unroll
            for (int a = 0; a < 2; ++a)
                fa[a] = *(const i32x4 *)(pa + 32 * a * LS + 32 * ks);
#pragma unroll
            for (int s = 0; s < 2; ++s)
                fb[s] = *(const i32x4 *)(pbq + 32 * s * LS + 32 * ks);
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int s = 0; s < 2; ++s)
                    acc[a][s] = M::mma(fa[a], fb[s], acc[a][s]);
        }
        if (more)
            stage_store(buf ^ 1, st);
        __syncthreads();
    }

    const uint32_t prow0 = p0 + 64 * wr;
    V nmin = big_val<V>();
    if constexpr (NEED_NORMS) {
        const V *np = (const V *)g.norm_p;
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const uint32_t i = prow0 + 32 * a + 8 * (r >> 2) + 4 * half + (r & 3);
                if (i < g.n_p)
                    nmin = vmin(nmin, np[i]);
            }
    }
    const uint64_t blk = (uint64_t)(pt * n_qt + qt) * 4 + wave;
    uint64_t blk_run = 0;
    if constexpr (MODE == MODE_EMIT)
        blk_run = g.block_offsets[blk];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const uint32_t j = q0 + 64 * wc + 32 * s + c32;
        V ny = V(0);
        if constexpr (NEED_NORMS)
            ny = j < g.n_q ? ((const V *)g.norm_q)[j] : big_val<V>();
        const acc_t blk_acc[2] = {acc[0][s], acc[1][s]};
        epilogue<DT, MET, MODE, 2>(blk_acc, prow0, j, half, lane, nmin, ny, g, blk_run);
    }
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

constexpr int RES_NW = 4;
constexpr int RES_BN = 64;
template <int DT, int KS>
constexpr int res_wmb()
{
    return (DT == DT_I8 && KS <= 2) ? 4 : 2;
}

template <int DT, int MET, int MODE, int V>
hipError_t launch_resident_v(const Plan &p, const JoinArgs &g, uint32_t al, hipStream_t st)
{
    constexpr int KS = ResidentCfg<DT>::KS[V];
    constexpr int WMB = res_wmb<DT, KS>();
    hipLaunchKernelGGL((join_resident<DT, MET, MODE, KS, WMB, RES_NW, RES_BN>), dim3(p.grid),
                       dim3(RES_NW * 64), 0, st, g, al);
    return hipGetLastError();
}

template <int DT, int MET, int MODE>
hipError_t launch_mode(const Plan &p, const JoinArgs &g, uint32_t al, hipStream_t st)
{
    if (p.family == FAM_STREAMED) {
        hipLaunchKernelGGL((join_streamed<DT, MET, MODE>), dim3(p.grid), dim3(256), 0, st, g, al);
        return hipGetLastError();
    }
    switch (p.variant) {
    case 0: return launch_resident_v<DT, MET, MODE, 0>(p, g, al, st);
    case 1: return launch_resident_v<DT, MET, MODE, 1>(p, g, al, st);
    case 2: return launch_resident_v<DT, MET, MODE, 2>(p, g, al, st);
    case 3: return launch_resident_v<DT, MET, MODE, 3>(p, g, al, st);
    default: return hipErrorInvalidValue;
    }
}

template <int DT>
hipError_t launch_dtype(const Plan &p, int metric, int mode, bool aligned, const JoinArgs &g,
                        hipStream_t st)
{
    const uint32_t al = aligned ? 1u : 0u;
    if (metric == MET_IP) {
        switch (mode) {
        case MODE_SINGLE: return launch_mode<DT, MET_IP, MODE_SINGLE>(p, g, al, st);
        case MODE_COUNT: return launch_mode<DT, MET_IP, MODE_COUNT>(p, g, al, st);
        case MODE_EMIT: return launch_mode<DT, MET_IP, MODE_EMIT>(p, g, al, st);
        }
    } else if (metric == MET_L2) {
        switch (mode) {
        case MODE_SINGLE: return launch_mode<DT, MET_L2, MODE_SINGLE>(p, g, al, st);
        case MODE_COUNT: return launch_mode<DT, MET_L2, MODE_COUNT>(p, g, al, st);
        case MODE_EMIT: return launch_mode<DT, MET_L2, MODE_EMIT>(p, g, al, st);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace sjk
