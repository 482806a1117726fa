// sj_lsh.hip -- gfx950 kernels of the LSH-bucketed join (Ahle & Silvestri,
// "Similarity Search with Tensor Core Units", Section 4, the LSH method of
// Theorem 3): hash every point into L tables, bring each table's equal keys
// together with a radix sort, list the buckets that P and Q share, and run the
// exact join inside every shared bucket on the matrix cores.
//
// The bucket join is the brute-force join of Section 4 restricted to a pair of
// buckets: Theorem 3's cost is the sum over tables and shared buckets of
// |P bucket| x |Q bucket| inner products, each bucket pair handled as a
// blocked product on 64 x 64 workgroup tiles (32 x 32 MFMA blocks), with the
// same fused threshold test and wave-ballot compaction as the all-pairs join.
#include "sj_lsh.h"

#include <hipcub/hipcub.hpp>

#include "sj_internal.h"
#include "sj_join_kernels.h"

namespace sjl {
namespace {

using sjk::DT_BF16;
using sjk::DT_F16;
using sjk::DT_I8;
using sjk::i32x4;
using sjk::MET_IP;
using sjk::MET_L2;

// ----------------------------------------------------------------- keys

// The E stored elements of one 16-byte chunk as exact values.
template <int DT>
struct Chunk;

template <>
struct Chunk<DT_F16> {
    static constexpr int E = 8;
    typedef double acc_t;
    static __device__ __forceinline__ double at(const i32x4 &v, int e)
    {
        const uint16_t h = (uint16_t)((uint32_t)v[e >> 1] >> (16 * (e & 1)));
        return (double)(float)__builtin_bit_cast(_Float16, h);
    }
};

template <>
struct Chunk<DT_BF16> {
    static constexpr int E = 8;
    typedef double acc_t;
    static __device__ __forceinline__ double at(const i32x4 &v, int e)
    {
        const uint32_t h = ((uint32_t)v[e >> 1] >> (16 * (e & 1))) & 0xffffu;
        return (double)__builtin_bit_cast(float, h << 16);
    }
};

template <>
struct Chunk<DT_I8> {
    static constexpr int E = 16;
    typedef int32_t acc_t;   // |z| <= 32768 * 128 * 128 = 2^29: exact
    static __device__ __forceinline__ int32_t at(const i32x4 &v, int e)
    {
        return (int32_t)(int8_t)((uint32_t)v[e >> 2] >> (8 * (e & 3)));
    }
};

// Functions evaluated per pass over a row.
constexpr int KG = 4;

// One thread per (row, table): z_f = sum_m A[f][m] x_m in ascending m (exact
// products; for fp16/bf16 a double sum in that order, for int8 an exact int32
// sum), then the function value and the key (see launch_keys).
template <int DT>
__global__ void __launch_bounds__(256) keys_kernel(Rows r, uint32_t d, uint32_t k,
                                                   const int8_t *A, const int32_t *B, int32_t w,
                                                   uint64_t *keys)
{
    typedef Chunk<DT> C;
    typedef typename C::acc_t acc_t;
    const uint32_t row = blockIdx.x * 256 + threadIdx.x;
    const uint32_t t = blockIdx.y;
    if (row >= r.n)
        return;
    const uint8_t *x = r.X + (size_t)row * r.row_bytes;
    const uint32_t nch = (d + C::E - 1) / C::E;
    const uint32_t beta = k ? 64 / k : 64;
    const uint64_t low = beta >= 64 ? ~0ull : (1ull << beta) - 1;
    uint64_t key = 0;
    for (uint32_t u0 = 0; u0 < k; u0 += KG) {
        acc_t z[KG];
#pragma unroll
        for (int g = 0; g < KG; ++g)
            z[g] = acc_t(0);
        const int8_t *a = A + (size_t)(t * k + u0) * d;
        for (uint32_t c = 0; c < nch; ++c) {
            const i32x4 v = *(const i32x4 *)(x + 16 * c);
#pragma unroll
            for (int e = 0; e < C::E; ++e) {
                const uint32_t m = c * C::E + e;
                if (m < d) {
                    const acc_t xe = C::at(v, e);
#pragma unroll
                    for (int g = 0; g < KG; ++g)
                        if (u0 + g < k)
                            z[g] += acc_t(a[(size_t)g * d + m]) * xe;
                }
            }
        }
#pragma unroll
        for (int g = 0; g < KG; ++g) {
            const uint32_t u = u0 + g;
            if (u < k) {
                if (w == 0) {
                    key |= (uint64_t)(z[g] >= acc_t(0)) << u;
                } else {
                    const double q = ((double)z[g] + (double)B[t * k + u]) / (double)w;
                    const int64_t v = (int64_t)floor(q);
                    key |= ((uint64_t)v & low) << (beta * u);
                }
            }
        }
    }
    keys[(size_t)t * r.n + row] = key;
}

__global__ void iota_kernel(uint32_t *v, uint32_t n)
{
    const uint32_t i = blockIdx.x * 256 + threadIdx.x;
    if (i < n)
        v[i] = i;
}

// ------------------------------------------------------------ bucket pairs

// First sorted position in [lo, hi) whose key is > key (keys ascending).
__device__ __forceinline__ uint32_t upper_bound(const uint64_t *s, uint32_t lo, uint32_t hi,
                                                uint64_t key)
{
    while (lo < hi) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (s[mid] <= key)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

__device__ __forceinline__ uint32_t lower_bound(const uint64_t *s, uint32_t lo, uint32_t hi,
                                                uint64_t key)
{
    while (lo < hi) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (s[mid] < key)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// One thread per (sorted position of P, table): the first position of each P
// bucket looks its key up in Q's sorted keys and, when Q has it, appends the
// bucket pair.
__global__ void __launch_bounds__(256) bucket_pairs_kernel(const uint64_t *sorted_p,
                                                           uint32_t n_p,
                                                           const uint64_t *sorted_q,
                                                           uint32_t n_q, BucketPairs bp)
{
    const uint32_t p = blockIdx.x * 256 + threadIdx.x;
    const uint32_t t = blockIdx.y;
    if (p >= n_p)
        return;
    const uint64_t *sp = sorted_p + (size_t)t * n_p;
    const uint64_t *sq = sorted_q + (size_t)t * n_q;
    const uint64_t key = sp[p];
    if (p > 0 && sp[p - 1] == key)
        return;
    const uint32_t pe = upper_bound(sp, p + 1, n_p, key);
    const uint32_t q0 = lower_bound(sq, 0, n_q, key);
    const uint32_t qe = upper_bound(sq, q0, n_q, key);
    if (q0 == qe)
        return;
    const uint32_t np = pe - p, nq = qe - q0;
    const uint64_t tiles = (uint64_t)((np + TILE - 1) / TILE) * ((nq + TILE - 1) / TILE);
    const unsigned long long old =
        atomicAdd(&bp.counters[0], (1ull << TILE_BITS) | (unsigned long long)tiles);
    atomicAdd(&bp.counters[1], (unsigned long long)tiles);
    atomicAdd(&bp.counters[2], (unsigned long long)np * nq);
    const uint64_t slot = old >> TILE_BITS;
    if (slot < bp.cap) {
        bp.head[slot] = make_uint4(t, p, np, q0);
        bp.nq[slot] = nq;
        bp.tile0[slot] = old & ((1ull << TILE_BITS) - 1);
    }
}

// ------------------------------------------------------------ bucket join

template <int DT, int MET>
__device__ __forceinline__ bool matches(typename sjk::Mma<DT>::val_t acc,
                                        typename sjk::Mma<DT>::val_t nx,
                                        typename sjk::Mma<DT>::val_t ny, const JoinArgs &g)
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

// A workgroup of 4 waves takes 64 x 64 tiles of bucket pairs (grid-stride):
// the tile's rows of P and Q are gathered through the tables' sorted
// permutations into LDS in chunks of 128 bytes of each row (16-byte chunks,
// rows padded by one chunk), wave (wr, wc) multiplies its 32 x 32 block on the
// matrix cores over the chunk's k-steps, and the epilogue applies the exact
// test, drops pairs that share a bucket in an earlier table (so every pair is
// reported once) and appends the rest with one atomic per wave.
template <int DT, int MET>
__global__ void __launch_bounds__(256) join_kernel(JoinArgs g)
{
    typedef sjk::Mma<DT> M;
    typedef typename M::acc_t acc_t;
    typedef typename M::val_t V;
    constexpr int CS = 9;    // LDS positions per tile row: 8 chunks + 1 pad
    __shared__ i32x4 sA[TILE * CS], sB[TILE * CS];
    __shared__ uint32_t sIP[TILE], sIQ[TILE];
    __shared__ V sNP[TILE], sNQ[TILE];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1, half = lane >> 5, c32 = lane & 31;
    const uint32_t rb = g.P.row_bytes;   // == g.Q.row_bytes
    const uint32_t lc = tid & 7, lr = tid >> 3;   // this thread's load chunk and rows lr, lr + 32

    for (uint64_t T = blockIdx.x; T < g.n_tiles; T += gridDim.x) {
        uint32_t lo = 0, hi = g.n_bp;
        while (hi - lo > 1) {
            const uint32_t mid = (lo + hi) >> 1;
            if (g.tile0[mid] <= T)
                lo = mid;
            else
                hi = mid;
        }
        const uint4 h = g.head[lo];
        const uint32_t t = h.x, nq = g.nq[lo];
        const uint64_t local = T - g.tile0[lo];
        const uint32_t ntq = (nq + TILE - 1) / TILE;
        const uint32_t tp = (uint32_t)(local / ntq), tq = (uint32_t)(local % ntq);
        const uint32_t rows_p = min(h.z - tp * TILE, TILE), rows_q = min(nq - tq * TILE, TILE);

        __syncthreads();   // the previous tile's reads of sIP/sIQ/sA/sB are done
        if (tid < (int)TILE) {
            const bool ok = (uint32_t)tid < rows_p;
            const uint32_t i = ok ? g.perm_p[(size_t)t * g.P.n + h.y + tp * TILE + tid] : 0u;
            sIP[tid] = i;
            if constexpr (MET == MET_L2)
                sNP[tid] = ok ? ((const V *)g.norm_p)[i] : V(0);
        } else if (tid < (int)(2 * TILE)) {
            const int c = tid - TILE;
            const bool ok = (uint32_t)c < rows_q;
            const uint32_t j = ok ? g.perm_q[(size_t)t * g.Q.n + h.w + tq * TILE + c] : 0u;
            sIQ[c] = j;
            if constexpr (MET == MET_L2)
                sNQ[c] = ok ? ((const V *)g.norm_q)[j] : V(0);
        }
        __syncthreads();
        const uint8_t *pa0 = g.P.X + (size_t)sIP[lr] * rb;
        const uint8_t *pa1 = g.P.X + (size_t)sIP[lr + 32] * rb;
        const uint8_t *pb0 = g.Q.X + (size_t)sIQ[lr] * rb;
        const uint8_t *pb1 = g.Q.X + (size_t)sIQ[lr + 32] * rb;
        const bool va0 = lr < rows_p, va1 = lr + 32 < rows_p;
        const bool vb0 = lr < rows_q, vb1 = lr + 32 < rows_q;

        acc_t acc = acc_t{};
        for (uint32_t kc = 0; kc < rb; kc += 128) {
            const uint32_t off = kc + 16 * lc;
            const i32x4 z = {0, 0, 0, 0};
            const bool in = off < rb;
            const i32x4 a0 = va0 && in ? *(const i32x4 *)(pa0 + off) : z;
            const i32x4 a1 = va1 && in ? *(const i32x4 *)(pa1 + off) : z;
            const i32x4 b0 = vb0 && in ? *(const i32x4 *)(pb0 + off) : z;
            const i32x4 b1 = vb1 && in ? *(const i32x4 *)(pb1 + off) : z;
            if (kc)
                __syncthreads();   // the previous chunk's fragments are read
            sA[lr * CS + lc] = a0;
            sA[(lr + 32) * CS + lc] = a1;
            sB[lr * CS + lc] = b0;
            sB[(lr + 32) * CS + lc] = b1;
            __syncthreads();
            const uint32_t nks = min(4u, (rb - kc + 31) / 32);
#pragma unroll
            for (uint32_t ks = 0; ks < 4; ++ks)
                if (ks < nks) {
                    const i32x4 a = sA[(wr * 32 + c32) * CS + 2 * ks + half];
                    const i32x4 b = sB[(wc * 32 + c32) * CS + 2 * ks + half];
                    acc = M::mma(a, b, acc);
                }
        }

        // epilogue: result register r of this lane is (row wr*32 + 8(r/4) +
        // 4 half + r%4, column wc*32 + c32) of the tile
        const uint32_t jl = wc * 32 + c32;
        const bool jok = jl < rows_q;
        const uint32_t j = sIQ[jl];
        const V ny = MET == MET_L2 ? sNQ[jl] : V(0);
        uint32_t m = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const uint32_t il = wr * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
            const V nx = MET == MET_L2 ? sNP[il] : V(0);
            const bool ok = jok && il < rows_p && matches<DT, MET>(acc[r], nx, ny, g);
            m |= ok ? (1u << r) : 0u;
        }
        if (t > 0 && m != 0) {
            uint32_t mm = m;
            while (mm) {
                const int r = __builtin_ctz(mm);
                mm &= mm - 1;
                const uint32_t i = sIP[wr * 32 + 8 * (r >> 2) + 4 * half + (r & 3)];
                for (uint32_t t2 = 0; t2 < t; ++t2)
                    if (g.keys_p[(size_t)t2 * g.P.n + i] == g.keys_q[(size_t)t2 * g.Q.n + j]) {
                        m &= ~(1u << r);
                        break;
                    }
            }
        }
        const uint32_t cnt = (uint32_t)__builtin_popcount(m);
        uint32_t tot = 0, pre = 0;
#pragma unroll
        for (int b = 0; b < 5; ++b) {
            const uint64_t bits = __ballot((cnt >> b) & 1);
            tot += (uint32_t)__popcll(bits) << b;
            pre += sjk::lanes_below(bits) << b;
        }
        if (tot != 0) {
            unsigned long long base = 0;
            if (lane == 0)
                base = atomicAdd(g.counter, (unsigned long long)tot);
            uint64_t pos = sjk::first_lane_u64(base) + pre;
            while (m) {
                const int r = __builtin_ctz(m);
                m &= m - 1;
                if (pos < g.cap) {
                    const uint32_t i = sIP[wr * 32 + 8 * (r >> 2) + 4 * half + (r & 3)];
                    ((sjk::global_pair *)g.pairs)[pos] = sjk::pack_pair(i, j);
                }
                ++pos;
            }
        }
    }
}

template <int DT>
hipError_t launch_keys_t(const Rows &r, uint32_t d, uint32_t L, uint32_t k, const int8_t *A,
                         const int32_t *B, int32_t w, uint64_t *keys, hipStream_t s)
{
    const dim3 grid((r.n + 255) / 256, L);
    hipLaunchKernelGGL(keys_kernel<DT>, grid, dim3(256), 0, s, r, d, k, A, B, w, keys);
    return hipGetLastError();
}

template <int DT, int MET>
hipError_t launch_join_t(const JoinArgs &g, int num_cus, hipStream_t s)
{
    const uint64_t want = (uint64_t)num_cus * 8;
    const uint32_t grid = (uint32_t)(g.n_tiles < want ? g.n_tiles : want);
    hipLaunchKernelGGL((join_kernel<DT, MET>), dim3(grid), dim3(256), 0, s, g);
    return hipGetLastError();
}

}  // namespace

uint32_t key_bits(uint32_t k, int32_t w)
{
    if (k == 0)
        return 1;
    if (w == 0)
        return k;
    const uint32_t b = (64 / k) * k;
    return b > 64 ? 64 : b;
}

hipError_t launch_keys(int dtype, const Rows &r, uint32_t d, uint32_t L, uint32_t k,
                       const int8_t *A, const int32_t *B, int32_t w, uint64_t *keys,
                       hipStream_t s)
{
    if (r.n == 0 || L == 0)
        return hipSuccess;
    switch (dtype) {
    case DT_F16:
        return launch_keys_t<DT_F16>(r, d, L, k, A, B, w, keys, s);
    case DT_BF16:
        return launch_keys_t<DT_BF16>(r, d, L, k, A, B, w, keys, s);
    default:
        return launch_keys_t<DT_I8>(r, d, L, k, A, B, w, keys, s);
    }
}

size_t sort_temp_bytes(uint32_t n, uint32_t bits)
{
    size_t bytes = 0;
    (void)hipcub::DeviceRadixSort::SortPairs(nullptr, bytes, (const uint64_t *)nullptr,
                                             (uint64_t *)nullptr, (const uint32_t *)nullptr,
                                             (uint32_t *)nullptr, n, 0, (int)bits);
    return bytes;
}

hipError_t sort_tables(const uint64_t *keys, uint64_t *sorted, uint32_t *perm, uint32_t *iota,
                       uint32_t n, uint32_t L, uint32_t bits, void *temp, size_t temp_bytes,
                       hipStream_t s)
{
    if (n == 0)
        return hipSuccess;
    hipLaunchKernelGGL(iota_kernel, dim3((n + 255) / 256), dim3(256), 0, s, iota, n);
    hipError_t e = hipGetLastError();
    for (uint32_t t = 0; t < L && e == hipSuccess; ++t) {
        size_t tb = temp_bytes;
        e = hipcub::DeviceRadixSort::SortPairs(temp, tb, keys + (size_t)t * n,
                                               sorted + (size_t)t * n, iota,
                                               perm + (size_t)t * n, n, 0, (int)bits, s);
    }
    return e;
}

hipError_t launch_bucket_pairs(const uint64_t *sorted_p, uint32_t n_p, const uint64_t *sorted_q,
                               uint32_t n_q, uint32_t L, const BucketPairs &bp, hipStream_t s)
{
    if (n_p == 0 || n_q == 0 || L == 0)
        return hipSuccess;
    hipLaunchKernelGGL(bucket_pairs_kernel, dim3((n_p + 255) / 256, L), dim3(256), 0, s,
                       sorted_p, n_p, sorted_q, n_q, bp);
    return hipGetLastError();
}

hipError_t launch_join(int dtype, int metric, const JoinArgs &g, int num_cus, hipStream_t s)
{
    if (g.n_tiles == 0)
        return hipSuccess;
    const bool l2 = metric == MET_L2;
    switch (dtype) {
    case DT_F16:
        return l2 ? launch_join_t<DT_F16, MET_L2>(g, num_cus, s)
                  : launch_join_t<DT_F16, MET_IP>(g, num_cus, s);
    case DT_BF16:
        return l2 ? launch_join_t<DT_BF16, MET_L2>(g, num_cus, s)
                  : launch_join_t<DT_BF16, MET_IP>(g, num_cus, s);
    default:
        return l2 ? launch_join_t<DT_I8, MET_L2>(g, num_cus, s)
                  : launch_join_t<DT_I8, MET_IP>(g, num_cus, s);
    }
}

}  // namespace sjl
