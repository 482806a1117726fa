// sj_lsh.hip -- gfx950 kernels of the LSH-bucketed join (Ahle & Silvestri,
// "Similarity Search with Tensor Core Units", Section 4, the LSH method of
// Theorem 3): hash every point into L tables, bring each table's equal keys
// together with a radix sort, list the buckets that P and Q share, and run the
// exact join inside every shared bucket on the matrix cores.
//
// The bucket join is the brute-force join of Section 4 restricted to a pair of
// buckets: Theorem 3's cost is the sum over tables and shared buckets of
// |P bucket| x |Q bucket| inner products, each bucket pair handled as a
// blocked product on 128 x 128 workgroup tiles (32 x 32 MFMA blocks), with the
// same fused threshold test and wave-ballot compaction as the all-pairs join.
#include "sj_lsh.h"


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

// The E stored elements of one 16-byte chunk as exact values; `acc_t` is the
// projection's accumulator and `a_t` the type the projection entries are
// converted to once, before the hash (so that the inner loop is one fused
// multiply-add per element and function, its entry read through the scalar
// path: the entries are the same for every row of a workgroup).
template <int DT>
struct Chunk;

template <>
struct Chunk<DT_F16> {
    static constexpr int E = 8;
    typedef double acc_t;
    typedef double a_t;
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
    typedef double a_t;
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
    typedef int32_t a_t;
    static __device__ __forceinline__ int32_t at(const i32x4 &v, int e)
    {
        return (int32_t)(int8_t)((uint32_t)v[e >> 2] >> (8 * (e & 3)));
    }
};

// Projection rows are widened with their length padded to a multiple of the
// chunk's E elements (zeros past d): together with the zero padding of the
// rows this adds only exact zeros to each sum, and the inner loop needs no
// bounds test.
template <int DT>
constexpr uint32_t padded_d(uint32_t d)
{
    return (d + Chunk<DT>::E - 1) / Chunk<DT>::E * Chunk<DT>::E;
}

template <typename T>
__global__ void widen_kernel(const int8_t *A, T *out, uint32_t d, uint32_t dp, uint64_t n_out)
{
    const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n_out) {
        const uint64_t f = i / dp, m = i - f * dp;
        out[i] = m < d ? T(A[f * d + m]) : T(0);
    }
}

// Rows a workgroup of the key kernel stages in LDS at once (one per lane of a
// wave), and the bytes of a row it stages per pass.
constexpr int KROWS = 64;
constexpr int KSEG = 512;

// G consecutive functions of one row segment: z[g] += sum_m A[f0 + g][m0 + m] x_m
// over the segment's nch chunks (x: this lane's row in LDS) in ascending m.
// The entries' addresses are the same for every lane (the compiler reads them
// with scalar loads).
template <int DT, int G>
__device__ __forceinline__ void project(const uint8_t *x, uint32_t nch, uint32_t dp,
                                        const typename Chunk<DT>::a_t *a,
                                        typename Chunk<DT>::acc_t (&z)[G])
{
    typedef Chunk<DT> C;
    typedef typename C::acc_t acc_t;
    for (uint32_t c = 0; c < nch; ++c) {
        const i32x4 v = *(const i32x4 *)(x + 16 * c);
        acc_t xe[C::E];
#pragma unroll
        for (int e = 0; e < C::E; ++e)
            xe[e] = C::at(v, e);
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const typename C::a_t *ag = a + (size_t)g * dp + c * C::E;
#pragma unroll
            for (int e = 0; e < C::E; ++e)
                z[g] += acc_t(ag[e]) * xe[e];
        }
    }
}

// Function u's value folded into the key (see launch_keys).
template <typename T>
__device__ __forceinline__ void fold_value(uint64_t &key, T z, uint32_t u, uint32_t beta,
                                           uint64_t low, const int32_t *B, uint32_t f,
                                           int32_t w)
{
    if (w == 0) {
        key |= (uint64_t)(z >= T(0)) << u;
    } else {
        const double q = ((double)z + (double)B[f]) / (double)w;
        const int64_t v = (int64_t)floor(q);
        key |= ((uint64_t)v & low) << (beta * u);
    }
}

// A workgroup of 4 waves takes KROWS rows: it stages them in LDS in segments
// of KSEG bytes per row (coalesced loads; rows padded by 16 bytes so that the
// lanes' 16-byte reads of their own rows hit distinct banks) and each lane
// computes the keys of its row; wave v takes the tables v, v + 4, ...  Per
// table: z_f = sum_m A[f][m] x_m in ascending m (exact products; for
// fp16/bf16 a double sum in that order, for int8 an exact int32 sum), then the
// function values and the key (see launch_keys).  Rows of at
// most KSEG bytes are staged once for every table; longer rows once per table
// and segment, with the partial sums kept for at most 16 functions per pass.
template <int DT, bool LONG>
__global__ void __launch_bounds__(256) keys_kernel(Rows r, uint32_t d, uint32_t L, uint32_t k,
                                                   const typename Chunk<DT>::a_t *A,
                                                   const int32_t *B, int32_t w,
                                                   uint64_t *keys)
{
    typedef Chunk<DT> C;
    typedef typename C::acc_t acc_t;
    constexpr int RS = KSEG + 16;   // LDS row stride
    __shared__ __attribute__((aligned(16))) uint8_t xs[KROWS * RS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t row0 = blockIdx.x * KROWS;
    const uint32_t rows = min(r.n - row0, (uint32_t)KROWS);
    const uint32_t dp = padded_d<DT>(d);
    const uint32_t rb = dp * (DT == DT_I8 ? 1 : 2);   // bytes hashed per row (<= row_bytes)
    const uint32_t beta = k ? 64 / k : 64;
    const uint64_t low = beta >= 64 ? ~0ull : (1ull << beta) - 1;

    auto stage = [&](uint32_t seg0, uint32_t segb) {
        // segb bytes of every row from byte seg0; 16 bytes per lane per step
        const uint32_t cpr = segb / 16;
        for (uint32_t q = tid; q < KROWS * cpr; q += 256) {
            const uint32_t rr = q / cpr, cc = q - rr * cpr;
            i32x4 v = {0, 0, 0, 0};
            if (rr < rows)
                v = *(const i32x4 *)(r.X + (size_t)(row0 + rr) * r.row_bytes + seg0 + 16 * cc);
            *(i32x4 *)(xs + rr * RS + 16 * cc) = v;
        }
    };
    const uint8_t *mine = xs + lane * RS;
    if constexpr (!LONG) {
        if (rb)
            stage(0, rb);
        __syncthreads();
        const uint32_t nch = rb / 16;
        for (uint32_t t = wave; t < L; t += 4) {
            uint64_t key = 0ull;
            uint32_t u = 0;
            for (; u + 4 <= k; u += 4) {
                acc_t z[4] = {};
                project<DT, 4>(mine, nch, dp, A + (size_t)(t * k + u) * dp, z);
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    fold_value(key, z[g], u + g, beta, low, B, t * k + u + g, w);
            }
            if (u + 2 <= k) {
                acc_t z[2] = {};
                project<DT, 2>(mine, nch, dp, A + (size_t)(t * k + u) * dp, z);
#pragma unroll
                for (int g = 0; g < 2; ++g)
                    fold_value(key, z[g], u + g, beta, low, B, t * k + u + g, w);
                u += 2;
            }
            if (u < k) {
                acc_t z[1] = {};
                project<DT, 1>(mine, nch, dp, A + (size_t)(t * k + u) * dp, z);
                fold_value(key, z[0], u, beta, low, B, t * k + u, w);
            }
            if ((uint32_t)lane < rows)
                keys[(size_t)t * r.n + row0 + lane] = key;
        }
        return;
    } else {
    // long rows: segments of KSEG bytes, every wave takes table t = wave + 4 j
    // in turn (all waves pass every barrier: the table loop is uniform)
    const uint32_t tl = (L + 3) / 4 * 4;
    for (uint32_t t0 = 0; t0 < tl; t0 += 4) {
        const uint32_t t = t0 + wave;
        uint64_t key = 0ull;
        for (uint32_t u = 0; u < k; u += 16) {
            acc_t z[16] = {};
            for (uint32_t seg0 = 0; seg0 < rb; seg0 += KSEG) {
                const uint32_t segb = min(rb - seg0, (uint32_t)KSEG);
                __syncthreads();   // the previous segment is consumed
                stage(seg0, segb);
                __syncthreads();
                if (t < L) {
                    const typename C::a_t *a = A + (size_t)(t * k + u) * dp +
                                               seg0 / 16 * C::E;
                    if (u + 16 <= k)
                        project<DT, 16>(mine, segb / 16, dp, a, z);
                    else
#pragma unroll
                        for (int g = 0; g < 16; ++g)
                            if (u + g < k) {
                                acc_t zg[1] = {z[g]};
                                project<DT, 1>(mine, segb / 16, dp, a + (size_t)g * dp, zg);
                                z[g] = zg[0];
                            }
                }
            }
#pragma unroll
            for (int g = 0; g < 16; ++g)
                if (t < L && u + g < k)
                    fold_value(key, z[g], u + g, beta, low, B, t * k + u + g, w);
        }
        if (t < L && (uint32_t)lane < rows)
            keys[(size_t)t * r.n + row0 + lane] = key;
    }
    }
}

// ------------------------------------------------ keys on the matrix cores
//
// For rows of at most 512 bytes and at most HF_MAX functions in all: the
// projections z_f(x) of 32 rows by 32 functions come from one MFMA block
// (int8: exact int32 sums, so every decision is taken here; fp16 / bf16:
// products exact in fp32, sums rounded).  A
// decision (sign, or floor((z + B) / w)) is taken from the fp32 value only when
// it is certain: the fp32 sum and the double sum in ascending m both differ
// from the exact sum by at most gamma(d) sum_m |A_m x_m| <= gamma(d) ||A|| ||x||
// (any summation order; gamma(d) = d u / (1 - d u)), so when |z| exceeds twice
// the sum of both bounds the sign is the double sum's, and when the interval
// z +- that margin maps to one bucket the quantised value is.  A (row, table)
// with uncertain functions is queued with their mask, and fix_kernel computes
// those with the exact double evaluation, so the keys equal keys_kernel's.
constexpr int HF_MAX = 512;

template <int DT>
__global__ void widen_h_kernel(const int8_t *A, uint16_t *Ah, uint32_t d, uint32_t rl,
                               uint64_t n_out)
{
    const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n_out) {
        const uint64_t f = i / rl, m = i - f * rl;
        const float a = m < d ? (float)A[f * d + m] : 0.0f;   // |a| <= 128: exact in both
        if constexpr (DT == DT_F16)
            Ah[i] = __builtin_bit_cast(uint16_t, (_Float16)a);
        else
            Ah[i] = (uint16_t)(__builtin_bit_cast(uint32_t, a) >> 16);
    }
}

// int8 projection rows copied into rows of rb bytes (zero padded): the int8
// matrix cores' operand layout.
__global__ void pad_b_kernel(const int8_t *A, int8_t *Ab, uint32_t d, uint32_t rb,
                             uint64_t n_out)
{
    const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n_out) {
        const uint64_t f = i / rb, m = i - f * rb;
        Ab[i] = m < d ? A[f * d + m] : (int8_t)0;
    }
}

// Upper bounds of Euclidean norms: rows of A (int8, d entries) or of X
// (stored rows); the double sum is rounded up by a relative 2^-20.
__global__ void anorm_kernel(const int8_t *A, uint32_t d, uint32_t n_fn, float *out)
{
    const uint32_t f = blockIdx.x * 256 + threadIdx.x;
    if (f < n_fn) {
        double s = 0.0;
        for (uint32_t m = 0; m < d; ++m)
            s += (double)A[(uint64_t)f * d + m] * A[(uint64_t)f * d + m];
        out[f] = (float)(sqrt(s) * (1.0 + 0x1p-20));
    }
}

template <int DT>
__global__ void xnorm_kernel(Rows r, uint32_t d, float *out)
{
    const uint32_t row = blockIdx.x * 256 + threadIdx.x;
    if (row < r.n) {
        const uint8_t *x = r.X + (size_t)row * r.row_bytes;
        double s = 0.0;
        for (uint32_t c = 0; c < padded_d<DT>(d) / Chunk<DT>::E; ++c) {
            const i32x4 v = *(const i32x4 *)(x + 16 * c);
#pragma unroll
            for (int e = 0; e < Chunk<DT>::E; ++e) {
                const double xe = (double)Chunk<DT>::at(v, e);
                s += xe * xe;
            }
        }
        out[row] = (float)(sqrt(s) * (1.0 + 0x1p-20));
    }
}

// A wave takes 32 rows (A-fragments of KS k-steps in registers) and sweeps the
// L k functions in MFMA blocks of 32; each lane folds its function's value
// into the (row, table) key in LDS (64-bit atomic OR), and marks uncertain
// ones; then the wave writes the keys and queues each (row, table) with its
// mask of uncertain functions (one queue atomic per wave).
template <int DT, int KS>
__global__ void __launch_bounds__(256) keys_mfma_kernel(
    Rows r, uint32_t L, uint32_t k, const uint8_t *Ah, const float *anorm, const float *xnorm,
    const int32_t *B, int32_t w, float gam, uint64_t *keys, uint4 *fix,
    unsigned long long *nfix)
{
    typedef sjk::Mma<DT> M;
    typedef typename M::acc_t acc_t;
    __shared__ unsigned long long skey[4][32 * 64];
    __shared__ unsigned long long sunc[4][32][HF_MAX / 64];   // uncertain (row, function)
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int h = lane >> 5, c32 = lane & 31;
    const uint32_t row0 = (blockIdx.x * 4 + wave) * 32;
    const uint32_t nf = L * k;
    const uint32_t beta = 64 / k;
    const uint64_t low = beta >= 64 ? ~0ull : (1ull << beta) - 1;
    unsigned long long *kk = skey[wave];
    for (uint32_t i = lane; i < 32 * L; i += 64)
        kk[i] = 0ull;
    for (uint32_t i = lane; i < 32 * (HF_MAX / 64); i += 64)
        sunc[wave][i / (HF_MAX / 64)][i % (HF_MAX / 64)] = 0ull;
    i32x4 af[KS];
    const uint32_t arow = row0 + c32;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const uint32_t off = 32 * ks + 16 * h;
        af[ks] = arow < r.n && off < r.row_bytes
                     ? *(const i32x4 *)(r.X + (size_t)arow * r.row_bytes + off)
                     : i32x4{0, 0, 0, 0};
    }
    float xn[16] = {};
    if constexpr (DT != DT_I8) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const uint32_t R = row0 + 8 * (q >> 2) + 4 * h + (q & 3);
            xn[q] = R < r.n ? xnorm[R] : 0.0f;
        }
    }
    __builtin_amdgcn_wave_barrier();
    for (uint32_t f0 = 0; f0 < nf; f0 += 32) {
        const uint32_t f = f0 + c32;
        acc_t acc = acc_t{};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const uint32_t off = 32 * ks + 16 * h;
            const i32x4 b = f < nf && off < r.row_bytes
                                ? *(const i32x4 *)(Ah + (size_t)f * r.row_bytes + off)
                                : i32x4{0, 0, 0, 0};
            acc = M::mma(af[ks], b, acc);
        }
        if (f >= nf)
            continue;
        const uint32_t t = f / k, u = f - t * k;
        const float na = DT == DT_I8 ? 0.0f : anorm[f];
        const double bf = w > 0 ? (double)B[f] : 0.0;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int Rl = 8 * (q >> 2) + 4 * h + (q & 3);
            uint64_t contrib;
            bool sure;
            if constexpr (DT == DT_I8) {
                // int8 products summed exactly in int32: every decision is the
                // exact one (and the double evaluation's, which is exact too)
                const int32_t z = acc[q];
                sure = true;
                if (w == 0)
                    contrib = (uint64_t)(z >= 0) << u;
                else
                    contrib = ((uint64_t)(int64_t)floor(((double)z + bf) / (double)w) & low)
                              << (beta * u);
            } else {
                const float z = acc[q];
                const float e = gam * na * xn[q];
                if (w == 0) {
                    sure = __builtin_fabsf(z) > e;
                    contrib = (uint64_t)(z >= 0.0f) << u;
                } else {
                    const double lo = floor(((double)z - (double)e + bf) / (double)w);
                    const double hi = floor(((double)z + (double)e + bf) / (double)w);
                    sure = lo == hi;
                    contrib = ((uint64_t)(int64_t)lo & low) << (beta * u);
                }
            }
            if (sure)
                atomicOr(&kk[Rl * L + t], (unsigned long long)contrib);
            else
                atomicOr(&sunc[wave][Rl][f >> 6], 1ull << (f & 63));
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    // the uncertain functions of (row Rl, table t): bits t k .. t k + k - 1 of
    // the row's function mask
    auto umask = [&](uint32_t Rl, uint32_t t) -> uint64_t {
        const uint32_t b0 = t * k;
        const unsigned long long *m = sunc[wave][Rl];
        uint64_t v = m[b0 >> 6] >> (b0 & 63);
        if ((b0 & 63) != 0 && (b0 >> 6) + 1 < HF_MAX / 64)
            v |= m[(b0 >> 6) + 1] << (64 - (b0 & 63));
        return k >= 64 ? v : v & ((1ull << k) - 1);
    };
    // keys (certain bits), then the queue entries of the wave with one atomic
    uint32_t total = 0;
    for (uint32_t i0 = 0; i0 < 32 * L; i0 += 64) {
        const uint32_t i = i0 + lane;
        bool q = false;
        if (i < 32 * L) {
            const uint32_t Rl = i / L, t = i - Rl * L;
            const uint32_t R = row0 + Rl;
            if (R < r.n) {
                keys[(size_t)t * r.n + R] = kk[i];
                q = umask(Rl, t) != 0;
            }
        }
        total += (uint32_t)__popcll(__ballot(q));
    }
    if (total == 0)
        return;
    unsigned long long base = 0;
    if (lane == 0)
        base = atomicAdd(nfix, (unsigned long long)total);
    base = sjk::first_lane_u64(base);
    for (uint32_t i0 = 0; i0 < 32 * L; i0 += 64) {
        const uint32_t i = i0 + lane;
        uint64_t m = 0;
        uint32_t Rl = 0, t = 0;
        if (i < 32 * L) {
            Rl = i / L;
            t = i - Rl * L;
            if (row0 + Rl < r.n)
                m = umask(Rl, t);
        }
        const uint64_t bits = __ballot(m != 0);
        if (m != 0)
            fix[base + sjk::lanes_below(bits)] =
                make_uint4(row0 + Rl, t, (uint32_t)m, (uint32_t)(m >> 32));
        base += (uint32_t)__popcll(bits);
    }
}

// The queued (row, table) keys: the functions the matrix-core pass could not
// decide, recomputed exactly as keys_kernel does (the row read from global
// memory), OR-ed into the key (whose bits for them are still zero); one
// thread per entry, grid-stride over the queue's length read from device
// memory.
template <int DT>
__global__ void __launch_bounds__(256) fix_kernel(Rows r, uint32_t d, uint32_t k,
                                                  const typename Chunk<DT>::a_t *A,
                                                  const int32_t *B, int32_t w,
                                                  const uint4 *fix,
                                                  const unsigned long long *nfix, uint64_t *keys)
{
    typedef Chunk<DT> C;
    typedef typename C::acc_t acc_t;
    const uint64_t n_fix = *nfix;
    const uint32_t dp = padded_d<DT>(d), nch = dp / C::E;
    const uint32_t beta = k ? 64 / k : 64;
    const uint64_t low = beta >= 64 ? ~0ull : (1ull << beta) - 1;
    for (uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x; i < n_fix;
         i += (uint64_t)gridDim.x * 256) {
        const uint4 e = fix[i];
        const uint32_t row = e.x, t = e.y;
        uint64_t m = (uint64_t)e.z | ((uint64_t)e.w << 32);
        const uint8_t *x = r.X + (size_t)row * r.row_bytes;
        uint64_t key = 0;
        while (m) {
            const uint32_t u = (uint32_t)__builtin_ctzll(m);
            m &= m - 1;
            const typename C::a_t *a = A + (size_t)(t * k + u) * dp;
            acc_t z = acc_t(0);
            for (uint32_t c = 0; c < nch; ++c) {
                const i32x4 v = *(const i32x4 *)(x + 16 * c);
#pragma unroll
                for (int q = 0; q < C::E; ++q)
                    z += acc_t(a[c * C::E + q]) * C::at(v, q);
            }
            fold_value(key, z, u, beta, low, B, t * k + u, w);
        }
        keys[(size_t)t * r.n + row] |= key;
    }
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

// Position after the run of `key` that starts at p - 1 (keys ascending):
// doubling steps, then a binary search in the last step.
__device__ __forceinline__ uint32_t run_end(const uint64_t *s, uint32_t p, uint32_t n, uint64_t key)
{
    uint32_t lo = p, step = 1;
    while (lo + step <= n && s[lo + step - 1] == key) {
        lo += step;
        step *= 2;
    }
    return upper_bound(s, lo, min(lo + step, n), key);
}

// Per table and block of 256 sorted positions of P, the range of Q's sorted
// positions whose keys lie between the block's first and last keys: qr[t nb +
// b] = {first position with key >= the block's first, first with key > its
// last} (one thread each, so the searches of every block run at once).
__global__ void __launch_bounds__(256) qrange_kernel(const uint64_t *sorted_p, uint32_t n_p,
                                                     const uint64_t *sorted_q, uint32_t n_q,
                                                     uint32_t L, uint2 *qr)
{
    const uint32_t nb = (n_p + 255) / 256;
    const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (uint64_t)nb * L)
        return;
    const uint32_t t = (uint32_t)(i / nb), b = (uint32_t)(i - (uint64_t)t * nb);
    const uint64_t *sp = sorted_p + (size_t)t * n_p;
    const uint64_t *sq = sorted_q + (size_t)t * n_q;
    const uint32_t pf = 256 * b;
    qr[i] = make_uint2(lower_bound(sq, 0, n_q, sp[pf]),
                       upper_bound(sq, 0, n_q, sp[min(pf + 255, n_p - 1)]));
}

// One thread per (sorted position of P, table): a position that starts a P
// bucket looks its key up in Q's sorted keys within the block's range
// (qrange_kernel), staged in LDS when it holds at most QCAP keys, and, when Q
// has the key, marks the position with the bucket's sizes.
constexpr uint32_t QCAP = 2048;

__global__ void __launch_bounds__(256) bucket_find_kernel(const uint64_t *sorted_p, uint32_t n_p,
                                                          const uint64_t *sorted_q, uint32_t n_q,
                                                          const uint2 *qr, uint32_t *flag,
                                                          uint32_t *f_np, uint32_t *f_q0,
                                                          uint32_t *f_nq, ulonglong2 *part)
{
    __shared__ uint64_t s_q[QCAP];
    __shared__ unsigned long long s_cand[4], s_rows[4];
    const uint32_t t = blockIdx.y, tid = threadIdx.x;
    const uint32_t pf = blockIdx.x * 256, p = pf + tid;
    const uint64_t *sp = sorted_p + (size_t)t * n_p;
    const uint64_t *sq = sorted_q + (size_t)t * n_q;
    const uint2 range = qr[(size_t)t * gridDim.x + blockIdx.x];
    const uint32_t qa = range.x, qb = range.y;
    const bool staged = qb - qa <= QCAP;   // uniform
    if (staged) {
        for (uint32_t i = tid; i < qb - qa; i += 256)
            s_q[i] = sq[qa + i];
        __syncthreads();
    }
    uint64_t cand = 0, rows = 0;
    if (p < n_p) {
        const size_t at = (size_t)t * n_p + p;
        uint32_t fl = 0;
        const uint64_t key = sp[p];
        if (p == 0 || sp[p - 1] != key) {
            uint32_t q0, qe;
            if (staged) {
                // first position with key >= key, then first with key > key
                uint32_t lo = 0, hi = qb - qa;
                while (lo < hi) {
                    const uint32_t mid = lo + (hi - lo) / 2;
                    if (s_q[mid] < key)
                        lo = mid + 1;
                    else
                        hi = mid;
                }
                uint32_t e = lo;
                hi = qb - qa;
                while (e < hi) {
                    const uint32_t mid = e + (hi - e) / 2;
                    if (s_q[mid] <= key)
                        e = mid + 1;
                    else
                        hi = mid;
                }
                q0 = qa + lo;
                qe = qa + e;
            } else {
                q0 = lower_bound(sq, qa, qb, key);
                qe = upper_bound(sq, q0, qb, key);
            }
            if (q0 < qe) {
                const uint32_t np = run_end(sp, p + 1, n_p, key) - p;
                fl = 1;
                f_np[at] = np;
                f_q0[at] = q0;
                f_nq[at] = qe - q0;
                cand = (uint64_t)np * (qe - q0);
                rows = (uint64_t)np + (qe - q0);
            }
        }
        flag[at] = fl;
    }
    // the block's pair evaluations and rows, summed by sum_parts_kernel (one
    // counter updated by every block serialises the blocks on its address)
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        cand += __shfl_xor(cand, o, 64);
        rows += __shfl_xor(rows, o, 64);
    }
    if ((tid & 63) == 0) {
        s_cand[tid >> 6] = cand;
        s_rows[tid >> 6] = rows;
    }
    __syncthreads();
    if (tid == 0)
        part[(size_t)t * gridDim.x + blockIdx.x] =
            make_ulonglong2(s_cand[0] + s_cand[1] + s_cand[2] + s_cand[3],
                            s_rows[0] + s_rows[1] + s_rows[2] + s_rows[3]);
}

// One block of 1024 threads: out[0] = sum of the parts' pair evaluations,
// out[7] = sum of their rows (the counters' slots; written, not added to).
__global__ void __launch_bounds__(1024) sum_parts_kernel(const ulonglong2 *part, uint64_t n,
                                                         unsigned long long *out)
{
    __shared__ unsigned long long s_c[16], s_r[16];
    const uint32_t tid = threadIdx.x;
    unsigned long long c = 0, r = 0;
    for (uint64_t i = tid; i < n; i += 1024) {
        const ulonglong2 v = part[i];
        c += v.x;
        r += v.y;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        c += __shfl_xor(c, o, 64);
        r += __shfl_xor(r, o, 64);
    }
    if ((tid & 63) == 0) {
        s_c[tid >> 6] = c;
        s_r[tid >> 6] = r;
    }
    __syncthreads();
    if (tid == 0) {
        unsigned long long tc = 0, tr = 0;
        for (int w = 0; w < 16; ++w) {
            tc += s_c[w];
            tr += s_r[w];
        }
        out[0] = tc;
        out[7] = tr;
    }
}

__global__ void __launch_bounds__(256) bucket_write_kernel(uint32_t n_p, uint64_t total,
                                                           const uint32_t *flag,
                                                           const uint32_t *f_np,
                                                           const uint32_t *f_q0,
                                                           const uint32_t *f_nq,
                                                           const unsigned long long *rec_off,
                                                           Records rec)
{
    const uint64_t at = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (at >= total || !flag[at])
        return;
    const uint64_t r = rec_off[at];
    rec.t[r] = (uint32_t)(at / n_p);
    rec.pq[r] = make_uint4((uint32_t)(at % n_p), f_np[at], f_q0[at], f_nq[at]);
}

// One block per chunk of PACK_CHUNK records: the sizes go to LDS and the
// first thread walks them in order (greedy packing, see sj_lsh.h).
__global__ void __launch_bounds__(256) pack_kernel(Records rec, uint32_t n_rec, int write,
                                                   uint32_t *chunk_desc, uint32_t *chunk_tiles,
                                                   const unsigned long long *desc_off,
                                                   const unsigned long long *tile_off, Descs desc,
                                                   unsigned long long *overflow)
{
    static_assert(PACK_CHUNK == 256, "one record per thread");
    __shared__ uint4 spq[PACK_CHUNK];
    __shared__ uint32_t st[PACK_CHUNK];
    const uint32_t c = blockIdx.x, r0 = c * PACK_CHUNK, tid = threadIdx.x;
    const uint32_t rn = min((uint32_t)PACK_CHUNK, n_rec - r0);
    if (tid < rn) {
        spq[tid] = rec.pq[r0 + tid];
        st[tid] = rec.t[r0 + tid];
    }
    __syncthreads();
    if (tid != 0)
        return;
    const uint64_t dbase = write ? desc_off[c] : 0, tbase = write ? tile_off[c] : 0;
    uint32_t nd = 0;
    uint64_t nt = 0;
    uint32_t gs = 0, gp = 0, gq = 0, gc = 0;   // the open group: first, rows, records
    auto emit = [&](uint32_t first, uint32_t count, uint64_t tiles) {
        if (write) {
            desc.head[dbase + nd] = make_uint4(r0 + first, count, count ? 0u : st[first], 0u);
            if (count == 0)
                desc.pq[dbase + nd] = spq[first];
            desc.tile[dbase + nd] = tbase + nt;
        }
        ++nd;
        nt += tiles;
    };
    for (uint32_t i = 0; i < rn; ++i) {
        const uint32_t np = spq[i].y, nq = spq[i].w;
        if (np > TILE || nq > TILE) {
            if (gc) {
                emit(gs, gc, 1);
                gc = 0;
            }
            emit(i, 0, (uint64_t)((np + TILE - 1) / TILE) * ((nq + TILE - 1) / TILE));
            continue;
        }
        if (gc && (gp + np > TILE || gq + nq > TILE)) {
            emit(gs, gc, 1);
            gc = 0;
        }
        if (gc == 0) {
            gs = i;
            gp = gq = 0;
        }
        gp += np;
        gq += nq;
        ++gc;
    }
    if (gc)
        emit(gs, gc, 1);
    if (!write) {
        chunk_desc[c] = nd;
        chunk_tiles[c] = (uint32_t)min(nt, (uint64_t)0xffffffffu);
        if (nt > 0xffffffffull)
            atomicMax(overflow, 1ull);
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

// A workgroup of 4 waves takes a contiguous range of the tiles (see the
// descriptors in sj_lsh.h): a tile of a record tiled alone holds up to TILE
// of its P rows and TILE of its Q rows; a packed tile holds the P rows and
// the Q rows of a group of records, each row tagged with its record's place
// in the group, and only pairs with equal tags (the same bucket) are
// candidates.  The rows are gathered through the tables' sorted permutations
// into LDS in chunks of 128 bytes of each row (16-byte chunks, rows padded by
// one chunk), wave (wr, wc) multiplies its 64 x 64 quarter (2 x 2 blocks of
// 32 x 32: per k-step two A- and two B-fragments for four MFMAs) over the
// chunk's k-steps, and the epilogue applies the exact test to the candidates,
// drops pairs that share a bucket in an earlier table (so every pair is
// reported once) and appends the rest with one atomic per wave and block.
// With row records (REC) each row comes with its fingerprint and norm in one
// 128-byte line: the load of a row's 8 chunks brings all three into LDS.
template <int DT, int MET, bool REC>
__global__ void __launch_bounds__(256, 4) join_kernel(JoinArgs g)
{
    typedef sjk::Mma<DT> M;
    typedef typename M::acc_t acc_t;
    typedef typename M::val_t V;
    constexpr int CS = 9;            // LDS positions per tile row: 8 chunks + 1 pad
    constexpr int LPT = TILE / 32;   // rows each thread loads per operand and chunk
    __shared__ i32x4 sA[TILE * CS], sB[TILE * CS];
    __shared__ uint32_t sIP[TILE], sIQ[TILE];
    __shared__ V sNP[TILE], sNQ[TILE];
    __shared__ uint8_t sGP[TILE], sGQ[TILE];                 // row's record in the group
    __shared__ uint32_t sRT[TILE];                           // group record's table
    // With row records each wave stages up to OUTW of its pairs here and
    // reserves their slots with one atomic per flush (the records leave room
    // in LDS); otherwise it reserves once per tile with matches.
    constexpr uint32_t OUTW = REC ? 64 : 1;
    __shared__ uint64_t sOut[4][OUTW];
    // used only while a packed tile's row indices are gathered, before the
    // rows themselves go to sA: the group's row prefix sums and its records'
    // first positions
    uint2 *const sR0 = (uint2 *)sA;
    uint32_t *const sPS = (uint32_t *)(sR0 + TILE), *const sQS = sPS + (TILE + 1);
    static_assert(2 * TILE + 2 * (TILE + 1) <= TILE * CS * 4, "group tables fit sA");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1, half = lane >> 5, c32 = lane & 31;
    const uint32_t rb = g.P.row_bytes;   // == g.Q.row_bytes
    const uint32_t lc = tid & 7, lr = tid >> 3;   // load chunk; rows lr + 32 e
    // tables with a fingerprint byte: a record's chunks fc0 .. 6 hold 16 each
    // (fc0: past the k-steps' 32-byte reads of the row); otherwise the first 16
    const uint32_t fc0 = rec_fp_chunk(rb);
    const uint32_t FT = REC ? 16 * (7 - fc0) : 16u;

    // a contiguous range of tiles per workgroup: one search for the
    // descriptor of its first tile, then a walk
    const uint64_t per = (g.n_tiles + gridDim.x - 1) / gridDim.x;
    const uint64_t T0 = (uint64_t)blockIdx.x * per;
    const uint64_t T1 = min(T0 + per, g.n_tiles);
    if (T0 >= T1)
        return;   // the whole workgroup: no barrier is skipped by part of it
    uint32_t dsc = 0;
    {
        uint32_t hi = g.n_desc;
        while (hi - dsc > 1) {
            const uint32_t mid = (dsc + hi) >> 1;
            if (g.desc.tile[mid] <= T0)
                dsc = mid;
            else
                hi = mid;
        }
    }
    uint64_t local = T0 - g.desc.tile[dsc];
    uint32_t staged = 0;   // wave-uniform: pairs in sOut[wave]
    // one reservation for the wave's staged pairs, then each lane writes a
    // share of them
    auto flush = [&]() {
        unsigned long long base = 0;
        if (lane == 0)
            base = atomicAdd(g.counter, (unsigned long long)staged);
        base = sjk::first_lane_u64(base);
        for (uint32_t l = lane; l < staged; l += 64)
            if (base + l < g.cap)
                ((sjk::global_pair *)g.pairs)[base + l] = sOut[wave][l];
        staged = 0;
    };
    for (uint64_t T = T0; T < T1; ++T) {
        const uint4 hd = g.desc.head[dsc];
        const uint32_t first = hd.x, ngrp = hd.y;
        uint32_t rows_p, rows_q;
        __syncthreads();   // the previous tile's reads of the LDS tables are done
        if (ngrp == 0) {
            // a record tiled alone: sub-tile (tp, tq) of its ntp x ntq tiles
            const uint32_t t = hd.z;
            const uint4 rq = g.desc.pq[dsc];
            const uint32_t np = rq.y, nq = rq.w;
            const uint32_t ntq = (nq + TILE - 1) / TILE, ntp = (np + TILE - 1) / TILE;
            const uint32_t tp = (uint32_t)(local / ntq), tq = (uint32_t)(local % ntq);
            rows_p = min(np - tp * TILE, TILE);
            rows_q = min(nq - tq * TILE, TILE);
            if (++local == (uint64_t)ntp * ntq) {
                local = 0;
                ++dsc;
            }
            if (tid < (int)TILE) {
                const bool okp = (uint32_t)tid < rows_p;
                sIP[tid] = okp ? g.perm_p[(size_t)t * g.P.n + rq.x + tp * TILE + tid] : 0u;
                const bool okq = (uint32_t)tid < rows_q;
                sIQ[tid] = okq ? g.perm_q[(size_t)t * g.Q.n + rq.z + tq * TILE + tid] : 0u;
                sGP[tid] = 0;
                sGQ[tid] = 0;
                if (tid == 0)
                    sRT[0] = t;
            }
        } else {
            // a packed group of ngrp records, one tile: the records' row
            // counts, prefix-summed by the first two waves (ngrp <= TILE)
            ++dsc;
            local = 0;
            uint32_t np = 0, nq = 0;
            if (tid < (int)ngrp) {
                const uint4 rq = g.rec.pq[first + tid];
                np = rq.y;
                nq = rq.w;
                sRT[tid] = g.rec.t[first + tid];
                sR0[tid] = make_uint2(rq.x, rq.z);
            }
            uint32_t ip = np, iq = nq;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t up = __shfl_up(ip, o, 64), uq = __shfl_up(iq, o, 64);
                if (lane >= o) {
                    ip += up;
                    iq += uq;
                }
            }
            if (tid == 63) {
                sPS[TILE] = ip;   // first wave's totals, for the second wave
                sQS[TILE] = iq;
            }
            __syncthreads();
            if (tid >= 64 && tid < (int)TILE) {
                ip += sPS[TILE];
                iq += sQS[TILE];
            }
            __syncthreads();
            if (tid < (int)TILE) {
                sPS[tid + 1] = ip;   // inclusive sums: row prefix of record tid + 1
                sQS[tid + 1] = iq;
            }
            if (tid == 0)
                sPS[0] = sQS[0] = 0;
            __syncthreads();
            rows_p = sPS[ngrp];
            rows_q = sQS[ngrp];
            if (tid < (int)TILE) {
                // this thread's P row and Q row: the record holding it (the last
                // prefix at or below it), then its sorted position
                uint32_t gi = 0, gj = 0, lo, hi;
                if ((uint32_t)tid < rows_p) {
                    lo = 0, hi = ngrp;
                    while (hi - lo > 1) {
                        const uint32_t mid = (lo + hi) >> 1;
                        if (sPS[mid] <= (uint32_t)tid)
                            lo = mid;
                        else
                            hi = mid;
                    }
                    gi = lo;
                    sIP[tid] = g.perm_p[(size_t)sRT[gi] * g.P.n + sR0[gi].x + (tid - sPS[gi])];
                } else {
                    sIP[tid] = 0u;
                }
                if ((uint32_t)tid < rows_q) {
                    lo = 0, hi = ngrp;
                    while (hi - lo > 1) {
                        const uint32_t mid = (lo + hi) >> 1;
                        if (sQS[mid] <= (uint32_t)tid)
                            lo = mid;
                        else
                            hi = mid;
                    }
                    gj = lo;
                    sIQ[tid] = g.perm_q[(size_t)sRT[gj] * g.Q.n + sR0[gj].y + (tid - sQS[gj])];
                } else {
                    sIQ[tid] = 0u;
                }
                sGP[tid] = (uint8_t)gi;
                sGQ[tid] = (uint8_t)gj;
            }
        }
        __syncthreads();
        if constexpr (MET == MET_L2 && !REC) {
            if (tid < (int)TILE) {
                sNP[tid] = (uint32_t)tid < rows_p ? ((const V *)g.norm_p)[sIP[tid]] : V(0);
                sNQ[tid] = (uint32_t)tid < rows_q ? ((const V *)g.norm_q)[sIQ[tid]] : V(0);
            }
            __syncthreads();
        }
        const bool packed = ngrp != 0;

        acc_t acc[2][2];
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
                acc[a][b] = acc_t{};
        // rows are addressed through the tile's indices in LDS at every load
        // (no per-thread row pointers: fewer registers, four waves per SIMD)
        for (uint32_t kc = 0; kc < rb; kc += 128) {
            if constexpr (REC) {
                // whole records straight into LDS (one pass: rows of at most
                // REC_ROW bytes).  A wave's load fills 64 consecutive 16-byte
                // positions; position p holds chunk p % CS of the record of
                // tile row p / CS (the pad position reloads chunk 0).  Rows
                // past the tile's (index 0) load row 0: their results are
                // never read.
                constexpr int NLD = TILE * CS / 64;
#pragma unroll
                for (int k = 0; k < (NLD + 3) / 4; ++k) {
                    const int kk = 4 * k + wave;
                    if (kk < NLD) {
                        const uint32_t pos = 64 * kk + lane, row = pos / CS, ch = pos % CS;
                        const uint32_t cb = 16 * (ch == CS - 1 ? 0 : ch);
                        sjk::buffer_load_lds16(g.rec_p, g.P.n * REC_BYTES, sIP[row] * REC_BYTES + cb,
                                               (uint8_t *)sA + 1024 * kk);
                        sjk::buffer_load_lds16(g.rec_q, g.Q.n * REC_BYTES, sIQ[row] * REC_BYTES + cb,
                                               (uint8_t *)sB + 1024 * kk);
                    }
                }
                __builtin_amdgcn_s_waitcnt(0);   // this wave's loads landed
                __syncthreads();
            } else {
                const uint32_t off = kc + 16 * lc;
                const i32x4 z = {0, 0, 0, 0};
                const bool in = off < rb;
                i32x4 la[LPT], lb[LPT];
#pragma unroll
                for (int e = 0; e < LPT; ++e) {
                    const uint32_t rr = lr + 32 * e;
                    la[e] = rr < rows_p && in
                                ? *(const i32x4 *)(g.P.X + (size_t)sIP[rr] * rb + off) : z;
                    lb[e] = rr < rows_q && in
                                ? *(const i32x4 *)(g.Q.X + (size_t)sIQ[rr] * rb + off) : z;
                }
                if (kc)
                    __syncthreads();   // the previous chunk's fragments are read
#pragma unroll
                for (int e = 0; e < LPT; ++e) {
                    sA[(lr + 32 * e) * CS + lc] = la[e];
                    sB[(lr + 32 * e) * CS + lc] = lb[e];
                }
                __syncthreads();
            }
            const uint32_t nks = min(4u, (rb - kc + 31) / 32);
#pragma unroll
            for (uint32_t ks = 0; ks < 4; ++ks)
                if (ks < nks) {
                    i32x4 fa[2], fb[2];
#pragma unroll
                    for (int a = 0; a < 2; ++a) {
                        fa[a] = sA[(wr * 64 + 32 * a + c32) * CS + 2 * ks + half];
                        fb[a] = sB[(wc * 64 + 32 * a + c32) * CS + 2 * ks + half];
                    }
#pragma unroll
                    for (int a = 0; a < 2; ++a)
#pragma unroll
                        for (int b = 0; b < 2; ++b)
                            acc[a][b] = M::mma(fa[a], fb[b], acc[a][b]);
                }
        }

        // epilogue.  Result register r of block (a, b) of this lane is (row
        // wr*64 + 32a + 8(r/4) + 4 half + r%4, column wc*64 + 32b + c32).
        // First the exact test of every result (in a packed tile also the
        // bucket tags of its matches); then, only in a wave with a match, the
        // first-table rule from the rows' key fingerprints, which the wave
        // stages in the operand LDS the MFMAs no longer read.
        // A record's norm is the first word of its chunk 7, its fingerprints
        // chunks fc0..6 (the MFMAs read only the row's chunks).
        auto norm_p = [&](uint32_t il) {
            if constexpr (REC)
                return *(const V *)&sA[il * CS + 7];
            else
                return sNP[il];
        };
        auto norm_q = [&](uint32_t jl) {
            if constexpr (REC)
                return *(const V *)&sB[jl * CS + 7];
            else
                return sNQ[jl];
        };
        uint32_t mk[2][2];
        bool any = false;
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const uint32_t jl = wc * 64 + 32 * b + c32;
            const bool jok = jl < rows_q;
            const V ny = MET == MET_L2 ? norm_q(jl) : V(0);
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                const uint32_t ib = wr * 64 + 32 * a + 4 * half;
                uint32_t m = 0;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const uint32_t il = ib + 8 * (r >> 2) + (r & 3);
                    const V nx = MET == MET_L2 ? norm_p(il) : V(0);
                    const bool ok = jok && il < rows_p && matches<DT, MET>(acc[a][b][r], nx, ny, g);
                    m |= ok ? (1u << r) : 0u;
                }
                mk[a][b] = m;
                any |= m != 0;
            }
        }
        if constexpr (!REC)
            __syncthreads();   // every wave's MFMAs are done with sA and sB
        if (__ballot(any) == 0)
            continue;
        uint4 *const wf = (uint4 *)sA + wave * 128;   // fingerprints: 64 P rows, 64 Q rows
        if (!REC && g.L > 1) {
            const uint32_t pr = wr * 64 + lane, qr = wc * 64 + lane;
            const uint4 z4 = make_uint4(0u, 0u, 0u, 0u);
            wf[lane] = pr < rows_p ? g.fp_p[sIP[pr]] : z4;
            wf[64 + lane] = qr < rows_q ? g.fp_q[sIQ[qr]] : z4;
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        }
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const uint32_t jl = wc * 64 + 32 * b + c32;
            const uint32_t j = sIQ[jl];
            const uint32_t gq = sGQ[jl];
            const uint32_t t = sRT[gq];   // the pair's table (its bucket's)
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                const uint32_t ib = wr * 64 + 32 * a + 4 * half;
                uint32_t m = mk[a][b];
                if (__ballot(m != 0) == 0)
                    continue;
                if (packed) {
                    // candidates of a packed tile: rows of the same bucket
                    uint32_t mm = m;
                    while (mm) {
                        const int r = __builtin_ctz(mm);
                        mm &= mm - 1;
                        if (sGP[ib + 8 * (r >> 2) + (r & 3)] != gq)
                            m &= ~(1u << r);
                    }
                }
                if (t > 0 && m != 0) {
                    // the first-table rule: drop the pair when its keys agree
                    // in an earlier table.  Tables below FT by fingerprint (a
                    // byte per table; equal keys give equal bytes), each equal
                    // byte confirmed with the keys; later tables by their
                    // keys, 8 tables per round of independent loads.
                    const uint32_t tf = t < FT ? t : FT;
                    uint32_t mm = m;
                    while (mm) {
                        const int r = __builtin_ctz(mm);
                        mm &= mm - 1;
                        const uint32_t il = ib + 8 * (r >> 2) + (r & 3);
                        const uint32_t i = sIP[il];
                        bool same = false;
                        for (uint32_t c = 0; 16 * c < tf && !same; ++c) {
                            const uint4 fi = REC ? ((const uint4 *)sA)[il * CS + fc0 + c]
                                                 : wf[il - wr * 64];
                            const uint4 fj = REC ? ((const uint4 *)sB)[jl * CS + fc0 + c]
                                                 : wf[64 + (jl - wc * 64)];
                            const uint32_t xw[4] = {fi.x ^ fj.x, fi.y ^ fj.y, fi.z ^ fj.z,
                                                    fi.w ^ fj.w};
                            uint32_t eq = 0;   // bit u: byte u (table 16 c + u) equal
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                const uint32_t x = xw[q];
                                const uint32_t y =
                                    ~(((x & 0x7f7f7f7fu) + 0x7f7f7f7fu) | x | 0x7f7f7f7fu);
                                eq |= (((y >> 7) & 1u) | ((y >> 14) & 2u) | ((y >> 21) & 4u) |
                                       ((y >> 28) & 8u)) << (4 * q);
                            }
                            const uint32_t rem = tf - 16 * c;
                            eq &= rem >= 16 ? 0xffffu : (1u << rem) - 1u;
                            while (eq && !same) {
                                const uint32_t t2 = 16 * c + __builtin_ctz(eq);
                                eq &= eq - 1;
                                same = g.keys_p[(size_t)t2 * g.P.n + i] ==
                                       g.keys_q[(size_t)t2 * g.Q.n + j];
                            }
                        }
                        for (uint32_t t2 = FT; t2 < t && !same; t2 += 8) {
#pragma unroll
                            for (uint32_t u = 0; u < 8; ++u) {
                                const uint32_t tt = t2 + u < t ? t2 + u : t - 1;
                                same |= g.keys_p[(size_t)tt * g.P.n + i] ==
                                        g.keys_q[(size_t)tt * g.Q.n + j];
                            }
                        }
                        if (same)
                            m &= ~(1u << r);
                    }
                }
                mk[a][b] = m;
            }
        }
        // one slot reservation for the wave's matches of the whole tile: the
        // lanes' counts (at most 64) give the wave's total and each lane's
        // prefix through seven ballots, and each lane writes its pairs in
        // (block, register) order
        const uint32_t cnt = (uint32_t)(__builtin_popcount(mk[0][0]) + __builtin_popcount(mk[1][0]) +
                                        __builtin_popcount(mk[0][1]) + __builtin_popcount(mk[1][1]));
        uint32_t tot = 0, pre = 0;
#pragma unroll
        for (int bit = 0; bit < 7; ++bit) {
            const uint64_t bits = __ballot((cnt >> bit) & 1);
            tot += (uint32_t)__popcll(bits) << bit;
            pre += sjk::lanes_below(bits) << bit;
        }
        if (tot == 0)
            continue;
        if constexpr (REC) {
            if (staged + tot > OUTW) {
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                flush();
            }
            if (tot <= OUTW) {
                // stage: each lane's pairs at its prefix, in (block, register) order
                uint32_t at = staged + pre;
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    const uint32_t j = sIQ[wc * 64 + 32 * b + c32];
#pragma unroll
                    for (int a = 0; a < 2; ++a) {
                        const uint32_t ib = wr * 64 + 32 * a + 4 * half;
                        uint32_t m = mk[a][b];
                        while (m) {
                            const int r = __builtin_ctz(m);
                            m &= m - 1;
                            sOut[wave][at++] = sjk::pack_pair(sIP[ib + 8 * (r >> 2) + (r & 3)], j);
                        }
                    }
                }
                staged += tot;
                continue;
            }
        }
        unsigned long long base = 0;
        if (lane == 0)
            base = atomicAdd(g.counter, (unsigned long long)tot);
        uint64_t pos = sjk::first_lane_u64(base) + pre;
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const uint32_t j = sIQ[wc * 64 + 32 * b + c32];
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                const uint32_t ib = wr * 64 + 32 * a + 4 * half;
                uint32_t m = mk[a][b];
                while (m) {
                    const int r = __builtin_ctz(m);
                    m &= m - 1;
                    if (pos < g.cap) {
                        const uint32_t i = sIP[ib + 8 * (r >> 2) + (r & 3)];
                        ((sjk::global_pair *)g.pairs)[pos] = sjk::pack_pair(i, j);
                    }
                    ++pos;
                }
            }
        }
    }
    if constexpr (REC) {
        if (staged) {
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            flush();
        }
    }
}

// Fingerprints of the keys of the first min(L, 16) tables: byte t of fp[row]
// is the top byte of keys[t n + row] times an odd constant, so rows with equal
// keys in table t have equal bytes t (and rows with different keys rarely do).
__global__ void __launch_bounds__(256) fingerprint_kernel(const uint64_t *keys, uint32_t n,
                                                          uint32_t L, uint4 *fp)
{
    const uint32_t row = blockIdx.x * 256 + threadIdx.x;
    if (row >= n)
        return;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    const uint32_t tl = L < 16 ? L : 16;
    for (uint32_t t = 0; t < tl; ++t) {
        const uint32_t byte = (uint32_t)((keys[(size_t)t * n + row] * 0x9E3779B97F4A7C15ull) >> 56);
        w[t >> 2] |= byte << (8 * (t & 3));
    }
    fp[row] = make_uint4(w[0], w[1], w[2], w[3]);
}

// Row records (sj_lsh.h): thread per row (the lanes' key loads are
// coalesced over consecutive rows).  Chunk c in fc0 .. 6 holds the
// fingerprint bytes of tables 16 (c - fc0) .. + 15 (byte u: the top byte of
// the table's key times an odd constant), chunk 7 the norm.
__global__ void __launch_bounds__(256) rowrec_kernel(Rows r, const uint32_t *norm,
                                                     const uint64_t *keys, uint32_t L, i32x4 *out)
{
    const uint32_t row = blockIdx.x * 256 + threadIdx.x;
    if (row >= r.n)
        return;
    const uint32_t fc0 = rec_fp_chunk(r.row_bytes);
    i32x4 *o = out + (size_t)row * (REC_BYTES / 16);
    for (uint32_t c = 0; c < REC_BYTES / 16; ++c) {
        i32x4 v = {0, 0, 0, 0};
        if (16 * c < r.row_bytes) {
            v = *(const i32x4 *)(r.X + (size_t)row * r.row_bytes + 16 * c);
        } else if (c >= fc0 && c < 7) {
            const uint32_t t0 = 16 * (c - fc0);
            uint32_t w[4] = {0u, 0u, 0u, 0u};
            for (uint32_t u = 0; u < 16 && t0 + u < L; ++u) {
                const uint32_t byte =
                    (uint32_t)((keys[(size_t)(t0 + u) * r.n + row] * 0x9E3779B97F4A7C15ull) >> 56);
                w[u >> 2] |= byte << (8 * (u & 3));
            }
            v = i32x4{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
        } else if (c == 7 && norm) {
            v[0] = (int)norm[row];
        }
        o[c] = v;
    }
}

template <int DT>
hipError_t launch_keys_t(const Rows &r, uint32_t d, uint32_t L, uint32_t k, const void *Aw,
                         const int32_t *B, int32_t w, uint64_t *keys,
                         hipStream_t s)
{
    const dim3 grid((r.n + KROWS - 1) / KROWS);
    const uint32_t rb = padded_d<DT>(d) * (DT == DT_I8 ? 1 : 2);
    if (rb <= KSEG)
        hipLaunchKernelGGL((keys_kernel<DT, false>), grid, dim3(256), 0, s, r, d, L, k,
                           (const typename Chunk<DT>::a_t *)Aw, B, w, keys);
    else
        hipLaunchKernelGGL((keys_kernel<DT, true>), grid, dim3(256), 0, s, r, d, L, k,
                           (const typename Chunk<DT>::a_t *)Aw, B, w, keys);
    return hipGetLastError();
}

template <int DT, int MET>
hipError_t launch_join_t(const JoinArgs &g, int num_cus, hipStream_t s)
{
    const uint64_t want = (uint64_t)num_cus * 8;
    const uint32_t grid = (uint32_t)(g.n_tiles < want ? g.n_tiles : want);
    if (g.rec_p)
        hipLaunchKernelGGL((join_kernel<DT, MET, true>), dim3(grid), dim3(256), 0, s, g);
    else
        hipLaunchKernelGGL((join_kernel<DT, MET, false>), dim3(grid), dim3(256), 0, s, g);
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

size_t widened_bytes(int dtype, uint32_t L, uint32_t k, uint32_t d)
{
    return dtype == DT_I8 ? (size_t)L * k * padded_d<DT_I8>(d) * 4
                          : (size_t)L * k * padded_d<DT_F16>(d) * 8;
}

hipError_t launch_keys(int dtype, const Rows &r, uint32_t d, uint32_t L, uint32_t k,
                       const void *Aw, const int32_t *B, int32_t w,
                       uint64_t *keys, hipStream_t s)
{
    if (r.n == 0 || L == 0)
        return hipSuccess;
    switch (dtype) {
    case DT_F16:
        return launch_keys_t<DT_F16>(r, d, L, k, Aw, B, w, keys, s);
    case DT_BF16:
        return launch_keys_t<DT_BF16>(r, d, L, k, Aw, B, w, keys, s);
    default:
        return launch_keys_t<DT_I8>(r, d, L, k, Aw, B, w, keys, s);
    }
}

bool keys_fast_applies(int dtype, uint32_t row_bytes, uint32_t L, uint32_t k, int32_t w)
{
    return row_bytes <= 512 && k >= 1 &&
           (uint64_t)L * k <= HF_MAX && L <= 64 && (w == 0 || k >= 2);
}

size_t keys_fast_bytes(uint32_t n_max, uint32_t L, uint32_t k, uint32_t row_bytes)
{
    // fp16 / bf16 projection rows, their norms, row norms, the fix queue
    return (size_t)L * k * row_bytes + 256 + (size_t)L * k * 4 + 256 + (size_t)n_max * 4 + 256 +
           (size_t)L * n_max * 16;
}

template <int DT, int KS>
static void launch_mfma_t(const Rows &r, uint32_t L, uint32_t k, const uint8_t *Ah,
                          const float *an, const float *xn, const int32_t *B, int32_t w, float gam, uint64_t *keys, uint4 *fix,
                          unsigned long long *nfix, hipStream_t s)
{
    hipLaunchKernelGGL((keys_mfma_kernel<DT, KS>), dim3((r.n + 127) / 128), dim3(256), 0, s, r,
                       L, k, Ah, an, xn, B, w, gam, keys, fix, nfix);
}

template <int DT>
static hipError_t keys_fast_t(const Rows &r, uint32_t d, uint32_t L, uint32_t k,
                              const int8_t *A, const void *Aw, const int32_t *B, int32_t w, uint64_t *keys, uint8_t *ws, bool widen,
                              unsigned long long *nfix, hipStream_t s)
{
    const uint32_t nf = L * k;
    uint8_t *Ah = ws;
    float *an = (float *)(ws + (((size_t)nf * r.row_bytes + 255) & ~(size_t)255));
    float *xn = (float *)((uint8_t *)an + (((size_t)nf * 4 + 255) & ~(size_t)255));
    uint4 *fix = (uint4 *)((uint8_t *)xn + (((size_t)r.n * 4 + 255) & ~(size_t)255));
    if constexpr (DT == DT_I8) {
        // the projection rows as int8 operand rows; sums exact: no norms, no queue
        if (widen) {
            const uint64_t n_out = (uint64_t)nf * r.row_bytes;
            hipLaunchKernelGGL(pad_b_kernel, dim3((unsigned)((n_out + 255) / 256)), dim3(256), 0,
                               s, A, (int8_t *)Ah, d, r.row_bytes, n_out);
        }
    } else {
        if (widen) {
            const uint32_t rl = r.row_bytes / 2;
            const uint64_t n_out = (uint64_t)nf * rl;
            hipLaunchKernelGGL(widen_h_kernel<DT>, dim3((unsigned)((n_out + 255) / 256)),
                               dim3(256), 0, s, A, (uint16_t *)Ah, d, rl, n_out);
            hipLaunchKernelGGL(anorm_kernel, dim3((nf + 255) / 256), dim3(256), 0, s, A, d, nf,
                               an);
        }
        hipLaunchKernelGGL(xnorm_kernel<DT>, dim3((r.n + 255) / 256), dim3(256), 0, s, r, d, xn);
    }
    // twice the fp32 and double summation bounds for d terms
    const double dd = d ? (double)d : 1.0;
    const double g24 = dd * 0x1p-24 / (1.0 - dd * 0x1p-24);
    const double g53 = dd * 0x1p-53 / (1.0 - dd * 0x1p-53);
    const float gam = (float)(2.0 * (g24 + g53) * (1.0 + 0x1p-10));
    const uint32_t ks = (r.row_bytes + 31) / 32;
    if (ks <= 2)
        launch_mfma_t<DT, 2>(r, L, k, Ah, an, xn, B, w, gam, keys, fix, nfix, s);
    else if (ks <= 4)
        launch_mfma_t<DT, 4>(r, L, k, Ah, an, xn, B, w, gam, keys, fix, nfix, s);
    else if (ks <= 8)
        launch_mfma_t<DT, 8>(r, L, k, Ah, an, xn, B, w, gam, keys, fix, nfix, s);
    else
        launch_mfma_t<DT, 16>(r, L, k, Ah, an, xn, B, w, gam, keys, fix, nfix, s);
    if constexpr (DT != DT_I8)
        hipLaunchKernelGGL(fix_kernel<DT>, dim3(512), dim3(256), 0, s, r, d, k,
                           (const typename Chunk<DT>::a_t *)Aw, B, w, fix,
                           (const unsigned long long *)nfix, keys);
    return hipGetLastError();
}

hipError_t launch_keys_fast(int dtype, const Rows &r, uint32_t d, uint32_t L, uint32_t k,
                            const int8_t *A, const void *Aw, const int32_t *B, int32_t w, uint64_t *keys, void *ws, bool widen,
                            unsigned long long *nfix, hipStream_t s)
{
    if (r.n == 0)
        return hipSuccess;
    if (dtype == DT_F16)
        return keys_fast_t<DT_F16>(r, d, L, k, A, Aw, B, w, keys, (uint8_t *)ws, widen,
                                   nfix, s);
    if (dtype == DT_I8)
        return keys_fast_t<DT_I8>(r, d, L, k, A, Aw, B, w, keys, (uint8_t *)ws, widen,
                                  nfix, s);
    return keys_fast_t<DT_BF16>(r, d, L, k, A, Aw, B, w, keys, (uint8_t *)ws, widen,
                                nfix, s);
}

hipError_t launch_widen(int dtype, const int8_t *A, uint32_t n_fn, uint32_t d, void *out,
                        hipStream_t s)
{
    const uint32_t dp = dtype == DT_I8 ? padded_d<DT_I8>(d) : padded_d<DT_F16>(d);
    const uint64_t n = (uint64_t)n_fn * dp;
    if (n == 0)
        return hipSuccess;
    const dim3 grid((unsigned)((n + 255) / 256));
    if (dtype == DT_I8)
        hipLaunchKernelGGL(widen_kernel<int32_t>, grid, dim3(256), 0, s, A, (int32_t *)out, d,
                           dp, n);
    else
        hipLaunchKernelGGL(widen_kernel<double>, grid, dim3(256), 0, s, A, (double *)out, d, dp,
                           n);
    return hipGetLastError();
}

hipError_t launch_fingerprints(const uint64_t *keys, uint32_t n, uint32_t L, uint4 *fp,
                               hipStream_t s)
{
    if (n == 0)
        return hipSuccess;
    hipLaunchKernelGGL(fingerprint_kernel, dim3((n + 255) / 256), dim3(256), 0, s, keys, n, L, fp);
    return hipGetLastError();
}

hipError_t launch_rowrec(const Rows &r, const void *norm, const uint64_t *keys, uint32_t L,
                         uint8_t *out, hipStream_t s)
{
    if (r.n == 0)
        return hipSuccess;
    if (r.row_bytes > REC_ROW)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(rowrec_kernel, dim3((r.n + 255) / 256), dim3(256), 0, s, r,
                       (const uint32_t *)norm, keys, L, (i32x4 *)out);
    return hipGetLastError();
}

hipError_t launch_bucket_find(const uint64_t *sorted_p, uint32_t n_p, const uint64_t *sorted_q,
                              uint32_t n_q, uint32_t L, void *ws, uint32_t *flag, uint32_t *f_np,
                              uint32_t *f_q0, uint32_t *f_nq, unsigned long long *n_cand,
                              hipStream_t s)
{
    if (n_p == 0 || n_q == 0 || L == 0)
        return hipSuccess;
    const uint32_t nb = (n_p + 255) / 256;
    const uint64_t nr = (uint64_t)nb * L;
    // workspace: the block sums, then the block ranges of Q
    ulonglong2 *part = (ulonglong2 *)ws;
    uint2 *qr = (uint2 *)(part + nr);
    hipLaunchKernelGGL(qrange_kernel, dim3((uint32_t)((nr + 255) / 256)), dim3(256), 0, s,
                       sorted_p, n_p, sorted_q, n_q, L, qr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(bucket_find_kernel, dim3(nb, L), dim3(256), 0, s, sorted_p, n_p, sorted_q,
                       n_q, (const uint2 *)qr, flag, f_np, f_q0, f_nq, part);
    e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(sum_parts_kernel, dim3(1), dim3(1024), 0, s, (const ulonglong2 *)ws,
                       (uint64_t)nb * L, n_cand);
    return hipGetLastError();
}

hipError_t launch_bucket_write(uint32_t n_p, uint32_t L, const uint32_t *flag,
                               const uint32_t *f_np, const uint32_t *f_q0, const uint32_t *f_nq,
                               const unsigned long long *rec_off, const Records &rec,
                               hipStream_t s)
{
    const uint64_t total = (uint64_t)n_p * L;
    if (total == 0)
        return hipSuccess;
    hipLaunchKernelGGL(bucket_write_kernel, dim3((uint32_t)((total + 255) / 256)), dim3(256), 0,
                       s, n_p, total, flag, f_np, f_q0, f_nq, rec_off, rec);
    return hipGetLastError();
}

hipError_t launch_pack(const Records &rec, uint32_t n_rec, bool write, uint32_t *chunk_desc,
                       uint32_t *chunk_tiles, const unsigned long long *desc_off,
                       const unsigned long long *tile_off, const Descs &desc,
                       unsigned long long *overflow, hipStream_t s)
{
    if (n_rec == 0)
        return hipSuccess;
    hipLaunchKernelGGL(pack_kernel, dim3((n_rec + PACK_CHUNK - 1) / PACK_CHUNK), dim3(256), 0, s,
                       rec, n_rec, write ? 1 : 0, chunk_desc, chunk_tiles, desc_off, tile_off,
                       desc, overflow);
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
