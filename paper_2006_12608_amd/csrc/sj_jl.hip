// sj_jl.hip -- the TCU Johnson-Lindenstrauss transform of Ahle & Silvestri,
// "Similarity Search with Tensor Core Units", Lemma 3 / Theorem 2, on gfx950.
//
// M = (I_{r_l} (x) A_l) ... (I_{r_1} (x) A_1): since I_r (x) A is A copied
// r times along the diagonal, a batch of n row vectors of length r_i c_i,
// read as n r_i rows of c_i entries, is multiplied by A_i^T as one dense
// product, and the result (n r_i rows of k_i entries) read back as n rows of
// r_i k_i entries is the next level's input -- no data moves between levels.
// Each level is one fp32 product Y = X A_i^T on the matrix cores
// (v_mfma_f32_32x32x2_f32) with its operands staged through LDS; the first
// level decodes fp16 / bf16 / int8 rows exactly to fp32.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sj_internal.h"

namespace sjj {

using sjk::DT_BF16;
using sjk::DT_F16;
using sjk::DT_I8;

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int SRC_F32 = 0;

// Rows per workgroup tile and entries of K per LDS chunk (the column blocks
// of 32 a wave keeps accumulators for at once, NCB, are a template argument:
// as many as the level's N needs, up to 4).
constexpr int NCBMAX = 4;
constexpr int TR = 128;
constexpr int KC = 32;
constexpr int XS = KC + 1;   // LDS row stride (floats): lanes of a fragment read distinct banks

// Raw source bits of one entry / four consecutive entries (idx a multiple
// of 4, the row 4-entry aligned), decoded by dec1 / dec4 once they are used:
// loads in flight hold only the raw words.
template <int SRC>
__device__ __forceinline__ uint32_t raw1(const void *X, uint64_t idx)
{
    if constexpr (SRC == SRC_F32)
        return __builtin_bit_cast(uint32_t, ((const float *)X)[idx]);
    else if constexpr (SRC == DT_I8)
        return (uint32_t)(uint8_t)((const int8_t *)X)[idx];
    else
        return ((const uint16_t *)X)[idx];
}

template <int SRC>
__device__ __forceinline__ float dec1(uint32_t w)
{
    if constexpr (SRC == SRC_F32)
        return __builtin_bit_cast(float, w);
    else if constexpr (SRC == DT_I8)
        return (float)(int8_t)w;
    else if constexpr (SRC == DT_F16)
        return (float)__builtin_bit_cast(_Float16, (uint16_t)w);
    else
        return __builtin_bit_cast(float, w << 16);
}

template <int SRC>
__device__ __forceinline__ uint4 raw4(const void *X, uint64_t idx)
{
    if constexpr (SRC == SRC_F32) {
        return *(const uint4 *)((const float *)X + idx);
    } else if constexpr (SRC == DT_I8) {
        return make_uint4(*(const uint32_t *)((const int8_t *)X + idx), 0u, 0u, 0u);
    } else {
        const uint2 w = *(const uint2 *)((const uint16_t *)X + idx);
        return make_uint4(w.x, w.y, 0u, 0u);
    }
}

template <int SRC>
__device__ __forceinline__ void dec4(uint4 w, float (&v)[4])
{
    if constexpr (SRC == SRC_F32) {
        v[0] = __builtin_bit_cast(float, w.x), v[1] = __builtin_bit_cast(float, w.y);
        v[2] = __builtin_bit_cast(float, w.z), v[3] = __builtin_bit_cast(float, w.w);
    } else if constexpr (SRC == DT_I8) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            v[j] = (float)(int8_t)(w.x >> (8 * j));
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            v[j] = dec1<SRC>(((j < 2 ? w.x : w.y) >> (16 * (j & 1))) & 0xffffu);
    }
}

// Y (rows x N, fp32) = X (rows x K) A^T, A N x K fp32 row-major.  A workgroup
// of 4 waves owns TR rows; for each group of NCB column blocks it walks K in
// chunks of KC entries, staging the chunk of its TR rows and of the group's
// rows of A in LDS as fp32 (consecutive threads load consecutive entries of
// a row: coalesced), and wave w multiplies rows 32 w .. 32 w + 31 on the
// matrix cores (per k-step, lane l supplies X[row l % 32][k + l / 32] and
// A[column l % 32][k + l / 32]).  The next chunk's entries are loaded into
// registers (raw) while the current chunk's MFMAs run.  Entries past the
// matrices read as zero; results outside rows x N are not stored.
template <int SRC, bool VEC, int NCB>
__global__ void __launch_bounds__(256, NCB >= 4 ? 2 : 4) jl_level(const void *X, uint64_t rows, uint32_t K,
                                                   const float *A, uint32_t N, float *Y)
{
    __shared__ float sx[TR * XS];
    __shared__ float sa[32 * NCB * XS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = lane >> 5, c32 = lane & 31;
    const uint64_t tile0 = (uint64_t)blockIdx.x * TR;
    const uint64_t row0 = tile0 + 32 * wave;
    // per thread: XQ quads (VEC) or XE entries of X, AE entries of A per chunk
    constexpr int XQ = TR * KC / 4 / 256, XE = TR * KC / 256, AE = 32 * NCB * KC / 256;
    for (uint32_t cb0 = 0; cb0 < N; cb0 += 32 * NCB) {
        // only the column blocks this group uses (whole blocks of 32 rows)
        const uint32_t arows = min((N - cb0 + 31) / 32 * 32, 32u * NCB);
        uint4 rq[VEC ? XQ : 1];
        uint32_t re[VEC ? 1 : XE];
        float ra[AE];
        // this thread's entries: X rows xr + XRS u at column xc (quads: 4
        // entries from xc), A rows ar + 8 u at column ac; element indices from
        // one base per chunk (opaque to the optimiser, so the per-load
        // addresses are not all computed up front and kept)
        constexpr uint32_t XRS = VEC ? 256 / (KC / 4) : 256 / KC;
        const uint32_t xr = VEC ? tid / (KC / 4) : tid / KC;
        const uint32_t xc = VEC ? 4 * (tid % (KC / 4)) : tid % KC;
        const uint32_t ar = tid / KC, ac = tid % KC;
        auto fetch = [&](uint32_t k0) {
            uint64_t xb = (tile0 + xr) * K + k0 + xc;
            asm volatile("" : "+v"(xb));
            const uint64_t xs = (uint64_t)XRS * K;
            const bool kx = k0 + xc < K;
            if constexpr (VEC) {
#pragma unroll
                for (int u = 0; u < XQ; ++u)
                    rq[u] = kx && tile0 + xr + XRS * u < rows ? raw4<SRC>(X, xb + xs * u)
                                                               : make_uint4(0u, 0u, 0u, 0u);
            } else {
#pragma unroll
                for (int u = 0; u < XE; ++u)
                    re[u] = kx && tile0 + xr + XRS * u < rows ? raw1<SRC>(X, xb + xs * u) : 0u;
            }
            uint64_t ab = (uint64_t)(cb0 + ar) * K + k0 + ac;
            asm volatile("" : "+v"(ab));
            const bool ka = k0 + ac < K;
#pragma unroll
            for (int u = 0; u < AE; ++u) {
                const uint32_t r = ar + 8 * u;
                ra[u] = ka && r < arows && cb0 + r < N ? A[ab + (uint64_t)8 * u * K] : 0.0f;
            }
        };
        auto put = [&]() {
            if constexpr (VEC) {
#pragma unroll
                for (int u = 0; u < XQ; ++u) {
                    const int q = tid + 256 * u, r = q / (KC / 4), e = 4 * (q % (KC / 4));
                    float v[4];
                    dec4<SRC>(rq[u], v);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        sx[r * XS + e + j] = v[j];
                }
            } else {
#pragma unroll
                for (int u = 0; u < XE; ++u) {
                    const int q = tid + 256 * u;
                    sx[(q / KC) * XS + q % KC] = dec1<SRC>(re[u]);
                }
            }
#pragma unroll
            for (int u = 0; u < AE; ++u) {
                const int q = tid + 256 * u;
                sa[(q / KC) * XS + q % KC] = ra[u];
            }
        };
        f32x16 acc[NCB];
#pragma unroll
        for (int b = 0; b < NCB; ++b)
            acc[b] = f32x16{};
        fetch(0);
        for (uint32_t k0 = 0; k0 < K; k0 += KC) {
            __syncthreads();   // the previous chunk is consumed
            put();
            if (k0 + KC < K)
                fetch(k0 + KC);   // lands while this chunk's MFMAs run
            __syncthreads();
#pragma unroll
            for (int ks = 0; ks < KC / 2; ++ks) {
                const float a = sx[(32 * wave + c32) * XS + 2 * ks + h];
#pragma unroll
                for (int b = 0; b < NCB; ++b)
                    if (cb0 + 32 * b < N) {   // uniform
                        const float bv = sa[(32 * b + c32) * XS + 2 * ks + h];
                        acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bv, acc[b], 0, 0, 0);
                    }
            }
        }
        // register r of lane l: (row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32)
#pragma unroll
        for (int b = 0; b < NCB; ++b) {
            const uint32_t col = cb0 + 32 * b + c32;
            if (cb0 + 32 * b >= N || col >= N)
                continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const uint64_t orow = row0 + 8 * (r >> 2) + 4 * h + (r & 3);
                if (orow < rows)
                    Y[orow * N + col] = acc[b][r];
            }
        }
    }
}

template <int SRC, int NCB>
void launch_level_n(bool vec, uint64_t blocks, const void *X, uint64_t rows, uint32_t K,
                    const float *A, uint32_t N, float *Y, hipStream_t s)
{
    if (vec)
        hipLaunchKernelGGL((jl_level<SRC, true, NCB>), dim3((uint32_t)blocks), dim3(256), 0, s, X,
                           rows, K, A, N, Y);
    else
        hipLaunchKernelGGL((jl_level<SRC, false, NCB>), dim3((uint32_t)blocks), dim3(256), 0, s,
                           X, rows, K, A, N, Y);
}

template <int SRC>
hipError_t launch_level_t(const void *X, uint64_t rows, uint32_t K, const float *A, uint32_t N,
                          float *Y, hipStream_t s)
{
    const uint64_t blocks = (rows + TR - 1) / TR;
    const size_t esz = SRC == SRC_F32 ? 4 : SRC == DT_I8 ? 1 : 2;
    const bool vec = K % 4 == 0 && (uintptr_t)X % (4 * esz) == 0;
    if (N <= 32)
        launch_level_n<SRC, 1>(vec, blocks, X, rows, K, A, N, Y, s);
    else if (N <= 64)
        launch_level_n<SRC, 2>(vec, blocks, X, rows, K, A, N, Y, s);
    else
        launch_level_n<SRC, NCBMAX>(vec, blocks, X, rows, K, A, N, Y, s);
    return hipGetLastError();
}

// One level: Y (rows x N) = X (rows x K) A^T; src = 0 for fp32 rows, else the
// dtype code of the caller's rows.
hipError_t launch_level(int src, const void *X, uint64_t rows, uint32_t K, const float *A,
                        uint32_t N, float *Y, hipStream_t s)
{
    if (rows == 0 || N == 0)
        return hipSuccess;
    switch (src) {
    case SRC_F32: return launch_level_t<SRC_F32>(X, rows, K, A, N, Y, s);
    case DT_F16: return launch_level_t<DT_F16>(X, rows, K, A, N, Y, s);
    case DT_BF16: return launch_level_t<DT_BF16>(X, rows, K, A, N, Y, s);
    case DT_I8: return launch_level_t<DT_I8>(X, rows, K, A, N, Y, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace sjj
