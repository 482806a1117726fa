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

// Four consecutive entries from idx (idx a multiple of 4, the row 4-entry
// aligned) decoded to fp32.
template <int SRC>
__device__ __forceinline__ void load4(const void *X, uint64_t idx, float (&v)[4])
{
    if constexpr (SRC == SRC_F32) {
        const float4 f = *(const float4 *)((const float *)X + idx);
        v[0] = f.x, v[1] = f.y, v[2] = f.z, v[3] = f.w;
    } else if constexpr (SRC == DT_I8) {
        const uint32_t w = *(const uint32_t *)((const int8_t *)X + idx);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            v[j] = (float)(int8_t)(w >> (8 * j));
    } else {
        const uint2 w = *(const uint2 *)((const uint16_t *)X + idx);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t hbits = ((j < 2 ? w.x : w.y) >> (16 * (j & 1))) & 0xffffu;
            if constexpr (SRC == DT_F16)
                v[j] = (float)__builtin_bit_cast(_Float16, (uint16_t)hbits);
            else
                v[j] = __builtin_bit_cast(float, hbits << 16);
        }
    }
}

template <int SRC>
__device__ __forceinline__ float load_elem(const void *X, uint64_t idx)
{
    if constexpr (SRC == SRC_F32) {
        return ((const float *)X)[idx];
    } else if constexpr (SRC == DT_F16) {
        return (float)((const _Float16 *)X)[idx];
    } else if constexpr (SRC == DT_BF16) {
        const uint32_t h = ((const uint16_t *)X)[idx];
        return __builtin_bit_cast(float, h << 16);
    } else {
        return (float)((const int8_t *)X)[idx];
    }
}

// Column blocks of 32 a wave keeps accumulators for at once, rows per
// workgroup tile and entries of K per LDS chunk.
constexpr int NCB = 4;
constexpr int TR = 128;
constexpr int KC = 32;
constexpr int XS = KC + 1;   // LDS row stride (floats): lanes of a fragment read distinct banks

// Y (rows x N, fp32) = X (rows x K) A^T, A N x K fp32 row-major.  A workgroup
// of 4 waves owns TR rows; for each group of NCB column blocks it walks K in
// chunks of KC entries, staging the chunk of its TR rows and of the group's
// rows of A in LDS as fp32 (consecutive threads load consecutive entries of
// a row: coalesced), and wave w multiplies rows 32 w .. 32 w + 31 on the
// matrix cores (per k-step, lane l supplies X[row l % 32][k + l / 32] and
// A[column l % 32][k + l / 32]).  Entries past the matrices read as zero;
// results outside rows x N are not stored.
template <int SRC, bool VEC>
__global__ void __launch_bounds__(256) jl_level(const void *X, uint64_t rows, uint32_t K,
                                                const float *A, uint32_t N, float *Y)
{
    __shared__ float sx[TR * XS];
    __shared__ float sa[32 * NCB * XS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = lane >> 5, c32 = lane & 31;
    const uint64_t tile0 = (uint64_t)blockIdx.x * TR;
    const uint64_t row0 = tile0 + 32 * wave;
    for (uint32_t cb0 = 0; cb0 < N; cb0 += 32 * NCB) {
        f32x16 acc[NCB];
#pragma unroll
        for (int b = 0; b < NCB; ++b)
            acc[b] = f32x16{};
        for (uint32_t k0 = 0; k0 < K; k0 += KC) {
            __syncthreads();   // the previous chunk is consumed
            if constexpr (VEC) {
                // K is a multiple of 4 and X aligned for 4-entry loads
#pragma unroll
                for (int q = tid; q < TR * KC / 4; q += 256) {
                    const int r = q / (KC / 4), e = 4 * (q % (KC / 4));
                    const uint64_t row = tile0 + r;
                    const uint32_t k = k0 + e;
                    float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                    if (row < rows && k < K)
                        load4<SRC>(X, row * K + k, v);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        sx[r * XS + e + j] = v[j];
                }
            } else {
#pragma unroll
                for (int q = tid; q < TR * KC; q += 256) {
                    const int r = q / KC, e = q % KC;
                    const uint64_t row = tile0 + r;
                    const uint32_t k = k0 + e;
                    sx[r * XS + e] = row < rows && k < K ? load_elem<SRC>(X, row * K + k) : 0.0f;
                }
            }
            // only the column blocks this group uses (whole blocks of 32 rows)
            const uint32_t arows = min((N - cb0 + 31) / 32 * 32, 32u * NCB);
            for (uint32_t q = tid; q < arows * KC; q += 256) {
                const int r = q / KC, e = q % KC;
                const uint32_t col = cb0 + r, k = k0 + e;
                sa[r * XS + e] = col < N && k < K ? A[(uint64_t)col * K + k] : 0.0f;
            }
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

template <int SRC>
hipError_t launch_level_t(const void *X, uint64_t rows, uint32_t K, const float *A, uint32_t N,
                          float *Y, hipStream_t s)
{
    const uint64_t blocks = (rows + TR - 1) / TR;
    const size_t esz = SRC == SRC_F32 ? 4 : SRC == DT_I8 ? 1 : 2;
    const bool vec = K % 4 == 0 && (uintptr_t)X % (4 * esz) == 0;
    if (vec)
        hipLaunchKernelGGL((jl_level<SRC, true>), dim3((uint32_t)blocks), dim3(256), 0, s, X, rows,
                           K, A, N, Y);
    else
        hipLaunchKernelGGL((jl_level<SRC, false>), dim3((uint32_t)blocks), dim3(256), 0, s, X,
                           rows, K, A, N, Y);
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
