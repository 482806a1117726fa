// sj_jl.hip -- the TCU Johnson-Lindenstrauss transform of Ahle & Silvestri,
// "Similarity Search with Tensor Core Units", Lemma 3 / Theorem 2, on gfx950.
//
// M = (I_{r_l} (x) A_l) ... (I_{r_1} (x) A_1): since I_r (x) A is A copied
// r times along the diagonal, a batch of n row vectors of length r_i c_i,
// read as n r_i rows of c_i entries, is multiplied by A_i^T as one dense
// product, and the result (n r_i rows of k_i entries) read back as n rows of
// r_i k_i entries is the next level's input -- no data moves between levels.
// Each level is one fp32 product Y = X A_i^T on the matrix cores
// (v_mfma_f32_32x32x2_f32); the first level decodes fp16 / bf16 / int8 rows
// exactly to fp32.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sj_internal.h"

namespace sjj {

using sjk::DT_BF16;
using sjk::DT_F16;
using sjk::DT_I8;

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int SRC_F32 = 0;

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

// Column blocks of 32 a wave keeps accumulators for at once.
constexpr int NCB = 4;

// Y (rows x N, fp32) = X (rows x K) A^T, A N x K fp32 row-major.  A wave owns
// 32 rows and sweeps the columns NCB blocks of 32 at a time; per k-step
// (two entries of K) lane l supplies X[row l % 32][k + l / 32] and
// A[column l % 32][k + l / 32].  Rows past `rows`, columns past N and entries
// past K read as zero; results outside rows x N are not stored.
template <int SRC>
__global__ void __launch_bounds__(256) jl_level(const void *X, uint64_t rows, uint32_t K,
                                                const float *A, uint32_t N, float *Y)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int h = lane >> 5, c32 = lane & 31;
    const uint64_t row0 = ((uint64_t)blockIdx.x * 4 + wave) * 32;
    if (row0 >= rows)
        return;
    const uint64_t row = row0 + c32;
    const bool rok = row < rows;
    for (uint32_t cb0 = 0; cb0 < N; cb0 += 32 * NCB) {
        f32x16 acc[NCB];
#pragma unroll
        for (int b = 0; b < NCB; ++b)
            acc[b] = f32x16{};
        for (uint32_t k = 0; k < K; k += 2) {
            const uint32_t kk = k + h;
            const float a = rok && kk < K ? load_elem<SRC>(X, row * K + kk) : 0.0f;
#pragma unroll
            for (int b = 0; b < NCB; ++b) {
                const uint32_t col = cb0 + 32 * b + c32;
                if (cb0 + 32 * b < N) {   // uniform
                    const float bv = col < N && kk < K ? A[(uint64_t)col * K + kk] : 0.0f;
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
    const uint64_t blocks = (rows + 127) / 128;
    hipLaunchKernelGGL(jl_level<SRC>, dim3((uint32_t)blocks), dim3(256), 0, s, X, rows, K, A, N,
                       Y);
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
