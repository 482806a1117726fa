// sj_front.hip -- Section 4's ip-distance front ends on gfx950: the rows the
// join's matrix-core kernels read for cosine similarity (f = g = x / ||x||)
// and for the Hamming distance (f(x) = (x, 1 - x), g(y) = (1 - y, y) on
// {0, 1}^d).  Both are O(n d) passes over the rows, bound by HBM.
#include "sj_internal.h"

namespace sjk {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// ------------------------------------------------------------------ cosine
// Exact value of element k of a row of dtype DT.
template <int DT>
__device__ __forceinline__ double elem_value(const uint8_t *row, uint32_t k)
{
    if constexpr (DT == DT_I8) {
        return (double)(int8_t)row[k];
    } else if constexpr (DT == DT_F16) {
        return (double)(float)((const _Float16 *)row)[k];
    } else {
        const uint32_t b = (uint32_t)((const uint16_t *)row)[k] << 16;
        return (double)__uint_as_float(b);
    }
}

// The nearest value with P significand bits (binary16: P = 11, smallest
// normal exponent -14; bfloat16: P = 8, -126) of a double, ties to even, as a
// 16-bit pattern.  From the double's bit pattern: the value is sig * 2^e2
// with an integer significand; the result's quantum is 2^q with q = max(lg -
// (P - 1), EMIN - (P - 1)) where lg = floor(log2 |v|); the bits of sig below
// the quantum are dropped and decide the rounding (above half: up; exactly
// half: up when the kept part is odd).  The pattern is then
// ((q - EMIN + P) << (P - 1)) + kept - 2^(P - 1) for normal and subnormal
// results alike, a kept significand of 2^P carrying into the exponent field;
// |v| at or above 2^(EMAX + 1) is infinity.
template <int P, int EMIN, int EMAX>
__device__ __forceinline__ uint16_t round_double_rne(double v)
{
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
    const uint32_t E = (uint32_t)(b >> 52) & 0x7ffu;
    const uint64_t frac = b & ((1ull << 52) - 1);
    if (E == 0 && frac == 0)
        return sign;
    const uint64_t sig = E == 0 ? frac : (frac | (1ull << 52));
    const int e2 = (E == 0 ? 1 : (int)E) - 1075;
    const int lg = 63 - __clzll((long long)sig) + e2;
    if (lg > EMAX)
        return sign | (uint16_t)(((EMAX - EMIN + 2) << (P - 1)));   // infinity
    const int q = lg - (P - 1) > EMIN - (P - 1) ? lg - (P - 1) : EMIN - (P - 1);
    const int shift = q - e2;   // > 0: a double has more significand bits
    if (shift >= 64)
        return sign;            // far below half the smallest subnormal
    const uint64_t kept0 = sig >> shift;
    const uint64_t rem = sig & ((1ull << shift) - 1);
    const uint64_t half = 1ull << (shift - 1);
    const uint64_t kept = kept0 + ((rem > half || (rem == half && (kept0 & 1))) ? 1 : 0);
    const uint32_t bits =
        ((uint32_t)(q - EMIN + P) << (P - 1)) + (uint32_t)kept - (1u << (P - 1));
    return sign | (uint16_t)bits;
}

// Norm of every row: sqrt of the sum of the squares in double, ascending k
// (one thread per row; every square of a decoded element is exact).
template <int DT>
__global__ void __launch_bounds__(256) row_norms_f64(const uint8_t *X, uint32_t n, uint32_t d,
                                                     uint32_t row_bytes, double *norm)
{
    const uint32_t i = blockIdx.x * 256 + threadIdx.x;
    if (i >= n)
        return;
    const uint8_t *row = X + (size_t)i * row_bytes;
    double s = 0.0;
    for (uint32_t k = 0; k < d; ++k) {
        const double x = elem_value<DT>(row, k);
        s += x * x;
    }
    norm[i] = __builtin_sqrt(s);
}

// y = x / ||x|| rounded to the output type (binary16 for fp16 and int8 rows,
// bfloat16 for bfloat16 rows); a row of norm 0 is written as +0.
template <int DT>
__global__ void __launch_bounds__(256) normalize_rows(const uint8_t *X, uint32_t n, uint32_t d,
                                                      uint32_t row_bytes, const double *norm,
                                                      uint16_t *Y)
{
    const uint64_t total = (uint64_t)n * d;
    for (uint64_t t = (uint64_t)blockIdx.x * 256 + threadIdx.x; t < total;
         t += (uint64_t)gridDim.x * 256) {
        const uint32_t i = (uint32_t)(t / d), k = (uint32_t)(t - (uint64_t)i * d);
        const double nr = norm[i];
        uint16_t y = 0;
        if (nr != 0.0) {
            const double q = elem_value<DT>(X + (size_t)i * row_bytes, k) / nr;
            y = DT == DT_BF16 ? round_double_rne<8, -126, 127>(q) : round_double_rne<11, -14, 15>(q);
        }
        Y[t] = y;
    }
}

template <int DT>
static hipError_t normalize_dt(const uint8_t *X, uint32_t n, uint32_t d, double *norm, uint16_t *Y,
                               hipStream_t st)
{
    const uint32_t row_bytes = d * (DT == DT_I8 ? 1u : 2u);
    hipLaunchKernelGGL((row_norms_f64<DT>), dim3((n + 255) / 256), dim3(256), 0, st, X, n, d,
                       row_bytes, norm);
    const uint64_t total = (uint64_t)n * d;
    const uint64_t blocks = (total + 255) / 256;
    hipLaunchKernelGGL((normalize_rows<DT>), dim3((uint32_t)(blocks < 65536 ? blocks : 65536)),
                       dim3(256), 0, st, X, n, d, row_bytes, norm, Y);
    return hipGetLastError();
}

hipError_t launch_normalize(int dtype, const void *X, uint32_t n, uint32_t d, double *norm,
                            void *Y, hipStream_t stream)
{
    if (n == 0 || d == 0)
        return hipSuccess;
    const uint8_t *x = (const uint8_t *)X;
    uint16_t *y = (uint16_t *)Y;
    switch (dtype) {
    case DT_F16: return normalize_dt<DT_F16>(x, n, d, norm, y, stream);
    case DT_BF16: return normalize_dt<DT_BF16>(x, n, d, norm, y, stream);
    case DT_I8: return normalize_dt<DT_I8>(x, n, d, norm, y, stream);
    }
    return hipErrorInvalidValue;
}

// ----------------------------------------------------------------- Hamming
// Bit rows (coordinate m in bit m % 8 of byte m / 8, ceil(d / 8) bytes per
// row) unpacked to int8 rows of out_bytes bytes (a multiple of 16, >= 2 d):
//   side 0 (P):  f(x)  = (x_0 .. x_{d-1}, 1 - x_0 .. 1 - x_{d-1}, 0 ...)
//   side 1 (Q): -g(y)  = (y_0 - 1 .. y_{d-1} - 1, -y_0 .. -y_{d-1}, 0 ...)
// so that <f(x), -g(y)> = -sum_m (x_m (1 - y_m) + (1 - x_m) y_m) = -Ham(x, y).
// One thread per 4-byte word of the output.
__global__ void __launch_bounds__(256) unpack_hamming(const uint8_t *bits, uint32_t n, uint32_t d,
                                                      uint32_t out_bytes, int side, uint8_t *out)
{
    const uint32_t in_stride = (d + 7) / 8;
    const uint32_t wpr = out_bytes / 4;
    const uint64_t words = (uint64_t)n * wpr;
    for (uint64_t w = (uint64_t)blockIdx.x * 256 + threadIdx.x; w < words;
         w += (uint64_t)gridDim.x * 256) {
        const uint64_t row = w / wpr;
        const uint32_t col = (uint32_t)(w - row * wpr) * 4;
        const uint8_t *rb = bits + row * in_stride;
        uint32_t v = 0;
#pragma unroll
        for (uint32_t b = 0; b < 4; ++b) {
            const uint32_t c = col + b;
            int e = 0;
            if (c < 2 * d) {
                const uint32_t m = c < d ? c : c - d;
                const int x = (rb[m >> 3] >> (m & 7)) & 1;
                if (side == 0)
                    e = c < d ? x : 1 - x;
                else
                    e = c < d ? x - 1 : -x;
            }
            v |= (uint32_t)(uint8_t)(int8_t)e << (8 * b);
        }
        *(uint32_t *)(out + row * out_bytes + col) = v;
    }
}

hipError_t launch_unpack_hamming(const uint8_t *bits, uint32_t n, uint32_t d, uint32_t out_bytes,
                                 int side, uint8_t *out, hipStream_t stream)
{
    if (n == 0)
        return hipSuccess;
    const uint64_t words = (uint64_t)n * (out_bytes / 4);
    const uint64_t blocks = (words + 255) / 256;
    hipLaunchKernelGGL(unpack_hamming, dim3((uint32_t)(blocks < 65536 ? blocks : 65536)),
                       dim3(256), 0, stream, bits, n, d, out_bytes, side, out);
    return hipGetLastError();
}

}  // namespace sjk
