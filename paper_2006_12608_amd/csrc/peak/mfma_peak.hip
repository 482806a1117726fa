// mfma_peak.hip -- measurement only: the MFMA-only throughput this GPU
// sustains (no memory traffic, no epilogue), the reference the join kernels'
// fraction of peak can be read against next to the spec figure.  Built into
// its own library (libsj_peak.so); bench.py is its only caller.
//
//   extern "C" int sj_peak_mfma(int dtype, int waves_per_simd, double target_ms,
//                               const void *operands, uint64_t n_bytes,
//                               double *tops, double *ms);
//
// dtype: 1 = fp16, 2 = bf16 (v_mfma_f32_32x32x16_*), 3 = int8
// (v_mfma_i32_32x32x32_i8).  Every wave runs four independent accumulator
// chains over four A and four B fragments per lane, rotated so consecutive
// MFMAs see different data, as the join's streamed B-fragments do.  The
// fragments are 16-byte chunks taken from `operands` (device memory of
// n_bytes, e.g. the workload's own rows: the matrix cores' power, and so the
// clock they sustain, depends on the data), or random finite values when
// operands is null.  One launch of about target_ms is timed with HIP events
// after a short calibration launch; *tops receives TFLOP/s (TOP/s for int8),
// *ms the time.  Returns 0, or -1 on a bad argument, -4 on a HIP error.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

template <int DT>
struct Op;
template <>
struct Op<1> {
    typedef f32x16 acc_t;
    static __device__ __forceinline__ acc_t mma(i32x4 a, i32x4 b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    }
};
template <>
struct Op<2> {
    typedef f32x16 acc_t;
    static __device__ __forceinline__ acc_t mma(i32x4 a, i32x4 b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
};
template <>
struct Op<3> {
    typedef i32x16 acc_t;
    static __device__ __forceinline__ acc_t mma(i32x4 a, i32x4 b, acc_t c)
    {
        return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
    }
};

constexpr int kFrags = 4;   // A and B fragments per lane, and accumulator chains

template <int DT>
__global__ void __launch_bounds__(256) mfma_loop(const i32x4 *in, int n_in, float *out, int iters)
{
    typedef typename Op<DT>::acc_t acc_t;
    const int t = blockIdx.x * 256 + threadIdx.x;
    i32x4 a[kFrags], b[kFrags];
#pragma unroll
    for (int f = 0; f < kFrags; ++f) {
        a[f] = in[(t * 2 * kFrags + f) % n_in];
        b[f] = in[(t * 2 * kFrags + kFrags + f) % n_in];
    }
    acc_t acc[kFrags];
#pragma unroll
    for (int c = 0; c < kFrags; ++c)
        acc[c] = acc_t{};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int r = 0; r < kFrags; ++r)          // four rounds, B rotated each round
#pragma unroll
            for (int c = 0; c < kFrags; ++c)
                acc[c] = Op<DT>::mma(a[c], b[(c + r) % kFrags], acc[c]);
    }
    float s = 0.0f;
#pragma unroll
    for (int c = 0; c < kFrags; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            s += (float)acc[c][r];
    out[t] = s;   // keeps the chains live
}

template <int DT>
hipError_t launch(int grid, const i32x4 *in, int n_in, float *out, int iters)
{
    hipLaunchKernelGGL((mfma_loop<DT>), dim3(grid), dim3(256), 0, 0, in, n_in, out, iters);
    return hipGetLastError();
}

hipError_t launch_dt(int dt, int grid, const i32x4 *in, int n_in, float *out, int iters)
{
    switch (dt) {
    case 1: return launch<1>(grid, in, n_in, out, iters);
    case 2: return launch<2>(grid, in, n_in, out, iters);
    default: return launch<3>(grid, in, n_in, out, iters);
    }
}

// Random operand bits of the element type's ordinary range: fp16 / bf16
// values of magnitude below 2 (no inf / NaN), any int8.
void fill_random(std::vector<uint32_t> &v, int dt)
{
    uint64_t x = 0x9E3779B97F4A7C15ull;
    for (auto &w : v) {
        x ^= x << 13;
        x ^= x >> 7;
        x ^= x << 17;
        uint32_t r = (uint32_t)(x >> 16);
        if (dt == 1)
            r &= 0xBBFFBBFFu;   // clears each fp16 half's top exponent bit
        else if (dt == 2)
            r &= 0xBF7FBF7Fu;   // clears each bf16 half's top exponent bit
        w = r;
    }
}

}  // namespace

extern "C" int sj_peak_mfma(int dtype, int waves_per_simd, double target_ms,
                            const void *operands, uint64_t n_bytes, double *tops, double *ms)
{
    if (dtype < 1 || dtype > 3 || waves_per_simd < 1 || waves_per_simd > 8 || !(target_ms > 0) ||
        !tops || !ms || (operands && n_bytes < 16))
        return -1;
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return -4;
    const int grid = cus * waves_per_simd;   // 4 waves per workgroup = one per SIMD
    const bool own = operands == nullptr;
    const uint64_t chunks = own ? (1u << 16) : n_bytes / 16;
    const int n_in = (int)(chunks < (1u << 30) ? chunks : (1u << 30));
    std::vector<uint32_t> host(own ? (size_t)n_in * 4 : 0);
    if (own)
        fill_random(host, dtype);
    i32x4 *in = own ? nullptr : (i32x4 *)operands;
    float *out = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int st = 0;
    float el = 0.0f;
    int iters = 64;
    if ((own && (hipMalloc(&in, host.size() * 4) != hipSuccess ||
                 hipMemcpy(in, host.data(), host.size() * 4, hipMemcpyHostToDevice) !=
                     hipSuccess)) ||
        hipMalloc(&out, (size_t)grid * 256 * sizeof(float)) != hipSuccess ||
        hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
        st = -4;
        goto done;
    }
    // calibration launch (also warms the clocks), then one timed launch
    for (int pass = 0; pass < 2; ++pass) {
        if (hipEventRecord(e0, 0) != hipSuccess ||
            launch_dt(dtype, grid, in, n_in, out, iters) != hipSuccess ||
            hipEventRecord(e1, 0) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
            hipEventElapsedTime(&el, e0, e1) != hipSuccess) {
            st = -4;
            goto done;
        }
        if (pass == 0) {
            const double scale = target_ms / (el > 1e-3 ? el : 1e-3);
            const double want = iters * scale;
            iters = want < 1 ? 1 : want > 2e8 ? 200000000 : (int)want;
        }
    }
    {
        const double per_mfma = dtype == 3 ? 65536.0 : 32768.0;   // ops of one 32x32 MFMA
        const double mfmas = (double)grid * 4 * iters * kFrags * kFrags;
        *ms = el;
        *tops = mfmas * per_mfma / (el * 1e-3) / 1e12;
    }
done:
    if (e0)
        (void)hipEventDestroy(e0);
    if (e1)
        (void)hipEventDestroy(e1);
    if (own && in)
        (void)hipFree(in);
    if (out)
        (void)hipFree(out);
    return st;
}
