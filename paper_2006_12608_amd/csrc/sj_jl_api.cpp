// sj_jl_api.cpp -- host side of the TCU Johnson-Lindenstrauss transform
// (sj_jl; contract in include/sj.h): size-chain checks, scratch for the
// intermediate levels, one matrix-core product per level on the context's
// stream (kernels in sj_jl.hip).
#include <hip/hip_runtime.h>

#include "sj.h"
#include "sj_host.h"

using namespace sjh;

namespace sjj {
hipError_t launch_level(int src, const void *X, uint64_t rows, uint32_t K, const float *A,
                        uint32_t N, float *Y, hipStream_t s);
}

extern "C" int sj_jl(sj_ctx *c, int dtype, const void *X, uint32_t n, uint32_t d,
                     uint32_t levels, const uint32_t *shape, const float *A, float *Y)
{
    g_err.clear();
    if (!c)
        return fail(SJ_E_INVAL, "context is NULL");
    if (dtype != SJ_F16 && dtype != SJ_BF16 && dtype != SJ_I8)
        return fail(SJ_E_INVAL, "unknown dtype %d", dtype);
    if (levels < 1 || levels > 32 || !shape)
        return fail(SJ_E_INVAL, "levels = %u: 1 <= levels <= 32 with a shape array", levels);
    // the size chain of Lemma 3: d = r_1 c_1, r_i k_i = r_{i+1} c_{i+1}
    uint64_t len = d, a_elems = 0, tmp = 0;
    for (uint32_t i = 0; i < levels; ++i) {
        const uint64_t k = shape[3 * i], cc = shape[3 * i + 1], r = shape[3 * i + 2];
        if (k == 0 || cc == 0 || r == 0)
            return fail(SJ_E_INVAL, "level %u: sizes must be positive", i + 1);
        if (r * cc != len)
            return fail(SJ_E_INVAL, "level %u: r c = %llu does not match the input length %llu",
                        i + 1, (unsigned long long)(r * cc), (unsigned long long)len);
        if (k > 65536 || cc > 65536)
            return fail(SJ_E_UNSUPPORTED, "level %u: k or c above 65536", i + 1);
        a_elems += k * cc;
        len = r * k;
        // n * len elements per level (and 4 n len bytes) must not wrap: at
        // most 2^48, far beyond any device memory
        if (len > ((uint64_t)1 << 48) / (n ? n : 1))
            return fail(SJ_E_UNSUPPORTED, "level %u: n * r * k = %u * %llu elements is too large",
                        i + 1, n, (unsigned long long)len);
        if (i + 1 < levels)
            tmp = tmp > (uint64_t)n * len ? tmp : (uint64_t)n * len;
    }
    int st;
    if ((st = check_device_ptr(c, X, (size_t)n * d * esize(dtype), "X")) != SJ_OK)
        return st;
    if ((st = check_device_ptr(c, A, (size_t)a_elems * 4, "A")) != SJ_OK)
        return st;
    if ((st = check_device_ptr(c, Y, (size_t)n * len * 4, "Y")) != SJ_OK)
        return st;
    c->stats = sj_stats{};
    if (n == 0)
        return SJ_OK;
    const size_t half = align_up((size_t)tmp * 4);
    if ((st = grow_scratch(c, 2 * half + 256)) != SJ_OK)
        return st;
    float *buf[2] = {(float *)c->scratch, (float *)((uint8_t *)c->scratch + half)};
    hipStream_t s = c->stream;
    SJ_HIP(hipSetDevice(c->device));
    SJ_HIP(hipEventRecord(c->ev[0], s));
    const void *in = X;
    int src = dtype;
    const float *a = A;
    for (uint32_t i = 0; i < levels; ++i) {
        const uint32_t k = shape[3 * i], cc = shape[3 * i + 1], r = shape[3 * i + 2];
        float *out = i + 1 == levels ? Y : buf[i & 1];
        SJ_HIP(sjj::launch_level(src, in, (uint64_t)n * r, cc, a, k, out, s));
        in = out;
        src = 0;
        a += (size_t)k * cc;
    }
    SJ_HIP(hipEventRecord(c->ev[1], s));
    SJ_HIP(hipStreamSynchronize(s));
    c->stats.ms_join = elapsed_ms(c->ev[0], c->ev[1]);
    c->stats.timed = 1;
    return SJ_OK;
}
