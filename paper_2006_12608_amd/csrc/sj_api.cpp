// sj_api.cpp -- host side of libsj.so: argument checking, threshold conversion,
// scratch management and the single-pass / count-then-emit protocols around
// the gfx950 kernels.  Public contract: include/sj.h.
#include "sj.h"

#include <hip/hip_runtime.h>

#include <cfloat>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include <mutex>

#include "sj_host.h"
#include "sj_internal.h"

// Device scratch of sj_join_noalloc, for callers that cannot allocate: the
// match counter and scan total (first 256 bytes), then the row norms,
// repacked rows and block counts / offsets of one call.  Each GPU the library
// runs on holds its own copy until the process ends; host code reaches it only
// through the address looked up once per device (sj_create), never through
// this name.
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

namespace sjh {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(SJ_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

size_t esize(int dtype) { return dtype == SJ_I8 ? 1 : 2; }

int check_device_ptr(const sj_ctx *c, const void *p, size_t bytes, const char *name)
{
    if (bytes == 0)
        return SJ_OK;
    if (!p)
        return fail(SJ_E_INVAL, "%s is NULL", name);
    hipPointerAttribute_t a;
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();
        return fail(SJ_E_INVAL, "%s is not a pointer known to HIP", name);
    }
    if (a.type != hipMemoryTypeDevice && a.type != hipMemoryTypeManaged)
        return fail(SJ_E_INVAL, "%s is not device memory", name);
    if (a.device != c->device)
        return fail(SJ_E_INVAL, "%s lives on device %d, the context on %d", name, a.device,
                    c->device);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p) == hipSuccess && base) {
        const uintptr_t b = (uintptr_t)base, q = (uintptr_t)p;
        if (q < b || q - b > size || size - (q - b) < bytes)
            return fail(SJ_E_INVAL, "%s: %zu bytes needed but its allocation holds %zu from there",
                        name, bytes, (size_t)(size - (q - b)));
    } else {
        (void)hipGetLastError();
    }
    return SJ_OK;
}

// Smallest float >= s (so acc >= s32 <=> acc >= s for every float acc).
float float_at_or_above(double s)
{
    if (std::isinf(s))
        return (float)s;
    if (s > (double)FLT_MAX)
        return INFINITY;
    float f = (float)s;
    if ((double)f < s)
        f = std::nextafter(f, INFINITY);
    return f;
}

// Largest float <= r (so x <= r32 <=> x <= r for every float x).
float float_at_or_below(double r)
{
    if (std::isinf(r))
        return (float)r;
    if (r < -(double)FLT_MAX)
        return -INFINITY;
    float f = (float)r;
    if ((double)f > r)
        f = std::nextafter(f, -INFINITY);
    return f;
}

int grow_scratch(sj_ctx *c, size_t bytes)
{
    if (bytes <= c->scratch_bytes)
        return SJ_OK;
    if (c->scratch) {
        (void)hipStreamSynchronize(c->stream);
        (void)hipFree(c->scratch);
        c->scratch = nullptr;
        c->scratch_bytes = 0;
    }
    size_t want = bytes + bytes / 4;
    if (hipMalloc(&c->scratch, want) != hipSuccess) {
        (void)hipGetLastError();
        c->scratch = nullptr;
        if (hipMalloc(&c->scratch, bytes) != hipSuccess) {
            (void)hipGetLastError();
            c->scratch = nullptr;
            return fail(SJ_E_NOMEM, "cannot allocate %zu bytes of device scratch", bytes);
        }
        want = bytes;
    }
    c->scratch_bytes = want;
    return SJ_OK;
}

int grow_front(sj_ctx *c, size_t bytes)
{
    if (bytes <= c->front_bytes)
        return SJ_OK;
    if (c->front) {
        (void)hipStreamSynchronize(c->stream);
        (void)hipFree(c->front);
        c->front = nullptr;
        c->front_bytes = 0;
    }
    if (hipMalloc(&c->front, bytes) != hipSuccess) {
        (void)hipGetLastError();
        c->front = nullptr;
        return fail(SJ_E_NOMEM, "cannot allocate %zu bytes of device memory for the rows of "
                    "the front end", bytes);
    }
    c->front_bytes = bytes;
    return SJ_OK;
}

double elapsed_ms(hipEvent_t a, hipEvent_t b)
{
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, a, b) != hipSuccess) {
        (void)hipGetLastError();
        return 0.0;
    }
    return ms;
}

}  // namespace sjh

namespace {

using namespace sjh;

struct Request {
    int metric, dtype;
    const void *P, *Q;
    uint32_t n_p, n_q, d;
    double thr;
    uint32_t *pairs;
    uint64_t cap;
    bool two_pass, count_only, timing, recompute;
    // the score matrix is symmetric although P and Q are different buffers
    // (the Hamming front end's f(x) and -g(x)): a single pass computes the
    // upper triangle only and mirrors its pairs, as for P == Q
    bool symmetric = false;
};

// Largest match-bit buffer the two-pass mode keeps (bytes); beyond it, or
// when it cannot be allocated, the second pass recomputes the product.
const size_t kMaxMaskBytes = (size_t)64 << 30;
// Room for match records (resident kernel's two-pass mode), split evenly over
// the first pass's workgroups: at most 4 Mi records (640 MiB) in all, and per
// workgroup at most its number of 32x32 blocks; a workgroup that finds more
// blocks with matches makes the second pass recompute.
const uint64_t kMaxRecords = (uint64_t)4 << 20;

// Per-device address of `scratch` (hipGetSymbolAddress with the device
// current, at sj_create); null until looked up or when the lookup failed.
constexpr int kMaxDevices = 64;
std::mutex g_fixed_mu;
uint8_t *g_fixed[kMaxDevices] = {};
int g_fixed_err[kMaxDevices] = {};

// Looks up this device's copy of `scratch` once; the device must be current.
void lookup_fixed_scratch(int device)
{
    if (device < 0 || device >= kMaxDevices)
        return;
    std::lock_guard<std::mutex> lock(g_fixed_mu);
    if (g_fixed[device] || g_fixed_err[device])
        return;
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
        (void)hipGetLastError();
        g_fixed_err[device] = e != hipSuccess ? (int)e : -1;
        return;
    }
    g_fixed[device] = (uint8_t *)ptr;
}

// A caller-independent scratch region: `base` (device) of `bytes` bytes whose
// first 256 bytes hold the call's counters.  Null base: the context's own,
// growing scratch and counters.
struct Fixed {
    uint8_t *base;
    size_t bytes;
};
const size_t kFixedHead = 256;

int run(sj_ctx *c, const Request &rq, uint64_t *n_out, const Fixed *fx = nullptr)
{
    if (!c)
        return fail(SJ_E_INVAL, "context is NULL");
    if (!n_out)
        return fail(SJ_E_INVAL, "result pointer is NULL");
    *n_out = 0;
    if (rq.dtype != SJ_F16 && rq.dtype != SJ_BF16 && rq.dtype != SJ_I8)
        return fail(SJ_E_INVAL, "unknown dtype %d", rq.dtype);
    if (rq.metric != SJ_IP && rq.metric != SJ_L2)
        return fail(SJ_E_INVAL, "unknown metric %d", rq.metric);
    if (std::isnan(rq.thr))
        return fail(SJ_E_INVAL, "threshold is NaN");
    if (rq.d > (rq.dtype == SJ_I8 ? 32768u : 65536u))
        return fail(SJ_E_UNSUPPORTED, "d = %u is above the limit for this dtype", rq.d);
    const size_t row_bytes = (size_t)rq.d * esize(rq.dtype);
    const size_t bytes_p = (size_t)rq.n_p * row_bytes, bytes_q = (size_t)rq.n_q * row_bytes;
    int st;
    if ((st = check_device_ptr(c, rq.P, bytes_p, "P")) != SJ_OK)
        return st;
    if ((st = check_device_ptr(c, rq.Q, bytes_q, "Q")) != SJ_OK)
        return st;
    if (!rq.count_only && rq.cap > 0) {
        if (rq.cap > (uint64_t)SIZE_MAX / 8)
            return fail(SJ_E_INVAL, "cap too large");
        if ((st = check_device_ptr(c, rq.pairs, (size_t)rq.cap * 8, "pairs")) != SJ_OK)
            return st;
        if ((uintptr_t)rq.pairs % 8 != 0)
            return fail(SJ_E_INVAL, "pairs must be 8-byte aligned");
    }
    c->stats = sj_stats{};
    if (rq.n_p == 0 || rq.n_q == 0)
        return SJ_OK;

    sjk::Plan plan;
    if (!sjk::plan_join(rq.dtype, rq.metric, rq.n_p, rq.n_q,
                        (uint32_t)(row_bytes == 0 ? 16 : (row_bytes + 15) & ~(size_t)15),
                        c->num_cus, &plan))
        return fail(SJ_E_UNSUPPORTED, "shape %u x %u x %u is too large for one launch", rq.n_p,
                    rq.n_q, rq.d);
    // The kernels read rows as 16-byte chunks: inputs whose rows are not
    // 16-byte aligned are first repacked into zero-padded rows (zero columns
    // change neither inner products nor squared distances).
    // d = 0 takes the same path: one zero chunk per row (every score is 0).
    const bool aligned = row_bytes > 0 && row_bytes % 16 == 0 && ((uintptr_t)rq.P % 16) == 0 &&
                         ((uintptr_t)rq.Q % 16) == 0;
    const size_t krow = row_bytes == 0 ? 16 : (row_bytes + 15) & ~(size_t)15;
    const bool self = rq.P == rq.Q && rq.n_p == rq.n_q;
    const bool l2 = rq.metric == SJ_L2;
    const bool blocks = rq.two_pass || rq.count_only;
    // Count-then-emit with the K-streamed kernel keeps the first pass's match
    // bits (one per result) when they fit, so the second pass does not repeat
    // the product.
    const size_t mask_bytes = (size_t)plan.n_blocks * sjk::ST_MASK_WORDS * 2;
    bool use_masks = rq.two_pass && !rq.count_only && !rq.recompute &&
                     plan.family == sjk::FAM_STREAMED && plan.n_blocks <= kMaxMaskBytes / 1024 &&
                     mask_bytes <= kMaxMaskBytes;
    // With the resident kernel it appends a record per 32x32 block with
    // matches instead (its outputs are sparse next to its products).
    bool use_records = rq.two_pass && !rq.count_only && !rq.recompute &&
                       plan.family == sjk::FAM_RESIDENT;
    if (fx) {
        // the fixed region holds no match bits or records: the second pass
        // recomputes the product
        use_masks = false;
        use_records = false;
    }
    uint64_t rec_cap = kMaxRecords / plan.grid;
    rec_cap = rec_cap < plan.wg_blocks32 ? rec_cap : plan.wg_blocks32;
    if (rec_cap == 0)
        use_records = false;
    const size_t rec_bytes = align_up((size_t)rec_cap * plan.grid * sizeof(sjk::MatchRecord)) +
                             (size_t)plan.grid * 4;

    // scratch layout: [repacked P][repacked Q][norms P][norms Q][block counts]
    //                 [block offsets][scan partials][match bits]
    size_t off_rp = 0, off_rq = 0, off_mask = 0;
    size_t off_np = 0, off_nq = 0, off_cnt = 0, off_offs = 0, off_part = 0, need = 0;
    if (!aligned) {
        off_rp = need;
        need = align_up(need + (size_t)rq.n_p * krow);
        off_rq = self ? off_rp : need;
        if (!self)
            need = align_up(need + (size_t)rq.n_q * krow);
    }
    if (l2) {
        off_np = need;
        need = align_up(need + (size_t)rq.n_p * 4);
        off_nq = self ? off_np : need;
        if (!self)
            need = align_up(need + (size_t)rq.n_q * 4);
    }
    if (blocks) {
        off_cnt = need;
        need = align_up(need + plan.n_blocks * 4);
        off_offs = need;
        need = align_up(need + plan.n_blocks * 8);
        off_part = need;
        need = align_up(need + sjk::scan_partials_size(plan.n_blocks) * 8);
    }
    off_mask = need;   // match bits or match records
    uint8_t *scr;
    unsigned long long *d_small = c->d_small;
    if (fx) {
        if (need > fx->bytes - kFixedHead)
            return fail(SJ_E_UNSUPPORTED,
                        "this call needs %zu bytes of device scratch; the fixed scratch of "
                        "sj_join_noalloc holds %zu",
                        need, fx->bytes - kFixedHead);
        d_small = (unsigned long long *)fx->base;
        scr = fx->base + kFixedHead;
    } else {
        const size_t extra = use_masks ? mask_bytes : use_records ? rec_bytes : 0;
        if (extra) {
            const std::string prev_err = g_err;
            if (grow_scratch(c, need + extra) != SJ_OK) {
                use_masks = use_records = false;   // recompute instead
                g_err = prev_err;
            }
        }
        if ((st = grow_scratch(c, use_masks || use_records ? need + extra : need)) != SJ_OK)
            return st;
        scr = (uint8_t *)c->scratch;
    }

    sjk::JoinArgs g = {};
    g.P = aligned ? (const uint8_t *)rq.P : scr + off_rp;
    g.Q = aligned ? (const uint8_t *)rq.Q : scr + off_rq;
    g.n_p = rq.n_p;
    g.n_q = rq.n_q;
    g.row_bytes = (uint32_t)krow;
    if (rq.dtype == SJ_I8) {
        if (!l2) {
            const double s = std::ceil(rq.thr);
            g.thr_i = s < -1073741824.0 ? -1073741824 : s > 1073741824.0 ? 1073741824 : (int32_t)s;
        } else {
            const double r = std::floor(rq.thr);
            g.thr_i = r < -1.0 ? -1 : r > 2147483647.0 ? 2147483647 : (int32_t)r;
        }
    } else {
        g.thr_f = l2 ? float_at_or_below(rq.thr) : float_at_or_above(rq.thr);
    }
    g.norm_p = scr + off_np;
    g.norm_q = scr + off_nq;
    g.pairs = rq.count_only ? nullptr : rq.pairs;
    g.cap = rq.count_only ? 0 : rq.cap;
    g.counter = d_small;
    g.block_counts = (uint32_t *)(scr + off_cnt);
    g.block_offsets = (const unsigned long long *)(scr + off_offs);
    g.masks = use_masks ? (uint16_t *)(scr + off_mask) : nullptr;
    g.records = use_records ? (sjk::MatchRecord *)(scr + off_mask) : nullptr;
    g.rec_cap = use_records ? (uint32_t)rec_cap : 0;
    g.rec_counts = use_records ? (uint32_t *)(scr + off_mask +
                                              align_up((size_t)rec_cap * plan.grid *
                                                       sizeof(sjk::MatchRecord)))
                               : nullptr;
    g.rec_max = d_small + 2;
    g.qsplit = plan.qsplit;

    hipStream_t s = c->stream;
    SJ_HIP(hipSetDevice(c->device));
    if (fx) {
        // the fixed region keeps the previous call's contents: clear the
        // counters (the count pass writes every block count itself)
        SJ_HIP(sjk::launch_zero_u64(d_small, 4, s));
    } else {
        if (!blocks)
            SJ_HIP(hipMemsetAsync(c->d_small, 0, sizeof(unsigned long long), s));
        if (use_records)
            SJ_HIP(hipMemsetAsync(c->d_small + 2, 0, sizeof(unsigned long long), s));
    }
    if (rq.timing)
        SJ_HIP(hipEventRecord(c->ev[0], s));
    if (!aligned) {
        SJ_HIP(sjk::launch_repack((const uint8_t *)rq.P, rq.n_p, (uint32_t)row_bytes,
                                  scr + off_rp, (uint32_t)krow, s));
        if (!self)
            SJ_HIP(sjk::launch_repack((const uint8_t *)rq.Q, rq.n_q, (uint32_t)row_bytes,
                                      scr + off_rq, (uint32_t)krow, s));
    }
    if (l2) {
        SJ_HIP(sjk::launch_norms(rq.dtype, g.P, rq.n_p, g.row_bytes, scr + off_np, s));
        if (!self)
            SJ_HIP(sjk::launch_norms(rq.dtype, g.Q, rq.n_q, g.row_bytes, scr + off_nq, s));
    }
    if (rq.timing)
        SJ_HIP(hipEventRecord(c->ev[1], s));

    uint64_t total = 0;
    bool emit_from_bits = false;
    if (!blocks) {
        // a self-join computes the upper triangle only and mirrors its pairs
        const bool tri = (self || rq.symmetric) && rq.n_p == rq.n_q;
        const int mode = tri ? sjk::MODE_TRI : sjk::MODE_SINGLE;
        SJ_HIP(sjk::launch_join(plan, rq.dtype, rq.metric, mode, g, s));
        if (rq.timing)
            SJ_HIP(hipEventRecord(c->ev[2], s));
        SJ_HIP(hipMemcpyAsync(c->h_small, d_small, sizeof(unsigned long long),
                              hipMemcpyDeviceToHost, s));
        SJ_HIP(hipStreamSynchronize(s));
        total = c->h_small[0];
        if (rq.timing) {
            c->stats.ms_norms = l2 ? elapsed_ms(c->ev[0], c->ev[1]) : 0.0;
            c->stats.ms_join = elapsed_ms(c->ev[1], c->ev[2]);
        }
    } else {
        SJ_HIP(sjk::launch_join(plan, rq.dtype, rq.metric,
                                use_masks     ? sjk::MODE_MASK
                                : use_records ? sjk::MODE_RECORD
                                              : sjk::MODE_COUNT,
                                g, s));
        if (rq.timing)
            SJ_HIP(hipEventRecord(c->ev[2], s));
        SJ_HIP(sjk::launch_scan(g.block_counts, plan.n_blocks,
                                (unsigned long long *)(scr + off_offs),
                                (unsigned long long *)(scr + off_part), d_small + 1, s));
        if (rq.timing)
            SJ_HIP(hipEventRecord(c->ev[3], s));
        SJ_HIP(hipMemcpyAsync(c->h_small + 1, d_small + 1, 2 * sizeof(unsigned long long),
                              hipMemcpyDeviceToHost, s));
        SJ_HIP(hipStreamSynchronize(s));
        total = c->h_small[1];
        if (use_records && c->h_small[2] > rec_cap)
            use_records = false;   // some blocks have no record: recompute
        if (rq.timing) {
            c->stats.ms_norms = l2 ? elapsed_ms(c->ev[0], c->ev[1]) : 0.0;
            c->stats.ms_count = elapsed_ms(c->ev[1], c->ev[2]);
            c->stats.ms_scan = elapsed_ms(c->ev[2], c->ev[3]);
        }
        if (!rq.count_only && total <= rq.cap && total > 0) {
            if (rq.timing)
                SJ_HIP(hipEventRecord(c->ev[4], s));
            if (use_masks)
                SJ_HIP(sjk::launch_emit_masks(plan, g, s));
            else if (use_records)
                SJ_HIP(sjk::launch_emit_records(g, plan.grid, s));
            else
                SJ_HIP(sjk::launch_join(plan, rq.dtype, rq.metric, sjk::MODE_EMIT, g, s));
            emit_from_bits = use_masks || use_records;
            if (rq.timing)
                SJ_HIP(hipEventRecord(c->ev[5], s));
            SJ_HIP(hipStreamSynchronize(s));
            if (rq.timing)
                c->stats.ms_emit = elapsed_ms(c->ev[4], c->ev[5]);
        }
    }
    c->stats.total = total;
    c->stats.kernel = (uint32_t)plan.family;
    c->stats.emit_from_bits = emit_from_bits ? 1u : 0u;
    c->stats.timed = rq.timing ? 1u : 0u;
    *n_out = total;
    if (!rq.count_only && total > rq.cap)
        return fail(SJ_E_OVERFLOW, "%llu matches exceed the capacity of %llu pairs",
                    (unsigned long long)total, (unsigned long long)rq.cap);
    return SJ_OK;
}

// Section 4's cosine ip-distance: P and Q normalised (f = g = x / ||x||) into
// the front-end buffer, then the inner-product join of the normalised rows.
int cosine_join(sj_ctx *c, Request rq, uint64_t *n_out)
{
    if (!c)
        return fail(SJ_E_INVAL, "context is NULL");
    if (!n_out)
        return fail(SJ_E_INVAL, "result pointer is NULL");
    *n_out = 0;
    if (rq.dtype != SJ_F16 && rq.dtype != SJ_BF16 && rq.dtype != SJ_I8)
        return fail(SJ_E_INVAL, "unknown dtype %d", rq.dtype);
    if (rq.d > 65536)
        return fail(SJ_E_UNSUPPORTED, "d = %u is above the limit", rq.d);
    const size_t es = esize(rq.dtype);
    int st;
    if ((st = check_device_ptr(c, rq.P, (size_t)rq.n_p * rq.d * es, "P")) != SJ_OK)
        return st;
    if ((st = check_device_ptr(c, rq.Q, (size_t)rq.n_q * rq.d * es, "Q")) != SJ_OK)
        return st;
    if (es == 2 && (((uintptr_t)rq.P | (uintptr_t)rq.Q) & 1))
        return fail(SJ_E_INVAL, "fp16 / bf16 rows must be 2-byte aligned");
    if (rq.n_p == 0 || rq.n_q == 0 || rq.d == 0) {
        // nothing to normalise: the join's own handling of empty inputs and
        // of d = 0 (every score 0) applies
        rq.dtype = rq.dtype == SJ_BF16 ? SJ_BF16 : SJ_F16;
        return run(c, rq, n_out);
    }
    const bool self = rq.P == rq.Q && rq.n_p == rq.n_q;
    const size_t bp = align_up((size_t)rq.n_p * rq.d * 2);
    const size_t bq = self ? 0 : align_up((size_t)rq.n_q * rq.d * 2);
    const size_t bn = (size_t)(rq.n_p > rq.n_q ? rq.n_p : rq.n_q) * sizeof(double);
    if ((st = grow_front(c, bp + bq + bn)) != SJ_OK)
        return st;
    uint8_t *f = (uint8_t *)c->front;
    double *norm = (double *)(f + bp + bq);
    SJ_HIP(hipSetDevice(c->device));
    SJ_HIP(sjk::launch_normalize(rq.dtype, rq.P, rq.n_p, rq.d, norm, f, c->stream));
    if (!self)
        SJ_HIP(sjk::launch_normalize(rq.dtype, rq.Q, rq.n_q, rq.d, norm, f + bp, c->stream));
    rq.P = f;
    rq.Q = self ? f : f + bp;
    rq.dtype = rq.dtype == SJ_BF16 ? SJ_BF16 : SJ_F16;
    return run(c, rq, n_out);
}

}  // namespace

extern "C" {

int sj_create(sj_ctx **out, int device, void *stream)
{
    g_err.clear();
    if (!out)
        return fail(SJ_E_INVAL, "ctx pointer is NULL");
    *out = nullptr;
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return hip_fail(e, "hipGetDeviceCount");
    }
    if (device < 0 || device >= n)
        return fail(SJ_E_INVAL, "device %d does not exist (%d visible)", device, n);
    hipDeviceProp_t prop;
    SJ_HIP(hipGetDeviceProperties(&prop, device));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(SJ_E_UNSUPPORTED, "device %d is %s; this library is built for gfx950", device,
                    prop.gcnArchName);
    SJ_HIP(hipSetDevice(device));
    sj_ctx *c = new (std::nothrow) sj_ctx();
    if (!c)
        return fail(SJ_E_NOMEM, "out of host memory");
    c->device = device;
    c->stream = (hipStream_t)stream;
    c->num_cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 256;
    if (hipMalloc(&c->d_small, 4 * sizeof(unsigned long long)) != hipSuccess ||
        hipHostMalloc(&c->h_small, 4 * sizeof(unsigned long long), hipHostMallocDefault) !=
            hipSuccess) {
        (void)hipGetLastError();
        sj_destroy(c);
        return fail(SJ_E_NOMEM, "cannot allocate the match counter");
    }
    for (auto &ev : c->ev)
        if (hipEventCreate(&ev) != hipSuccess) {
            (void)hipGetLastError();
            ev = nullptr;
            sj_destroy(c);
            return fail(SJ_E_HIP, "hipEventCreate failed");
        }
    // this device's copy of the no-allocation scratch, looked up once (a
    // failure only disables sj_join_noalloc, which then reports it)
    lookup_fixed_scratch(device);
    *out = c;
    return SJ_OK;
}

int sj_join_ip(sj_ctx *ctx, int dtype, const void *P, uint32_t n_p, const void *Q, uint32_t n_q,
               uint32_t d, double s, uint32_t *pairs, uint64_t cap, uint64_t *n_out,
               unsigned flags)
{
    g_err.clear();
    if (flags & ~(unsigned)(SJ_FLAG_TWO_PASS | SJ_FLAG_TIMING | SJ_FLAG_RECOMPUTE | SJ_FLAG_COSINE))
        return fail(SJ_E_INVAL, "unknown flags 0x%x", flags);
    Request rq{SJ_IP, dtype, P, Q, n_p, n_q, d, s, pairs, cap,
               (flags & SJ_FLAG_TWO_PASS) != 0, false, (flags & SJ_FLAG_TIMING) != 0,
               (flags & SJ_FLAG_RECOMPUTE) != 0};
    if (flags & SJ_FLAG_COSINE)
        return cosine_join(ctx, rq, n_out);
    return run(ctx, rq, n_out);
}

int sj_normalize(sj_ctx *ctx, int dtype, const void *X, uint32_t n, uint32_t d, void *Y)
{
    g_err.clear();
    if (!ctx)
        return fail(SJ_E_INVAL, "context is NULL");
    if (dtype != SJ_F16 && dtype != SJ_BF16 && dtype != SJ_I8)
        return fail(SJ_E_INVAL, "unknown dtype %d", dtype);
    if (d > 65536)
        return fail(SJ_E_UNSUPPORTED, "d = %u is above the limit", d);
    const size_t es = esize(dtype);
    int st;
    if ((st = check_device_ptr(ctx, X, (size_t)n * d * es, "X")) != SJ_OK)
        return st;
    if ((st = check_device_ptr(ctx, Y, (size_t)n * d * 2, "Y")) != SJ_OK)
        return st;
    if (((uintptr_t)Y & 1) || (es == 2 && ((uintptr_t)X & 1)))
        return fail(SJ_E_INVAL, "16-bit rows must be 2-byte aligned");
    ctx->stats = sj_stats{};
    if (n == 0 || d == 0)
        return SJ_OK;
    if ((st = grow_scratch(ctx, (size_t)n * sizeof(double))) != SJ_OK)
        return st;
    SJ_HIP(hipSetDevice(ctx->device));
    SJ_HIP(sjk::launch_normalize(dtype, X, n, d, (double *)ctx->scratch, Y, ctx->stream));
    SJ_HIP(hipStreamSynchronize(ctx->stream));
    return SJ_OK;
}

int sj_join_hamming(sj_ctx *ctx, const void *P, uint32_t n_p, const void *Q, uint32_t n_q,
                    uint32_t d, double r, uint32_t *pairs, uint64_t cap, uint64_t *n_out,
                    unsigned flags)
{
    g_err.clear();
    if (!ctx)
        return fail(SJ_E_INVAL, "context is NULL");
    if (!n_out)
        return fail(SJ_E_INVAL, "result pointer is NULL");
    *n_out = 0;
    if (std::isnan(r))
        return fail(SJ_E_INVAL, "radius is NaN");
    if (flags & ~(unsigned)(SJ_FLAG_TWO_PASS | SJ_FLAG_TIMING | SJ_FLAG_RECOMPUTE))
        return fail(SJ_E_INVAL, "unknown flags 0x%x", flags);
    if (d > 16384)
        return fail(SJ_E_UNSUPPORTED, "d = %u bits is above the limit of 16384", d);
    const size_t in_row = (d + 7) / 8;
    int st;
    if ((st = check_device_ptr(ctx, P, (size_t)n_p * in_row, "P")) != SJ_OK)
        return st;
    if ((st = check_device_ptr(ctx, Q, (size_t)n_q * in_row, "Q")) != SJ_OK)
        return st;
    Request rq{SJ_IP, SJ_I8, P, Q, n_p, n_q, 0, -r, pairs, cap,
               (flags & SJ_FLAG_TWO_PASS) != 0, false, (flags & SJ_FLAG_TIMING) != 0,
               (flags & SJ_FLAG_RECOMPUTE) != 0};
    if (n_p == 0 || n_q == 0 || d == 0)
        return run(ctx, rq, n_out);   // no pairs, or every distance 0 (d = 0)
    // f(x) and -g(y) as int8 rows of 2 d values, padded with zeros to 16 bytes
    const uint32_t rb = (uint32_t)((2 * (size_t)d + 15) & ~(size_t)15);
    const size_t bp = align_up((size_t)n_p * rb), bq = align_up((size_t)n_q * rb);
    if ((st = grow_front(ctx, bp + bq)) != SJ_OK)
        return st;
    uint8_t *f = (uint8_t *)ctx->front;
    SJ_HIP(hipSetDevice(ctx->device));
    SJ_HIP(sjk::launch_unpack_hamming((const uint8_t *)P, n_p, d, rb, 0, f, ctx->stream));
    SJ_HIP(sjk::launch_unpack_hamming((const uint8_t *)Q, n_q, d, rb, 1, f + bp, ctx->stream));
    rq.P = f;
    rq.Q = f + bp;
    rq.d = rb;
    rq.symmetric = P == Q && n_p == n_q;
    return run(ctx, rq, n_out);
}

int sj_join_l2(sj_ctx *ctx, int dtype, const void *P, uint32_t n_p, const void *Q, uint32_t n_q,
               uint32_t d, double r2, uint32_t *pairs, uint64_t cap, uint64_t *n_out,
               unsigned flags)
{
    g_err.clear();
    if (flags & ~(unsigned)(SJ_FLAG_TWO_PASS | SJ_FLAG_TIMING | SJ_FLAG_RECOMPUTE))
        return fail(SJ_E_INVAL, "flags 0x%x: sj_join_l2 takes SJ_FLAG_TWO_PASS, SJ_FLAG_TIMING "
                    "and SJ_FLAG_RECOMPUTE", flags);
    Request rq{SJ_L2, dtype, P, Q, n_p, n_q, d, r2, pairs, cap,
               (flags & SJ_FLAG_TWO_PASS) != 0, false, (flags & SJ_FLAG_TIMING) != 0,
               (flags & SJ_FLAG_RECOMPUTE) != 0};
    return run(ctx, rq, n_out);
}

int sj_count(sj_ctx *ctx, int metric, int dtype, const void *P, uint32_t n_p, const void *Q,
             uint32_t n_q, uint32_t d, double threshold, uint64_t *count)
{
    g_err.clear();
    Request rq{metric, dtype, P, Q, n_p, n_q, d, threshold, nullptr, 0, true, true, false, false};
    return run(ctx, rq, count);
}

int sj_join_noalloc(sj_ctx *ctx, int metric, int dtype, const void *P, uint32_t n_p,
                    const void *Q, uint32_t n_q, uint32_t d, double threshold, uint32_t *pairs,
                    uint64_t cap, uint64_t *n_out, unsigned flags)
{
    g_err.clear();
    if (!ctx)
        return fail(SJ_E_INVAL, "context is NULL");
    if (flags & ~(unsigned)(SJ_FLAG_TWO_PASS | SJ_FLAG_TIMING | SJ_FLAG_RECOMPUTE))
        return fail(SJ_E_INVAL, "unknown flags 0x%x", flags);
    uint8_t *base = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_fixed_mu);
        if (ctx->device >= 0 && ctx->device < kMaxDevices)
            base = g_fixed[ctx->device];
    }
    if (!base)
        return fail(SJ_E_HIP, "the fixed scratch of device %d is not available", ctx->device);
    const Fixed fx{base, kNoAllocScratchBytes};
    Request rq{metric, dtype, P, Q, n_p, n_q, d, threshold, pairs, cap,
               (flags & SJ_FLAG_TWO_PASS) != 0, false, (flags & SJ_FLAG_TIMING) != 0, true};
    return run(ctx, rq, n_out, &fx);
}

void sj_destroy(sj_ctx *c)
{
    if (!c)
        return;
    (void)hipSetDevice(c->device);
    if (c->stream || c->d_small)
        (void)hipStreamSynchronize(c->stream);
    for (auto &ev : c->ev)
        if (ev)
            (void)hipEventDestroy(ev);
    if (c->scratch)
        (void)hipFree(c->scratch);
    if (c->front)
        (void)hipFree(c->front);
    if (c->d_small)
        (void)hipFree(c->d_small);
    if (c->h_small)
        (void)hipHostFree(c->h_small);
    delete c;
}

int sj_get_stats(const sj_ctx *ctx, sj_stats *out)
{
    if (!ctx || !out)
        return fail(SJ_E_INVAL, "NULL argument");
    *out = ctx->stats;
    return SJ_OK;
}

const char *sj_last_error(void) { return g_err.c_str(); }

}  // extern "C"
