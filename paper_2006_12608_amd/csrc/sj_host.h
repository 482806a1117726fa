// sj_host.h -- host-side state and helpers shared by the library's entry
// points (sj_api.cpp: the all-pairs join; sj_lsh_api.cpp: the LSH-bucketed join).
// Not part of the public C-ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>

#include "sj.h"

struct sj_ctx {
    int device = 0;
    hipStream_t stream = nullptr;
    int num_cus = 256;
    unsigned long long *d_small = nullptr;  // [0] match counter, [1] scan total,
                                            // [2] largest per-workgroup record count
    unsigned long long *h_small = nullptr;  // pinned host copy of d_small
    void *scratch = nullptr;
    size_t scratch_bytes = 0;
    void *front = nullptr;        // rows made by the front ends (normalised or
    size_t front_bytes = 0;       // unpacked), kept apart from the join's scratch
    hipEvent_t ev[6] = {};
    sj_stats stats = {};
};

namespace sjh {

// Message of the calling thread's last failure (sj_last_error).
extern thread_local std::string g_err;

// Records the message and returns `code`.
int fail(int code, const char *fmt, ...);
int hip_fail(hipError_t e, const char *what);

#define SJ_HIP(call)                                \
    do {                                            \
        hipError_t e_ = (call);                     \
        if (e_ != hipSuccess)                       \
            return sjh::hip_fail(e_, #call);        \
    } while (0)

// Bytes per element of a dtype code.
size_t esize(int dtype);

// `p` must be device memory of the context's GPU holding at least `bytes`
// bytes from p on (checked against its allocation's range).
int check_device_ptr(const sj_ctx *c, const void *p, size_t bytes, const char *name);

// Smallest float >= s / largest float <= r.
float float_at_or_above(double s);
float float_at_or_below(double r);

// Grows the context's scratch to at least `bytes` (contents not kept).
int grow_scratch(sj_ctx *c, size_t bytes);

// Grows the context's front-end buffer to at least `bytes` (contents not kept).
int grow_front(sj_ctx *c, size_t bytes);

inline size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

double elapsed_ms(hipEvent_t a, hipEvent_t b);

}  // namespace sjh
