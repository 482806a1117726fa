// sj_lsh_api.cpp -- host side of the LSH-bucketed join (sj_join_lsh; contract in
// include/sj.h): argument checks, scratch layout and the sequence
// hash -> sort -> bucket pairs -> bucket join on the context's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "sj.h"
#include "sj_host.h"
#include "sj_internal.h"
#include "sj_lsh.h"

using namespace sjh;

namespace {

// Tables and records are addressed with 32-bit positions.
const uint64_t kMaxTableRows = (uint64_t)1 << 32;
const uint32_t kMaxTables = 256;

}  // namespace

extern "C" int sj_join_lsh(sj_ctx *c, int metric, int dtype, const void *P, uint32_t n_p,
                           const void *Q, uint32_t n_q, uint32_t d, double thr, uint32_t L,
                           uint32_t k, const int8_t *A, const int32_t *B, int32_t w,
                           uint32_t *pairs, uint64_t cap, uint64_t *n_out, uint64_t *n_cand)
{
    g_err.clear();
    if (!c)
        return fail(SJ_E_INVAL, "context is NULL");
    if (!n_out)
        return fail(SJ_E_INVAL, "result pointer is NULL");
    *n_out = 0;
    if (n_cand)
        *n_cand = 0;
    if (dtype != SJ_F16 && dtype != SJ_BF16 && dtype != SJ_I8)
        return fail(SJ_E_INVAL, "unknown dtype %d", dtype);
    if (metric != SJ_IP && metric != SJ_L2)
        return fail(SJ_E_INVAL, "unknown metric %d", metric);
    if (std::isnan(thr))
        return fail(SJ_E_INVAL, "threshold is NaN");
    if (L < 1 || L > kMaxTables)
        return fail(SJ_E_INVAL, "L = %u tables: 1 <= L <= %u", L, kMaxTables);
    if (k > 64)
        return fail(SJ_E_INVAL, "k = %u functions per table: k <= 64", k);
    if (w < 0)
        return fail(SJ_E_INVAL, "bucket width w = %d is negative", w);
    if (d > (dtype == SJ_I8 ? 32768u : 65536u))
        return fail(SJ_E_UNSUPPORTED, "d = %u is above the limit for this dtype", d);
    const uint64_t n_max = n_p > n_q ? n_p : n_q;
    if ((uint64_t)L * n_max >= kMaxTableRows)
        return fail(SJ_E_UNSUPPORTED, "L * max(n_p, n_q) = %llu is not below 2^32",
                    (unsigned long long)L * n_max);
    const size_t row_bytes = (size_t)d * esize(dtype);
    int st;
    if ((st = check_device_ptr(c, P, (size_t)n_p * row_bytes, "P")) != SJ_OK)
        return st;
    if ((st = check_device_ptr(c, Q, (size_t)n_q * row_bytes, "Q")) != SJ_OK)
        return st;
    if ((st = check_device_ptr(c, A, (size_t)L * k * d, "A")) != SJ_OK)
        return st;
    if (w > 0 && (st = check_device_ptr(c, B, (size_t)L * k * 4, "B")) != SJ_OK)
        return st;
    if (cap > 0) {
        if (cap > (uint64_t)SIZE_MAX / 8)
            return fail(SJ_E_INVAL, "cap too large");
        if ((st = check_device_ptr(c, pairs, (size_t)cap * 8, "pairs")) != SJ_OK)
            return st;
        if ((uintptr_t)pairs % 8 != 0)
            return fail(SJ_E_INVAL, "pairs must be 8-byte aligned");
    }
    c->stats = sj_stats{};
    if (n_p == 0 || n_q == 0)
        return SJ_OK;

    // Rows as the kernels read them (16-byte aligned, zero-padded to a
    // multiple of 16 bytes; repacked when the caller's are not).
    const bool aligned = row_bytes > 0 && row_bytes % 16 == 0 && (uintptr_t)P % 16 == 0 &&
                         (uintptr_t)Q % 16 == 0;
    const size_t krow = row_bytes == 0 ? 16 : (row_bytes + 15) & ~(size_t)15;
    const bool self = P == Q && n_p == n_q;
    const bool l2 = metric == SJ_L2;
    const uint32_t bits = sjl::key_bits(k, w);
    // records: at most min(n_p, n_q) per table (a table has at most that
    // many keys shared by P and Q); packing chunks of them
    const uint64_t bp_cap = (uint64_t)L * (n_p < n_q ? n_p : n_q);
    const uint64_t chunk_cap = (bp_cap + sjl::PACK_CHUNK - 1) / sjl::PACK_CHUNK;
    const uint64_t pos_p = (uint64_t)L * n_p;   // sorted positions of P, all tables
    // one sort workspace, used by P and then by Q
    const size_t temp_bytes = std::max(sjl::sort_temp_bytes(n_max, L),
                                       sjl::bucket_find_ws_bytes(n_p, L));
    const size_t a_bytes = sjl::widened_bytes(dtype, L, k, d);

    // scratch: [rows P][rows Q][norms P][norms Q][keys P][keys Q][sorted P]
    //          [sorted Q][perm P][perm Q][fingerprints P, Q][row records P, Q]
    //          [bucket marks, sizes and numbers]
    //          [records][chunk counts and offsets][descriptors][scan partials]
    //          [counters][sort temp][widened projections]
    size_t need = 0;
    auto take = [&](size_t bytes) {
        const size_t at = need;
        need = align_up(need + bytes);
        return at;
    };
    const size_t off_rp = aligned ? 0 : take((size_t)n_p * krow);
    const size_t off_rq = aligned || self ? off_rp : take((size_t)n_q * krow);
    const size_t off_np = l2 ? take((size_t)n_p * 4) : 0;
    const size_t off_nq = l2 && !self ? take((size_t)n_q * 4) : off_np;
    const size_t off_kp = take((size_t)L * n_p * 8);
    const size_t off_kq = self ? off_kp : take((size_t)L * n_q * 8);
    const size_t off_sp = take((size_t)L * n_p * 8);
    const size_t off_sq = self ? off_sp : take((size_t)L * n_q * 8);
    const size_t off_pp = take((size_t)L * n_p * 4);
    const size_t off_pq = self ? off_pp : take((size_t)L * n_q * 4);
    // short rows travel to the bucket join as records with their norm and
    // fingerprints (one cache line per row); longer ones with 16 fingerprint
    // bytes per row in an array of their own
    const bool use_rec = krow <= sjl::REC_ROW && n_max * sjl::REC_BYTES <= 0xffffffffull;
    const size_t off_fpp = use_rec ? 0 : take((size_t)n_p * 16);
    const size_t off_fpq = use_rec || self ? off_fpp : take((size_t)n_q * 16);
    const size_t off_recp = use_rec ? take((size_t)n_p * sjl::REC_BYTES) : 0;
    const size_t off_recq = use_rec && !self ? take((size_t)n_q * sjl::REC_BYTES) : off_recp;
    const size_t off_flag = take(pos_p * 4);
    const size_t off_fnp = take(pos_p * 4);
    const size_t off_fq0 = take(pos_p * 4);
    const size_t off_fnq = take(pos_p * 4);
    const size_t off_roff = take(pos_p * 8);
    const size_t off_rect = take(bp_cap * 4);
    const size_t off_recpq = take(bp_cap * 16);
    const size_t off_cdesc = take(chunk_cap * 4);
    const size_t off_ctile = take(chunk_cap * 4);
    const size_t off_doff = take(chunk_cap * 8);
    const size_t off_toff = take(chunk_cap * 8);
    const size_t off_dhead = take(bp_cap * 16);
    const size_t off_dpq = take(bp_cap * 16);
    const size_t off_dtile = take(bp_cap * 8);
    const size_t off_part = take(sjk::scan_partials_size(pos_p > chunk_cap ? pos_p : chunk_cap) * 8);
    // counters: [0] pair evaluations, [1] records, [2] descriptors, [3] [4]
    // the hash's fix queues, [5] tiles, [6] tile overflow, [7] bucket rows
    const size_t off_cnt = take(8 * 8);
    const size_t off_temp = take(temp_bytes);
    const size_t off_aw = take(a_bytes);
    // keys on the matrix cores where they apply
    const bool fast = sjl::keys_fast_applies(dtype, (uint32_t)krow, L, k, w);
    const size_t off_ws = fast ? take(sjl::keys_fast_bytes((uint32_t)n_max, L, k, (uint32_t)krow)) : 0;
    if ((st = grow_scratch(c, need)) != SJ_OK)
        return st;
    uint8_t *scr = (uint8_t *)c->scratch;
    hipStream_t s = c->stream;
    SJ_HIP(hipSetDevice(c->device));

    sjl::Rows rp{aligned ? (const uint8_t *)P : scr + off_rp, n_p, (uint32_t)krow};
    sjl::Rows rq{aligned ? (const uint8_t *)Q : scr + off_rq, n_q, (uint32_t)krow};
    unsigned long long *cnt = (unsigned long long *)(scr + off_cnt);
    SJ_HIP(hipMemsetAsync(cnt, 0, 8 * 8, s));
    SJ_HIP(hipMemsetAsync(c->d_small, 0, sizeof(unsigned long long), s));
    SJ_HIP(hipEventRecord(c->ev[0], s));
    if (!aligned) {
        SJ_HIP(sjk::launch_repack((const uint8_t *)P, n_p, (uint32_t)row_bytes, scr + off_rp,
                                  (uint32_t)krow, s));
        if (!self)
            SJ_HIP(sjk::launch_repack((const uint8_t *)Q, n_q, (uint32_t)row_bytes,
                                      scr + off_rq, (uint32_t)krow, s));
    }
    if (l2) {
        SJ_HIP(sjk::launch_norms(dtype, rp.X, n_p, rp.row_bytes, scr + off_np, s));
        if (!self)
            SJ_HIP(sjk::launch_norms(dtype, rq.X, n_q, rq.row_bytes, scr + off_nq, s));
    }
    uint64_t *keys_p = (uint64_t *)(scr + off_kp), *keys_q = (uint64_t *)(scr + off_kq);
    SJ_HIP(sjl::launch_widen(dtype, A, L * k, d, scr + off_aw, s));
    if (fast) {
        SJ_HIP(sjl::launch_keys_fast(dtype, rp, d, L, k, A, scr + off_aw, B, w, keys_p,
                                     scr + off_ws, true, cnt + 3, s));
        if (!self)
            SJ_HIP(sjl::launch_keys_fast(dtype, rq, d, L, k, A, scr + off_aw, B, w,
                                         keys_q, scr + off_ws, false, cnt + 4, s));
    } else {
        SJ_HIP(sjl::launch_keys(dtype, rp, d, L, k, scr + off_aw, B, w, keys_p, s));
        if (!self)
            SJ_HIP(sjl::launch_keys(dtype, rq, d, L, k, scr + off_aw, B, w, keys_q, s));
    }
    uint4 *fp_p = (uint4 *)(scr + off_fpp), *fp_q = (uint4 *)(scr + off_fpq);
    if (use_rec) {
        SJ_HIP(sjl::launch_rowrec(rp, l2 ? scr + off_np : nullptr, keys_p, L, scr + off_recp, s));
        if (!self)
            SJ_HIP(sjl::launch_rowrec(rq, l2 ? scr + off_nq : nullptr, keys_q, L,
                                      scr + off_recq, s));
    } else if (L > 1) {
        SJ_HIP(sjl::launch_fingerprints(keys_p, n_p, L, fp_p, s));
        if (!self)
            SJ_HIP(sjl::launch_fingerprints(keys_q, n_q, L, fp_q, s));
    }
    SJ_HIP(hipEventRecord(c->ev[1], s));
    uint64_t *sorted_p = (uint64_t *)(scr + off_sp), *sorted_q = (uint64_t *)(scr + off_sq);
    uint32_t *perm_p = (uint32_t *)(scr + off_pp), *perm_q = (uint32_t *)(scr + off_pq);
    SJ_HIP(sjl::sort_tables(keys_p, sorted_p, perm_p, n_p, L, bits, scr + off_temp, s));
    if (!self)
        SJ_HIP(sjl::sort_tables(keys_q, sorted_q, perm_q, n_q, L, bits, scr + off_temp, s));
    // the buckets P and Q share, as records in key order, then their tiles
    uint32_t *flag = (uint32_t *)(scr + off_flag);
    // (its per-block sums in the sorts' workspace, free by now)
    SJ_HIP(sjl::launch_bucket_find(sorted_p, n_p, sorted_q, n_q, L, scr + off_temp, flag,
                                   (uint32_t *)(scr + off_fnp), (uint32_t *)(scr + off_fq0),
                                   (uint32_t *)(scr + off_fnq), cnt, s));
    unsigned long long *part = (unsigned long long *)(scr + off_part);
    SJ_HIP(sjk::launch_scan(flag, pos_p, (unsigned long long *)(scr + off_roff), part, cnt + 1, s));
    const sjl::Records rec{(uint32_t *)(scr + off_rect), (uint4 *)(scr + off_recpq)};
    SJ_HIP(sjl::launch_bucket_write(n_p, L, flag, (const uint32_t *)(scr + off_fnp),
                                    (const uint32_t *)(scr + off_fq0),
                                    (const uint32_t *)(scr + off_fnq),
                                    (const unsigned long long *)(scr + off_roff), rec, s));
    SJ_HIP(hipMemcpyAsync(c->h_small, cnt + 1, 8, hipMemcpyDeviceToHost, s));
    SJ_HIP(hipStreamSynchronize(s));
    const uint64_t n_rec = c->h_small[0];
    const uint64_t n_chunk = (n_rec + sjl::PACK_CHUNK - 1) / sjl::PACK_CHUNK;
    const sjl::Descs desc{(uint4 *)(scr + off_dhead), (uint4 *)(scr + off_dpq),
                          (unsigned long long *)(scr + off_dtile)};
    uint32_t *cdesc = (uint32_t *)(scr + off_cdesc), *ctile = (uint32_t *)(scr + off_ctile);
    unsigned long long *doff = (unsigned long long *)(scr + off_doff);
    unsigned long long *toff = (unsigned long long *)(scr + off_toff);
    SJ_HIP(sjl::launch_pack(rec, (uint32_t)n_rec, false, cdesc, ctile, nullptr, nullptr, desc,
                            cnt + 6, s));
    if (n_chunk) {
        SJ_HIP(sjk::launch_scan(cdesc, n_chunk, doff, part, cnt + 2, s));
        SJ_HIP(sjk::launch_scan(ctile, n_chunk, toff, part, cnt + 5, s));
    }
    SJ_HIP(sjl::launch_pack(rec, (uint32_t)n_rec, true, cdesc, ctile, doff, toff, desc, cnt + 6,
                            s));
    SJ_HIP(hipEventRecord(c->ev[2], s));
    unsigned long long hc[8];
    SJ_HIP(hipMemcpyAsync(hc, cnt, sizeof hc, hipMemcpyDeviceToHost, s));
    SJ_HIP(hipStreamSynchronize(s));
    if (hc[6])
        return fail(SJ_E_UNSUPPORTED, "a chunk of buckets needs more than 2^32 tiles");

    sjl::JoinArgs g = {};
    const uint64_t n_tiles = hc[5], cand = hc[0];
    g.P = rp;
    g.Q = rq;
    g.L = L;
    g.perm_p = perm_p;
    g.perm_q = perm_q;
    g.keys_p = keys_p;
    g.keys_q = keys_q;
    g.fp_p = use_rec ? nullptr : fp_p;
    g.fp_q = use_rec ? nullptr : fp_q;
    g.rec_p = use_rec ? scr + off_recp : nullptr;
    g.rec_q = use_rec ? scr + off_recq : nullptr;
    g.rec = rec;
    g.desc = desc;
    g.n_desc = (uint32_t)hc[2];
    g.n_tiles = n_tiles;
    if (dtype == SJ_I8) {
        if (!l2) {
            const double sc = std::ceil(thr);
            g.thr_i = sc < -1073741824.0 ? -1073741824 : sc > 1073741824.0 ? 1073741824
                                                                          : (int32_t)sc;
        } else {
            const double r = std::floor(thr);
            g.thr_i = r < -1.0 ? -1 : r > 2147483647.0 ? 2147483647 : (int32_t)r;
        }
    } else {
        g.thr_f = l2 ? float_at_or_below(thr) : float_at_or_above(thr);
    }
    g.norm_p = scr + off_np;
    g.norm_q = scr + off_nq;
    g.pairs = pairs;
    g.cap = cap;
    g.counter = c->d_small;
    SJ_HIP(sjl::launch_join(dtype, metric, g, c->num_cus, s));
    SJ_HIP(hipEventRecord(c->ev[3], s));
    SJ_HIP(hipMemcpyAsync(c->h_small, c->d_small, 8, hipMemcpyDeviceToHost, s));
    SJ_HIP(hipStreamSynchronize(s));
    const uint64_t total = c->h_small[0];
    c->stats.total = total;
    c->stats.ms_norms = elapsed_ms(c->ev[0], c->ev[1]);
    c->stats.ms_scan = elapsed_ms(c->ev[1], c->ev[2]);
    c->stats.ms_join = elapsed_ms(c->ev[2], c->ev[3]);
    c->stats.kernel = 3;
    c->stats.timed = 1;
    c->stats.lsh_rows = hc[7];
    *n_out = total;
    if (n_cand)
        *n_cand = cand;
    if (total > cap)
        return fail(SJ_E_OVERFLOW, "%llu matches exceed the capacity of %llu pairs",
                    (unsigned long long)total, (unsigned long long)cap);
    return SJ_OK;
}

// The grouping of the LSH-bucketed join's tables on its own (Section 4: the
// points of each table grouped by bucket); contract in include/sj.h.
extern "C" int sj_lsh_sort(sj_ctx *c, const uint64_t *keys, uint32_t n, uint32_t L,
                           uint32_t bits, uint32_t *perm)
{
    g_err.clear();
    if (!c)
        return fail(SJ_E_INVAL, "context is NULL");
    if (bits > 64)
        return fail(SJ_E_INVAL, "bits = %u: at most 64", bits);
    const uint64_t total = (uint64_t)L * n;
    if (total >= kMaxTableRows)
        return fail(SJ_E_UNSUPPORTED, "L * n = %llu is not below 2^32",
                    (unsigned long long)total);
    c->stats = sj_stats{};
    if (total == 0)
        return SJ_OK;
    int st;
    if ((st = check_device_ptr(c, keys, total * 8, "keys")) != SJ_OK)
        return st;
    if ((st = check_device_ptr(c, perm, total * 4, "perm")) != SJ_OK)
        return st;
    if ((uintptr_t)keys % 8 != 0 || (uintptr_t)perm % 4 != 0)
        return fail(SJ_E_INVAL, "keys must be 8-byte and perm 4-byte aligned");
    const size_t off_sorted = 0;
    const size_t off_temp = align_up(total * 8);
    if ((st = grow_scratch(c, off_temp + sjl::sort_temp_bytes(n, L))) != SJ_OK)
        return st;
    uint8_t *scr = (uint8_t *)c->scratch;
    hipStream_t s = c->stream;
    SJ_HIP(hipSetDevice(c->device));
    SJ_HIP(sjl::sort_tables(keys, (uint64_t *)(scr + off_sorted), perm, n, L, bits,
                            scr + off_temp, s));
    SJ_HIP(hipStreamSynchronize(s));
    return SJ_OK;
}

// Section 4's parameter choice for the LSH-bucketed join (host only).
extern "C" double sj_lsh_collision(int32_t w, double sigma, double dist)
{
    if (std::isnan(dist) || dist < 0.0 || w < 0)
        return std::nan("");
    if (w == 0) {
        // random hyperplane through the origin: it separates two vectors at
        // angle theta with probability theta / pi
        if (dist > M_PI)
            return std::nan("");
        return 1.0 - dist / M_PI;
    }
    // floor((<a, x> + b) / w) with a ~ N(0, sigma^2 I), b ~ U[0, w): the
    // projections of two points at distance dist differ by u Z, u = sigma dist,
    // Z ~ N(0, 1), and collide with probability E[max(0, 1 - u |Z| / w)] =
    // 1 - 2 Phi(-w / u) - 2 u / (sqrt(2 pi) w) (1 - exp(-w^2 / (2 u^2)))
    if (!(sigma > 0.0))
        return std::nan("");
    const double u = sigma * dist;
    if (u == 0.0)
        return 1.0;
    const double c = (double)w / u;
    const double phi = 0.5 * std::erfc(c / std::sqrt(2.0));   // Phi(-c)
    return 1.0 - 2.0 * phi - 2.0 / (std::sqrt(2.0 * M_PI) * c) * (1.0 - std::exp(-0.5 * c * c));
}

extern "C" int sj_lsh_plan(double p1, double p2, uint64_t n, uint32_t tile, double recall,
                           uint32_t *k, uint32_t *L_inst, uint32_t *reps)
{
    g_err.clear();
    if (!k || !L_inst || !reps)
        return fail(SJ_E_INVAL, "NULL output");
    if (!(p2 > 0.0 && p2 < p1 && p1 < 1.0))
        return fail(SJ_E_INVAL, "need 0 < p2 < p1 < 1 (p1 = %g, p2 = %g)", p1, p2);
    if (!(recall > 0.0 && recall < 1.0))
        return fail(SJ_E_INVAL, "recall %g is not in (0, 1)", recall);
    if (tile == 0 || n == 0)
        return fail(SJ_E_INVAL, "tile and n must be positive");
    // p2^k <= tile / n: a point collides with at most `tile` far points per
    // table in expectation (one tile of the matrix cores); k = 0 when n <= tile
    uint32_t kk = 0;
    const double target = (double)tile / (double)n;
    double pk = 1.0;
    while (pk > target) {
        pk *= p2;
        if (++kk > 64)
            return fail(SJ_E_UNSUPPORTED, "more than 64 functions per table needed");
    }
    // one instance: L = ceil(1 / p1^k) tables find a pair at the threshold
    // with probability 1 - (1 - p1^k)^L >= 1 - 1/e
    const double q = std::pow(p1, (double)kk);
    const double L = std::ceil(1.0 / q - 1e-9);
    if (L > 4294967295.0)
        return fail(SJ_E_UNSUPPORTED, "1 / p1^k = %g tables", 1.0 / q);
    // R independent instances merged miss it with probability <= e^-R
    const double R = std::ceil(-std::log(1.0 - recall) - 1e-12);
    *k = kk;
    *L_inst = (uint32_t)L;
    *reps = (uint32_t)(R < 1.0 ? 1.0 : R);
    return SJ_OK;
}
