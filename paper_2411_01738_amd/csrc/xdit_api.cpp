// C ABI of the library (declared in include/xdit.h): argument validation,
// the per-thread stream and error message, and dispatch to the HIP kernels.
// Every check runs before any HIP call, so a rejected call touches neither the
// device nor the caller's buffers.
#include <cmath>
#include "../../include/xdit.h"

#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <map>
#include <mutex>
#include <tuple>

#include "kernels.h"

namespace {

thread_local hipStream_t g_stream = nullptr;
thread_local char g_error[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof(g_error), fmt, ap);
    va_end(ap);
    return code;
}

void clear_error() { g_error[0] = '\0'; }

constexpr int64_t kMaxDim = INT32_MAX;

int esize_of(int32_t dtype) { return dtype == XDIT_BF16 ? 2 : 4; }

int check_dtype_dim(int32_t dtype, int64_t head_dim) {
    if (dtype != XDIT_BF16 && dtype != XDIT_F32)
        return fail(XDIT_ERR_DTYPE, "unknown dtype %d (expected XDIT_BF16=0 or XDIT_F32=1)", dtype);
    if (head_dim != 64 && head_dim != 72 && head_dim != 128)
        return fail(XDIT_ERR_UNSUPPORTED, "head_dim %lld not supported (64, 72 or 128)",
                    (long long)head_dim);
    return XDIT_OK;
}

int check_dims(const char* what, int64_t B, int64_t n1, int64_t n2, int64_t H) {
    if (B < 0 || n1 < 0 || n2 < 0 || H < 0)
        return fail(XDIT_ERR_SHAPE, "%s: negative dimension", what);
    if (B > kMaxDim || n1 > kMaxDim || n2 > kMaxDim || H > kMaxDim)
        return fail(XDIT_ERR_SHAPE, "%s: dimension exceeds 2^31-1", what);
    // keep every tensor below 2^40 elements so offsets never overflow
    if ((double)B * (double)(n1 > n2 ? n1 : n2) * (double)H * 128.0 > 1099511627776.0)
        return fail(XDIT_ERR_SHAPE, "%s: tensor too large", what);
    return XDIT_OK;
}

// The kernels address each batch's rows with 32-bit byte offsets, plus up to
// one tile (256 rows) of look-ahead past the end.
int check_batch_bytes(const char* what, int64_t rows, int64_t heads, int64_t head_dim, int esize) {
    const int64_t row = heads * head_dim * esize;
    if ((rows + 256) * row >= ((int64_t)1 << 31))
        return fail(XDIT_ERR_SHAPE, "%s: one batch of a tensor exceeds 2 GiB", what);
    return XDIT_OK;
}

struct Span {
    const void* p;
    int64_t bytes;
    const char* name;
};

bool overlap(const Span& a, const Span& b) {
    if (a.bytes <= 0 || b.bytes <= 0) return false;
    const uintptr_t a0 = (uintptr_t)a.p, b0 = (uintptr_t)b.p;
    return a0 < b0 + (uintptr_t)b.bytes && b0 < a0 + (uintptr_t)a.bytes;
}

int check_ptr(const Span& s) {
    if (s.bytes > 0 && s.p == nullptr) return fail(XDIT_ERR_NULL, "%s is NULL", s.name);
    if (s.bytes > 0 && ((uintptr_t)s.p & 15u) != 0)
        return fail(XDIT_ERR_LAYOUT, "%s is not 16-byte aligned", s.name);
    return XDIT_OK;
}

int check_no_overlap(const Span& out, const Span& in) {
    if (overlap(out, in)) return fail(XDIT_ERR_ALIAS, "%s overlaps %s", out.name, in.name);
    return XDIT_OK;
}

int hip_status(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(XDIT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return XDIT_OK;
}

#define XDIT_TRY(expr)            \
    do {                          \
        const int rc_ = (expr);   \
        if (rc_ != XDIT_OK) return rc_; \
    } while (0)

}  // namespace

extern "C" {

int xdit_set_stream(void* stream) {
    g_stream = (hipStream_t)stream;
    return XDIT_OK;
}

void* xdit_get_stream(void) { return (void*)g_stream; }

const char* xdit_last_error(void) { return g_error; }

const char* xdit_version(void) { return "xdit-mi355x 0.1 (gfx950)"; }

struct SplitArgs {
    int32_t splits = 1;        // requested (<= 0: the library picks)
    void* workspace = nullptr;
    int64_t workspace_bytes = 0;
};

static constexpr int kCUs = 256;
static constexpr int kPartRows = xdit::kPartSlotRows;  // query rows per tile of a partitioned launch

static int64_t align256(int64_t x) { return (x + 255) / 256 * 256; }

// Query tiles of a partitioned launch (128 rows) over the batch and heads.
static int64_t part_pairs(int64_t batch, int64_t q_len, int64_t heads) {
    return (q_len + kPartRows - 1) / kPartRows * batch * heads;
}

// A work partition of a bf16 launch (see xdit::AttnParams): `whole`
// workgroups sweep query tiles whole, `parts` workgroups take the cut ranges
// of the rest; parts = 0: one workgroup per query tile.
struct Partition {
    int64_t whole = 0, parts = 0;
};

// Workspace of a partitioned launch: one partial slot (O and LSE in float32)
// per cut range, two when ranges may cross query tiles.
static int64_t part_ws_bytes(const Partition& pt, int64_t pairs, int64_t head_dim) {
    if (pt.parts <= 0) return 0;
    const int64_t slots = pt.parts % (pairs - pt.whole) == 0 ? pt.parts : 2 * pt.parts;
    return align256(slots * kPartRows * (head_dim + 1) * 4);
}

// The library's partition for `pairs` query tiles over kv_len keys.  Time
// model in units of one 128-key tile of one workgroup: a workgroup's sweep
// (or part of one) costs a fixed ~5 tiles (prologue, pipeline fill,
// epilogue) plus its tiles; each round of workgroups over the CUs costs its
// longest member; cut sweeps add the fix-up launch (~3 tiles).  Candidates:
//   * one workgroup per query tile (of 128 rows, or of 64 at d <= 72);
//   * every sweep cut into s even parts (s = 2..XDIT_MAX_SPLITS), for query
//     tiles that leave CUs idle;
//   * the query tiles of the full rounds whole and each of the r left over
//     cut into s = min(16, 256 / r) parts, so that the last round is full
//     (K/V reuse among the query tiles of one head is kept in the rounds of
//     whole sweeps).
// A partition is taken only when the model saves at least 10 %.  The model
// counts rounds of one workgroup per CU; at d = 128 the kernel runs two
// 4-wave workgroups per CU, for which flux's measured alternatives (whole
// rounds of 512 with the rest cut, 512 equal ranges) were no faster than
// this choice.
// XDIT_PARTITION=balanced instead cuts the whole launch into 256 equal
// ranges (ranges cross query tiles; it loses the K/V reuse, so it is never
// chosen; tests use it), XDIT_PARTITION=none forces no partition.
static Partition pick_parts(int64_t pairs, int64_t kv_len, int64_t head_dim) {
    Partition none;
    const char* force = getenv("XDIT_PARTITION");
    if (force && strcmp(force, "none") == 0) return none;
    const int64_t bn = head_dim > 96 ? 64 : 128;  // kernel K/V tile
    const int64_t T = (kv_len + bn - 1) / bn > 1 ? (kv_len + bn - 1) / bn : 1;
    if (force && strcmp(force, "balanced") == 0) {
        // every sweep may meet at most kMaxSweepParts ranges
        if (pairs * T / kCUs * (xdit::kMaxSweepParts - 1) >= T) {
            Partition b;
            b.parts = kCUs;
            return b;
        }
        return none;
    }
    const double t = (double)((kv_len + 127) / 128 > 1 ? (kv_len + 127) / 128 : 1);
    const double ovh = 5.0, fix = 3.0;
    auto rounds = [](int64_t n) { return (double)((n + kCUs - 1) / kCUs); };
    // unpartitioned: 128-row query tiles, or at d <= 72 64-row ones (twice
    // the workgroups, half the work per tile)
    double plain = rounds(pairs) * (t + ovh);
    if (head_dim <= 72 && rounds(2 * pairs) * (t / 2 + ovh) < plain) plain = rounds(2 * pairs) * (t / 2 + ovh);
    double best = plain;
    Partition pick;
    for (int s = 2; s <= XDIT_MAX_SPLITS && t >= 4.0 * s; ++s) {
        const double c = rounds(pairs * s) * (ovh + t / s) + fix;
        if (c < best) {
            best = c;
            pick.whole = 0;
            pick.parts = pairs * s;
        }
    }
    const int64_t full = pairs / kCUs * kCUs, r = pairs - full;
    const int64_t s = r > 0 ? (kCUs / r < XDIT_MAX_SPLITS ? kCUs / r : XDIT_MAX_SPLITS) : 0;
    if (full > 0 && s >= 2 && t >= 2.0 * s) {
        const double c = (double)(full / kCUs) * (t + ovh) + (ovh + t / s) + fix;
        if (c < best) {
            best = c;
            pick.whole = full;
            pick.parts = r * s;
        }
    }
    return best < 0.9 * plain ? pick : none;
}

// The partition of a call: none for float32 (not partitioned) or for
// sweeps of at most one K/V tile (nothing to cut: a part would sweep its
// query tile whole), every sweep in `splits` even parts for splits > 1, the
// library's choice for splits <= 0.
static Partition call_parts(int32_t dtype, int64_t pairs, int64_t kv_len, int64_t head_dim, int32_t splits) {
    Partition pt;
    const int64_t bn = head_dim > 96 ? 64 : 128;  // kernel K/V tile of a partitioned launch
    if (dtype != XDIT_BF16 || pairs == 0 || kv_len <= bn) return pt;
    if (splits > 1) pt.parts = pairs * splits;
    else if (splits <= 0) pt = pick_parts(pairs, kv_len, head_dim);
    return pt;
}

// Resolve the partition and check the workspace; returns XDIT_OK and sets
// *pt_out.
static int resolve_parts(const char* fn, const SplitArgs& sa, int32_t dtype, int64_t batch, int64_t q_len,
                         int64_t kv_len, int64_t heads, int64_t head_dim, Partition* pt_out) {
    if (sa.splits > XDIT_MAX_SPLITS)
        return fail(XDIT_ERR_RANGE, "%s: splits = %d above %d", fn, sa.splits, XDIT_MAX_SPLITS);
    const int64_t pairs = part_pairs(batch, q_len, heads);
    const Partition pt = call_parts(dtype, pairs, kv_len, head_dim, sa.splits);
    if (pt.parts > 0) {
        const int64_t need = part_ws_bytes(pt, pairs, head_dim);
        if (sa.workspace == nullptr || sa.workspace_bytes < need)
            return fail(XDIT_ERR_RANGE, "%s: workspace of %lld bytes, the partition needs %lld", fn,
                        (long long)sa.workspace_bytes, (long long)need);
        if ((uintptr_t)sa.workspace & 255u) return fail(XDIT_ERR_LAYOUT, "%s: workspace not 256-byte aligned", fn);
    }
    *pt_out = pt;
    return XDIT_OK;
}

// Launch a partitioned attention: the sweep workgroups, then the fix-up of
// cut sweeps (both inside launch_attn_bf16).
static hipError_t launch_parts(xdit::AttnParams p, const Partition& pt, void* workspace) {
    p.whole = pt.whole;
    p.parts = pt.parts;
    p.part = (float*)workspace;
    return xdit::launch_attn_bf16(p, g_stream);
}

static int chunk_impl(const char* fn, const void* q, const void* k, const void* v, void* out,
                      float* lse, int64_t batch, int64_t q_len, int64_t kv_len, int64_t heads,
                      int64_t head_dim, int32_t dtype, int accum, const SplitArgs& sa = SplitArgs()) {
    XDIT_TRY(check_dtype_dim(dtype, head_dim));
    XDIT_TRY(check_dims(fn, batch, q_len, kv_len, heads));
    XDIT_TRY(check_batch_bytes(fn, q_len > kv_len ? q_len : kv_len, heads, head_dim,
                               esize_of(dtype)));
    const int64_t es = esize_of(dtype);
    const int64_t row = heads * head_dim * es;
    const Span sq{q, batch * q_len * row, "q"}, sk{k, batch * kv_len * row, "k"},
        sv{v, batch * kv_len * row, "v"}, so{out, batch * q_len * row, "out"},
        sl{lse, lse ? batch * heads * q_len * 4 : 0, "lse"};
    for (const Span* s : {&sq, &sk, &sv, &so}) XDIT_TRY(check_ptr(*s));
    if (accum && lse == nullptr && batch * heads * q_len > 0)
        return fail(XDIT_ERR_NULL, "%s: the running lse is required", fn);
    if (lse && ((uintptr_t)lse & 3u)) return fail(XDIT_ERR_LAYOUT, "lse is not 4-byte aligned");
    for (const Span* s : {&sq, &sk, &sv}) {
        XDIT_TRY(check_no_overlap(so, *s));
        XDIT_TRY(check_no_overlap(sl, *s));
    }
    XDIT_TRY(check_no_overlap(sl, so));
    Partition parts;
    XDIT_TRY(resolve_parts(fn, sa, dtype, batch, q_len, kv_len, heads, head_dim, &parts));
    if (parts.parts > 0) {
        const Span sw{sa.workspace, part_ws_bytes(parts, part_pairs(batch, q_len, heads), head_dim),
                      "workspace"};
        for (const Span* s : {&sq, &sk, &sv, &so, &sl}) XDIT_TRY(check_no_overlap(sw, *s));
    }
    if (batch == 0 || q_len == 0 || heads == 0) return XDIT_OK;

    xdit::AttnParams p{};
    p.q = q;
    p.k = k;
    p.v = v;
    p.out = out;
    p.lse = lse;
    p.B = (int)batch;
    p.H = (int)heads;
    p.Nq = (int)q_len;
    p.Nk = (int)kv_len;
    p.D = (int)head_dim;
    p.accum = accum;
    if (parts.parts > 0) return hip_status(launch_parts(p, parts, sa.workspace), fn);
    const hipError_t e = dtype == XDIT_BF16 ? xdit::launch_attn_bf16(p, g_stream)
                                            : xdit::launch_attn_f32(p, g_stream);
    return hip_status(e, fn);
}

int xdit_chunk_attn(const void* q, const void* k, const void* v, void* out, float* lse,
                    int64_t batch, int64_t q_len, int64_t kv_len, int64_t heads, int64_t head_dim,
                    int32_t dtype) {
    clear_error();
    return chunk_impl("xdit_chunk_attn", q, k, v, out, lse, batch, q_len, kv_len, heads, head_dim,
                      dtype, 0);
}

int xdit_chunk_attn_accum(const void* q, const void* k, const void* v, void* out, float* lse,
                          int64_t batch, int64_t q_len, int64_t kv_len, int64_t heads,
                          int64_t head_dim, int32_t dtype) {
    clear_error();
    return chunk_impl("xdit_chunk_attn_accum", q, k, v, out, lse, batch, q_len, kv_len, heads,
                      head_dim, dtype, 1);
}

static int check_patch_args(const char* fn, const void* q, void* kv_buf, int64_t patch_off,
                            int64_t patch_len, const void* fresh_k, const void* fresh_v,
                            const void* out, int64_t batch, int64_t seq_len, int64_t heads,
                            int64_t head_dim, int32_t dtype) {
    XDIT_TRY(check_dtype_dim(dtype, head_dim));
    XDIT_TRY(check_dims(fn, batch, seq_len, 0, heads));  // patch_len is bounded by the range check
    XDIT_TRY(check_batch_bytes(fn, seq_len, heads, head_dim, esize_of(dtype)));
    if (patch_off < 0 || patch_len < 0 || patch_off > seq_len - patch_len)
        return fail(XDIT_ERR_RANGE, "%s: slice [%lld, %lld) outside the buffer of %lld rows", fn,
                    (long long)patch_off, (long long)(patch_off + patch_len), (long long)seq_len);
    const int64_t row = heads * head_dim * esize_of(dtype);
    const Span sb{kv_buf, 2 * batch * seq_len * row, "kv_buf"},
        sk{fresh_k, batch * patch_len * row, "fresh_k"}, sv{fresh_v, batch * patch_len * row, "fresh_v"},
        sq{q, q ? batch * patch_len * row : 0, "q"}, so{out, out ? batch * patch_len * row : 0, "out"};
    for (const Span* s : {&sb, &sk, &sv, &sq, &so}) XDIT_TRY(check_ptr(*s));
    // the buffer is written while the queries and fresh rows are read
    XDIT_TRY(check_no_overlap(sk, sb));
    XDIT_TRY(check_no_overlap(sv, sb));
    XDIT_TRY(check_no_overlap(sq, sb));
    for (const Span* s : {&sq, &sb, &sk, &sv}) XDIT_TRY(check_no_overlap(so, *s));
    return XDIT_OK;
}

// The patch step in its general form: fresh rows over up to
// XDIT_MAX_RANGES disjoint row ranges, queries of their own.
static int patch_ranges_impl(const char* fn, const void* q, int64_t q_len, void* kv_buf,
                             int32_t n_ranges, const int64_t* range_off, const int64_t* range_len,
                             const void* fresh_k, const void* fresh_v, void* out, float* lse,
                             int64_t batch, int64_t seq_len, int64_t heads, int64_t head_dim,
                             int32_t dtype, const SplitArgs& sa = SplitArgs()) {
    XDIT_TRY(check_dtype_dim(dtype, head_dim));
    if (n_ranges < 0 || n_ranges > XDIT_MAX_RANGES)
        return fail(XDIT_ERR_RANGE, "%s: n_ranges = %d outside [0, %d]", fn, n_ranges, XDIT_MAX_RANGES);
    if (n_ranges > 0 && (range_off == nullptr || range_len == nullptr))
        return fail(XDIT_ERR_NULL, "%s: range_off / range_len host arrays are NULL", fn);
    XDIT_TRY(check_dims(fn, batch, seq_len, q_len, heads));
    int64_t off[XDIT_MAX_RANGES] = {0, 0}, len[XDIT_MAX_RANGES] = {0, 0};
    int64_t F = 0;
    for (int r = 0; r < n_ranges; ++r) {
        off[r] = range_off[r];
        len[r] = range_len[r];
        if (off[r] < 0 || len[r] < 0 || off[r] > seq_len - len[r])
            return fail(XDIT_ERR_RANGE, "%s: range %d [%lld, %lld) outside the buffer of %lld rows", fn, r,
                        (long long)off[r], (long long)(off[r] + len[r]), (long long)seq_len);
        for (int r2 = 0; r2 < r; ++r2)
            if (len[r] > 0 && len[r2] > 0 && off[r] < off[r2] + len[r2] && off[r2] < off[r] + len[r])
                return fail(XDIT_ERR_RANGE, "%s: ranges %d and %d overlap", fn, r2, r);
        F += len[r];
    }
    const int es = esize_of(dtype);
    int64_t most = seq_len > q_len ? seq_len : q_len;
    XDIT_TRY(check_batch_bytes(fn, most, heads, head_dim, es));
    const int64_t row = heads * head_dim * es;
    const Span sb{kv_buf, 2 * batch * seq_len * row, "kv_buf"}, sk{fresh_k, batch * F * row, "fresh_k"},
        sv{fresh_v, batch * F * row, "fresh_v"}, sq{q, batch * q_len * row, "q"},
        so{out, batch * q_len * row, "out"}, sl{lse, lse ? batch * heads * q_len * 4 : 0, "lse"};
    for (const Span* s : {&sb, &sk, &sv, &sq, &so}) XDIT_TRY(check_ptr(*s));
    if (lse && ((uintptr_t)lse & 3u)) return fail(XDIT_ERR_LAYOUT, "lse is not 4-byte aligned");
    // the buffer is written while the queries and fresh rows are read
    XDIT_TRY(check_no_overlap(sk, sb));
    XDIT_TRY(check_no_overlap(sv, sb));
    XDIT_TRY(check_no_overlap(sq, sb));
    for (const Span* s : {&sq, &sb, &sk, &sv}) {
        XDIT_TRY(check_no_overlap(so, *s));
        XDIT_TRY(check_no_overlap(sl, *s));
    }
    XDIT_TRY(check_no_overlap(sl, so));
    Partition parts;
    XDIT_TRY(resolve_parts(fn, sa, dtype, batch, q_len, seq_len, heads, head_dim, &parts));
    if (parts.parts > 0) {
        const Span sw{sa.workspace, part_ws_bytes(parts, part_pairs(batch, q_len, heads), head_dim),
                      "workspace"};
        for (const Span* s : {&sb, &sk, &sv, &sq, &so, &sl}) XDIT_TRY(check_no_overlap(sw, *s));
    }
    if (batch == 0 || heads == 0) return XDIT_OK;

    const int64_t plane = batch * seq_len * row;
    if (q_len == 0) {
        // no queries: only the update
        int64_t base = 0;
        for (int r = 0; r < n_ranges; ++r) {
            if (len[r] > 0) {
                xdit::UpdateParams u{};
                u.kv_buf = kv_buf;
                u.fresh_k = fresh_k;
                u.fresh_v = fresh_v;
                u.B = (int)batch;
                u.N = (int)seq_len;
                u.H = (int)heads;
                u.D = (int)head_dim;
                u.off = (int)off[r];
                u.len = (int)len[r];
                u.frows = (int)F;
                u.fbase = (int)base;
                u.esize = es;
                XDIT_TRY(hip_status(xdit::launch_kv_update(u, g_stream), fn));
            }
            base += len[r];
        }
        return XDIT_OK;
    }
    xdit::AttnParams p{};
    p.q = q;
    p.k = kv_buf;
    p.v = (const char*)kv_buf + plane;
    if (F > 0) {
        p.fresh_k = fresh_k;
        p.fresh_v = fresh_v;
        p.wk = kv_buf;
        p.wv = (char*)kv_buf + plane;
    }
    p.out = out;
    p.lse = lse;
    p.B = (int)batch;
    p.H = (int)heads;
    p.Nq = (int)q_len;
    p.Nk = (int)seq_len;
    p.D = (int)head_dim;
    p.off0 = (int)off[0];
    p.len0 = (int)len[0];
    p.off1 = (int)off[1];
    p.len1 = (int)len[1];
    if (parts.parts > 0) return hip_status(launch_parts(p, parts, sa.workspace), fn);
    const hipError_t e = dtype == XDIT_BF16 ? xdit::launch_attn_bf16(p, g_stream)
                                            : xdit::launch_attn_f32(p, g_stream);
    return hip_status(e, fn);
}

int xdit_patch_attn(const void* q, void* kv_buf, int64_t patch_off, int64_t patch_len,
                    const void* fresh_k, const void* fresh_v, void* out, int64_t batch,
                    int64_t seq_len, int64_t heads, int64_t head_dim, int32_t dtype) {
    clear_error();
    if (patch_len > 0 && (q == nullptr || out == nullptr))
        return fail(XDIT_ERR_NULL, "xdit_patch_attn: q and out are required");
    XDIT_TRY(check_patch_args("xdit_patch_attn", q, kv_buf, patch_off, patch_len, fresh_k,
                              fresh_v, out, batch, seq_len, heads, head_dim, dtype));
    if (batch == 0 || patch_len == 0 || heads == 0) return XDIT_OK;
    return patch_ranges_impl("xdit_patch_attn", q, patch_len, kv_buf, 1, &patch_off, &patch_len,
                             fresh_k, fresh_v, out, nullptr, batch, seq_len, heads, head_dim, dtype);
}

int xdit_patch_attn_ranges(const void* q, int64_t q_len, void* kv_buf, int32_t n_ranges,
                           const int64_t* range_off, const int64_t* range_len, const void* fresh_k,
                           const void* fresh_v, void* out, float* lse, int64_t batch,
                           int64_t seq_len, int64_t heads, int64_t head_dim, int32_t dtype) {
    clear_error();
    return patch_ranges_impl("xdit_patch_attn_ranges", q, q_len, kv_buf, n_ranges, range_off,
                             range_len, fresh_k, fresh_v, out, lse, batch, seq_len, heads, head_dim,
                             dtype);
}

int64_t xdit_split_workspace_bytes(int64_t batch, int64_t q_len, int64_t kv_len, int64_t heads,
                                   int64_t head_dim, int32_t dtype, int32_t splits) {
    clear_error();
    if (check_dtype_dim(dtype, head_dim) != XDIT_OK) return -1;
    if (check_dims("xdit_split_workspace_bytes", batch, q_len, kv_len, heads) != XDIT_OK) return -1;
    if (splits > XDIT_MAX_SPLITS) return -1;
    const int64_t pairs = part_pairs(batch, q_len, heads);
    return part_ws_bytes(call_parts(dtype, pairs, kv_len, head_dim, splits), pairs, head_dim);
}

int xdit_chunk_attn_split(const void* q, const void* k, const void* v, void* out, float* lse,
                          int32_t splits, void* workspace, int64_t workspace_bytes, int64_t batch,
                          int64_t q_len, int64_t kv_len, int64_t heads, int64_t head_dim,
                          int32_t dtype) {
    clear_error();
    SplitArgs sa;
    sa.splits = splits;
    sa.workspace = workspace;
    sa.workspace_bytes = workspace_bytes;
    return chunk_impl("xdit_chunk_attn_split", q, k, v, out, lse, batch, q_len, kv_len, heads,
                      head_dim, dtype, 0, sa);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Allocation-free form of xdit_chunk_attn_split: the partial slots of cut
// sweeps live in a fixed device array instead of a caller workspace.  Each
// GPU the library runs on holds its own copy of the array until the process
// ends, and every call on that GPU shares it: the kernels write every slot
// they read within the call, so nothing needs clearing, but two calls that
// overlap on one GPU (concurrent streams or threads) race on it.
namespace {

constexpr int64_t kScratchBytes = (int64_t)16 << 20;  // 16 MiB
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array.  The array's name is
// a host-side stand-in in host code: its device address comes from
// hipGetSymbolAddress, called once per device with that device current.
int scratch_of_current_device(const char* fn, void** out) {
    int dev = -1;
    XDIT_TRY(hip_status(hipGetDevice(&dev), fn));
    if (dev < 0 || dev >= kMaxDevices) return fail(XDIT_ERR_HIP, "%s: device %d out of range", fn, dev);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        XDIT_TRY(hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), fn));
        if (p == nullptr) return fail(XDIT_ERR_HIP, "%s: no device address for the scratch array", fn);
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return XDIT_OK;
}

}  // namespace

extern "C" {

int64_t xdit_noalloc_scratch_bytes(void) { return kScratchBytes; }

int xdit_chunk_attn_split_noalloc(const void* q, const void* k, const void* v, void* out, float* lse,
                                  int32_t splits, int64_t batch, int64_t q_len, int64_t kv_len,
                                  int64_t heads, int64_t head_dim, int32_t dtype) {
    clear_error();
    const char* fn = "xdit_chunk_attn_split_noalloc";
    // size checks first, on the host: the partition's slots must fit
    XDIT_TRY(check_dtype_dim(dtype, head_dim));
    XDIT_TRY(check_dims(fn, batch, q_len, kv_len, heads));
    if (splits > XDIT_MAX_SPLITS)
        return fail(XDIT_ERR_RANGE, "%s: splits = %d above %d", fn, splits, XDIT_MAX_SPLITS);
    const int64_t pairs = part_pairs(batch, q_len, heads);
    const int64_t need = part_ws_bytes(call_parts(dtype, pairs, kv_len, head_dim, splits), pairs, head_dim);
    if (need > kScratchBytes)
        return fail(XDIT_ERR_RANGE, "%s: the partition needs %lld bytes of scratch, above the %lld-byte maximum",
                    fn, (long long)need, (long long)kScratchBytes);
    SplitArgs sa;
    sa.splits = splits;
    sa.workspace_bytes = kScratchBytes;
    if (need > 0) XDIT_TRY(scratch_of_current_device(fn, &sa.workspace));
    return chunk_impl(fn, q, k, v, out, lse, batch, q_len, kv_len, heads, head_dim, dtype, 0, sa);
}

int xdit_chunk_attn_accum_split(const void* q, const void* k, const void* v, void* out, float* lse,
                                int32_t splits, void* workspace, int64_t workspace_bytes, int64_t batch,
                                int64_t q_len, int64_t kv_len, int64_t heads, int64_t head_dim,
                                int32_t dtype) {
    clear_error();
    SplitArgs sa;
    sa.splits = splits;
    sa.workspace = workspace;
    sa.workspace_bytes = workspace_bytes;
    return chunk_impl("xdit_chunk_attn_accum_split", q, k, v, out, lse, batch, q_len, kv_len, heads,
                      head_dim, dtype, 1, sa);
}

int xdit_patch_attn_split(const void* q, int64_t q_len, void* kv_buf, int32_t n_ranges,
                          const int64_t* range_off, const int64_t* range_len, const void* fresh_k,
                          const void* fresh_v, void* out, float* lse, int32_t splits,
                          void* workspace, int64_t workspace_bytes, int64_t batch, int64_t seq_len,
                          int64_t heads, int64_t head_dim, int32_t dtype) {
    clear_error();
    SplitArgs sa;
    sa.splits = splits;
    sa.workspace = workspace;
    sa.workspace_bytes = workspace_bytes;
    return patch_ranges_impl("xdit_patch_attn_split", q, q_len, kv_buf, n_ranges, range_off,
                             range_len, fresh_k, fresh_v, out, lse, batch, seq_len, heads,
                             head_dim, dtype, sa);
}

int xdit_kv_update(void* kv_buf, int64_t patch_off, int64_t patch_len, const void* fresh_k,
                   const void* fresh_v, int64_t batch, int64_t seq_len, int64_t heads,
                   int64_t head_dim, int32_t dtype) {
    clear_error();
    XDIT_TRY(check_patch_args("xdit_kv_update", nullptr, kv_buf, patch_off, patch_len, fresh_k,
                              fresh_v, nullptr, batch, seq_len, heads, head_dim, dtype));
    if (batch == 0 || patch_len == 0 || heads == 0) return XDIT_OK;
    xdit::UpdateParams p{};
    p.kv_buf = kv_buf;
    p.fresh_k = fresh_k;
    p.fresh_v = fresh_v;
    p.B = (int)batch;
    p.N = (int)seq_len;
    p.H = (int)heads;
    p.D = (int)head_dim;
    p.off = (int)patch_off;
    p.len = (int)patch_len;
    p.frows = (int)patch_len;
    p.fbase = 0;
    p.esize = esize_of(dtype);
    return hip_status(xdit::launch_kv_update(p, g_stream), "xdit_kv_update launch");
}

int xdit_lse_merge(const void* const* outs, const float* const* lses, int32_t n, void* out,
                   float* lse_out, int64_t batch, int64_t q_len, int64_t heads, int64_t head_dim,
                   int32_t dtype) {
    clear_error();
    XDIT_TRY(check_dtype_dim(dtype, head_dim));
    XDIT_TRY(check_dims("xdit_lse_merge", batch, q_len, 0, heads));
    XDIT_TRY(check_batch_bytes("xdit_lse_merge", q_len, heads, head_dim, esize_of(dtype)));
    if (n < 1 || n > XDIT_MAX_PARTIALS)
        return fail(XDIT_ERR_RANGE, "xdit_lse_merge: n = %d outside [1, %d]", n, XDIT_MAX_PARTIALS);
    if (outs == nullptr || lses == nullptr)
        return fail(XDIT_ERR_NULL, "xdit_lse_merge: outs / lses host arrays are NULL");
    const int64_t obytes = batch * q_len * heads * head_dim * esize_of(dtype);
    const int64_t lbytes = batch * heads * q_len * 4;
    const Span so{out, obytes, "out"}, slo{lse_out, lse_out ? lbytes : 0, "lse_out"};
    XDIT_TRY(check_ptr(so));
    if (lse_out && ((uintptr_t)lse_out & 3u)) return fail(XDIT_ERR_LAYOUT, "lse_out is not 4-byte aligned");
    XDIT_TRY(check_no_overlap(slo, so));
    for (int r = 0; r < n; ++r) {
        const Span sp{outs[r], obytes, "outs[r]"}, sl{lses[r], lbytes, "lses[r]"};
        XDIT_TRY(check_ptr(sp));
        if (lbytes > 0 && lses[r] == nullptr) return fail(XDIT_ERR_NULL, "lses[%d] is NULL", r);
        if (lbytes > 0 && ((uintptr_t)lses[r] & 3u))
            return fail(XDIT_ERR_LAYOUT, "lses[%d] is not 4-byte aligned", r);
        if (outs[r] != out) XDIT_TRY(check_no_overlap(so, sp));  // exact in-place is allowed
        XDIT_TRY(check_no_overlap(so, sl));
        XDIT_TRY(check_no_overlap(slo, sl));
        XDIT_TRY(check_no_overlap(slo, sp));
    }
    if (obytes == 0) return XDIT_OK;
    xdit::MergeParams p{};
    p.outs = outs;
    p.lses = lses;
    p.n = n;
    p.out = out;
    p.lse_out = lse_out;
    p.B = (int)batch;
    p.Nq = (int)q_len;
    p.H = (int)heads;
    p.D = (int)head_dim;
    const hipError_t e = dtype == XDIT_BF16 ? xdit::launch_merge_bf16(p, g_stream)
                                            : xdit::launch_merge_f32(p, g_stream);
    return hip_status(e, "xdit_lse_merge launch");
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The stage micro-step's projections: plain bf16 GEMMs with float32
// accumulation through hipBLASLt, one handle per device and one plan per
// shape, both created on first use and kept for the life of the process.  A
// plan holds the layouts and the fastest of hipBLASLt's candidate
// algorithms that need no workspace, timed on the first call's own operands
// (three rounds of a few runs each on the calling stream, which that first
// call therefore synchronises).
namespace {

struct GemmPlan {
    hipblasLtMatmulDesc_t desc = nullptr;
    hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, ld = nullptr;
    hipblasLtMatmulAlgo_t algo{};
};

std::mutex g_gemm_mutex;
std::map<int, hipblasLtHandle_t> g_handles;
// plans by (device, M, N, K, batch)
std::map<std::tuple<int, int64_t, int64_t, int64_t, int>, GemmPlan> g_plans;
constexpr int kNoAlgorithm = 1;  // gemm_bf16: hipBLASLt offers no algorithm for the shape

int blas_status(hipblasStatus_t st, const char* what) {
    if (st != HIPBLAS_STATUS_SUCCESS) return fail(XDIT_ERR_HIP, "%s: hipBLASLt status %d", what, (int)st);
    return XDIT_OK;
}

// Row-major C[M, N] = A[M, K] B[K, N], all bf16 and contiguous.  In
// hipBLASLt's column-major terms that is C^T (N x M) = B^T (N x K) A^T (K x M),
// where B^T and A^T are the row-major buffers read as column-major.  With
// batch > 1: C_i = A B_i for i < batch, the B_i and the C_i consecutive
// (one strided-batched launch; A is shared, batch stride 0).  Returns
// kNoAlgorithm, with no error set and nothing launched, when hipBLASLt has
// no algorithm for the shape.
int gemm_bf16(const char* fn, const void* A, const void* B, void* C, int64_t M, int64_t N, int64_t K,
              int batch = 1) {
    if (M == 0 || N == 0) return XDIT_OK;
    int dev = 0;
    XDIT_TRY(hip_status(hipGetDevice(&dev), fn));
    std::lock_guard<std::mutex> lock(g_gemm_mutex);
    auto hit = g_handles.find(dev);
    if (hit == g_handles.end()) {
        hipblasLtHandle_t h = nullptr;
        XDIT_TRY(blas_status(hipblasLtCreate(&h), "hipblasLtCreate"));
        hit = g_handles.emplace(dev, h).first;
    }
    const hipblasLtHandle_t handle = hit->second;
    const auto key = std::make_tuple(dev, M, N, K, batch);
    auto pit = g_plans.find(key);
    if (pit == g_plans.end()) {
        GemmPlan pl;
        XDIT_TRY(blas_status(hipblasLtMatmulDescCreate(&pl.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F),
                             "hipblasLtMatmulDescCreate"));
        const hipblasOperation_t op = HIPBLAS_OP_N;
        XDIT_TRY(blas_status(hipblasLtMatmulDescSetAttribute(pl.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &op, sizeof(op)),
                             "hipblasLtMatmulDescSetAttribute"));
        XDIT_TRY(blas_status(hipblasLtMatmulDescSetAttribute(pl.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &op, sizeof(op)),
                             "hipblasLtMatmulDescSetAttribute"));
        XDIT_TRY(blas_status(hipblasLtMatrixLayoutCreate(&pl.la, HIP_R_16BF, N, K, N), "hipblasLtMatrixLayoutCreate"));
        XDIT_TRY(blas_status(hipblasLtMatrixLayoutCreate(&pl.lb, HIP_R_16BF, K, M, K), "hipblasLtMatrixLayoutCreate"));
        XDIT_TRY(blas_status(hipblasLtMatrixLayoutCreate(&pl.ld, HIP_R_16BF, N, M, N), "hipblasLtMatrixLayoutCreate"));
        if (batch > 1) {
            const int32_t bc = batch;
            const int64_t sb = N * K, sa = 0, sc = N * M;
            for (hipblasLtMatrixLayout_t l : {pl.la, pl.lb, pl.ld})
                XDIT_TRY(blas_status(hipblasLtMatrixLayoutSetAttribute(l, HIPBLASLT_MATRIX_LAYOUT_BATCH_COUNT, &bc,
                                                                       sizeof(bc)),
                                     "hipblasLtMatrixLayoutSetAttribute"));
            XDIT_TRY(blas_status(hipblasLtMatrixLayoutSetAttribute(pl.la, HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET,
                                                                   &sb, sizeof(sb)),
                                 "hipblasLtMatrixLayoutSetAttribute"));
            XDIT_TRY(blas_status(hipblasLtMatrixLayoutSetAttribute(pl.lb, HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET,
                                                                   &sa, sizeof(sa)),
                                 "hipblasLtMatrixLayoutSetAttribute"));
            XDIT_TRY(blas_status(hipblasLtMatrixLayoutSetAttribute(pl.ld, HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET,
                                                                   &sc, sizeof(sc)),
                                 "hipblasLtMatrixLayoutSetAttribute"));
        }
        hipblasLtMatmulPreference_t pref = nullptr;
        XDIT_TRY(blas_status(hipblasLtMatmulPreferenceCreate(&pref), "hipblasLtMatmulPreferenceCreate"));
        uint64_t ws = 0;
        hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws, sizeof(ws));
        constexpr int kCands = 16;
        hipblasLtMatmulHeuristicResult_t res[kCands];
        int nres = 0;
        const hipblasStatus_t st = hipblasLtMatmulAlgoGetHeuristic(handle, pl.desc, pl.la, pl.lb, pl.ld, pl.ld, pref,
                                                                   kCands, res, &nres);
        hipblasLtMatmulPreferenceDestroy(pref);
        if (batch > 1 && (st != HIPBLAS_STATUS_SUCCESS || nres < 1)) {
            hipblasLtMatrixLayoutDestroy(pl.la);
            hipblasLtMatrixLayoutDestroy(pl.lb);
            hipblasLtMatrixLayoutDestroy(pl.ld);
            hipblasLtMatmulDescDestroy(pl.desc);
            return kNoAlgorithm;
        }
        XDIT_TRY(blas_status(st, "hipblasLtMatmulAlgoGetHeuristic"));
        if (nres < 1)
            return fail(XDIT_ERR_HIP, "%s: hipBLASLt has no algorithm for a %lld x %lld x %lld bf16 GEMM", fn,
                        (long long)M, (long long)N, (long long)K);
        pl.algo = res[0].algo;
        if (nres > 1) {
            hipEvent_t e0 = nullptr, e1 = nullptr;
            XDIT_TRY(hip_status(hipEventCreate(&e0), fn));
            XDIT_TRY(hip_status(hipEventCreate(&e1), fn));
            const float one = 1.f, zero = 0.f;
            // three rounds over the candidates, each candidate's best round
            // counts: the GPU clocks are still rising during the first calls
            // of a process, which would favour the candidates timed last
            float cand_ms[kCands];
            for (int i = 0; i < kCands; ++i) cand_ms[i] = 1e30f;
            for (int round = 0; round < 3; ++round)
                for (int i = 0; i < nres; ++i) {
                    if (res[i].state != HIPBLAS_STATUS_SUCCESS || res[i].workspaceSize != 0) continue;
                    bool ok = true;
                    for (int r = 0; r < 8 && ok; ++r) {
                        if (r == 2) ok = hipEventRecord(e0, g_stream) == hipSuccess;
                        ok = ok && hipblasLtMatmul(handle, pl.desc, &one, B, pl.la, A, pl.lb, &zero, C, pl.ld, C,
                                                   pl.ld, &res[i].algo, nullptr, 0,
                                                   g_stream) == HIPBLAS_STATUS_SUCCESS;
                    }
                    float ms = 0.f;
                    ok = ok && hipEventRecord(e1, g_stream) == hipSuccess && hipEventSynchronize(e1) == hipSuccess &&
                         hipEventElapsedTime(&ms, e0, e1) == hipSuccess;
                    if (ok && ms < cand_ms[i]) cand_ms[i] = ms;
                }
            float best = 1e30f;
            for (int i = 0; i < nres; ++i)
                if (cand_ms[i] < best) {
                    best = cand_ms[i];
                    pl.algo = res[i].algo;
                }
            (void)hipEventDestroy(e0);
            (void)hipEventDestroy(e1);
        }
        if (batch > 1) {
            // a batched plan is kept only if its algorithm runs (a shared
            // operand with batch stride 0 is not taken by every kernel)
            const float one = 1.f, zero = 0.f;
            if (hipblasLtMatmul(handle, pl.desc, &one, B, pl.la, A, pl.lb, &zero, C, pl.ld, C, pl.ld, &pl.algo,
                                nullptr, 0, g_stream) != HIPBLAS_STATUS_SUCCESS) {
                hipblasLtMatrixLayoutDestroy(pl.la);
                hipblasLtMatrixLayoutDestroy(pl.lb);
                hipblasLtMatrixLayoutDestroy(pl.ld);
                hipblasLtMatmulDescDestroy(pl.desc);
                return kNoAlgorithm;
            }
        }
        pit = g_plans.emplace(key, pl).first;
    }
    const GemmPlan& pl = pit->second;
    const float alpha = 1.f, beta = 0.f;
    return blas_status(hipblasLtMatmul(handle, pl.desc, &alpha, B, pl.la, A, pl.lb, &beta, C, pl.ld, C, pl.ld,
                                       &pl.algo, nullptr, 0, g_stream),
                       fn);
}

}  // namespace

extern "C" int xdit_stage_step(const void* x, const void* wq, const void* wk, const void* wv,
                               const void* wo, void* kv_buf, int64_t patch_off, int64_t patch_len,
                               void* q, void* k, void* v, void* o, void* y, int64_t batch,
                               int64_t seq_len, int64_t heads, int64_t head_dim, int64_t hidden,
                               int32_t dtype) {
    clear_error();
    const char* fn = "xdit_stage_step";
    XDIT_TRY(check_dtype_dim(dtype, head_dim));
    if (dtype != XDIT_BF16) return fail(XDIT_ERR_UNSUPPORTED, "%s: bf16 only", fn);
    if (hidden <= 0 || hidden > 65536) return fail(XDIT_ERR_SHAPE, "%s: hidden = %lld outside [1, 65536]", fn,
                                                   (long long)hidden);
    XDIT_TRY(check_patch_args(fn, q, kv_buf, patch_off, patch_len, k, v, o, batch, seq_len, heads, head_dim,
                              dtype));
    const int64_t HD = heads * head_dim, M = batch * patch_len;
    const Span sx{x, M * hidden * 2, "x"}, sy{y, M * hidden * 2, "y"}, swq{wq, hidden * HD * 2, "wq"},
        swk{wk, hidden * HD * 2, "wk"}, swv{wv, hidden * HD * 2, "wv"}, swo{wo, HD * hidden * 2, "wo"},
        sb{kv_buf, 2 * batch * seq_len * HD * 2, "kv_buf"}, sq{q, M * HD * 2, "q"}, sk{k, M * HD * 2, "k"},
        sv{v, M * HD * 2, "v"}, so{o, M * HD * 2, "o"};
    const Span* ins[] = {&sx, &swq, &swk, &swv, &swo};
    const Span* outs[] = {&sq, &sk, &sv, &so, &sy};
    for (const Span* s : ins) XDIT_TRY(check_ptr(*s));
    for (const Span* s : outs) XDIT_TRY(check_ptr(*s));
    for (int i = 0; i < 5; ++i) {
        XDIT_TRY(check_no_overlap(*outs[i], sb));
        for (const Span* s : ins) XDIT_TRY(check_no_overlap(*outs[i], *s));
        for (int j = 0; j < i; ++j) XDIT_TRY(check_no_overlap(*outs[i], *outs[j]));
    }
    if (M == 0 || heads == 0) return XDIT_OK;
    // The three projections as one strided-batched GEMM when the weights
    // are consecutive [3, C, H*d] and q, k, v consecutive [3, B, L, H, d];
    // otherwise (or if hipBLASLt has no batched algorithm) three GEMMs.
    const int64_t wbytes = hidden * HD * 2, obytes = M * HD * 2;
    const char *cq = (const char*)q, *cwq = (const char*)wq;
    int rc = kNoAlgorithm;
    if ((const char*)wk == cwq + wbytes && (const char*)wv == cwq + 2 * wbytes && (const char*)k == cq + obytes &&
        (const char*)v == cq + 2 * obytes)
        rc = gemm_bf16(fn, x, wq, q, M, HD, hidden, 3);
    if (rc == kNoAlgorithm) {
        XDIT_TRY(gemm_bf16(fn, x, wq, q, M, HD, hidden));
        XDIT_TRY(gemm_bf16(fn, x, wk, k, M, HD, hidden));
        XDIT_TRY(gemm_bf16(fn, x, wv, v, M, HD, hidden));
    } else {
        XDIT_TRY(rc);
    }
    XDIT_TRY(patch_ranges_impl(fn, q, patch_len, kv_buf, 1, &patch_off, &patch_len, k, v, o, nullptr, batch,
                               seq_len, heads, head_dim, dtype));
    return gemm_bf16(fn, o, wo, y, M, hidden, HD);
}
