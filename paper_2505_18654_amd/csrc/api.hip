// C ABI of the library: argument validation (pure host code, before any HIP call),
// workspace layout and kernel launches.  See include/mtgr_hstu.h and include/mtgr_embedding.h
// for the contract.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "../../include/mtgr_embedding.h"
#include "../../include/mtgr_hstu.h"
#include "mtgr_internal.h"

namespace {

thread_local std::string g_last_error;

mtgr_status_t fail(mtgr_status_t st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
mtgr_status_t fail(mtgr_status_t st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

mtgr_status_t ok() {
    g_last_error.clear();
    return MTGR_SUCCESS;
}

mtgr_status_t device_fail(hipError_t e, const char* where) {
    return fail(MTGR_ERROR_DEVICE, "%s: %s", where, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

constexpr int MAX_SEQLEN = (mtgr::SCHED_BUCKETS - 1) * 64;

// The vector-ALU kernels serve fp32 and bf16 at head_dim 16; the MFMA kernels the rest.
bool vec_path(const mtgr_hstu_problem_t* p) {
    return p->dtype == MTGR_DTYPE_FP32 || p->head_dim == 16;
}

struct AttnLayout {
    int tile;            // rows per work item
    int ntile;           // 64-token summary tiles per user
    long long slots;     // physical work-list entries (= grid size)
    size_t off_summ, off_items, off_sorted, off_code, off_dsoff, total;
    size_t off_ds, total_bwd;   // stored-dS region (backward = 1 size)
};

AttnLayout attn_layout(const mtgr_hstu_problem_t* p) {
    AttnLayout L{};
    L.tile = vec_path(p) ? mtgr::ATTN_TILE_F32 : mtgr::ATTN_TILE_BF16;
    L.ntile = (p->max_seqlen + 63) / 64;
    L.slots = mtgr::schedule_slots(p->total_tokens, p->num_users, p->max_seqlen, p->num_heads, L.tile);
    L.off_summ = 0;
    L.off_items = align256((size_t)p->num_users * L.ntile * sizeof(int4));
    L.off_sorted = L.off_items + align256((size_t)L.slots * sizeof(int2));
    L.off_code = L.off_sorted + align256((size_t)p->num_users * sizeof(int));
    L.off_dsoff = L.off_code + align256((size_t)p->total_tokens * sizeof(int));
    L.total = L.off_dsoff + align256((size_t)(p->num_users + 1) * sizeof(long long));
    // sum_b ceil(n_b/64)^2 <= ceil(max_seqlen/64) * sum_b ceil(n_b/64) <= ntile * (T/64 + B)
    L.off_ds = L.total;
    const size_t blocks = (size_t)p->num_heads * (size_t)L.ntile *
                          (size_t)((p->total_tokens + 63) / 64 + p->num_users);
    L.total_bwd = vec_path(p) ? L.total : L.off_ds + blocks * mtgr::DS_BLOCK_BYTES;
    return L;
}

mtgr_status_t check_problem(const mtgr_hstu_problem_t* p) {
    if (!p) return fail(MTGR_ERROR_NULL_POINTER, "problem is NULL");
    if (p->dtype != MTGR_DTYPE_BF16 && p->dtype != MTGR_DTYPE_FP32)
        return fail(MTGR_ERROR_UNSUPPORTED, "dtype %d is not supported", p->dtype);
    if (p->num_users < 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "num_users %d < 0", p->num_users);
    if (p->total_tokens < 0 || p->total_tokens >= (1ll << 31))
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "total_tokens %lld outside [0, 2^31)",
                    (long long)p->total_tokens);
    if (p->max_seqlen < 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "max_seqlen %d < 0", p->max_seqlen);
    if (p->num_users > 0 && p->total_tokens > 0 && p->max_seqlen == 0)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "max_seqlen is 0 with tokens present");
    if (p->total_tokens > 0 && p->num_users == 0)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "total_tokens > 0 with no users");
    if (p->max_seqlen > MAX_SEQLEN)
        return fail(MTGR_ERROR_UNSUPPORTED, "max_seqlen %d above %d", p->max_seqlen, MAX_SEQLEN);
    if (p->num_heads < 1 || p->num_heads > MTGR_MAX_HEADS)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "num_heads %d outside 1..%d", p->num_heads,
                    MTGR_MAX_HEADS);
    const int dh = p->head_dim;
    const bool dh_ok = dh == 16 || dh == 32 || dh == 64 || dh == 128;
    if (!dh_ok)
        return fail(MTGR_ERROR_UNSUPPORTED, "head_dim %d not supported for %s", dh,
                    p->dtype == MTGR_DTYPE_BF16 ? "bf16" : "fp32");
    if (p->num_rab_buckets < 0 || p->num_rab_buckets > MTGR_MAX_RAB_BUCKETS)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "num_rab_buckets %d outside 0..%d",
                    p->num_rab_buckets, MTGR_MAX_RAB_BUCKETS);
    if (p->flags & ~(MTGR_ATTN_PLANNED | MTGR_BWD_SKIP_DQ | MTGR_BWD_SKIP_DKDV | MTGR_BWD_KEEP_DS |
                     MTGR_BWD_DS_READY | MTGR_FWD_CAND_ROWS))
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "unknown flags 0x%x", p->flags);
    if (!std::isfinite(p->alpha)) return fail(MTGR_ERROR_INVALID_ARGUMENT, "alpha is not finite");
    const long long row = (long long)p->num_heads * dh;
    const int esz = p->dtype == MTGR_DTYPE_BF16 ? 2 : 4;
    const long long lds[4] = {p->ld_q, p->ld_k, p->ld_v, p->ld_o};
    const char* names[4] = {"ld_q", "ld_k", "ld_v", "ld_o"};
    for (int i = 0; i < 4; i++) {
        if (lds[i] < row)
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "%s %lld below num_heads*head_dim %lld", names[i],
                        lds[i], row);
        if ((lds[i] * esz) % 16 != 0)
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "%s %lld is not a multiple of 16 bytes", names[i],
                        lds[i]);
        if (lds[i] > MTGR_MAX_LD)
            return fail(MTGR_ERROR_UNSUPPORTED, "%s %lld above %lld elements", names[i], lds[i],
                        (long long)MTGR_MAX_LD);
    }
    // Every attention kernel launches one 256-thread workgroup per work-list slot, and a grid
    // holds at most 2^32 - 1 work-items.
    if (mtgr::schedule_slots(p->total_tokens, p->num_users, p->max_seqlen, p->num_heads,
                             vec_path(p) ? mtgr::ATTN_TILE_F32 : mtgr::ATTN_TILE_BF16) >= (1ll << 24))
        return fail(MTGR_ERROR_UNSUPPORTED, "problem too large for one launch (2^24 work items or more)");
    return MTGR_SUCCESS;
}

#define REQUIRE_PTR(ptr, name)                                                        \
    do {                                                                              \
        if (!(ptr)) return fail(MTGR_ERROR_NULL_POINTER, "%s is NULL", name);         \
        if (!aligned16(ptr))                                                          \
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "%s is not 16-byte aligned", name); \
    } while (0)

mtgr_status_t check_attn_common(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                const int8_t* seg, const int32_t* ts, const float* rab,
                                void* workspace, size_t ws_bytes) {
    mtgr_status_t st = check_problem(p);
    if (st != MTGR_SUCCESS) return st;
    if (rab && p->num_rab_buckets == 0)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "rab given but num_rab_buckets is 0");
    if (p->num_users > 0) {
        if (!offsets) return fail(MTGR_ERROR_NULL_POINTER, "offsets is NULL");
        if (((uintptr_t)offsets & 3u) != 0)
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "offsets is not 4-byte aligned");
    }
    if (p->total_tokens > 0) {
        if (!seg) return fail(MTGR_ERROR_NULL_POINTER, "seg is NULL");
        if (!ts) return fail(MTGR_ERROR_NULL_POINTER, "ts is NULL");
        if (((uintptr_t)ts & 3u) != 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "ts is not 4-byte aligned");
    }
    if (rab && ((uintptr_t)rab & 3u) != 0)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "rab is not 4-byte aligned");
    const AttnLayout L = attn_layout(p);
    if (p->num_users > 0 && p->total_tokens > 0) {
        if (ws_bytes < L.total)
            return fail(MTGR_ERROR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws_bytes,
                        L.total);
        if (!workspace) return fail(MTGR_ERROR_NULL_POINTER, "workspace is NULL");
        if (((uintptr_t)workspace & 255u) != 0)
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "workspace is not 256-byte aligned");
    }
    return MTGR_SUCCESS;
}

mtgr::AttnArgs make_args(const mtgr_hstu_problem_t* p, const AttnLayout& L, const int32_t* offsets,
                         const int8_t* seg, const int32_t* ts, void* workspace) {
    mtgr::AttnArgs a{};
    a.offsets = offsets;
    a.seg = seg;
    a.ts = ts;
    a.ld_q = p->ld_q;
    a.ld_k = p->ld_k;
    a.ld_v = p->ld_v;
    a.ld_o = p->ld_o;
    char* ws = (char*)workspace;
    a.summ = (const int4*)(ws + L.off_summ);
    a.tok_code = (const int*)(ws + L.off_code);
    a.items = (const int2*)(ws + L.off_items);
    a.ds_off = (const long long*)(ws + L.off_dsoff);
    a.ds = (uint16_t*)(ws + L.off_ds);
    a.ntile = L.ntile;
    a.heads = p->num_heads;
    a.alpha = p->alpha;
    a.nbuckets = p->num_rab_buckets;
    return a;
}

// Tile summaries + work list into the workspace.
mtgr_status_t schedule(const mtgr_hstu_problem_t* p, const AttnLayout& L, const int32_t* offsets,
                       const int8_t* seg, const int32_t* ts, void* workspace, hipStream_t s) {
    char* ws = (char*)workspace;
    hipError_t e = mtgr::launch_tile_summaries(offsets, seg, ts, p->num_users, L.ntile,
                                               (int4*)(ws + L.off_summ), (int*)(ws + L.off_code), s);
    if (e != hipSuccess) return device_fail(e, "tile summaries");
    e = mtgr::launch_build_schedule(offsets, p->num_users, p->num_heads, L.tile,
                                    (int2*)(ws + L.off_items), (int)L.slots, (int*)(ws + L.off_sorted), s);
    if (e != hipSuccess) return device_fail(e, "schedule");
    e = mtgr::launch_ds_offsets(offsets, p->num_users, p->num_heads, (long long*)(ws + L.off_dsoff), s);
    if (e != hipSuccess) return device_fail(e, "dS offsets");
    return MTGR_SUCCESS;
}

// Plan storage of mtgr_hstu_attn_fwd_noalloc: a file-scope device array, one per GPU the library
// runs on, held until the process ends.  In host code `scratch` names a host-side stand-in, so
// host code only ever uses the device address hipGetSymbolAddress returns for it.
__device__ __align__(256) unsigned char scratch[MTGR_NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[MAX_DEVICES] = {};

// Device address of `scratch` on the current device: looked up once per device (with that device
// current, at its first call) and kept.
mtgr_status_t scratch_of_current_device(void** ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return device_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= MAX_DEVICES)
        return fail(MTGR_ERROR_UNSUPPORTED, "device %d above the %d devices with a scratch address", dev,
                    MAX_DEVICES);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return device_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(MTGR_ERROR_DEVICE, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return MTGR_SUCCESS;
}

// Forward after check_attn_common passed on (workspace, its size).
mtgr_status_t attn_fwd_checked(const mtgr_hstu_problem_t* p, const int32_t* offsets, const int8_t* seg,
                               const int32_t* ts, const void* q, const void* k, const void* v,
                               const float* rab, void* out, void* workspace, hipStream_t s) {
    if (p->num_users == 0 || p->total_tokens == 0) return ok();
    REQUIRE_PTR(q, "q");
    REQUIRE_PTR(k, "k");
    REQUIRE_PTR(v, "v");
    REQUIRE_PTR(out, "out");
    const AttnLayout L = attn_layout(p);
    if (!(p->flags & MTGR_ATTN_PLANNED)) {
        mtgr_status_t st = schedule(p, L, offsets, seg, ts, workspace, s);
        if (st != MTGR_SUCCESS) return st;
    }
    mtgr::AttnArgs a = make_args(p, L, offsets, seg, ts, workspace);
    a.q = q;
    a.k = k;
    a.v = v;
    a.rab = rab;
    a.out = out;
    a.cand_rows = (p->flags & MTGR_FWD_CAND_ROWS) ? 1 : 0;
    // bf16 at head_dim 16 goes to the vector kernel inside launch_attn_fwd_bf16
    hipError_t e = p->dtype == MTGR_DTYPE_BF16 ? mtgr::launch_attn_fwd_bf16(a, p->head_dim, (int)L.slots, s)
                                               : mtgr::launch_attn_fwd_f32(a, p->head_dim, (int)L.slots, s);
    if (e != hipSuccess) return device_fail(e, "attention forward");
    return ok();
}

}  // namespace

extern "C" {

mtgr_status_t mtgr_hstu_attn_plan(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                  const int8_t* seg, const int32_t* ts, void* workspace,
                                  size_t workspace_bytes, mtgr_stream_t stream) {
    mtgr_status_t st = check_attn_common(p, offsets, seg, ts, nullptr, workspace, workspace_bytes);
    if (st != MTGR_SUCCESS) return st;
    if (p->num_users == 0 || p->total_tokens == 0) return ok();
    st = schedule(p, attn_layout(p), offsets, seg, ts, workspace, (hipStream_t)stream);
    if (st != MTGR_SUCCESS) return st;
    return ok();
}

mtgr_status_t mtgr_hstu_attn_workspace_size(const mtgr_hstu_problem_t* p, int backward, size_t* bytes) {
    if (!bytes) return fail(MTGR_ERROR_NULL_POINTER, "bytes is NULL");
    mtgr_status_t st = check_problem(p);
    if (st != MTGR_SUCCESS) return st;
    const AttnLayout L = attn_layout(p);
    *bytes = (p->num_users > 0 && p->total_tokens > 0) ? (backward ? L.total_bwd : L.total) : 0;
    return ok();
}

mtgr_status_t mtgr_hstu_attn_fwd(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                 const int8_t* seg, const int32_t* ts, const void* q, const void* k,
                                 const void* v, const float* rab, void* out, void* workspace,
                                 size_t workspace_bytes, mtgr_stream_t stream) {
    mtgr_status_t st = check_attn_common(p, offsets, seg, ts, rab, workspace, workspace_bytes);
    if (st != MTGR_SUCCESS) return st;
    return attn_fwd_checked(p, offsets, seg, ts, q, k, v, rab, out, workspace, (hipStream_t)stream);
}

mtgr_status_t mtgr_hstu_attn_fwd_noalloc(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                         const int8_t* seg, const int32_t* ts, const void* q, const void* k,
                                         const void* v, const float* rab, void* out, mtgr_stream_t stream) {
    mtgr_status_t st = check_problem(p);
    if (st != MTGR_SUCCESS) return st;
    if (p->flags & MTGR_ATTN_PLANNED)
        return fail(MTGR_ERROR_INVALID_ARGUMENT,
                    "MTGR_ATTN_PLANNED: the no-alloc forward rebuilds its plan in the shared scratch on every call");
    if (p->num_users == 0 || p->total_tokens == 0) return ok();
    const AttnLayout L = attn_layout(p);
    if (L.total > (size_t)MTGR_NOALLOC_SCRATCH_BYTES)
        return fail(MTGR_ERROR_UNSUPPORTED, "the plan needs %zu bytes, above the %u-byte scratch", L.total,
                    (unsigned)MTGR_NOALLOC_SCRATCH_BYTES);
    hipStream_t s = (hipStream_t)stream;
    int cur = -1, sdev = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return device_fail(e, "hipGetDevice");
    if (s) {
        e = hipStreamGetDevice(s, &sdev);
        if (e != hipSuccess) return device_fail(e, "hipStreamGetDevice");
        if (sdev != cur)
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "stream of device %d while device %d is current", sdev, cur);
    }
    void* ws = nullptr;
    st = scratch_of_current_device(&ws);
    if (st != MTGR_SUCCESS) return st;
    st = check_attn_common(p, offsets, seg, ts, rab, ws, MTGR_NOALLOC_SCRATCH_BYTES);
    if (st != MTGR_SUCCESS) return st;
    return attn_fwd_checked(p, offsets, seg, ts, q, k, v, rab, out, ws, s);
}

mtgr_status_t mtgr_hstu_attn_fwd_cached(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                        const int8_t* seg, const int32_t* ts, const void* q, const void* k,
                                        const void* v, const float* rab, void* out,
                                        const mtgr_hstu_problem_t* pc, const int32_t* offsets_c,
                                        const int32_t* ts_c, const void* kc, const void* vc,
                                        const void* cache_plan, size_t cache_plan_bytes, void* workspace,
                                        size_t workspace_bytes, mtgr_stream_t stream) {
    mtgr_status_t st = check_attn_common(p, offsets, seg, ts, rab, workspace, workspace_bytes);
    if (st != MTGR_SUCCESS) return st;
    if (!pc) return fail(MTGR_ERROR_NULL_POINTER, "cache problem is NULL");
    st = check_problem(pc);
    if (st != MTGR_SUCCESS) return st;
    if (pc->num_users != p->num_users || pc->num_heads != p->num_heads || pc->head_dim != p->head_dim ||
        pc->dtype != p->dtype)
        return fail(MTGR_ERROR_INVALID_ARGUMENT,
                    "cache and request differ in num_users, num_heads, head_dim or dtype");
    if (vec_path(p))
        return fail(MTGR_ERROR_UNSUPPORTED, "the cached forward runs on the bf16 matrix cores (head_dim 32..128)");
    if (p->flags & ~MTGR_ATTN_PLANNED)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "only MTGR_ATTN_PLANNED applies to the cached forward");
    if (p->num_users == 0) return ok();
    if (!offsets_c) return fail(MTGR_ERROR_NULL_POINTER, "offsets_c is NULL");
    if (((uintptr_t)offsets_c & 3u) != 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "offsets_c is not 4-byte aligned");
    const AttnLayout Lc = attn_layout(pc);
    if (pc->total_tokens > 0) {
        if (!ts_c) return fail(MTGR_ERROR_NULL_POINTER, "ts_c is NULL");
        if (((uintptr_t)ts_c & 3u) != 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "ts_c is not 4-byte aligned");
        REQUIRE_PTR(kc, "kc");
        REQUIRE_PTR(vc, "vc");
        if (!cache_plan) return fail(MTGR_ERROR_NULL_POINTER, "cache_plan is NULL");
        if (((uintptr_t)cache_plan & 255u) != 0)
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "cache_plan is not 256-byte aligned");
        if (cache_plan_bytes < Lc.total)
            return fail(MTGR_ERROR_WORKSPACE_TOO_SMALL, "cache_plan %zu bytes, need %zu", cache_plan_bytes, Lc.total);
    }
    if (p->total_tokens == 0) return ok();
    REQUIRE_PTR(q, "q");
    REQUIRE_PTR(k, "k");
    REQUIRE_PTR(v, "v");
    REQUIRE_PTR(out, "out");
    hipStream_t s = (hipStream_t)stream;
    const AttnLayout L = attn_layout(p);
    if (!(p->flags & MTGR_ATTN_PLANNED)) {
        st = schedule(p, L, offsets, seg, ts, workspace, s);
        if (st != MTGR_SUCCESS) return st;
    }
    mtgr::AttnArgs a = make_args(p, L, offsets, seg, ts, workspace);
    a.q = q;
    a.k = k;
    a.v = v;
    a.rab = rab;
    a.out = out;
    a.kc = kc;
    a.vc = vc;
    a.ld_kc = pc->ld_k;
    a.ld_vc = pc->ld_v;
    a.offsets_k = offsets_c;
    a.ts_k = ts_c;
    const char* cp = (const char*)cache_plan;
    a.tok_code_k = pc->total_tokens > 0 ? (const int*)(cp + Lc.off_code) : nullptr;
    a.summ_k = pc->total_tokens > 0 ? (const int4*)(cp + Lc.off_summ) : nullptr;
    a.ntile_k = pc->total_tokens > 0 ? Lc.ntile : 0;
    hipError_t e = mtgr::launch_attn_fwd_cached_bf16(a, p->head_dim, (int)L.slots, s);
    if (e != hipSuccess) return device_fail(e, "cached attention forward");
    return ok();
}

mtgr_status_t mtgr_hstu_attn_bwd(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                 const int8_t* seg, const int32_t* ts, const void* q, const void* k,
                                 const void* v, const float* rab, const void* dout, void* dq,
                                 void* dk, void* dv, float* drab, void* workspace,
                                 size_t workspace_bytes, mtgr_stream_t stream) {
    mtgr_status_t st = check_attn_common(p, offsets, seg, ts, rab, workspace, workspace_bytes);
    if (st != MTGR_SUCCESS) return st;
    if (p->flags & MTGR_FWD_CAND_ROWS)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "MTGR_FWD_CAND_ROWS applies to the forward only");
    if (drab && !rab) return fail(MTGR_ERROR_INVALID_ARGUMENT, "drab given without rab");
    if (drab && ((uintptr_t)drab & 3u) != 0)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "drab is not 4-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    if (p->num_users == 0 || p->total_tokens == 0) {
        if (drab) {
            hipError_t e = mtgr::launch_fill_f32(drab, (long long)p->num_heads * p->num_rab_buckets, 0.f, s);
            if (e != hipSuccess) return device_fail(e, "drab fill");
        }
        return ok();
    }
    const bool want_dq = !(p->flags & MTGR_BWD_SKIP_DQ);
    const bool want_dkdv = !(p->flags & MTGR_BWD_SKIP_DKDV);
    const bool keep_ds = (p->flags & MTGR_BWD_KEEP_DS) != 0;
    const bool ds_ready = (p->flags & MTGR_BWD_DS_READY) != 0;
    if (keep_ds && want_dq)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "MTGR_BWD_KEEP_DS needs MTGR_BWD_SKIP_DQ");
    if (ds_ready && want_dkdv)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "MTGR_BWD_DS_READY needs MTGR_BWD_SKIP_DKDV");
    if (ds_ready && drab)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "drab is formed by the MTGR_BWD_KEEP_DS call");
    REQUIRE_PTR(q, "q");
    REQUIRE_PTR(k, "k");
    REQUIRE_PTR(v, "v");
    REQUIRE_PTR(dout, "dout");
    if (want_dq) REQUIRE_PTR(dq, "dq");
    if (want_dkdv) {
        REQUIRE_PTR(dk, "dk");
        REQUIRE_PTR(dv, "dv");
    }
    const AttnLayout L = attn_layout(p);
    // Stored-dS path: the MFMA kernels and a backward-size workspace.
    const bool vec = vec_path(p);
    const bool ds_path = !vec && L.total_bwd > L.total && workspace_bytes >= L.total_bwd;
    if ((keep_ds || ds_ready) && !ds_path)
        return fail(MTGR_ERROR_WORKSPACE_TOO_SMALL,
                    "MTGR_BWD_KEEP_DS / _DS_READY need a bf16 problem and %zu workspace bytes", L.total_bwd);
    if (!(p->flags & MTGR_ATTN_PLANNED)) {
        st = schedule(p, L, offsets, seg, ts, workspace, s);
        if (st != MTGR_SUCCESS) return st;
    }
    mtgr::BwdPlan plan{};
    plan.dkdv = want_dkdv;
    plan.store_ds = want_dkdv && ds_path && (want_dq || keep_ds);
    plan.dq_from_ds = want_dq && (ds_ready || (want_dkdv && ds_path));
    plan.dq_recompute = want_dq && !plan.dq_from_ds;
    // drab comes from the dk/dv kernel when it runs (MFMA kernels), else from the recomputing
    // dq kernel; the vector-ALU kernels form it in their dq kernel
    float* drab_out = !vec ? ((want_dkdv || plan.dq_recompute) ? drab : nullptr)
                           : (want_dq ? drab : nullptr);
    if (drab_out) {
        hipError_t e = mtgr::launch_fill_f32(drab_out, (long long)p->num_heads * p->num_rab_buckets, 0.f, s);
        if (e != hipSuccess) return device_fail(e, "drab fill");
    }
    mtgr::AttnArgs a = make_args(p, L, offsets, seg, ts, workspace);
    a.q = q;
    a.k = k;
    a.v = v;
    a.rab = rab;
    a.dout = dout;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.drab = drab_out;
    hipError_t e = !vec ? mtgr::launch_attn_bwd_bf16(a, p->head_dim, (int)L.slots, plan, s)
                        : mtgr::launch_attn_bwd_vec(a, p->dtype == MTGR_DTYPE_BF16, p->head_dim, (int)L.slots,
                                                    want_dq, want_dkdv, s);
    if (e != hipSuccess) return device_fail(e, "attention backward");
    return ok();
}

}  // extern "C"

namespace {

mtgr_status_t check_gln(const mtgr_gln_problem_t* p) {
    if (!p) return fail(MTGR_ERROR_NULL_POINTER, "problem is NULL");
    if (p->dtype != MTGR_DTYPE_BF16 && p->dtype != MTGR_DTYPE_FP32)
        return fail(MTGR_ERROR_UNSUPPORTED, "dtype %d is not supported", p->dtype);
    if (p->num_tokens < 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "num_tokens < 0");
    // The forward launches 16 work-items per token (a wave per four tokens); a grid holds at
    // most 2^32 - 1 work-items.
    if (p->num_tokens >= (1ll << 28))
        return fail(MTGR_ERROR_UNSUPPORTED, "num_tokens %lld above 2^28 - 1", (long long)p->num_tokens);
    const int vec = p->dtype == MTGR_DTYPE_BF16 ? 8 : 4;
    const int dmax = p->dtype == MTGR_DTYPE_BF16 ? 4096 : 2048;
    if (p->dim <= 0 || p->dim % vec != 0)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "dim %d must be a positive multiple of %d", p->dim, vec);
    if (p->dim > dmax) return fail(MTGR_ERROR_UNSUPPORTED, "dim %d above %d", p->dim, dmax);
    if (p->num_groups < 1 || p->num_groups > MTGR_MAX_GROUPS)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "num_groups %d outside 1..%d", p->num_groups,
                    MTGR_MAX_GROUPS);
    if (!(p->eps > 0.f) || !std::isfinite(p->eps))
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "eps must be positive and finite");
    const int esz = p->dtype == MTGR_DTYPE_BF16 ? 2 : 4;
    const long long lds[3] = {p->ld_x, p->ld_u, p->ld_y};
    const char* names[3] = {"ld_x", "ld_u", "ld_y"};
    for (int i = 0; i < 3; i++) {
        if (lds[i] < p->dim)
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "%s %lld below dim %d", names[i], lds[i], p->dim);
        if ((lds[i] * esz) % 16 != 0)
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "%s %lld is not a multiple of 16 bytes", names[i],
                        lds[i]);
        if (lds[i] > MTGR_MAX_LD)
            return fail(MTGR_ERROR_UNSUPPORTED, "%s %lld above %lld elements", names[i], lds[i],
                        (long long)MTGR_MAX_LD);
    }
    return MTGR_SUCCESS;
}

mtgr::GlnArgs gln_args(const mtgr_gln_problem_t* p) {
    mtgr::GlnArgs a{};
    a.T = p->num_tokens;
    a.d = p->dim;
    a.G = p->num_groups;
    a.eps = p->eps;
    a.ld_x = p->ld_x;
    a.ld_u = p->ld_u;
    a.ld_y = p->ld_y;
    return a;
}

}  // namespace

extern "C" {

mtgr_status_t mtgr_group_layernorm_workspace_size(const mtgr_gln_problem_t* p, int backward,
                                                  size_t* bytes) {
    if (!bytes) return fail(MTGR_ERROR_NULL_POINTER, "bytes is NULL");
    mtgr_status_t st = check_gln(p);
    if (st != MTGR_SUCCESS) return st;
    *bytes = (backward && p->num_tokens > 0)
                 ? align256(mtgr::gln_bwd_workspace_bytes(p->num_tokens, p->dim, p->num_groups))
                 : 0;
    return ok();
}

mtgr_status_t mtgr_group_layernorm_fwd(const mtgr_gln_problem_t* p, const void* x, const void* u,
                                       const int8_t* group_ids, const float* gamma, const float* beta,
                                       void* y, float* mean, float* rstd, mtgr_stream_t stream) {
    mtgr_status_t st = check_gln(p);
    if (st != MTGR_SUCCESS) return st;
    REQUIRE_PTR(gamma, "gamma");
    REQUIRE_PTR(beta, "beta");
    if (p->num_tokens == 0) return ok();
    REQUIRE_PTR(x, "x");
    REQUIRE_PTR(y, "y");
    if (u && !aligned16(u)) return fail(MTGR_ERROR_INVALID_ARGUMENT, "u is not 16-byte aligned");
    if (!group_ids) return fail(MTGR_ERROR_NULL_POINTER, "group_ids is NULL");
    if ((mean && ((uintptr_t)mean & 3u)) || (rstd && ((uintptr_t)rstd & 3u)))
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "mean/rstd not 4-byte aligned");
    mtgr::GlnArgs a = gln_args(p);
    a.x = x;
    a.u = u;
    a.gid = group_ids;
    a.gamma = gamma;
    a.beta = beta;
    a.y = y;
    a.mean = mean;
    a.rstd = rstd;
    hipError_t e = mtgr::launch_gln_fwd(a, p->dtype == MTGR_DTYPE_BF16, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "group layernorm forward");
    return ok();
}

mtgr_status_t mtgr_group_layernorm_bwd(const mtgr_gln_problem_t* p, const void* dy, const void* x,
                                       const void* u, const int8_t* group_ids, const float* gamma,
                                       const float* mean, const float* rstd, void* dx, void* du,
                                       float* dgamma, float* dbeta, void* workspace,
                                       size_t workspace_bytes, mtgr_stream_t stream) {
    mtgr_status_t st = check_gln(p);
    if (st != MTGR_SUCCESS) return st;
    REQUIRE_PTR(gamma, "gamma");
    REQUIRE_PTR(dgamma, "dgamma");
    REQUIRE_PTR(dbeta, "dbeta");
    if ((u == nullptr) != (du == nullptr))
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "du must be given exactly when u is given");
    if (p->num_tokens > 0) {
        const size_t need = align256(mtgr::gln_bwd_workspace_bytes(p->num_tokens, p->dim, p->num_groups));
        if (workspace_bytes < need)
            return fail(MTGR_ERROR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", workspace_bytes, need);
        REQUIRE_PTR(workspace, "workspace");
    }
    if (p->num_tokens > 0) {
        REQUIRE_PTR(dy, "dy");
        REQUIRE_PTR(x, "x");
        REQUIRE_PTR(dx, "dx");
        if (u) {
            REQUIRE_PTR(u, "u");
            REQUIRE_PTR(du, "du");
        }
        if (!group_ids) return fail(MTGR_ERROR_NULL_POINTER, "group_ids is NULL");
        if (!mean) return fail(MTGR_ERROR_NULL_POINTER, "mean is NULL");
        if (!rstd) return fail(MTGR_ERROR_NULL_POINTER, "rstd is NULL");
    }
    mtgr::GlnArgs a = gln_args(p);
    a.dy = dy;
    a.x = x;
    a.u = u;
    a.gid = group_ids;
    a.gamma = gamma;
    a.mean = const_cast<float*>(mean);
    a.rstd = const_cast<float*>(rstd);
    a.dx = dx;
    a.du = du;
    a.dgamma = dgamma;
    a.dbeta = dbeta;
    a.workspace = (float*)workspace;
    hipError_t e = mtgr::launch_gln_bwd(a, p->dtype == MTGR_DTYPE_BF16, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "group layernorm backward");
    return ok();
}

static mtgr_status_t check_pointwise(int64_t rows, int32_t cols, mtgr_dtype_t dtype,
                                     const void* const* mats, const int64_t* lds, const char* const* names,
                                     int n, const float* bias) {
    if (dtype != MTGR_DTYPE_BF16 && dtype != MTGR_DTYPE_FP32) return fail(MTGR_ERROR_UNSUPPORTED, "dtype %d", (int)dtype);
    const int esz = dtype == MTGR_DTYPE_BF16 ? 2 : 4, per = 16 / esz;
    if (rows < 0 || cols <= 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "rows = %lld, cols = %d", (long long)rows, cols);
    if (cols % per != 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "cols = %d is not a multiple of %d", cols, per);
    if (rows > 0) {
        for (int i = 0; i < n; i++) {
            if (mats[i] == nullptr) return fail(MTGR_ERROR_NULL_POINTER, "%s is NULL", names[i]);
            if (!aligned16(mats[i])) return fail(MTGR_ERROR_INVALID_ARGUMENT, "%s is not 16-byte aligned", names[i]);
            if (lds[i] < cols || (lds[i] * esz) % 16 != 0)
                return fail(MTGR_ERROR_INVALID_ARGUMENT, "ld of %s = %lld (needs >= cols and 16-byte rows)", names[i],
                            (long long)lds[i]);
        }
        if (bias != nullptr && ((uintptr_t)bias & 3u) != 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "bias is not 4-byte aligned");
    }
    return MTGR_SUCCESS;
}

mtgr_status_t mtgr_bias_silu_fwd(int64_t rows, int32_t cols, mtgr_dtype_t dtype, const void* h, int64_t ld_h,
                                 const float* bias, void* out, int64_t ld_out, mtgr_stream_t stream) {
    const void* mats[2] = {h, out};
    const int64_t lds[2] = {ld_h, ld_out};
    const char* names[2] = {"h", "out"};
    mtgr_status_t st = check_pointwise(rows, cols, dtype, mats, lds, names, 2, bias);
    if (st != MTGR_SUCCESS) return st;
    hipError_t e = mtgr::launch_bias_silu(rows, cols, dtype == MTGR_DTYPE_BF16, false, h, ld_h, bias, nullptr, 0,
                                          out, ld_out, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "bias silu forward");
    return ok();
}

mtgr_status_t mtgr_bias_silu_bwd(int64_t rows, int32_t cols, mtgr_dtype_t dtype, const void* h, int64_t ld_h,
                                 const float* bias, const void* dout, int64_t ld_dout, void* dh, int64_t ld_dh,
                                 mtgr_stream_t stream) {
    const void* mats[3] = {h, dout, dh};
    const int64_t lds[3] = {ld_h, ld_dout, ld_dh};
    const char* names[3] = {"h", "dout", "dh"};
    mtgr_status_t st = check_pointwise(rows, cols, dtype, mats, lds, names, 3, bias);
    if (st != MTGR_SUCCESS) return st;
    hipError_t e = mtgr::launch_bias_silu(rows, cols, dtype == MTGR_DTYPE_BF16, true, h, ld_h, bias, dout, ld_dout,
                                          dh, ld_dh, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "bias silu backward");
    return ok();
}

mtgr_status_t mtgr_add(int64_t rows, int32_t cols, mtgr_dtype_t dtype, const void* a, int64_t ld_a, const void* b,
                       int64_t ld_b, void* out, int64_t ld_out, mtgr_stream_t stream) {
    const void* mats[3] = {a, b, out};
    const int64_t lds[3] = {ld_a, ld_b, ld_out};
    const char* names[3] = {"a", "b", "out"};
    mtgr_status_t st = check_pointwise(rows, cols, dtype, mats, lds, names, 3, nullptr);
    if (st != MTGR_SUCCESS) return st;
    hipError_t e = mtgr::launch_add(rows, cols, dtype == MTGR_DTYPE_BF16, a, ld_a, b, ld_b, out, ld_out,
                                    (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "add");
    return ok();
}

}  // extern "C"

namespace {

constexpr long long GEMM_MAX_LD = 1ll << 22;   // 32-bit per-lane copy offsets over 256 rows

mtgr_status_t check_gemm(int layout, int64_t M, int64_t N, int64_t K, int epilogue) {
    if (layout < MTGR_GEMM_NN || layout > MTGR_GEMM_TN)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "layout %d is not MTGR_GEMM_NN / _NT / _TN", layout);
    if (epilogue < MTGR_GEMM_EPI_NONE || epilogue > MTGR_GEMM_EPI_BIAS_RESIDUAL)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "epilogue %d unknown", epilogue);
    if (layout == MTGR_GEMM_TN && epilogue != MTGR_GEMM_EPI_NONE)
        return fail(MTGR_ERROR_UNSUPPORTED, "MTGR_GEMM_TN takes no epilogue");
    if (M < 0 || N < 0 || K < 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "negative size");
    if (M >= (1ll << 31) || N >= (1ll << 31) || K >= (1ll << 31))
        return fail(MTGR_ERROR_UNSUPPORTED, "sizes must be below 2^31");
    if (N % 8 != 0) return fail(MTGR_ERROR_UNSUPPORTED, "N = %lld is not a multiple of 8", (long long)N);
    if (layout != MTGR_GEMM_TN && K % 32 != 0)
        return fail(MTGR_ERROR_UNSUPPORTED, "K = %lld is not a multiple of 32", (long long)K);
    if (layout == MTGR_GEMM_TN && M % 8 != 0)
        return fail(MTGR_ERROR_UNSUPPORTED, "M = %lld is not a multiple of 8 (MTGR_GEMM_TN)", (long long)M);
    int mb, nb, s, per;
    mtgr::gemm_plan(layout, M, N, K, &mb, &nb, &s, &per);
    if ((long long)((mb + mtgr::XCDS - 1) / mtgr::XCDS) * mtgr::XCDS * nb * s >= (1ll << 24))
        return fail(MTGR_ERROR_UNSUPPORTED, "problem too large for one launch");
    return MTGR_SUCCESS;
}

mtgr_status_t check_ld(const void* p, const char* name, int64_t ld, int64_t min_ld) {
    if (!p) return fail(MTGR_ERROR_NULL_POINTER, "%s is NULL", name);
    if (!aligned16(p)) return fail(MTGR_ERROR_INVALID_ARGUMENT, "%s is not 16-byte aligned", name);
    if (ld < min_ld || ld % 8 != 0)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "ld of %s = %lld (needs >= %lld and a multiple of 8)", name,
                    (long long)ld, (long long)min_ld);
    if (ld >= GEMM_MAX_LD)
        return fail(MTGR_ERROR_UNSUPPORTED, "ld of %s = %lld above %lld", name, (long long)ld, GEMM_MAX_LD);
    return MTGR_SUCCESS;
}

}  // namespace

extern "C" {

mtgr_status_t mtgr_gemm_workspace_size(int32_t layout, int64_t M, int64_t N, int64_t K, size_t* bytes) {
    if (!bytes) return fail(MTGR_ERROR_NULL_POINTER, "bytes is NULL");
    mtgr_status_t st = check_gemm(layout, M, N, K, MTGR_GEMM_EPI_NONE);
    if (st != MTGR_SUCCESS) return st;
    *bytes = (M > 0 && N > 0 && K > 0) ? align256(mtgr::gemm_workspace_bytes(layout, M, N, K)) : 0;
    return ok();
}

mtgr_status_t mtgr_gemm_bf16(int32_t layout, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                             const void* B, int64_t ldb, void* C, int64_t ldc, int32_t epilogue, const float* bias,
                             const void* R, int64_t ldr, void* C2, int64_t ldc2, float* colsum, void* workspace,
                             size_t workspace_bytes, mtgr_stream_t stream) {
    mtgr_status_t st = check_gemm(layout, M, N, K, epilogue);
    if (st != MTGR_SUCCESS) return st;
    if (colsum && layout != MTGR_GEMM_TN)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "colsum is formed by MTGR_GEMM_TN only");
    if (colsum && ((uintptr_t)colsum & 3u) != 0)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "colsum is not 4-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    if (M == 0 || N == 0) return ok();
    if (K == 0) return fail(MTGR_ERROR_UNSUPPORTED, "K = 0");
    const bool a_kr = layout == MTGR_GEMM_TN, b_kr = layout != MTGR_GEMM_NT;
    if ((st = check_ld(A, "A", lda, a_kr ? M : K)) != MTGR_SUCCESS) return st;
    if ((st = check_ld(B, "B", ldb, b_kr ? N : K)) != MTGR_SUCCESS) return st;
    if ((st = check_ld(C, "C", ldc, N)) != MTGR_SUCCESS) return st;
    if (epilogue != MTGR_GEMM_EPI_NONE) {
        if (!bias) return fail(MTGR_ERROR_NULL_POINTER, "bias is NULL");
        if (!aligned16(bias)) return fail(MTGR_ERROR_INVALID_ARGUMENT, "bias is not 16-byte aligned");
    }
    if (epilogue == MTGR_GEMM_EPI_BIAS_SILU && (st = check_ld(C2, "C2", ldc2, N)) != MTGR_SUCCESS) return st;
    if (epilogue == MTGR_GEMM_EPI_BIAS_RESIDUAL && (st = check_ld(R, "R", ldr, N)) != MTGR_SUCCESS) return st;
    mtgr::GemmArgs g{};
    g.layout = layout;
    g.epilogue = epilogue;
    g.M = M;
    g.N = N;
    g.K = K;
    g.A = A;
    g.lda = lda;
    g.B = B;
    g.ldb = ldb;
    g.C = C;
    g.ldc = ldc;
    g.C2 = C2;
    g.ldc2 = ldc2;
    g.R = R;
    g.ldr = ldr;
    g.bias = bias;
    g.colsum = colsum;
    mtgr::gemm_plan(layout, M, N, K, &g.mblocks, &g.nblocks, &g.splits, &g.ks_per_split);
    if (layout == MTGR_GEMM_TN) {
        const size_t need = align256(mtgr::gemm_workspace_bytes(layout, M, N, K));
        if (workspace_bytes < need)
            return fail(MTGR_ERROR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", workspace_bytes, need);
        if (!workspace) return fail(MTGR_ERROR_NULL_POINTER, "workspace is NULL");
        if (!aligned16(workspace)) return fail(MTGR_ERROR_INVALID_ARGUMENT, "workspace is not 16-byte aligned");
        g.partial = (float*)workspace;
        g.colsum_partial = g.partial + (size_t)g.splits * M * N;
    }
    hipError_t e = mtgr::launch_gemm_bf16(g, s);
    if (e != hipSuccess) return device_fail(e, "gemm");
    return ok();
}

mtgr_status_t mtgr_debug_clock_probe(int32_t mfma_iterations, int32_t blocks, int64_t* out,
                                     int32_t* wall_clock_khz, mtgr_stream_t stream) {
    if (mfma_iterations < 1 || blocks < 1 || blocks > 65536)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "mfma_iterations = %d, blocks = %d", mfma_iterations, blocks);
    if (!out || !wall_clock_khz) return fail(MTGR_ERROR_NULL_POINTER, "out or wall_clock_khz is NULL");
    if (((uintptr_t)out & 7u) != 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "out is not 8-byte aligned");
    int dev = 0, khz = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (e != hipSuccess) return device_fail(e, "wall clock rate");
    *wall_clock_khz = khz;
    e = mtgr::launch_clock_probe(mfma_iterations, blocks, (long long*)out, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "clock probe");
    return ok();
}

mtgr_status_t mtgr_debug_validate_inputs(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                         const int8_t* seg, const int8_t* group_ids,
                                         int32_t num_groups, void* scratch, size_t scratch_bytes,
                                         mtgr_stream_t stream) {
    static_assert(MTGR_VALIDATE_SCRATCH_BYTES >= mtgr::VALIDATE_CONDITIONS * 8, "scratch size");
    if (p == nullptr) return fail(MTGR_ERROR_NULL_POINTER, "p is NULL");
    if (p->num_users < 0 || p->total_tokens < 0 || p->max_seqlen < 0)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "num_users, total_tokens and max_seqlen must be >= 0");
    if (offsets == nullptr) return fail(MTGR_ERROR_NULL_POINTER, "offsets is NULL");
    if (p->total_tokens > 0 && seg == nullptr) return fail(MTGR_ERROR_NULL_POINTER, "seg is NULL");
    if (group_ids != nullptr && (num_groups < 1 || num_groups > 127))
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "num_groups = %d outside 1..127", num_groups);
    if (scratch == nullptr) return fail(MTGR_ERROR_NULL_POINTER, "scratch is NULL");
    if (scratch_bytes < MTGR_VALIDATE_SCRATCH_BYTES)
        return fail(MTGR_ERROR_WORKSPACE_TOO_SMALL, "scratch has %zu bytes, needs %d", scratch_bytes,
                    MTGR_VALIDATE_SCRATCH_BYTES);
    if (((uintptr_t)scratch & 7u) != 0) return fail(MTGR_ERROR_INVALID_ARGUMENT, "scratch is not 8-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    unsigned long long* first = (unsigned long long*)scratch;
    hipError_t e = mtgr::launch_validate(offsets, p->num_users, p->total_tokens, p->max_seqlen, seg,
                                         group_ids, num_groups, first, s);
    if (e != hipSuccess) return device_fail(e, "validate inputs");
    unsigned long long h[mtgr::VALIDATE_CONDITIONS];
    e = hipMemcpyAsync(h, first, sizeof(h), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return device_fail(e, "validate inputs (copy back)");
    static const char* const what[mtgr::VALIDATE_CONDITIONS] = {
        "offsets[0] != 0", "offsets decrease after user", "offsets[num_users] != total_tokens",
        "sequence longer than max_seqlen: user", "seg outside 0..3 at token", "group id outside 0..G-1 at token"};
    std::string msg;
    for (int c = 0; c < mtgr::VALIDATE_CONDITIONS; c++) {
        if (h[c] == ~0ull) continue;
        char buf[96];
        snprintf(buf, sizeof(buf), "%s%s %llu", msg.empty() ? "" : "; ", what[c], h[c]);
        msg += buf;
    }
    if (!msg.empty()) return fail(MTGR_ERROR_INVALID_ARGUMENT, "%s", msg.c_str());
    return ok();
}

const char* mtgr_status_string(mtgr_status_t status) {
    switch (status) {
        case MTGR_SUCCESS: return "success";
        case MTGR_ERROR_NULL_POINTER: return "null pointer";
        case MTGR_ERROR_INVALID_ARGUMENT: return "invalid argument";
        case MTGR_ERROR_UNSUPPORTED: return "unsupported";
        case MTGR_ERROR_WORKSPACE_TOO_SMALL: return "workspace too small";
        case MTGR_ERROR_DEVICE: return "device error";
        default: return "unknown status";
    }
}

const char* mtgr_last_error_message(void) { return g_last_error.c_str(); }

int32_t mtgr_version(void) { return MTGR_HSTU_VERSION; }


}  // extern "C"

// ------------------------------------------------------------------------ embedding table
namespace {

constexpr long long EMB_MAX_BATCH = 1ll << 30;   // IDs per dedup call (int32 positions)

mtgr_status_t check_table(const mtgr_embedding_table_t* t, mtgr::EmbArgs* a) {
    if (!t) return fail(MTGR_ERROR_NULL_POINTER, "table is NULL");
    if (t->dtype != MTGR_DTYPE_BF16 && t->dtype != MTGR_DTYPE_FP32)
        return fail(MTGR_ERROR_UNSUPPORTED, "dtype %d is not supported", t->dtype);
    if (t->key_capacity < 2 || t->key_capacity > (1ll << 40) || (t->key_capacity & (t->key_capacity - 1)))
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "key_capacity %lld is not a power of two in 2 .. 2^40",
                    (long long)t->key_capacity);
    if (t->row_capacity < 1 || t->row_capacity > 0x7fffffffll)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "row_capacity %lld outside 1 .. 2^31 - 1",
                    (long long)t->row_capacity);
    if (t->key_capacity < t->row_capacity + 1)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "key_capacity %lld below row_capacity + 1",
                    (long long)t->key_capacity);
    if (t->dim < 8 || t->dim > 1024 || t->dim % 8)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "dim %d is not a multiple of 8 in 8 .. 1024", t->dim);
    REQUIRE_PTR(t->keys, "keys");
    REQUIRE_PTR(t->key_rows, "key_rows");
    REQUIRE_PTR(t->values, "values");
    REQUIRE_PTR(t->counts, "counts");
    REQUIRE_PTR(t->last_ts, "last_ts");
    REQUIRE_PTR(t->free_rows, "free_rows");
    REQUIRE_PTR(t->state, "state");
    a->key_capacity = t->key_capacity;
    a->row_capacity = (int)t->row_capacity;
    a->dim = t->dim;
    a->esize = t->dtype == MTGR_DTYPE_BF16 ? 2 : 4;
    a->keys = t->keys;
    a->key_rows = t->key_rows;
    a->values = t->values;
    a->counts = t->counts;
    a->last_ts = t->last_ts;
    a->free_rows = t->free_rows;
    a->state = t->state;
    return MTGR_SUCCESS;
}

mtgr_status_t check_count(long long n, long long max, const char* name) {
    if (n < 0 || n > max) return fail(MTGR_ERROR_INVALID_ARGUMENT, "%s %lld outside 0 .. %lld", name, n, max);
    return MTGR_SUCCESS;
}

}  // namespace

extern "C" {

mtgr_status_t mtgr_embedding_init(const mtgr_embedding_table_t* t, mtgr_stream_t stream) {
    mtgr::EmbArgs a;
    mtgr_status_t st = check_table(t, &a);
    if (st != MTGR_SUCCESS) return st;
    hipError_t e = mtgr::launch_emb_init(a, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "embedding init");
    return ok();
}

mtgr_status_t mtgr_embedding_dedup_workspace_size(int64_t n, size_t* bytes) {
    if (!bytes) return fail(MTGR_ERROR_NULL_POINTER, "bytes is NULL");
    mtgr_status_t st = check_count(n, EMB_MAX_BATCH, "n");
    if (st != MTGR_SUCCESS) return st;
    *bytes = mtgr::dedup_workspace_bytes(n);
    return ok();
}

mtgr_status_t mtgr_embedding_dedup(int64_t n, const uint64_t* ids, uint64_t* unique, int32_t* occurrences,
                                   int32_t* inverse, int64_t* num_unique, void* workspace,
                                   size_t workspace_bytes, mtgr_stream_t stream) {
    mtgr_status_t st = check_count(n, EMB_MAX_BATCH, "n");
    if (st != MTGR_SUCCESS) return st;
    REQUIRE_PTR(num_unique, "num_unique");
    REQUIRE_PTR(workspace, "workspace");
    if (n > 0) {
        REQUIRE_PTR(ids, "ids");
        REQUIRE_PTR(unique, "unique");
        REQUIRE_PTR(inverse, "inverse");
        if (occurrences && !aligned16(occurrences))
            return fail(MTGR_ERROR_INVALID_ARGUMENT, "occurrences is not 16-byte aligned");
    }
    const size_t need = mtgr::dedup_workspace_bytes(n);
    if (workspace_bytes < need)
        return fail(MTGR_ERROR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", workspace_bytes, need);
    hipError_t e = mtgr::launch_emb_dedup(n, ids, unique, occurrences, inverse, (long long*)num_unique, workspace,
                                          (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "embedding dedup");
    return ok();
}

mtgr_status_t mtgr_embedding_lookup_workspace_size(int64_t n_max, size_t* bytes) {
    if (!bytes) return fail(MTGR_ERROR_NULL_POINTER, "bytes is NULL");
    mtgr_status_t st = check_count(n_max, EMB_MAX_BATCH, "n_max");
    if (st != MTGR_SUCCESS) return st;
    *bytes = mtgr::lookup_workspace_bytes(n_max);
    return ok();
}

mtgr_status_t mtgr_embedding_lookup(const mtgr_embedding_table_t* t, int64_t n_max, const uint64_t* unique,
                                    const int32_t* occurrences, const int64_t* num_unique, int32_t now,
                                    int32_t insert, int32_t* rows, void* workspace, size_t workspace_bytes,
                                    mtgr_stream_t stream) {
    mtgr::EmbArgs a;
    mtgr_status_t st = check_table(t, &a);
    if (st != MTGR_SUCCESS) return st;
    st = check_count(n_max, EMB_MAX_BATCH, "n_max");
    if (st != MTGR_SUCCESS) return st;
    if (n_max == 0) return ok();
    REQUIRE_PTR(unique, "unique");
    REQUIRE_PTR(num_unique, "num_unique");
    REQUIRE_PTR(rows, "rows");
    REQUIRE_PTR(workspace, "workspace");
    if (occurrences && !aligned16(occurrences))
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "occurrences is not 16-byte aligned");
    const size_t need = mtgr::lookup_workspace_bytes(n_max);
    if (workspace_bytes < need)
        return fail(MTGR_ERROR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", workspace_bytes, need);
    hipError_t e = mtgr::launch_emb_lookup(a, n_max, unique, occurrences, (const long long*)num_unique, now,
                                           insert ? 1 : 0, rows, workspace, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "embedding lookup");
    return ok();
}

mtgr_status_t mtgr_embedding_gather(const mtgr_embedding_table_t* t, int64_t n, const int32_t* inverse,
                                    const int32_t* rows, void* out, int64_t ld_out, mtgr_stream_t stream) {
    mtgr::EmbArgs a;
    mtgr_status_t st = check_table(t, &a);
    if (st != MTGR_SUCCESS) return st;
    st = check_count(n, 0x7fffffffll, "n");
    if (st != MTGR_SUCCESS) return st;
    if (ld_out < t->dim || ld_out % 8)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "ld_out %lld is below dim or not a multiple of 8",
                    (long long)ld_out);
    if (n == 0) return ok();
    REQUIRE_PTR(inverse, "inverse");
    REQUIRE_PTR(rows, "rows");
    REQUIRE_PTR(out, "out");
    hipError_t e = mtgr::launch_emb_gather(a, n, inverse, rows, out, ld_out, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "embedding gather");
    return ok();
}

mtgr_status_t mtgr_embedding_sgd_workspace_size(int64_t n, int64_t n_max, int32_t dim, size_t* bytes) {
    if (!bytes) return fail(MTGR_ERROR_NULL_POINTER, "bytes is NULL");
    mtgr_status_t st = check_count(n, EMB_MAX_BATCH, "n");
    if (st != MTGR_SUCCESS) return st;
    st = check_count(n_max, EMB_MAX_BATCH, "n_max");
    if (st != MTGR_SUCCESS) return st;
    if (dim < 8 || dim > 1024 || dim % 8)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "dim %d is not a multiple of 8 in 8 .. 1024", dim);
    *bytes = mtgr::sgd_workspace_bytes(n, n_max, dim);
    return ok();
}

mtgr_status_t mtgr_embedding_sgd(const mtgr_embedding_table_t* t, int64_t n, const int32_t* inverse,
                                 const int32_t* occurrences, const void* grad_out, int64_t ld_grad, int64_t n_max,
                                 const int32_t* rows, const int64_t* num_unique, float lr, void* workspace,
                                 size_t workspace_bytes, mtgr_stream_t stream) {
    mtgr::EmbArgs a;
    mtgr_status_t st = check_table(t, &a);
    if (st != MTGR_SUCCESS) return st;
    st = check_count(n, EMB_MAX_BATCH, "n");
    if (st != MTGR_SUCCESS) return st;
    st = check_count(n_max, EMB_MAX_BATCH, "n_max");
    if (st != MTGR_SUCCESS) return st;
    if (!std::isfinite(lr)) return fail(MTGR_ERROR_INVALID_ARGUMENT, "lr is not finite");
    if (ld_grad < t->dim || ld_grad % 8)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "ld_grad %lld is below dim or not a multiple of 8",
                    (long long)ld_grad);
    if (n_max == 0) return ok();
    if (n > 0) {
        REQUIRE_PTR(inverse, "inverse");
        REQUIRE_PTR(occurrences, "occurrences");
        REQUIRE_PTR(grad_out, "grad_out");
    }
    REQUIRE_PTR(rows, "rows");
    REQUIRE_PTR(num_unique, "num_unique");
    REQUIRE_PTR(workspace, "workspace");
    const size_t need = mtgr::sgd_workspace_bytes(n, n_max, t->dim);
    if (workspace_bytes < need)
        return fail(MTGR_ERROR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", workspace_bytes, need);
    hipError_t e = mtgr::launch_emb_sgd(a, n, inverse, occurrences, grad_out, ld_grad, n_max, rows,
                                        (const long long*)num_unique, lr, workspace, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "embedding sgd");
    return ok();
}

mtgr_status_t mtgr_embedding_evict(const mtgr_embedding_table_t* t, int32_t threshold, uint32_t min_count,
                                   int64_t* num_evicted, mtgr_stream_t stream) {
    mtgr::EmbArgs a;
    mtgr_status_t st = check_table(t, &a);
    if (st != MTGR_SUCCESS) return st;
    REQUIRE_PTR(num_evicted, "num_evicted");
    hipError_t e = mtgr::launch_emb_evict(a, threshold, min_count, (long long*)num_evicted, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "embedding evict");
    return ok();
}

mtgr_status_t mtgr_embedding_rehash(const mtgr_embedding_table_t* from, const mtgr_embedding_table_t* to,
                                    mtgr_stream_t stream) {
    mtgr::EmbArgs a, b;
    mtgr_status_t st = check_table(from, &a);
    if (st != MTGR_SUCCESS) return st;
    st = check_table(to, &b);
    if (st != MTGR_SUCCESS) return st;
    if (from->values != to->values || from->counts != to->counts || from->last_ts != to->last_ts ||
        from->free_rows != to->free_rows || from->state != to->state)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "from and to must share the value store and state");
    if (from->row_capacity != to->row_capacity || from->dim != to->dim || from->dtype != to->dtype)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "from and to differ in row_capacity, dim or dtype");
    if (from->keys == to->keys || from->key_rows == to->key_rows)
        return fail(MTGR_ERROR_INVALID_ARGUMENT, "to needs a key store of its own");
    hipError_t e = mtgr::launch_emb_rehash(a, b, (hipStream_t)stream);
    if (e != hipSuccess) return device_fail(e, "embedding rehash");
    return ok();
}

}  // extern "C"
