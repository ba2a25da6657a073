// Host side of libspecverify: argument validation, workspace sizing, launches and
// error reporting for the C ABI declared in specverify.h. Every check runs before any
// HIP call, so an invalid call enqueues nothing (and needs no GPU to be rejected).
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <cstdint>

#include "sv_internal.h"

namespace {

thread_local char g_err[512] = "";

sv_status fail(sv_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

// SV_FAULT_INJECT=launch makes the next launch report a HIP failure without enqueuing,
// so callers' error paths can be exercised from the host.
bool inject_launch_fault() {
    const char* e = std::getenv("SV_FAULT_INJECT");
    return e && std::strcmp(e, "launch") == 0;
}

sv_status launched(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(SV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    g_err[0] = '\0';
    return SV_OK;
}

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

// every pointer must be NULL or aligned to `a` bytes (16 for the arrays read with 16-byte
// vector loads or LDS DMA, 4 for the int32 / fp32 arrays)
bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

sv_status check_budget(const sv_budget_desc* d, const float* conf, const int32_t* keep,
                       const int32_t* qo, const int32_t* sel) {
    if (!d) return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: desc is NULL");
    if (d->num_reqs < 1 || d->num_reqs > SV_MAX_BUDGET_REQS)
        return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: num_reqs %d outside [1, %d]", d->num_reqs, SV_MAX_BUDGET_REQS);
    if (d->block < 1 || d->block > SV_MAX_BLOCK)
        return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: block %d outside [1, %d]", d->block, SV_MAX_BLOCK);
    const long long N = (long long)d->num_reqs * d->block;
    if (N > SV_MAX_BUDGET_POSITIONS)
        return fail(SV_ERR_UNSUPPORTED, "sv_alloc_budget: num_reqs*block = %lld above %d", N, SV_MAX_BUDGET_POSITIONS);
    if (!keep || !qo || !sel) return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: keep/qo_indptr/sel must not be NULL");
    if (d->block > 1 && !conf) return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: conf is NULL");
    if (!aligned(conf, 4) || !aligned(keep, 4) || !aligned(qo, 4) || !aligned(sel, 4))
        return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: arrays must be 4-byte aligned");
    if (d->mode == SV_BUDGET_FIXED) {
        if (d->fixed_budget < d->num_reqs || d->fixed_budget > N)
            return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: fixed_budget %d outside [R=%d, R*b=%lld]",
                        d->fixed_budget, d->num_reqs, N);
    } else if (d->mode == SV_BUDGET_COST) {
        if (d->num_ratios < 1 || d->num_ratios > SV_MAX_RATIOS)
            return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: num_ratios %d outside [1, %d]", d->num_ratios, SV_MAX_RATIOS);
        for (int j = 0; j < d->num_ratios; j++) {
            if (d->ratio_permille[j] < 1 || d->ratio_permille[j] > 1000)
                return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: ratio_permille[%d] = %d outside (0, 1000]", j,
                            d->ratio_permille[j]);
            if (j > 0 && d->ratio_permille[j] <= d->ratio_permille[j - 1])
                return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: ratios must be strictly ascending");
            if (d->cost[j] == 0) return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: cost[%d] is 0", j);
        }
    } else {
        return fail(SV_ERR_INVALID_ARG, "sv_alloc_budget: unknown mode %d", d->mode);
    }
    return SV_OK;
}

sv_status check_attn(const sv_attn_desc* d) {
    if (!d) return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: desc is NULL");
    if (d->num_reqs < 1 || d->num_reqs > 65535)
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: num_reqs %d outside [1, 65535]", d->num_reqs);
    if (d->max_kv_len > (1 << 22))
        return fail(SV_ERR_UNSUPPORTED, "sv_verify_attn: max_kv_len %d above 2^22", d->max_kv_len);
    if (d->block < 1 || d->block > SV_MAX_BLOCK)
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: block %d outside [1, %d]", d->block, SV_MAX_BLOCK);
    if (d->total_q_max < 1) return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: total_q_max %d < 1", d->total_q_max);
    // the packed batch holds at most block rows per request, and the fp32 path launches one
    // workgroup per (row, head): both products in 64 bits
    if ((long long)d->total_q_max > (long long)d->num_reqs * d->block)
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: total_q_max %d above num_reqs*block = %lld", d->total_q_max,
                    (long long)d->num_reqs * d->block);
    if (d->num_q_heads > 0 && (long long)d->total_q_max * d->num_q_heads > 0x7FFFFFFFLL)
        return fail(SV_ERR_UNSUPPORTED, "sv_verify_attn: total_q_max*num_q_heads = %lld above 2^31-1",
                    (long long)d->total_q_max * d->num_q_heads);
    if (d->num_q_heads < 1 || d->num_kv_heads < 1 || d->num_q_heads % d->num_kv_heads != 0)
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: num_q_heads %d is not a multiple of num_kv_heads %d",
                    d->num_q_heads, d->num_kv_heads);
    if (!is_pow2(d->page_size) || d->page_size > 4096)
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: page_size %d is not a power of two <= 4096", d->page_size);
    if (d->max_pages_per_req < 1 || d->num_pages < 1 || d->max_kv_len < 1)
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: max_pages_per_req, num_pages and max_kv_len must be >= 1");
    if ((long long)d->max_pages_per_req * d->page_size < d->max_kv_len)
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: max_pages_per_req*page_size < max_kv_len");
    if (!(d->sm_scale >= 0.0f) || std::isinf(d->sm_scale))
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: sm_scale must be finite and >= 0");
    if (d->kv_split < 0 || d->kv_split % 64 != 0)
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: kv_split %d is not a non-negative multiple of 64", d->kv_split);
    const int G = d->num_q_heads / d->num_kv_heads;
    if (d->dtype == SV_BF16) {
        if (d->head_dim != 64 && d->head_dim != 128)
            return fail(SV_ERR_UNSUPPORTED, "sv_verify_attn: bf16 head_dim %d (supported: 64, 128)", d->head_dim);
        if ((long long)G * d->block > 1024)
            return fail(SV_ERR_UNSUPPORTED, "sv_verify_attn: group size * block = %d above 1024", G * d->block);
    } else if (d->dtype == SV_F32) {
        if (d->head_dim < 4 || d->head_dim > 256 || d->head_dim % 4 != 0)
            return fail(SV_ERR_UNSUPPORTED, "sv_verify_attn: fp32 head_dim %d (supported: multiples of 4 up to 256)",
                        d->head_dim);
    } else {
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: unknown dtype %d", d->dtype);
    }
    return SV_OK;
}

sv_status check_accept(const sv_accept_desc* d) {
    if (!d) return fail(SV_ERR_INVALID_ARG, "sv_spec_accept: desc is NULL");
    if (d->num_reqs < 1) return fail(SV_ERR_INVALID_ARG, "sv_spec_accept: num_reqs %d < 1", d->num_reqs);
    if (d->block < 1 || d->block > SV_MAX_BLOCK)
        return fail(SV_ERR_INVALID_ARG, "sv_spec_accept: block %d outside [1, %d]", d->block, SV_MAX_BLOCK);
    if (d->vocab < 1 || d->vocab > SV_MAX_VOCAB)
        return fail(SV_ERR_INVALID_ARG, "sv_spec_accept: vocab %d outside [1, %d]", d->vocab, SV_MAX_VOCAB);
    if (d->dtype != SV_F32 && d->dtype != SV_BF16)
        return fail(SV_ERR_INVALID_ARG, "sv_spec_accept: unknown dtype %d", d->dtype);
    if (d->kind == SV_PROBS) {
        if (d->dtype != SV_F32) return fail(SV_ERR_UNSUPPORTED, "sv_spec_accept: probability rows must be fp32");
    } else if (d->kind != SV_LOGITS) {
        return fail(SV_ERR_INVALID_ARG, "sv_spec_accept: unknown kind %d", d->kind);
    }
    if (!(d->temperature >= 0.0f) || std::isinf(d->temperature))
        return fail(SV_ERR_INVALID_ARG,
                    "sv_spec_accept: temperature must be finite and >= 0 (0 selects greedy verification)");
    if ((long long)d->num_reqs * d->block > (1LL << 30))
        return fail(SV_ERR_UNSUPPORTED, "sv_spec_accept: too many rows");
    // each kernel is one flat grid: its work-item count must fit the 32-bit dispatch size
    const sv::AcceptPlan p = sv::plan_accept(*d);
    const long long slots = (long long)d->num_reqs * (2LL * d->block - 1);
    if (slots * p.stats_chunks * 256 > 0xFFFFFFFFLL || (long long)d->num_reqs * p.res_chunks * 256 > 0xFFFFFFFFLL)
        return fail(SV_ERR_UNSUPPORTED, "sv_spec_accept: %d requests x vocab %d exceed one launch", d->num_reqs,
                    d->vocab);
    return SV_OK;
}

}  // namespace

extern "C" {

sv_status sv_alloc_budget(const sv_budget_desc* desc, const float* conf, int32_t* keep,
                          int32_t* qo_indptr, int32_t* sel, float* scores, uint64_t* utility,
                          void* stream) {
    sv_status st = check_budget(desc, conf, keep, qo_indptr, sel);
    if (st != SV_OK) return st;
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "sv_alloc_budget: injected launch failure");
    return launched(sv::launch_budget(*desc, conf, keep, qo_indptr, sel, scores, utility, (hipStream_t)stream),
                    "sv_alloc_budget");
}

size_t sv_verify_attn_workspace_size(const sv_attn_desc* desc) {
    if (check_attn(desc) != SV_OK) return 0;
    return sv::plan_attn(*desc).ws_bytes;
}

sv_status sv_verify_attn(const sv_attn_desc* desc, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* page_table, const int32_t* qo_indptr,
                         const int32_t* kv_lens, void* out, float* lse, void* ws, size_t ws_bytes,
                         void* stream) {
    sv_status st = check_attn(desc);
    if (st != SV_OK) return st;
    if (!q || !k_cache || !v_cache || !page_table || !qo_indptr || !kv_lens || !out)
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn: a required pointer is NULL");
    if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16) || !aligned(ws, 16) ||
        !aligned(page_table, 4) || !aligned(qo_indptr, 4) || !aligned(kv_lens, 4) || !aligned(lse, 4))
        return fail(SV_ERR_INVALID_ARG,
                    "sv_verify_attn: q, caches, out and ws must be 16-byte aligned, int32/fp32 arrays 4-byte aligned");
    const sv::AttnPlan p = sv::plan_attn(*desc);
    const size_t need = p.ws_bytes;
    if (need && (!ws || ws_bytes < need))
        return fail(SV_ERR_WORKSPACE, "sv_verify_attn: workspace of %zu bytes needed, %zu given", need,
                    ws ? ws_bytes : (size_t)0);
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "sv_verify_attn: injected launch failure");
    return launched(sv::launch_attn(*desc, p, q, k_cache, v_cache, page_table, qo_indptr, kv_lens, out, lse, ws,
                                    (hipStream_t)stream),
                    "sv_verify_attn");
}

sv_status sv_pack_verify(const sv_pack_desc* desc, const int32_t* block_tokens, const int32_t* ctx_lens,
                         const int32_t* qo_indptr, int32_t* tokens, int32_t* positions, int32_t* kv_lens,
                         void* stream) {
    if (!desc) return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: desc is NULL");
    const sv_pack_desc& d = *desc;
    if (d.num_reqs < 1) return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: num_reqs %d < 1", d.num_reqs);
    if (d.block < 1 || d.block > SV_MAX_BLOCK)
        return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: block %d outside [1, %d]", d.block, SV_MAX_BLOCK);
    if (d.total_max < 1) return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: total_max %d < 1", d.total_max);
    if ((long long)d.num_reqs * d.block > (1LL << 31) - 256)
        return fail(SV_ERR_UNSUPPORTED, "sv_pack_verify: too many block positions");
    if (!block_tokens || !ctx_lens || !qo_indptr || !tokens || !positions || !kv_lens)
        return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: a required pointer is NULL");
    if (!aligned(block_tokens, 4) || !aligned(ctx_lens, 4) || !aligned(qo_indptr, 4) || !aligned(tokens, 4) ||
        !aligned(positions, 4) || !aligned(kv_lens, 4))
        return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: arrays must be 4-byte aligned");
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "sv_pack_verify: injected launch failure");
    return launched(sv::launch_pack(d, block_tokens, ctx_lens, qo_indptr, tokens, positions, kv_lens,
                                    (hipStream_t)stream),
                    "sv_pack_verify");
}

sv_status sv_append_kv(const sv_append_desc* desc, const void* k_new, const void* v_new,
                       const int32_t* page_table, const int32_t* qo_indptr, const int32_t* ctx_lens,
                       void* k_cache, void* v_cache, void* stream) {
    if (!desc) return fail(SV_ERR_INVALID_ARG, "sv_append_kv: desc is NULL");
    const sv_append_desc& d = *desc;
    if (d.num_reqs < 1 || d.num_reqs > 65535)
        return fail(SV_ERR_INVALID_ARG, "sv_append_kv: num_reqs %d outside [1, 65535]", d.num_reqs);
    if (d.block < 1 || d.block > SV_MAX_BLOCK)
        return fail(SV_ERR_INVALID_ARG, "sv_append_kv: block %d outside [1, %d]", d.block, SV_MAX_BLOCK);
    if (d.total_max < 1 || d.num_kv_heads < 1 || d.num_kv_heads > 65535 || d.max_pages_per_req < 1 ||
        d.num_pages < 1)
        return fail(SV_ERR_INVALID_ARG, "sv_append_kv: total_max, num_kv_heads, max_pages_per_req and num_pages "
                                        "must be >= 1");
    if (!is_pow2(d.page_size) || d.page_size > 4096)
        return fail(SV_ERR_INVALID_ARG, "sv_append_kv: page_size %d is not a power of two <= 4096", d.page_size);
    if (d.dtype != SV_F32 && d.dtype != SV_BF16) return fail(SV_ERR_INVALID_ARG, "sv_append_kv: unknown dtype %d", d.dtype);
    const long long row_bytes = (long long)d.head_dim * (d.dtype == SV_F32 ? 4 : 2);
    if (d.head_dim < 1 || row_bytes % 16 != 0 || row_bytes > (1 << 16))
        return fail(SV_ERR_UNSUPPORTED, "sv_append_kv: head_dim %d (the row must be a multiple of 16 bytes)",
                    d.head_dim);
    if ((long long)d.num_reqs * d.block > 0x7FFFFFFFLL)
        return fail(SV_ERR_UNSUPPORTED, "sv_append_kv: too many block positions");
    if (!k_new || !v_new || !page_table || !qo_indptr || !ctx_lens || !k_cache || !v_cache)
        return fail(SV_ERR_INVALID_ARG, "sv_append_kv: a required pointer is NULL");
    if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) ||
        !aligned(page_table, 4) || !aligned(qo_indptr, 4) || !aligned(ctx_lens, 4))
        return fail(SV_ERR_INVALID_ARG, "sv_append_kv: rows and caches must be 16-byte aligned, int32 arrays 4-byte "
                                        "aligned");
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "sv_append_kv: injected launch failure");
    return launched(sv::launch_append(d, k_new, v_new, page_table, qo_indptr, ctx_lens, k_cache, v_cache,
                                      (hipStream_t)stream),
                    "sv_append_kv");
}

size_t sv_spec_accept_workspace_size(const sv_accept_desc* desc) {
    if (check_accept(desc) != SV_OK) return 0;
    return sv::plan_accept(*desc).total;
}

}  // extern "C"

namespace {

// ---- the no-allocation acceptance entry point ---------------------------------------
// A fixed device array stands in for the caller's workspace. Each GPU holds its own copy
// (loaded with the code object, kept until the process ends). Its device address is
// looked up once per device with hipGetSymbolAddress, with that device current; host code
// never passes the array's own name to a kernel.
constexpr size_t kScratchBytes = size_t(16) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

// device address of `scratch` on the device that owns `stream` (NULL: the current device)
sv_status scratch_for_stream(hipStream_t stream, void** out) {
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return fail(SV_ERR_HIP, "sv_spec_accept_noalloc: hipGetDevice: %s", hipGetErrorString(e));
    int dev = cur;
    if (stream) {
        e = hipStreamGetDevice(stream, &dev);
        if (e != hipSuccess)
            return fail(SV_ERR_HIP, "sv_spec_accept_noalloc: hipStreamGetDevice: %s", hipGetErrorString(e));
    }
    if (dev < 0 || dev >= kMaxDevices)
        return fail(SV_ERR_UNSUPPORTED, "sv_spec_accept_noalloc: device %d above %d", dev, kMaxDevices - 1);
    void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p) {
        *out = p;
        return SV_OK;
    }
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess)
        return fail(SV_ERR_HIP, "sv_spec_accept_noalloc: hipSetDevice: %s", hipGetErrorString(e));
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) {
        const hipError_t e2 = hipSetDevice(cur);
        if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess || !p)
        return fail(SV_ERR_HIP, "sv_spec_accept_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch_ptr[dev].store(p, std::memory_order_release);  // racing first calls store the same address
    *out = p;
    return SV_OK;
}

sv_status spec_accept(const char* name, const sv_accept_desc* desc, const void* target, const void* draft,
                      const float* draft_stats, const int32_t* draft_tokens, const int32_t* qo_indptr,
                      const float* u_accept, const float* u_sample, int32_t* accept_len, int32_t* out_tokens,
                      int32_t* flags, void* ws, size_t ws_bytes, void* stream, bool use_scratch = false,
                      float* dbg_pq = nullptr, float* dbg_row = nullptr) {
    sv_status st = check_accept(desc);
    if (st != SV_OK) return st;
    if (use_scratch) {  // the fixed device array takes the workspace's place
        ws = nullptr;
        ws_bytes = kScratchBytes;
        if (sv::plan_accept(*desc).total > kScratchBytes)
            return fail(SV_ERR_UNSUPPORTED,
                        "%s: this shape needs %zu bytes of scratch, above the fixed %zu; use sv_spec_accept with a "
                        "workspace",
                        name, sv::plan_accept(*desc).total, kScratchBytes);
    }
    const bool has_drafts = desc->block > 1;
    const bool greedy = desc->temperature == 0.0f;  // reads neither draft rows nor uniforms
    if (!target || !qo_indptr || !accept_len || !out_tokens || (has_drafts && !draft_tokens) ||
        (!greedy && (!u_sample || (has_drafts && (!draft || !u_accept)))))
        return fail(SV_ERR_INVALID_ARG, "%s: a required pointer is NULL", name);
    if (!aligned(target, 16) || !aligned(draft, 16) || !aligned(ws, 16) || !aligned(draft_tokens, 4) ||
        !aligned(qo_indptr, 4) || !aligned(u_accept, 4) || !aligned(u_sample, 4) || !aligned(accept_len, 4) ||
        !aligned(out_tokens, 4) || !aligned(flags, 4) || !aligned(draft_stats, 8))
        return fail(SV_ERR_INVALID_ARG,
                    "%s: target, draft and ws must be 16-byte aligned, draft_stats 8-byte aligned, int32/fp32 "
                    "arrays 4-byte aligned",
                    name);
    const sv::AcceptPlan p = sv::plan_accept(*desc);
    if (use_scratch && (st = scratch_for_stream((hipStream_t)stream, &ws)) != SV_OK) return st;
    if (!ws || ws_bytes < p.total)
        return fail(SV_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", name, p.total,
                    ws ? ws_bytes : (size_t)0);
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "%s: injected launch failure", name);
    return launched(sv::launch_accept(*desc, p, target, draft, draft_stats, draft_tokens, qo_indptr, u_accept,
                                      u_sample, accept_len, out_tokens, flags, ws, (hipStream_t)stream, dbg_pq,
                                      dbg_row),
                    name);
}

sv_status check_draft_stats(const sv_draft_stats_desc* d) {
    if (!d) return fail(SV_ERR_INVALID_ARG, "sv_draft_stats: desc is NULL");
    if (d->num_reqs < 1 || d->drafts < 1)
        return fail(SV_ERR_INVALID_ARG, "sv_draft_stats: num_reqs %d and drafts %d must be >= 1", d->num_reqs,
                    d->drafts);
    if (d->vocab < 1 || d->vocab > SV_MAX_VOCAB)
        return fail(SV_ERR_INVALID_ARG, "sv_draft_stats: vocab %d outside [1, %d]", d->vocab, SV_MAX_VOCAB);
    if (d->dtype != SV_F32 && d->dtype != SV_BF16)
        return fail(SV_ERR_INVALID_ARG, "sv_draft_stats: unknown dtype %d", d->dtype);
    if (!(d->temperature > 0.0f) || std::isinf(d->temperature))
        return fail(SV_ERR_INVALID_ARG, "sv_draft_stats: temperature must be finite and > 0");
    const long long rows = (long long)d->num_reqs * d->drafts;
    const int chunk = 256 * 4 * (d->dtype == SV_BF16 ? 8 : 4);  // the statistics chunk of sv_spec_accept
    const long long nc = ((long long)d->vocab + chunk - 1) / chunk;
    if (rows > (1LL << 30) || rows * nc * 256 > 0xFFFFFFFFLL)
        return fail(SV_ERR_UNSUPPORTED, "sv_draft_stats: %lld rows x vocab %d exceed one launch", rows, d->vocab);
    return SV_OK;
}

}  // namespace

extern "C" {

sv_status sv_spec_accept(const sv_accept_desc* desc, const void* target, const void* draft,
                         const int32_t* draft_tokens, const int32_t* qo_indptr,
                         const float* u_accept, const float* u_sample, int32_t* accept_len,
                         int32_t* out_tokens, int32_t* flags, void* ws, size_t ws_bytes,
                         void* stream) {
    return spec_accept("sv_spec_accept", desc, target, draft, nullptr, draft_tokens, qo_indptr, u_accept, u_sample,
                       accept_len, out_tokens, flags, ws, ws_bytes, stream);
}

sv_status sv_spec_accept_noalloc(const sv_accept_desc* desc, const void* target, const void* draft,
                                 const int32_t* draft_tokens, const int32_t* qo_indptr, const float* u_accept,
                                 const float* u_sample, int32_t* accept_len, int32_t* out_tokens, int32_t* flags,
                                 void* stream) {
    return spec_accept("sv_spec_accept_noalloc", desc, target, draft, nullptr, draft_tokens, qo_indptr, u_accept,
                       u_sample, accept_len, out_tokens, flags, nullptr, 0, stream, true);
}

sv_status sv_spec_accept_debug(const sv_accept_desc* desc, const void* target, const void* draft,
                               const int32_t* draft_tokens, const int32_t* qo_indptr, const float* u_accept,
                               const float* u_sample, int32_t* accept_len, int32_t* out_tokens, int32_t* flags,
                               float* dbg_pq, float* dbg_row, void* ws, size_t ws_bytes, void* stream) {
    if (desc && (desc->kind != SV_LOGITS || !(desc->temperature > 0.0f)))
        return fail(SV_ERR_INVALID_ARG,
                    "sv_spec_accept_debug: the export covers rejection sampling of logits (LOGITS, temperature > 0)");
    if (!dbg_pq || !dbg_row || !aligned(dbg_pq, 4) || !aligned(dbg_row, 4))
        return fail(SV_ERR_INVALID_ARG, "sv_spec_accept_debug: dbg_pq and dbg_row must be 4-byte aligned device arrays");
    return spec_accept("sv_spec_accept_debug", desc, target, draft, nullptr, draft_tokens, qo_indptr, u_accept,
                       u_sample, accept_len, out_tokens, flags, ws, ws_bytes, stream, false, dbg_pq, dbg_row);
}

sv_status sv_spec_accept_stats(const sv_accept_desc* desc, const void* target, const void* draft,
                               const float* draft_stats, const int32_t* draft_tokens, const int32_t* qo_indptr,
                               const float* u_accept, const float* u_sample, int32_t* accept_len,
                               int32_t* out_tokens, int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
    if (desc && (desc->kind != SV_LOGITS || !(desc->temperature > 0.0f)))
        return fail(SV_ERR_INVALID_ARG,
                    "sv_spec_accept_stats: draft statistics apply to rejection sampling (LOGITS, temperature > 0)");
    if (desc && desc->block > 1 && !draft_stats)
        return fail(SV_ERR_INVALID_ARG, "sv_spec_accept_stats: draft_stats is NULL");
    return spec_accept("sv_spec_accept_stats", desc, target, draft, desc && desc->block > 1 ? draft_stats : nullptr,
                       draft_tokens, qo_indptr, u_accept, u_sample, accept_len, out_tokens, flags, ws, ws_bytes,
                       stream);
}

size_t sv_draft_stats_workspace_size(const sv_draft_stats_desc* desc) {
    if (check_draft_stats(desc) != SV_OK) return 0;
    return sv::draft_stats_workspace(*desc);
}

sv_status sv_draft_stats(const sv_draft_stats_desc* desc, const void* draft_logits, float* stats, float* conf,
                         void* ws, size_t ws_bytes, void* stream) {
    sv_status st = check_draft_stats(desc);
    if (st != SV_OK) return st;
    if (!draft_logits || !stats) return fail(SV_ERR_INVALID_ARG, "sv_draft_stats: a required pointer is NULL");
    if (!aligned(draft_logits, 16) || !aligned(stats, 8) || !aligned(conf, 4) || !aligned(ws, 16))
        return fail(SV_ERR_INVALID_ARG,
                    "sv_draft_stats: logits and ws must be 16-byte aligned, stats 8-byte, conf 4-byte aligned");
    const size_t need = sv::draft_stats_workspace(*desc);
    if (!ws || ws_bytes < need)
        return fail(SV_ERR_WORKSPACE, "sv_draft_stats: workspace of %zu bytes needed, %zu given", need,
                    ws ? ws_bytes : (size_t)0);
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "sv_draft_stats: injected launch failure");
    return launched(sv::launch_draft_stats(*desc, draft_logits, stats, conf, ws, (hipStream_t)stream),
                    "sv_draft_stats");
}

const char* sv_status_string(int32_t status) {
    switch (status) {
        case SV_OK: return "SV_OK";
        case SV_ERR_INVALID_ARG: return "SV_ERR_INVALID_ARG";
        case SV_ERR_UNSUPPORTED: return "SV_ERR_UNSUPPORTED";
        case SV_ERR_WORKSPACE: return "SV_ERR_WORKSPACE";
        case SV_ERR_HIP: return "SV_ERR_HIP";
        default: return "SV_UNKNOWN_STATUS";
    }
}

const char* sv_last_error(void) { return g_err; }

int32_t sv_abi_version(void) { return SV_ABI_VERSION; }

}  // extern "C"
