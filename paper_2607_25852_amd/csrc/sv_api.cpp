// Host side of libspecverify: argument validation, workspace sizing, launches and
// error reporting for the C ABI declared in specverify.h. Every check runs before any
// HIP call, so an invalid call enqueues nothing (and needs no GPU to be rejected).
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <cstdint>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "sv_internal.h"

namespace {

using sv::aligned;
using sv::fail;

// A roctx range around every compute entry point (checks and launches): under
// `rocprofv3 --marker-trace` each call shows on the host timeline next to its kernels.
struct CallRange {
    explicit CallRange(const char* name) { roctxRangePushA(name); }
    ~CallRange() { roctxRangePop(); }
    CallRange(const CallRange&) = delete;
    CallRange& operator=(const CallRange&) = delete;
};

// SV_FAULT_INJECT=launch makes the next launch report a HIP failure without enqueuing,
// so callers' error paths can be exercised from the host.
bool inject_launch_fault() {
    const char* e = std::getenv("SV_FAULT_INJECT");
    return e && std::strcmp(e, "launch") == 0;
}

sv_status launched(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(SV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    sv::clear_error();
    return SV_OK;
}

}  // namespace

namespace {

// sv_verify_attn and sv_verify_attn_run: the same checks; `phases` says whether the
// work plan is built here (kAttnAll) or taken from the workspace (kAttnRun)
sv_status verify_attn(const char* name, int phases, const sv_attn_desc* desc, const void* q, const void* k_cache,
                      const void* v_cache, const int32_t* page_table, const int32_t* qo_indptr,
                      const int32_t* kv_lens, void* out, float* lse, void* ws, size_t ws_bytes, void* stream) {
    sv_status st = sv::check_attn(desc);
    if (st != SV_OK) return st;
    if (!q || !k_cache || !v_cache || !page_table || !qo_indptr || !kv_lens || !out)
        return fail(SV_ERR_INVALID_ARG, "%s: a required pointer is NULL", name);
    if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(out, 16) || !aligned(ws, 16) ||
        !aligned(page_table, 4) || !aligned(qo_indptr, 4) || !aligned(kv_lens, 4) || !aligned(lse, 4))
        return fail(SV_ERR_INVALID_ARG,
                    "%s: q, caches, out and ws must be 16-byte aligned, int32/fp32 arrays 4-byte aligned", name);
    const sv::AttnPlan p = sv::plan_attn(*desc);
    const size_t need = p.ws_bytes;
    if (need && (!ws || ws_bytes < need))
        return fail(SV_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", name, need,
                    ws ? ws_bytes : (size_t)0);
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "%s: injected launch failure", name);
    return launched(sv::launch_attn(*desc, p, q, k_cache, v_cache, page_table, qo_indptr, kv_lens, out, lse, ws,
                                    (hipStream_t)stream, phases),
                    name);
}

}  // namespace

extern "C" {

sv_status sv_alloc_budget(const sv_budget_desc* desc, const float* conf, int32_t* keep,
                          int32_t* qo_indptr, int32_t* sel, float* scores, uint64_t* utility,
                          void* stream) {
    CallRange range("sv_alloc_budget");
    sv_status st = sv::check_budget(desc, conf, keep, qo_indptr, sel);
    if (st != SV_OK) return st;
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "sv_alloc_budget: injected launch failure");
    return launched(sv::launch_budget(*desc, conf, keep, qo_indptr, sel, scores, utility, (hipStream_t)stream),
                    "sv_alloc_budget");
}

size_t sv_verify_attn_workspace_size(const sv_attn_desc* desc) {
    if (sv::check_attn(desc) != SV_OK) return 0;
    return sv::plan_attn(*desc).ws_bytes;
}


sv_status sv_verify_attn(const sv_attn_desc* desc, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* page_table, const int32_t* qo_indptr,
                         const int32_t* kv_lens, void* out, float* lse, void* ws, size_t ws_bytes,
                         void* stream) {
    CallRange range("sv_verify_attn");
    return verify_attn("sv_verify_attn", sv::kAttnAll, desc, q, k_cache, v_cache, page_table, qo_indptr, kv_lens, out,
                       lse, ws, ws_bytes, stream);
}

sv_status sv_verify_attn_run(const sv_attn_desc* desc, const void* q, const void* k_cache,
                             const void* v_cache, const int32_t* page_table, const int32_t* qo_indptr,
                             const int32_t* kv_lens, void* out, float* lse, void* ws, size_t ws_bytes,
                             void* stream) {
    CallRange range("sv_verify_attn_run");
    return verify_attn("sv_verify_attn_run", sv::kAttnRun, desc, q, k_cache, v_cache, page_table, qo_indptr, kv_lens,
                       out, lse, ws, ws_bytes, stream);
}

sv_status sv_verify_attn_plan(const sv_attn_desc* desc, const int32_t* qo_indptr, const int32_t* kv_lens, void* ws,
                              size_t ws_bytes, void* stream) {
    CallRange range("sv_verify_attn_plan");
    sv_status st = sv::check_attn(desc);
    if (st != SV_OK) return st;
    if (!qo_indptr || !kv_lens) return fail(SV_ERR_INVALID_ARG, "sv_verify_attn_plan: a required pointer is NULL");
    if (!aligned(qo_indptr, 4) || !aligned(kv_lens, 4) || !aligned(ws, 16))
        return fail(SV_ERR_INVALID_ARG, "sv_verify_attn_plan: int32 arrays 4-byte aligned, ws 16-byte aligned");
    const sv::AttnPlan p = sv::plan_attn(*desc);
    if (p.ws_bytes && (!ws || ws_bytes < p.ws_bytes))
        return fail(SV_ERR_WORKSPACE, "sv_verify_attn_plan: workspace of %zu bytes needed, %zu given", p.ws_bytes,
                    ws ? ws_bytes : (size_t)0);
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "sv_verify_attn_plan: injected launch failure");
    return launched(sv::launch_attn(*desc, p, nullptr, nullptr, nullptr, nullptr, qo_indptr, kv_lens, nullptr, nullptr,
                                    ws, (hipStream_t)stream, sv::kAttnPlan),
                    "sv_verify_attn_plan");
}

sv_status sv_prepare_round(const sv_budget_desc* bdesc, const float* conf, int32_t* keep, int32_t* qo_indptr,
                           int32_t* sel, float* scores, uint64_t* utility, const sv_pack_desc* pdesc,
                           const int32_t* block_tokens, const int32_t* ctx_lens, int32_t* tokens, int32_t* positions,
                           int32_t* kv_lens, const sv_attn_desc* adesc, void* attn_ws, size_t attn_ws_bytes,
                           void* stream) {
    CallRange range("sv_prepare_round");
    sv_status st = sv::check_budget(bdesc, conf, keep, qo_indptr, sel);
    if (st != SV_OK) return st;
    if ((st = sv::check_pack(pdesc)) != SV_OK) return st;
    if (pdesc->num_reqs != bdesc->num_reqs || pdesc->block != bdesc->block)
        return fail(SV_ERR_INVALID_ARG, "sv_prepare_round: the packing's num_reqs/block (%d, %d) differ from the "
                                        "budget's (%d, %d)",
                    pdesc->num_reqs, pdesc->block, bdesc->num_reqs, bdesc->block);
    if (!block_tokens || !ctx_lens || !tokens || !positions || !kv_lens)
        return fail(SV_ERR_INVALID_ARG, "sv_prepare_round: a required pointer is NULL");
    if (!aligned(block_tokens, 4) || !aligned(ctx_lens, 4) || !aligned(tokens, 4) || !aligned(positions, 4) ||
        !aligned(kv_lens, 4) || !aligned(attn_ws, 16))
        return fail(SV_ERR_INVALID_ARG, "sv_prepare_round: int32 arrays 4-byte aligned, attn_ws 16-byte aligned");
    if (adesc) {
        if ((st = sv::check_attn(adesc)) != SV_OK) return st;
        if (adesc->num_reqs != bdesc->num_reqs || adesc->block != bdesc->block)
            return fail(SV_ERR_INVALID_ARG, "sv_prepare_round: the attention's num_reqs/block (%d, %d) differ from "
                                            "the budget's (%d, %d)",
                        adesc->num_reqs, adesc->block, bdesc->num_reqs, bdesc->block);
        const size_t need = sv::plan_attn(*adesc).ws_bytes;
        if (need && (!attn_ws || attn_ws_bytes < need))
            return fail(SV_ERR_WORKSPACE, "sv_prepare_round: attention workspace of %zu bytes needed, %zu given",
                        need, attn_ws ? attn_ws_bytes : (size_t)0);
    }
    if (inject_launch_fault()) return fail(SV_ERR_HIP, "sv_prepare_round: injected launch failure");
    return launched(sv::launch_prepare(*bdesc, conf, keep, qo_indptr, sel, scores, utility, block_tokens, ctx_lens,
                                       tokens, positions, kv_lens, pdesc->total_max, adesc, attn_ws,
                                       (hipStream_t)stream),
                    "sv_prepare_round");
}

sv_status sv_pack_verify(const sv_pack_desc* desc, const int32_t* block_tokens, const int32_t* ctx_lens,
                         const int32_t* qo_indptr, int32_t* tokens, int32_t* positions, int32_t* kv_lens,
                         void* stream) {
    CallRange range("sv_pack_verify");
    sv_status st = sv::check_pack(desc);
    if (st != SV_OK) return st;
    const sv_pack_desc& d = *desc;
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
    CallRange range("sv_append_kv");
    sv_status st = sv::check_append(desc);
    if (st != SV_OK) return st;
    const sv_append_desc& d = *desc;
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
    if (sv::check_accept(desc) != SV_OK) return 0;
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
    sv_status st = sv::check_accept(desc);
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

}  // namespace

extern "C" {

sv_status sv_spec_accept(const sv_accept_desc* desc, const void* target, const void* draft,
                         const int32_t* draft_tokens, const int32_t* qo_indptr,
                         const float* u_accept, const float* u_sample, int32_t* accept_len,
                         int32_t* out_tokens, int32_t* flags, void* ws, size_t ws_bytes,
                         void* stream) {
    CallRange range("sv_spec_accept");
    return spec_accept("sv_spec_accept", desc, target, draft, nullptr, draft_tokens, qo_indptr, u_accept, u_sample,
                       accept_len, out_tokens, flags, ws, ws_bytes, stream);
}

sv_status sv_spec_accept_noalloc(const sv_accept_desc* desc, const void* target, const void* draft,
                                 const int32_t* draft_tokens, const int32_t* qo_indptr, const float* u_accept,
                                 const float* u_sample, int32_t* accept_len, int32_t* out_tokens, int32_t* flags,
                                 void* stream) {
    CallRange range("sv_spec_accept_noalloc");
    return spec_accept("sv_spec_accept_noalloc", desc, target, draft, nullptr, draft_tokens, qo_indptr, u_accept,
                       u_sample, accept_len, out_tokens, flags, nullptr, 0, stream, true);
}

sv_status sv_spec_accept_debug(const sv_accept_desc* desc, const void* target, const void* draft,
                               const int32_t* draft_tokens, const int32_t* qo_indptr, const float* u_accept,
                               const float* u_sample, int32_t* accept_len, int32_t* out_tokens, int32_t* flags,
                               float* dbg_pq, float* dbg_row, void* ws, size_t ws_bytes, void* stream) {
    CallRange range("sv_spec_accept_debug");
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
    CallRange range("sv_spec_accept_stats");
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
    if (sv::check_draft_stats(desc) != SV_OK) return 0;
    return sv::draft_stats_workspace(*desc);
}

sv_status sv_draft_stats(const sv_draft_stats_desc* desc, const void* draft_logits, float* stats, float* conf,
                         void* ws, size_t ws_bytes, void* stream) {
    CallRange range("sv_draft_stats");
    sv_status st = sv::check_draft_stats(desc);
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

const char* sv_last_error(void) { return sv::last_error(); }

int32_t sv_abi_version(void) { return SV_ABI_VERSION; }

}  // extern "C"
