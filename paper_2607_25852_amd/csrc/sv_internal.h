// Internal declarations shared by the host API and the kernel translation units of
// libspecverify. Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "specverify.h"

namespace sv {

// ---- budget -------------------------------------------------------------------
hipError_t launch_budget(const sv_budget_desc& d, const float* conf, int32_t* keep,
                         int32_t* qo_indptr, int32_t* sel, float* scores, uint64_t* utility,
                         hipStream_t stream);

// ---- verify attention -----------------------------------------------------------
struct AttnPlan {
    int kv_split;     // tokens per split-KV work item (multiple of 64)
    int max_splits;   // ceil(max_kv_len / kv_split)
    int waves;        // waves per workgroup (bf16 path)
    int halves;       // 2: a wave owns a 32-token half of each tile, 1: the whole tile
    int row_blocks;   // query-row blocks of (waves / halves) * 32 rows per (request, kv-head)
    size_t part_o_bytes;    // split partial outputs (fp32), offset 0
    size_t part_lse_bytes;  // split partial log-sum-exps, after part_o
    size_t off_groups;      // work list of the persistent kernel
    size_t off_ctr;         // {number of work items, work counter}
    size_t ws_bytes;        // total workspace (0 for the fp32 path)
};
AttnPlan plan_attn(const sv_attn_desc& d);
hipError_t launch_attn(const sv_attn_desc& d, const AttnPlan& plan, const void* q,
                       const void* k_cache, const void* v_cache, const int32_t* page_table,
                       const int32_t* qo_indptr, const int32_t* kv_lens, void* out, float* lse,
                       void* ws, hipStream_t stream);

// ---- acceptance -----------------------------------------------------------------
struct AcceptPlan {
    int stats_chunk;   // vocabulary elements per row-statistics workgroup
    int stats_chunks;  // chunks per row
    int res_chunk;     // vocabulary elements per residual workgroup
    int res_chunks;
    size_t off_cnt, off_stats_t, off_stats_q, off_plan, off_csum, off_tsum, total;  // off_tsum 0: none
};
AcceptPlan plan_accept(const sv_accept_desc& d);
hipError_t launch_accept(const sv_accept_desc& d, const AcceptPlan& plan, const void* target,
                         const void* draft, const float* draft_stats, const int32_t* draft_tokens,
                         const int32_t* qo_indptr, const float* u_accept, const float* u_sample,
                         int32_t* accept_len, int32_t* out_tokens, int32_t* flags, void* ws,
                         hipStream_t stream, float* dbg_pq = nullptr, float* dbg_row = nullptr);
size_t draft_stats_workspace(const sv_draft_stats_desc& d);
hipError_t launch_draft_stats(const sv_draft_stats_desc& d, const void* logits, float* stats, float* conf, void* ws,
                              hipStream_t stream);

hipError_t launch_pack(const sv_pack_desc& d, const int32_t* block_tokens, const int32_t* ctx_lens,
                       const int32_t* qo_indptr, int32_t* tokens, int32_t* positions, int32_t* kv_lens,
                       hipStream_t stream);
hipError_t launch_append(const sv_append_desc& d, const void* k_new, const void* v_new, const int32_t* page_table,
                         const int32_t* qo_indptr, const int32_t* ctx_lens, void* k_cache, void* v_cache,
                         hipStream_t stream);

}  // namespace sv
