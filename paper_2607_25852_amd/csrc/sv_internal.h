// Internal declarations shared by the host API and the kernel translation units of
// libspecverify: the launch functions (the GPU-free host logic is in sv_host.h). Not
// part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "specverify.h"
#include "sv_host.h"

namespace sv {

// ---- budget -------------------------------------------------------------------
hipError_t launch_budget(const sv_budget_desc& d, const float* conf, int32_t* keep,
                         int32_t* qo_indptr, int32_t* sel, float* scores, uint64_t* utility,
                         hipStream_t stream);
// the budget, the verify batch of the kept prefixes and (ad: bf16 attention) the
// verify-attention work plan in attn_ws, by one workgroup (sv_prepare_round)
hipError_t launch_prepare(const sv_budget_desc& d, const float* conf, int32_t* keep, int32_t* qo_indptr,
                          int32_t* sel, float* scores, uint64_t* utility, const int32_t* block_tokens,
                          const int32_t* ctx_lens, int32_t* tokens, int32_t* positions, int32_t* kv_lens,
                          int total_max, const sv_attn_desc* ad, void* attn_ws, hipStream_t stream);

// ---- verify attention -----------------------------------------------------------
// what launch_attn runs: the work plan, the attention (and the merge of split partials), or both
enum AttnPhases { kAttnPlan = 1, kAttnRun = 2, kAttnAll = 3 };
hipError_t launch_attn(const sv_attn_desc& d, const AttnPlan& plan, const void* q,
                       const void* k_cache, const void* v_cache, const int32_t* page_table,
                       const int32_t* qo_indptr, const int32_t* kv_lens, void* out, float* lse,
                       void* ws, hipStream_t stream, int phases = kAttnAll);

// ---- acceptance -----------------------------------------------------------------
hipError_t launch_accept(const sv_accept_desc& d, const AcceptPlan& plan, const void* target,
                         const void* draft, const float* draft_stats, const int32_t* draft_tokens,
                         const int32_t* qo_indptr, const float* u_accept, const float* u_sample,
                         int32_t* accept_len, int32_t* out_tokens, int32_t* flags, void* ws,
                         hipStream_t stream, float* dbg_pq = nullptr, float* dbg_row = nullptr);
hipError_t launch_draft_stats(const sv_draft_stats_desc& d, const void* logits, float* stats, float* conf, void* ws,
                              hipStream_t stream);

hipError_t launch_pack(const sv_pack_desc& d, const int32_t* block_tokens, const int32_t* ctx_lens,
                       const int32_t* qo_indptr, int32_t* tokens, int32_t* positions, int32_t* kv_lens,
                       hipStream_t stream);
hipError_t launch_append(const sv_append_desc& d, const void* k_new, const void* v_new, const int32_t* page_table,
                         const int32_t* qo_indptr, const int32_t* ctx_lens, void* k_cache, void* v_cache,
                         hipStream_t stream);

}  // namespace sv
