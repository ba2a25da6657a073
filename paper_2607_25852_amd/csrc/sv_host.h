// Host-side declarations of libspecverify that need no GPU runtime: argument checks,
// workspace layouts (and the acceptance layout constants the kernels share), the
// thread-local error message. Not part of the public ABI.
#pragma once
#include <cstddef>
#include <cstdint>

#include "specverify.h"

namespace sv {

// ---- acceptance layout, shared by accept.hip and the workspace plan ---------------
namespace acc {
constexpr int kThreads = 256;                       // threads of every acceptance workgroup
constexpr int kStatsLoads = 4;                      // 16-byte loads in flight per thread (16 KB chunks)
constexpr int kResChunk = 8192;                     // vocabulary chunk of the residual sums
constexpr int kResPer = kResChunk / kThreads;       // tokens per thread in a residual chunk
constexpr size_t kTsumMaxBytes = size_t(64) << 20;  // cap of the per-thread partial sums
constexpr int kCntStride = 32;                      // uint32 per request's arrival counter (a 128-byte line)

struct ReqPlan {
    int a, n, mode, flag;  // mode 0: residual after a rejection, 1: bonus, 2: nothing to draw
    int rowP, rowQ;        // target row of P_a (or P_n), draft row of Q_{a+1}
    float mP, iSP, mQ, iSQ;
};
}  // namespace acc

// ---- workspace layouts --------------------------------------------------------------
struct AttnPlan {
    int kv_split;     // tokens per split-KV work item (multiple of 64)
    int max_splits;   // ceil(max_kv_len / kv_split)
    int waves;        // waves per workgroup (bf16 path)
    int halves;       // 2: a wave owns a 32-token half of each tile, 1: the whole tile
    int row_blocks;   // query-row blocks of (waves / halves) * 32 rows per (request, kv-head)
    size_t part_o_bytes;    // split partial outputs (fp32), offset 0
    size_t part_lse_bytes;  // split partial log-sum-exps, after part_o
    size_t off_groups;      // work list of the persistent kernel
    size_t off_ctr;         // {number of work items, work counter, finished workgroups}
    size_t ws_bytes;        // total workspace (0 for the fp32 path)
};
struct AcceptPlan {
    int stats_chunk;   // vocabulary elements per row-statistics workgroup
    int stats_chunks;  // chunks per row
    int res_chunk;     // vocabulary elements per residual workgroup
    int res_chunks;
    size_t off_cnt, off_stats_t, off_stats_q, off_plan, off_csum, off_tsum, total;  // off_tsum 0: none
};
AttnPlan plan_attn(const sv_attn_desc& d);
AcceptPlan plan_accept(const sv_accept_desc& d);
size_t draft_stats_workspace(const sv_draft_stats_desc& d);

// ---- argument checks: SV_OK, or a status with the reason in last_error() ----------
sv_status fail(sv_status st, const char* fmt, ...);
void clear_error();
const char* last_error();
bool aligned(const void* p, size_t a);  // NULL counts as aligned
sv_status check_budget(const sv_budget_desc* d, const float* conf, const int32_t* keep, const int32_t* qo,
                       const int32_t* sel);
sv_status check_attn(const sv_attn_desc* d);
sv_status check_accept(const sv_accept_desc* d);
sv_status check_pack(const sv_pack_desc* d);
sv_status check_append(const sv_append_desc* d);
sv_status check_draft_stats(const sv_draft_stats_desc* d);

}  // namespace sv
