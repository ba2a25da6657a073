// Host-side logic of libspecverify that needs no GPU runtime: the argument checks every
// entry point runs before it enqueues anything, the workspace layouts, and the
// thread-local error message. The library links it; the sanitizer test also builds it on
// its own with g++ under AddressSanitizer and UndefinedBehaviorSanitizer.
#include "sv_host.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>

namespace sv {

namespace {
thread_local char g_err[512] = "";
}  // namespace

const char* last_error() { return g_err; }
void clear_error() { g_err[0] = '\0'; }

sv_status fail(sv_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

static bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

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
            return fail(SV_ERR_UNSUPPORTED, "sv_verify_attn: group size * block = %lld above 1024", (long long)G * d->block);
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

sv_status check_pack(const sv_pack_desc* desc) {
    if (!desc) return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: desc is NULL");
    const sv_pack_desc& d = *desc;
    if (d.num_reqs < 1) return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: num_reqs %d < 1", d.num_reqs);
    if (d.block < 1 || d.block > SV_MAX_BLOCK)
        return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: block %d outside [1, %d]", d.block, SV_MAX_BLOCK);
    if (d.total_max < 1) return fail(SV_ERR_INVALID_ARG, "sv_pack_verify: total_max %d < 1", d.total_max);
    if ((long long)d.num_reqs * d.block > (1LL << 31) - 256)
        return fail(SV_ERR_UNSUPPORTED, "sv_pack_verify: too many block positions");
    return SV_OK;
}

sv_status check_append(const sv_append_desc* desc) {
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
    return SV_OK;
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
    const int chunk = acc::kThreads * acc::kStatsLoads * (d->dtype == SV_BF16 ? 8 : 4);  // the statistics chunk
    const long long nc = ((long long)d->vocab + chunk - 1) / chunk;
    if (rows > (1LL << 30) || rows * nc * 256 > 0xFFFFFFFFLL)
        return fail(SV_ERR_UNSUPPORTED, "sv_draft_stats: %lld rows x vocab %d exceed one launch", rows, d->vocab);
    return SV_OK;
}

// ---- workspace layouts ----------------------------------------------------------

AttnPlan plan_attn(const sv_attn_desc& d) {
    AttnPlan p{};
    const int maxM = (d.num_q_heads / d.num_kv_heads) * d.block;
    // 8 waves. Up to 128 query rows per kv-head group: a wave owns (32-row group, 32-token
    // half of each tile), so 64 rows already keep all four SIMDs busy. Above 128 rows a
    // wave owns 32 rows over the whole tile (256 rows per workgroup), so a group of up to
    // 256 rows streams its KV once.
    p.waves = 8;
    p.halves = maxM > 128 ? 1 : 2;
    const int rows = (p.waves / p.halves) * 32;
    p.row_blocks = (maxM + rows - 1) / rows;
    if (d.dtype == SV_F32) {
        p.kv_split = 0;
        p.max_splits = 1;
        return p;
    }
    int split = d.kv_split;
    if (split <= 0) {
        // About 8 work items per compute unit if every request had the longest context:
        // R * Hkv * max_kv_len head-tokens over 256 CUs, divided by 8, at least 2048
        // tokens. Measured over split sizes 1024..24576, this picks the best or nearly the
        // best one on c64_b16 (8192), long_c32 (8192), the C5 c64 sweep (16384) and the
        // small rounds (2048 at 4..16 requests): fewer, longer items save per-item
        // prologues and merge work until the last items to finish start to dominate, and
        // below 2048 tokens the per-item costs outweigh the extra parallelism. The host
        // does not see the lengths themselves (they live on the device), so the bound
        // uses max_kv_len.
        long long want = (long long)d.num_reqs * d.num_kv_heads * d.max_kv_len / (256 * 8);
        if (want < 2048) want = 2048;
        split = (int)(((want + 63) / 64) * 64);
    }
    if (split > d.max_kv_len) split = ((d.max_kv_len + 63) / 64) * 64;
    // a split's page ids are staged in LDS: at most 1024 pages per split (a split of
    // n tokens starting on a 64-token boundary touches at most n / P + 2 pages)
    const long long max_split = 1022LL * d.page_size;
    if (split > max_split) split = (int)(max_split / 64 * 64);
    if (split < 64) split = 64;
    p.kv_split = split;
    p.max_splits = (d.max_kv_len + split - 1) / split;
    if (p.max_splits < 1) p.max_splits = 1;
    if (p.max_splits > 1) {
        p.part_o_bytes = (size_t)p.max_splits * d.total_q_max * d.num_q_heads * d.head_dim * sizeof(float);
        p.part_lse_bytes = (size_t)p.max_splits * d.total_q_max * d.num_q_heads * sizeof(float);
    }
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    p.off_groups = al(p.part_o_bytes + p.part_lse_bytes);
    p.off_ctr = al(p.off_groups + (size_t)d.num_reqs * p.max_splits * sizeof(int32_t));
    p.ws_bytes = p.off_ctr + 3 * sizeof(int32_t);  // work items, work counter, finished workgroups
    return p;
}

AcceptPlan plan_accept(const sv_accept_desc& d) {
    AcceptPlan p{};
    const int esz = d.dtype == SV_BF16 ? 2 : 4;
    const int vec = 16 / esz;
    p.stats_chunk = acc::kThreads * acc::kStatsLoads * vec;  // 16 KB of logits per workgroup
    p.stats_chunks = (d.vocab + p.stats_chunk - 1) / p.stats_chunk;
    p.res_chunk = acc::kResChunk;
    p.res_chunks = (d.vocab + p.res_chunk - 1) / p.res_chunk;
    const size_t R = d.num_reqs, b = d.block, D = b > 1 ? b - 1 : 1;
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    size_t off = 0;
    p.off_cnt = off;
    off = al(off + R * acc::kCntStride * sizeof(uint32_t));
    p.off_stats_t = off;
    off = al(off + R * b * p.stats_chunks * 2 * sizeof(float));
    p.off_stats_q = off;
    off = al(off + R * D * p.stats_chunks * 2 * sizeof(float));
    p.off_plan = off;
    off = al(off + R * sizeof(acc::ReqPlan));
    p.off_csum = off;
    off = al(off + R * p.res_chunks * 2 * sizeof(uint64_t));
    const size_t tsum_bytes = R * p.res_chunks * acc::kThreads * sizeof(uint64_t);
    p.off_tsum = tsum_bytes <= acc::kTsumMaxBytes ? off : 0;
    if (p.off_tsum) off = al(off + tsum_bytes);
    p.total = off;
    return p;
}

size_t draft_stats_workspace(const sv_draft_stats_desc& d) {
    const int esz = d.dtype == SV_BF16 ? 2 : 4;
    const int chunk = acc::kThreads * acc::kStatsLoads * (16 / esz);
    const size_t nc = ((size_t)d.vocab + chunk - 1) / chunk;
    return (size_t)d.num_reqs * d.drafts * nc * 2 * sizeof(float);
}

}  // namespace sv
