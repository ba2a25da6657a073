// Drives the library's host-side checks and workspace layouts (sv_host.cpp) over edge and
// seeded random descriptors, for the sanitizer test: built with g++ under
// AddressSanitizer and UndefinedBehaviorSanitizer (no recovery), any out-of-bounds access,
// signed overflow or other undefined behaviour aborts the run. Accepted descriptors must
// also give consistent workspace layouts; rejected ones must leave a reason.
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "sv_host.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next_u64() {  // splitmix64
    uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

const int kEdges[] = {INT_MIN, -65536, -1, 0, 1, 2, 3, 4, 5, 7, 8, 15, 16, 17, 31, 32, 63, 64, 65, 100, 127, 128,
                      129, 255, 256, 1000, 1001, 1023, 1024, 1025, 2048, 4095, 4096, 4097, 8191, 8192, 8193, 32768,
                      65535, 65536, 131072, (1 << 22) - 1, 1 << 22, (1 << 22) + 1, 1 << 30, INT_MAX - 1, INT_MAX};
constexpr int kNumEdges = sizeof(kEdges) / sizeof(kEdges[0]);

int pick() {
    const uint64_t r = next_u64();
    if (r % 3 == 0) return kEdges[(r >> 8) % kNumEdges];
    if (r % 3 == 1) return (int)((r >> 8) % 70000) - 100;
    return (int)(uint32_t)(r >> 16);
}

long g_accepted = 0, g_rejected = 0;

void expect(bool ok, const char* what) {
    if (!ok) {
        std::fprintf(stderr, "FAILED: %s\n", what);
        std::exit(2);
    }
}

void count(sv_status st) {
    if (st == SV_OK) {
        g_accepted++;
    } else {
        g_rejected++;
        expect(sv::last_error()[0] != '\0', "a rejected call leaves a reason");
        sv::clear_error();
    }
}

bool aligned256(size_t x) { return x % 256 == 0; }

void check_attn_layout(const sv_attn_desc& d) {
    const sv::AttnPlan p = sv::plan_attn(d);
    if (d.dtype == SV_F32) return;
    expect(p.kv_split >= 64 && p.kv_split % 64 == 0, "attention split is a positive multiple of 64");
    expect(p.max_splits >= 1, "at least one split");
    expect((long long)p.max_splits * p.kv_split >= d.max_kv_len, "splits cover the longest context");
    expect(p.off_groups >= p.part_o_bytes + p.part_lse_bytes && aligned256(p.off_groups), "work list after partials");
    expect(p.off_ctr >= p.off_groups + (size_t)d.num_reqs * p.max_splits * 4 && aligned256(p.off_ctr),
           "counter after the work list");
    expect(p.ws_bytes >= p.off_ctr + 8, "workspace holds the counters");
}

void check_accept_layout(const sv_accept_desc& d) {
    const sv::AcceptPlan p = sv::plan_accept(d);
    expect(p.stats_chunk > 0 && (long long)p.stats_chunks * p.stats_chunk >= d.vocab, "statistics chunks cover V");
    expect(p.res_chunk > 0 && (long long)p.res_chunks * p.res_chunk >= d.vocab, "residual chunks cover V");
    const size_t R = (size_t)d.num_reqs;
    expect(p.off_cnt == 0, "counters first");
    expect(p.off_stats_t >= R * sv::acc::kCntStride * 4 && aligned256(p.off_stats_t), "target statistics");
    expect(p.off_stats_q >= p.off_stats_t + R * d.block * p.stats_chunks * 8 && aligned256(p.off_stats_q),
           "draft statistics");
    expect(p.off_plan > p.off_stats_q && aligned256(p.off_plan), "plans");
    expect(p.off_csum >= p.off_plan + R * sizeof(sv::acc::ReqPlan) && aligned256(p.off_csum), "chunk sums");
    expect(p.total >= p.off_csum + R * p.res_chunks * 16, "total");
    if (p.off_tsum) expect(p.total >= p.off_tsum + R * p.res_chunks * sv::acc::kThreads * 8, "partial sums");
}

}  // namespace

int main() {
    // budget
    for (int it = 0; it < 20000; it++) {
        sv_budget_desc d{};
        d.num_reqs = pick();
        d.block = pick();
        d.mode = (int)(next_u64() % 3);
        d.fixed_budget = pick();
        d.num_ratios = (int)(next_u64() % 10) - 1;
        for (int j = 0; j < SV_MAX_RATIOS; j++) {
            d.ratio_permille[j] = it % 2 ? 250 * (j + 1) : pick();
            d.cost[j] = (uint32_t)pick();
        }
        static float conf[4];
        static int32_t keep[4], qo[4], sel[4];
        count(sv::check_budget(&d, conf, keep, qo, sel));
        count(sv::check_budget(&d, nullptr, keep, qo, sel));
    }
    count(sv::check_budget(nullptr, nullptr, nullptr, nullptr, nullptr));
    // attention
    for (int it = 0; it < 200000; it++) {
        sv_attn_desc d{};
        d.num_reqs = pick();
        d.total_q_max = pick();
        d.block = pick();
        d.num_q_heads = pick();
        d.num_kv_heads = it % 4 ? (int)(next_u64() % 16) + 1 : pick();
        d.head_dim = it % 3 ? 128 : pick();
        d.page_size = it % 3 ? 64 : pick();
        d.max_pages_per_req = pick();
        d.num_pages = pick();
        d.max_kv_len = pick();
        d.dtype = it % 5 == 0 ? (int)(next_u64() % 4) - 1 : (int)(next_u64() % 2);
        d.sm_scale = it % 7 == 0 ? NAN : (it % 11 == 0 ? INFINITY : 0.0f);
        d.kv_split = it % 2 ? 0 : pick();
        if (it % 2) {  // a valid shape with one field replaced
            int f[12] = {64, 1024, 16, 64, 8, 128, 64, 1 << 12, 1 << 18, 1 << 18, SV_BF16, 0};
            f[next_u64() % 12] = pick();
            d.num_reqs = f[0]; d.total_q_max = f[1]; d.block = f[2]; d.num_q_heads = f[3]; d.num_kv_heads = f[4];
            d.head_dim = f[5]; d.page_size = f[6]; d.max_pages_per_req = f[7]; d.num_pages = f[8];
            d.max_kv_len = f[9]; d.dtype = f[10]; d.kv_split = f[11]; d.sm_scale = 0.0f;
        }
        const sv_status st = sv::check_attn(&d);
        count(st);
        if (st == SV_OK) check_attn_layout(d);
    }
    // a realistic shape, and its edges
    {
        sv_attn_desc d{};
        d.num_reqs = 64; d.total_q_max = 1024; d.block = 16; d.num_q_heads = 64; d.num_kv_heads = 8;
        d.head_dim = 128; d.page_size = 64; d.max_pages_per_req = 1 << 16; d.num_pages = 1 << 20;
        d.max_kv_len = 1 << 22; d.dtype = SV_BF16; d.sm_scale = 0.0f; d.kv_split = 0;
        expect(sv::check_attn(&d) == SV_OK, "c64_b16-like attention accepted");
        check_attn_layout(d);
    }
    count(sv::check_attn(nullptr));
    // acceptance
    for (int it = 0; it < 200000; it++) {
        sv_accept_desc d{};
        d.num_reqs = pick();
        d.block = pick();
        d.vocab = pick();
        d.kind = it % 5 == 0 ? pick() : (int)(next_u64() % 2);
        d.dtype = it % 5 == 1 ? pick() : (int)(next_u64() % 2);
        const uint64_t r = next_u64() % 8;
        d.temperature = r == 0 ? NAN : r == 1 ? -1.0f : r == 2 ? INFINITY : r == 3 ? 0.0f : (float)(r - 3) * 0.5f;
        if (it % 2) {  // a valid shape with one field replaced
            int f[5] = {64, 16, 131072, SV_LOGITS, SV_BF16};
            f[next_u64() % 5] = pick();
            d.num_reqs = f[0]; d.block = f[1]; d.vocab = f[2]; d.kind = f[3]; d.dtype = f[4]; d.temperature = 1.0f;
        }
        const sv_status st = sv::check_accept(&d);
        count(st);
        if (st == SV_OK) check_accept_layout(d);
    }
    count(sv::check_accept(nullptr));
    // packing, append, drafter statistics
    for (int it = 0; it < 100000; it++) {
        sv_pack_desc p{};
        p.num_reqs = pick();
        p.block = pick();
        p.total_max = pick();
        count(sv::check_pack(&p));
        sv_append_desc a{};
        a.num_reqs = pick();
        a.block = pick();
        a.total_max = pick();
        a.num_kv_heads = pick();
        a.head_dim = pick();
        a.page_size = pick();
        a.max_pages_per_req = pick();
        a.num_pages = pick();
        a.dtype = (int)(next_u64() % 3);
        count(sv::check_append(&a));
        sv_draft_stats_desc s{};
        s.num_reqs = pick();
        s.drafts = pick();
        s.vocab = pick();
        s.dtype = (int)(next_u64() % 3);
        s.temperature = it % 3 ? 1.0f : (float)pick();
        const sv_status st = sv::check_draft_stats(&s);
        count(st);
        if (st == SV_OK) expect(sv::draft_stats_workspace(s) > 0, "drafter statistics workspace");
    }
    count(sv::check_pack(nullptr));
    count(sv::check_append(nullptr));
    count(sv::check_draft_stats(nullptr));
    std::printf("ok: %ld accepted, %ld rejected\n", g_accepted, g_rejected);
    return 0;
}
