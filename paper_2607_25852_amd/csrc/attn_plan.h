// Work list of the persistent verify-attention kernel, built by one workgroup. Every
// (request, split) group is bucketed by its tile count: full splits share the top bucket,
// a request's shorter last split lands in the bucket of its own length. The buckets are
// laid out in decreasing size (a counting sort), so the persistent workgroups take the
// long items early and the short ones fill the tail. The order inside a bucket is
// unspecified and does not affect any result: every item writes its own output rows or
// partial slot. Used by the attention call's own plan kernel and by the round set-up
// kernel (sv_prepare_round), so both build the same list.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace sv {

constexpr int kAttnTile = 64;         // KV tokens per tile of the attention kernel
constexpr int kPlanBuckets = 1024;    // tile counts 1..1024; longer splits share the last

struct AttnPlanArgs {
    int R, block, total_q, max_kv_len, split, Hkv, nrb;
    int32_t* groups;  // [R * max_splits] request << 16 | split
    int32_t* ctr;     // {work items, work counter, finished workgroups}
};

// splits of request i (0 when its packing is malformed) and the tile count of its last one
__device__ inline int plan_splits(const AttnPlanArgs& a, int q0, int k_i, int kv_len, int& last_tiles) {
    if (kv_len > a.max_kv_len) kv_len = a.max_kv_len;
    last_tiles = 0;
    if (!(k_i >= 1 && k_i <= a.block && kv_len - k_i >= 0 && q0 >= 0 && q0 + k_i <= a.total_q)) return 0;
    const int ns = (kv_len + a.split - 1) / a.split;
    last_tiles = (kv_len - (ns - 1) * a.split + kAttnTile - 1) / kAttnTile;
    return ns;
}

// NT threads of one workgroup (NT a multiple of 64 dividing kPlanBuckets); cursor:
// kPlanBuckets ints of LDS, wsum: NT / 64 ints of LDS. req(i, q0, k_i, kv_len) gives
// request i's packing and key count. Ends with a barrier-free store of the counters; the
// caller's kernel end publishes the list.
template <int NT, typename ReqFn>
__device__ inline void build_attn_plan(const AttnPlanArgs& a, ReqFn req, int* cursor, int* wsum) {
    static_assert(NT % 64 == 0 && kPlanBuckets % NT == 0, "plan threads");
    constexpr int BPT = kPlanBuckets / NT;  // buckets per thread in the scan
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int full_tiles = a.split / kAttnTile;
    auto bucket = [](int tiles) { return tiles < kPlanBuckets ? tiles - 1 : kPlanBuckets - 1; };
    const int fb = bucket(full_tiles);
    for (int k = tid; k < kPlanBuckets; k += NT) cursor[k] = 0;
    __syncthreads();
    // 1. histogram of group sizes (full splits summed per wave first: one shared bucket)
    for (int base = 0; base < a.R; base += NT) {
        const int i = base + tid;
        int last = 0, ns = 0;
        if (i < a.R) {
            int q0, k_i, kv;
            req(i, q0, k_i, kv);
            ns = plan_splits(a, q0, k_i, kv, last);
        }
        int full = ns > 1 ? ns - 1 : 0;
        for (int off = 32; off > 0; off >>= 1) full += __shfl_xor(full, off, 64);
        if (lane == 0 && full) atomicAdd(&cursor[fb], full);
        if (ns > 0) atomicAdd(&cursor[bucket(last)], 1);
    }
    __syncthreads();
    // 2. bucket starts in decreasing size: thread t scans positions t*BPT .. t*BPT+BPT-1 of
    //    the descending bucket order (bucket kPlanBuckets-1-position)
    int cnt[BPT];
    int loc = 0;
#pragma unroll
    for (int e = 0; e < BPT; e++) {
        cnt[e] = cursor[kPlanBuckets - 1 - (tid * BPT + e)];
        loc += cnt[e];
    }
    int incl = loc;
    for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off, 64);
        if (lane >= off) incl += v;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int pre = 0;
    for (int k = 0; k < w; k++) pre += wsum[k];
    int pos = pre + incl - loc;
#pragma unroll
    for (int e = 0; e < BPT; e++) {
        cursor[kPlanBuckets - 1 - (tid * BPT + e)] = pos;
        pos += cnt[e];
    }
    if (tid == NT - 1) {
        a.ctr[0] = pos * a.Hkv * a.nrb;
        a.ctr[1] = 0;
        a.ctr[2] = 0;
    }
    __syncthreads();
    // 3. place the groups (full splits: one atomic per wave, positions by a wave scan)
    for (int base = 0; base < a.R; base += NT) {
        const int i = base + tid;
        int last = 0, ns = 0;
        if (i < a.R) {
            int q0, k_i, kv;
            req(i, q0, k_i, kv);
            ns = plan_splits(a, q0, k_i, kv, last);
        }
        const int full = ns > 1 ? ns - 1 : 0;
        int fincl = full;
        for (int off = 1; off < 64; off <<= 1) {
            const int v = __shfl_up(fincl, off, 64);
            if (lane >= off) fincl += v;
        }
        int fbase = 0;
        if (lane == 63 && fincl) fbase = atomicAdd(&cursor[fb], fincl);
        fbase = __shfl(fbase, 63, 64);
        const int p0 = fbase + fincl - full;
        for (int t = 0; t < full; t++) a.groups[p0 + t] = (int32_t)(((uint32_t)i << 16) | (uint32_t)t);
        if (ns > 0) a.groups[atomicAdd(&cursor[bucket(last)], 1)] = (int32_t)(((uint32_t)i << 16) | (uint32_t)(ns - 1));
    }
}

}  // namespace sv
