// D-cut verification budget on one workgroup (AngelSpec Sec. 4.2).
//
// All R*b candidate positions fit in LDS (<= 8192). Each becomes a 64-bit key whose
// order is the selection order: fp32 score bits in the high word (scores are >= +0,
// so their bit patterns order like the values), then the depth inverted (shallower
// first on equal scores), then the request index inverted (lower request first).
// A bitonic sort in LDS ranks every key; the top K_j for every candidate ratio are
// then prefixes of the sorted order, so utilities, the ratio choice and the keep
// counts need no second selection.
#include "sv_internal.h"

#pragma clang fp contract(off)

namespace sv {
namespace {

constexpr int kThreads = 1024;
constexpr int kMaxKeys = SV_MAX_BUDGET_POSITIONS;
constexpr int kMaxReqs = SV_MAX_BUDGET_REQS;

struct BudgetArgs {
    int R, b, mode, fixed_K, nratios;
    int Kr[SV_MAX_RATIOS];      // K_j per ratio (computed on the host from the descriptor)
    uint32_t cost[SV_MAX_RATIOS];
};

__device__ inline float clamp_conf(float c) {
    if (!(c > 0.0f)) return 0.0f;  // NaN, negatives, -0
    return c > 1.0f ? 1.0f : c;
}

// floor(s * 2^40) for s in [0, 1]: exact (power-of-two scaling, fp64 holds it)
__device__ inline uint64_t score_fixed(float s) { return (uint64_t)((double)s * 1099511627776.0); }

__device__ inline uint64_t wave_sum_u64(uint64_t v) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__global__ __launch_bounds__(kThreads) void budget_kernel(BudgetArgs a, const float* __restrict__ conf,
                                                          int32_t* __restrict__ keep,
                                                          int32_t* __restrict__ qo_indptr,
                                                          int32_t* __restrict__ sel,
                                                          float* __restrict__ scores_out,
                                                          uint64_t* __restrict__ util_out) {
    __shared__ uint64_t keys[kMaxKeys];
    __shared__ int cnt[kMaxReqs];
    __shared__ uint64_t red[kThreads / 64][SV_MAX_RATIOS];
    __shared__ int s_K;
    __shared__ int scan_tmp[kThreads / 64];

    const int tid = threadIdx.x;
    const int R = a.R, b = a.b, N = R * b;
    int Npad = 2;
    while (Npad < N) Npad <<= 1;

    // 1. prefix scores, one request per thread, left to right in fp32 (eq. dcut-score)
    for (int i = tid; i < R; i += kThreads) {
        float s = 1.0f;
        for (int t = 0; t < b; t++) {
            if (t > 0) s = s * clamp_conf(conf[(size_t)i * (b - 1) + (t - 1)]);
            if (scores_out) scores_out[(size_t)i * b + t] = s;
            keys[i * b + t] = ((uint64_t)__float_as_uint(s) << 32) |
                              ((uint64_t)(0xFFFFu - (unsigned)t) << 16) | (uint64_t)(0xFFFFu - (unsigned)i);
        }
        cnt[i] = 0;
    }
    for (int p = N + tid; p < Npad; p += kThreads) keys[p] = 0;  // below every real key
    __syncthreads();

    // 2. bitonic sort, descending
    for (int k = 2; k <= Npad; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int p = tid; p < Npad; p += kThreads) {
                const int q = p ^ j;
                if (q > p) {
                    const uint64_t x = keys[p], y = keys[q];
                    const bool desc = (p & k) == 0;
                    if (desc ? (x < y) : (x > y)) {
                        keys[p] = y;
                        keys[q] = x;
                    }
                }
            }
            __syncthreads();
        }
    }

    // 3. utilities of every ratio: sums over prefixes of the sorted order
    const int nr = a.mode == SV_BUDGET_COST ? a.nratios : 1;
    uint64_t u[SV_MAX_RATIOS];
    for (int j = 0; j < SV_MAX_RATIOS; j++) u[j] = 0;
    for (int p = tid; p < N; p += kThreads) {
        const uint64_t f = score_fixed(__uint_as_float((uint32_t)(keys[p] >> 32)));
        for (int j = 0; j < nr; j++) {
            const int Kj = a.mode == SV_BUDGET_COST ? a.Kr[j] : a.fixed_K;
            if (p < Kj) u[j] += f;
        }
    }
    const int lane = tid & 63, wave = tid >> 6;
    for (int j = 0; j < nr; j++) {
        const uint64_t w = wave_sum_u64(u[j]);
        if (lane == 0) red[wave][j] = w;
    }
    __syncthreads();

    // 4. ratio choice (eq. dcut-select), exact cross-multiplication, ties -> smaller ratio
    if (tid == 0) {
        uint64_t U[SV_MAX_RATIOS];
        for (int j = 0; j < nr; j++) {
            uint64_t s = 0;
            for (int w = 0; w < kThreads / 64; w++) s += red[w][j];
            U[j] = s;
            if (util_out) util_out[j] = s;
        }
        int best = -1, K = a.fixed_K;
        if (a.mode == SV_BUDGET_COST) {
            best = 0;
            for (int j = 1; j < nr; j++) {
                const unsigned __int128 lhs = (unsigned __int128)U[j] * a.cost[best];
                const unsigned __int128 rhs = (unsigned __int128)U[best] * a.cost[j];
                if (lhs > rhs) best = j;
            }
            K = a.Kr[best];
        }
        s_K = K;
        sel[0] = K;
        sel[1] = best;
    }
    __syncthreads();

    // 5. kept positions per request: the first K keys of the sorted order
    const int K = s_K;
    for (int p = tid; p < K; p += kThreads) {
        const int i = 0xFFFF - (int)(keys[p] & 0xFFFFu);
        atomicAdd(&cnt[i], 1);
    }
    __syncthreads();

    // 6. keep = count - 1; qo_indptr = exclusive scan of the counts (block scan)
    constexpr int kPer = kMaxReqs / kThreads;  // 4 requests per thread
    int loc[kPer];
    int run = 0;
    for (int e = 0; e < kPer; e++) {
        const int i = tid * kPer + e;
        loc[e] = i < R ? cnt[i] : 0;
        run += loc[e];
    }
    // inclusive wave scan of run
    int incl = run;
    for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off, 64);
        if (lane >= off) incl += v;
    }
    if (lane == 63) scan_tmp[wave] = incl;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; w++) base += scan_tmp[w];
    int pos = base + incl - run;
    for (int e = 0; e < kPer; e++) {
        const int i = tid * kPer + e;
        if (i < R) {
            keep[i] = loc[e] - 1;
            qo_indptr[i] = pos;
        }
        pos += loc[e];
    }
    if (tid == kThreads - 1) qo_indptr[R] = pos;  // == K
}

}  // namespace

hipError_t launch_budget(const sv_budget_desc& d, const float* conf, int32_t* keep,
                         int32_t* qo_indptr, int32_t* sel, float* scores, uint64_t* utility,
                         hipStream_t stream) {
    BudgetArgs a{};
    a.R = d.num_reqs;
    a.b = d.block;
    a.mode = d.mode;
    a.fixed_K = d.fixed_budget;
    a.nratios = d.mode == SV_BUDGET_COST ? d.num_ratios : 0;
    const int64_t N = (int64_t)d.num_reqs * d.block;
    for (int j = 0; j < a.nratios; j++) {
        // eq. dcut-budget: K_j = max(R, ceil(rho_j * R * b)), rho_j = permille / 1000
        int64_t Kj = ((int64_t)d.ratio_permille[j] * N + 999) / 1000;
        if (Kj < d.num_reqs) Kj = d.num_reqs;
        if (Kj > N) Kj = N;
        a.Kr[j] = (int)Kj;
        a.cost[j] = d.cost[j];
    }
    hipLaunchKernelGGL(budget_kernel, dim3(1), dim3(kThreads), 0, stream, a, conf, keep, qo_indptr, sel,
                       scores, utility);
    return hipGetLastError();
}

}  // namespace sv
