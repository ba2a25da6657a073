// D-cut verification budget on one workgroup (AngelSpec Sec. 4.2).
//
// All R*b candidate positions (<= 8192) become 64-bit keys whose order is the selection
// order: fp32 score bits in the high word (scores are >= +0, so their bit patterns order
// like the values), then the depth inverted (shallower first on equal scores), then the
// request index inverted (lower request first). A bitonic sort ranks every key (held in
// registers; only strides of 64 threads or more go through LDS); the top K_j of every
// candidate ratio are then prefixes of the sorted order, so one prefix sum gives every
// utility, and the keep counts need no second selection.
#include "attn_plan.h"
#include "sv_internal.h"

#pragma clang fp contract(off)

namespace sv {
namespace {

constexpr int kThreads = 512;  // the workgroup of large rounds
constexpr int kWave = 64;      // the workgroup of small rounds: one wave
constexpr int kSmallMax = 128; // small rounds: R*b <= 128 (up to two keys per lane)
constexpr int kMaxKeys = SV_MAX_BUDGET_POSITIONS;
constexpr int kMaxReqs = SV_MAX_BUDGET_REQS;

struct BudgetArgs {
    int R, b, mode, fixed_K, nratios;
    int Kr[SV_MAX_RATIOS];      // K_j per ratio (computed on the host from the descriptor)
    uint32_t cost[SV_MAX_RATIOS];
};

// The rest of the round's set-up, run by the same workgroup after the budget
// (sv_prepare_round): the dense verify batch of the kept prefixes (sv_pack_verify's
// arithmetic) and, when `plan` is set, the verify-attention work plan over the key counts
// the packing produced (attn_plan.h).
struct PrepArgs {
    const int32_t* block_tokens;  // [R, b]
    const int32_t* ctx;           // [R]
    int32_t* tokens;              // [total_max]
    int32_t* positions;           // [total_max]
    int32_t* kv_lens;             // [R]
    int total_max;
    int plan;
    AttnPlanArgs pa;
};

__device__ inline float clamp_conf(float c) {
    if (!(c > 0.0f)) return 0.0f;  // NaN, negatives, -0
    return c > 1.0f ? 1.0f : c;
}

// floor(s * 2^40) for s in [0, 1]: exact (power-of-two scaling, fp64 holds it)
__device__ inline uint64_t score_fixed(float s) { return (uint64_t)((double)s * 1099511627776.0); }

// compare-exchange of a bitonic stage seen from element p holding x with partner value y
// (partner index p ^ j); k is the size of the bitonic blocks being merged. The final
// order is descending.
__device__ inline uint64_t cmpx(uint64_t x, uint64_t y, int p, int j, int k) {
    const bool desc = (p & k) == 0;
    const bool lower = (p & j) == 0;
    const bool keep_max = desc == lower;
    return keep_max ? (x > y ? x : y) : (x < y ? x : y);
}

__device__ inline uint64_t shfl_xor_u64(uint64_t v, int m) {
    const uint32_t lo = __shfl_xor((uint32_t)v, m, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m, 64);
    return ((uint64_t)hi << 32) | lo;
}

__device__ inline uint64_t shfl_up_u64(uint64_t v, int d) {
    const uint32_t lo = __shfl_up((uint32_t)v, d, 64);
    const uint32_t hi = __shfl_up((uint32_t)(v >> 32), d, 64);
    return ((uint64_t)hi << 32) | lo;
}

// NT threads, KPT keys per thread: thread t owns sorted positions t*KPT .. t*KPT+KPT-1.
// Bitonic stages with stride < KPT run in registers, < 64*KPT across lanes of a wave, the
// rest through LDS (ping-pong buffers, one barrier per stage). Small rounds run on one
// wave (NT = 64, at most 128 keys), where every stage stays in registers and shuffles
// and the barriers are a single wave's. (At 256 keys the one-wave form's sort is still
// faster, but its attention plan, 1024 buckets over 64 threads, costs more than that.)
template <int NT, int KPT, bool PREP>
__global__ __launch_bounds__(NT) void budget_kernel(BudgetArgs a, const float* __restrict__ conf,
                                                          int32_t* __restrict__ keep,
                                                          int32_t* __restrict__ qo_indptr,
                                                          int32_t* __restrict__ sel,
                                                          float* __restrict__ scores_out,
                                                          uint64_t* __restrict__ util_out, PrepArgs pr) {
    static_assert(NT == kThreads || (NT == kWave && KPT * NT <= kSmallMax), "budget workgroup");
    constexpr int NPAD = KPT * NT;
    // requests: up to kMaxReqs (large rounds) or kSmallMax (one wave); with PREP the
    // one-wave form keeps the attention plan's bucket cursors after them
    constexpr int NCNT = NT == kThreads ? kMaxReqs : kSmallMax + kPlanBuckets;
    __shared__ uint64_t lds[2][NPAD];
    __shared__ int cnt[NCNT];
    __shared__ uint64_t wtot[NT / 64];
    __shared__ uint64_t s_util[SV_MAX_RATIOS];
    __shared__ int s_K;
    __shared__ int scan_tmp[NT / 64];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int R = a.R, b = a.b, N = R * b;

    // 1. prefix scores, one request per thread, left to right in fp32 (eq. dcut-score);
    //    the confidences are first staged through LDS with coalesced loads (buffer 1 of
    //    the key storage is free until the first LDS stage of the sort)
    float* cst = (float*)&lds[1][0];
    for (int e = tid; e < R * (b - 1); e += NT) cst[e] = conf[e];
    __syncthreads();
    for (int i = tid; i < R; i += NT) {
        float s = 1.0f;
        for (int t = 0; t < b; t++) {
            if (t > 0) s = s * clamp_conf(cst[i * (b - 1) + (t - 1)]);
            if (scores_out) scores_out[(size_t)i * b + t] = s;
            lds[0][i * b + t] = ((uint64_t)__float_as_uint(s) << 32) |
                                ((uint64_t)(0xFFFFu - (unsigned)t) << 16) | (uint64_t)(0xFFFFu - (unsigned)i);
        }
        cnt[i] = 0;
    }
    for (int p = N + tid; p < NPAD; p += NT) lds[0][p] = 0;  // below every real key
    __syncthreads();
    uint64_t x[KPT];
#pragma unroll
    for (int e = 0; e < KPT; e++) x[e] = lds[0][tid * KPT + e];

    // 2. bitonic sort, descending, of NPAD keys
    int buf = 1;
#pragma unroll
    for (int k = 2; k <= NPAD; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            if (j < KPT) {
#pragma unroll
                for (int e = 0; e < KPT; e++) {
                    const int p = tid * KPT + e;
                    if ((e & j) == 0) {
                        const uint64_t y0 = x[e], y1 = x[e | j];
                        x[e] = cmpx(y0, y1, p, j, k);
                        x[e | j] = cmpx(y1, y0, p | j, j, k);
                    }
                }
            } else if (j < 64 * KPT) {
                const int m = j / KPT;
#pragma unroll
                for (int e = 0; e < KPT; e++) x[e] = cmpx(x[e], shfl_xor_u64(x[e], m), tid * KPT + e, j, k);
            } else {
#pragma unroll
                for (int e = 0; e < KPT; e++) lds[buf][tid * KPT + e] = x[e];
                __syncthreads();
#pragma unroll
                for (int e = 0; e < KPT; e++) {
                    const int p = tid * KPT + e;
                    x[e] = cmpx(x[e], lds[buf][p ^ j], p, j, k);
                }
                buf ^= 1;
            }
        }
    }

    // 3. inclusive prefix sums of the fixed-point scores in sorted order; the utility of
    //    budget K is the prefix at position K-1 (eq. dcut-batch-utility)
    uint64_t f[KPT], run = 0;
#pragma unroll
    for (int e = 0; e < KPT; e++) {
        run += score_fixed(__uint_as_float((uint32_t)(x[e] >> 32)));
        f[e] = run;
    }
    uint64_t incl = run;
    for (int d = 1; d < 64; d <<= 1) {
        const uint64_t v = shfl_up_u64(incl, d);
        if (lane >= d) incl += v;
    }
    if (lane == 63) wtot[wave] = incl;
    __syncthreads();
    uint64_t base = incl - run;
    for (int w = 0; w < wave; w++) base += wtot[w];
    const int nr = a.mode == SV_BUDGET_COST ? a.nratios : 1;
    for (int jr = 0; jr < nr; jr++) {
        const int Kj = a.mode == SV_BUDGET_COST ? a.Kr[jr] : a.fixed_K;
        const int q = Kj - 1 - tid * KPT;
        if (q >= 0 && q < KPT) s_util[jr] = base + f[q];
    }
    __syncthreads();

    // 4. ratio choice (eq. dcut-select), exact cross-multiplication, ties -> smaller ratio
    if (tid == 0) {
        int best = -1, K = a.fixed_K;
        if (a.mode == SV_BUDGET_COST) {
            best = 0;
            for (int jr = 1; jr < nr; jr++) {
                const unsigned __int128 lhs = (unsigned __int128)s_util[jr] * a.cost[best];
                const unsigned __int128 rhs = (unsigned __int128)s_util[best] * a.cost[jr];
                if (lhs > rhs) best = jr;
            }
            K = a.Kr[best];
        }
        if (util_out)
            for (int jr = 0; jr < nr; jr++) util_out[jr] = s_util[jr];
        s_K = K;
        sel[0] = K;
        sel[1] = best;
    }
    __syncthreads();

    // 5. kept positions per request: the first K keys of the sorted order
    const int K = s_K;
#pragma unroll
    for (int e = 0; e < KPT; e++)
        if (tid * KPT + e < K) atomicAdd(&cnt[0xFFFF - (int)(x[e] & 0xFFFFu)], 1);
    __syncthreads();

    // 6. keep = count - 1; qo_indptr = exclusive scan of the counts (block scan)
    constexpr int kPer = (NT == kThreads ? kMaxReqs : kSmallMax) / NT;  // requests per thread: 8 or 2
    int loc[kPer];
    int rsum = 0;
    for (int e = 0; e < kPer; e++) {
        const int i = tid * kPer + e;
        loc[e] = i < R ? cnt[i] : 0;
        rsum += loc[e];
    }
    int iscan = rsum;
    for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(iscan, off, 64);
        if (lane >= off) iscan += v;
    }
    if (lane == 63) scan_tmp[wave] = iscan;
    __syncthreads();
    int pos = iscan - rsum;
    for (int w = 0; w < wave; w++) pos += scan_tmp[w];
    // (with PREP the packing offsets also go to LDS, in the key buffers the sort is done with)
    int* qs = (int*)&lds[0][0];
    for (int e = 0; e < kPer; e++) {
        const int i = tid * kPer + e;
        if (i < R) {
            keep[i] = loc[e] - 1;
            qo_indptr[i] = pos;
            if (PREP) qs[i] = pos;
        }
        pos += loc[e];
    }
    if (tid == NT - 1) {
        qo_indptr[R] = pos;  // == K
        if (PREP) qs[R] = pos;
    }
    if constexpr (PREP) {
        __syncthreads();
        // 7. the verify batch (sv_pack_verify): row qo[i] + j carries block token j of request
        //    i at position L_i + j, and kv_lens[i] = L_i + k_i; every load is issued first
        int tk[KPT], Lc[KPT];
#pragma unroll
        for (int e = 0; e < KPT; e++) {
            const int p = tid + e * NT;
            tk[e] = p < N ? pr.block_tokens[p] : 0;
            Lc[e] = p < N ? pr.ctx[p / b] : 0;
        }
        int* kvs = cnt;  // key counts for the plan (the counts are no longer needed)
#pragma unroll
        for (int e = 0; e < KPT; e++) {
            const int p = tid + e * NT;
            if (p >= N) continue;
            const int i = p / b, j = p - i * b;
            const int q0 = qs[i], k_i = qs[i + 1] - q0;
            const int L = Lc[e];
            const bool ok = k_i >= 1 && k_i <= b && q0 >= 0 && q0 + k_i <= pr.total_max;
            if (j == 0) {
                pr.kv_lens[i] = ok ? L + k_i : L;
                kvs[i] = ok ? L + k_i : L;
            }
            if (ok && j < k_i) {
                pr.tokens[q0 + j] = tk[e];
                pr.positions[q0 + j] = L + j;
            }
        }
        if (!pr.plan) return;
        __syncthreads();
        // 8. the verify-attention work plan over those key counts
        int* cursor = NT == kThreads ? qs + ((R + 1 + 63) & ~63) : cnt + kSmallMax;
        build_attn_plan<NT>(pr.pa, [&](int i, int& q0, int& k_i, int& kv) {
            q0 = qs[i];
            k_i = qs[i + 1] - q0;
            kv = kvs[i];
        }, cursor, scan_tmp);
    }
}

}  // namespace

namespace {

BudgetArgs budget_args(const sv_budget_desc& d) {
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
    return a;
}

template <bool PREP>
hipError_t launch_budget_kernel(const sv_budget_desc& d, const float* conf, int32_t* keep, int32_t* qo_indptr,
                                int32_t* sel, float* scores, uint64_t* utility, const PrepArgs& pr,
                                hipStream_t stream) {
    const BudgetArgs a = budget_args(d);
    const int64_t N = (int64_t)d.num_reqs * d.block;
#define SV_LAUNCH_BUDGET(T, KP) \
    hipLaunchKernelGGL((budget_kernel<T, KP, PREP>), dim3(1), dim3(T), 0, stream, a, conf, keep, qo_indptr, sel, \
                       scores, utility, pr)
    if (N <= kSmallMax) {  // (R <= N)
        if (N <= kWave) SV_LAUNCH_BUDGET(kWave, 1);
        else SV_LAUNCH_BUDGET(kWave, 2);
    } else {
        const int64_t kpt = (N + kThreads - 1) / kThreads;
        if (kpt <= 1) SV_LAUNCH_BUDGET(kThreads, 1);
        else if (kpt <= 2) SV_LAUNCH_BUDGET(kThreads, 2);
        else if (kpt <= 4) SV_LAUNCH_BUDGET(kThreads, 4);
        else if (kpt <= 8) SV_LAUNCH_BUDGET(kThreads, 8);
        else SV_LAUNCH_BUDGET(kThreads, 16);
    }
#undef SV_LAUNCH_BUDGET
    return hipGetLastError();
}

}  // namespace

hipError_t launch_budget(const sv_budget_desc& d, const float* conf, int32_t* keep,
                         int32_t* qo_indptr, int32_t* sel, float* scores, uint64_t* utility,
                         hipStream_t stream) {
    return launch_budget_kernel<false>(d, conf, keep, qo_indptr, sel, scores, utility, PrepArgs{}, stream);
}

hipError_t launch_prepare(const sv_budget_desc& d, const float* conf, int32_t* keep, int32_t* qo_indptr,
                          int32_t* sel, float* scores, uint64_t* utility, const int32_t* block_tokens,
                          const int32_t* ctx_lens, int32_t* tokens, int32_t* positions, int32_t* kv_lens,
                          int total_max, const sv_attn_desc* ad, void* attn_ws, hipStream_t stream) {
    PrepArgs pr{};
    pr.block_tokens = block_tokens;
    pr.ctx = ctx_lens;
    pr.tokens = tokens;
    pr.positions = positions;
    pr.kv_lens = kv_lens;
    pr.total_max = total_max;
    if (ad && ad->dtype == SV_BF16) {  // the fp32 path has no work plan
        const AttnPlan p = plan_attn(*ad);
        pr.plan = 1;
        pr.pa = AttnPlanArgs{ad->num_reqs, ad->block, ad->total_q_max, ad->max_kv_len, p.kv_split, ad->num_kv_heads,
                             p.row_blocks, (int32_t*)((char*)attn_ws + p.off_groups),
                             (int32_t*)((char*)attn_ws + p.off_ctr)};
    }
    return launch_budget_kernel<true>(d, conf, keep, qo_indptr, sel, scores, utility, pr, stream);
}

}  // namespace sv
