// Speculative acceptance (rejection-sampling verification, AngelSpec Sec. 1; per-position
// acceptance probability min(1, p/q) whose expectation is the overlap of eq.
// mtp-acceptance-tv).
//
// Logits mode, two kernels on one stream, neither of which waits for another workgroup:
//   rowstats  streams every needed row once -- the n_i+1 target rows and n_i draft rows
//             of each request -- and writes per-chunk (max, sum of exponentials). This
//             is the HBM-bound pass.
//   draw      per (request, vocabulary chunk). Its first wave takes the request's
//             decision (decide_req): it merges the chunk statistics, evaluates the
//             acceptance test of every draft in its own lane (exact fp64 product
//             u*q < p) and finds the first rejection with a ballot; the chunk-0
//             workgroup writes the accepted prefix. Every workgroup of a request
//             computes the same decision from the same data, so none waits for another.
//             The workgroup then sums the integer weights floor(r * 2^40) of the
//             residual max(p - q, 0) (or of p for the bonus) over its chunk, stores the
//             sum device-coherently and counts itself on the request's arrival counter;
//             the last chunk workgroup of the request finds the token: Z, the threshold
//             floor(m * Z / 2^24), the chunk holding it and the exact token inside it.
// The arrival counters need no clearing launch: the statistics pass zeroes them.
// Probability mode has no statistics pass: the chunk-sum kernel takes the decision and
// sums the chunk, and a separate search kernel draws the token.
// Every sum that decides a token is an integer sum, so the result does not depend on
// how the vocabulary is split across threads.
#include "sv_internal.h"

#pragma clang fp contract(off)

namespace sv {
namespace {

using namespace acc;  // kThreads, kStatsLoads, kResChunk, kResPer, kCntStride, ReqPlan

constexpr float kLog2e = 1.4426950408889634f;

struct AcceptArgs {
    const void* target;
    const void* draft;
    const int32_t* tokens;
    const int32_t* qo;
    const float* ua;
    const float* us;
    int32_t* accept_len;
    int32_t* out_tokens;
    int32_t* flags;
    const float2* dstats;  // [R*D] (max, sum) of the draft rows from the drafter, or NULL
    float2* stats_t;  // [R*b][NC]
    float2* stats_q;  // [R*D][NC]
    ReqPlan* plan;    // [R]
    uint64_t* csum;   // [R][NCR][2]
    uint64_t* tsum;   // [R][NCR][kThreads] per-thread partial sums of column 0, or NULL
    uint32_t* cnt;    // [R][kCntStride] arrival counts of the draw's chunk workgroups (logits mode)
    float* dbg_pq;    // diagnostics or NULL: [2][R][D] the fp32 p(d_t), q(d_t) of every test
    float* dbg_row;   // diagnostics: [R][2][V] the fp32 P_a(v), Q_{a+1}(v) the draw weighs
    int R, b, D, V, NC, stats_chunk, NCR, res_chunk;
    float invT;
};

__device__ inline float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

__device__ inline float to_f(float x) { return x; }
__device__ inline float to_f(uint16_t h) { return bf2f(h); }

template <typename T>
__device__ inline float load_x(const T* row, int v) { return to_f(row[v]); }

// 16-byte load with the non-temporal hint, for rows streamed once per pass (the
// statistics and argmax passes): they would only evict reused lines from the caches
template <typename V>
__device__ inline V stream_load(const V* p) {
    return __builtin_nontemporal_load(p);
}

// fp32 probability of token v of a row: softmax(l / T) from its (max m, 1/sum) in logits
// mode, 2^(l * (log2e / T) - m * log2e) * (1/sum) with one fused multiply-add before the
// exponent; the stored value in probability mode. The draw's weights (weight_xy) compute
// the same expression.
template <bool LOGITS, typename T>
__device__ inline float prob_of(const T* row, int v, float m, float iS, float invT) {
    if (LOGITS) {
        return __builtin_amdgcn_exp2f(__builtin_fmaf(load_x<T>(row, v), invT * kLog2e, -m * kLog2e)) * iS;
    } else {
        return load_x<T>(row, v);
    }
}

// floor(min(r, 1) * 2^40) for r > 0 (0 for r <= 0 or NaN). v = min(r, 1) * 2^40 is exact
// (a power-of-two scaling) and below 2^41; its multiple of 2^32 (hi) and the remainder
// (lo = v - hi * 2^32, exact: both are multiples of the unit in the last place of v) are
// truncated to integers by the hardware conversion, so the result is floor(v) exactly.
__device__ inline uint64_t weight_of(float r) {
    r = r > 0.0f ? r : 0.0f;
    r = r < 1.0f ? r : 1.0f;
    const float v = r * 1099511627776.0f;                          // 2^40
    const float hf = __builtin_truncf(v * 2.3283064365386963e-10f);  // floor(v / 2^32)
    const float lf = v - hf * 4294967296.0f;
    return ((uint64_t)(uint32_t)hf << 32) | (uint64_t)(uint32_t)lf;
}

template <typename T>
__device__ inline const T* row_ptr(const void* base, long long row, int V) {
    return (const T*)base + row * (long long)V;
}

// Values handed from one workgroup to another inside a kernel go through device-coherent
// 8-byte stores and loads (agent scope: the XCDs' L2 caches are not coherent with each
// other). A writer waits for its stores to complete before it counts itself on an
// arrival counter, so the workgroup that sees the last count reads complete values.
__device__ inline void store_dev(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint64_t load_dev(const uint64_t* p) {
    return __hip_atomic_load((uint64_t*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// wait until every store this wave issued has completed (stores count in vmcnt on gfx9)
__device__ inline void wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ inline uint32_t arrive(uint32_t* ctr) {
    return __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Arrival counter of request i's draw: alone in a 128-byte cache line (kCntStride), because
// atomics on one line are serialised and a request's workgroups arrive close together.
__device__ inline size_t cnt_draw(int i) { return (size_t)i * kCntStride; }

// (max, sum of 2^((x - max) log2e)) of x = l * invT over the chunk [beg, end) of one row,
// valid in thread 0: every 16-byte load of the chunk is issued before any arithmetic
template <typename T>
__device__ inline float2 chunk_stats(const T* row, int beg, int end, int V, int stats_chunk, float invT,
                                     float* red) {
    constexpr int VEC = 16 / sizeof(T);
    typedef T vec_t __attribute__((ext_vector_type(VEC)));
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;

    float x[kStatsLoads * VEC];
    const bool vec_ok = (V % VEC) == 0 && (end - beg) == stats_chunk;
    if (vec_ok) {
        const vec_t* rv = (const vec_t*)(row + beg);
#pragma unroll
        for (int k = 0; k < kStatsLoads; k++) {
            const vec_t v = stream_load(rv + tid + k * kThreads);
#pragma unroll
            for (int e = 0; e < VEC; e++) x[k * VEC + e] = to_f(v[e]) * invT;
        }
    } else {
#pragma unroll
        for (int k = 0; k < kStatsLoads; k++)
#pragma unroll
            for (int e = 0; e < VEC; e++) {
                const int v = beg + (tid + k * kThreads) * VEC + e;
                x[k * VEC + e] = v < end ? load_x<T>(row, v) * invT : -INFINITY;
            }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < kStatsLoads * VEC; e++) mx = fmaxf(mx, x[e]);
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    if (lane == 0) red[w] = mx;
    __syncthreads();
    mx = red[0];
#pragma unroll
    for (int k = 1; k < kThreads / 64; k++) mx = fmaxf(mx, red[k]);
    __syncthreads();
    float s = 0.0f;
    if (mx != -INFINITY) {
#pragma unroll
        for (int e = 0; e < kStatsLoads * VEC; e++) s += __builtin_amdgcn_exp2f((x[e] - mx) * kLog2e);
    }
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) red[w] = s;
    __syncthreads();
    float tot = 0.0f;
    if (tid == 0)
        for (int k = 0; k < kThreads / 64; k++) tot += red[k];
    return make_float2(mx, tot);
}

// ----------------------------------------------------------------------------------
// rowstats: flat grid of (row slot, chunk), R*b + R*D slots of NC chunks (R*b when the
// draft rows' statistics are given): the packed target rows in order, then each
// request's draft rows. Its first R workgroups also zero the draw's arrival counters.
// ----------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void rowstats_kernel(AcceptArgs a) {
    __shared__ float red[kThreads / 64];
    const int slot = blockIdx.x / a.NC, c = blockIdx.x % a.NC;  // flat grid: (row slot, chunk)
    const int RB = a.R * a.b;
    if (blockIdx.x < (unsigned)a.R && threadIdx.x == 0) a.cnt[cnt_draw(blockIdx.x)] = 0;
    const T* row;
    float2* dst;
    if (slot < RB) {
        const int K = a.qo[a.R];
        if (slot >= K) return;
        row = row_ptr<T>(a.target, slot, a.V);
        dst = a.stats_t + (size_t)slot * a.NC;
    } else {
        const int s2 = slot - RB;
        const int i = s2 / a.D, t = s2 % a.D;
        const int n = a.qo[i + 1] - a.qo[i] - 1;
        if (t >= n) return;
        row = row_ptr<T>(a.draft, (long long)i * a.D + t, a.V);
        dst = a.stats_q + (size_t)(i * a.D + t) * a.NC;
    }
    const int beg = c * a.stats_chunk;
    const float2 st = chunk_stats<T>(row, beg, min(a.V, beg + a.stats_chunk), a.V, a.stats_chunk, a.invT, red);
    if (threadIdx.x == 0) dst[c] = st;
}

// combine the per-chunk (max, sum) of one row; chunk statistics are loaded 8 at a time
// so their latencies overlap
__device__ inline void merge_stats_ms(const float2* st, int NC, float& m, float& Sum) {
    float mm = -INFINITY, S = 0.0f;
    for (int c0 = 0; c0 < NC; c0 += 8) {
        float2 v[8];
#pragma unroll
        for (int k = 0; k < 8; k++) v[k] = c0 + k < NC ? st[c0 + k] : make_float2(-INFINITY, 0.0f);
        float bm = mm;
#pragma unroll
        for (int k = 0; k < 8; k++) bm = fmaxf(bm, v[k].x);
        if (bm != -INFINITY) {
            float acc = S * __builtin_amdgcn_exp2f((mm - bm) * kLog2e);
            if (mm == -INFINITY) acc = 0.0f;
#pragma unroll
            for (int k = 0; k < 8; k++)
                if (v[k].x != -INFINITY) acc += v[k].y * __builtin_amdgcn_exp2f((v[k].x - bm) * kLog2e);
            S = acc;
            mm = bm;
        }
    }
    m = mm;
    Sum = S;
}

__device__ inline float inv_sum(float S) { return S > 0.0f ? 1.0f / S : 0.0f; }

// (max, 1/sum) of one row from its chunk statistics
__device__ inline void merge_stats(const float2* st, int NC, float& m, float& iS) {
    float S;
    merge_stats_ms(st, NC, m, S);
    iS = inv_sum(S);
}

// ----------------------------------------------------------------------------------
// decision of request i, taken by one wavefront (lane = 0..63); the plan is valid in lane
// 0. With write set, the accepted prefix, accept_len, flags of a malformed request and
// the plan are stored.
// ----------------------------------------------------------------------------------
template <bool LOGITS, typename T>
__device__ inline ReqPlan decide_req(const AcceptArgs& a, const int i, const int lane, const bool write) {
    const int q0 = a.qo[i];
    const int n = a.qo[i + 1] - q0 - 1;
    const int K = a.qo[a.R];
    ReqPlan pl{};
    if (n < 0 || n > a.D || q0 < 0 || q0 + n + 1 > K || K > a.R * a.b) {  // malformed packing: nothing to draw
        pl.mode = 2;
        pl.flag = 2;
        if (write) {
            if (lane == 0) {
                a.plan[i] = pl;
                a.accept_len[i] = 0;
                if (a.flags) a.flags[i] = 2;
            }
            for (int t = lane; t < a.b; t += 64) a.out_tokens[(size_t)i * a.b + t] = -1;
        }
        return pl;
    }
    // per-row softmax statistics: lane r -> P_r (r <= n), lane 32+t -> Q_{t+1} (t < n)
    float m = 0.0f, iS = 0.0f;
    if (LOGITS) {
        if (lane <= n) merge_stats(a.stats_t + (size_t)(q0 + lane) * a.NC, a.NC, m, iS);
        else if (lane >= 32 && lane - 32 < n) {
            if (a.dstats) {  // the drafter's own (max, sum) of this row
                const float2 st = a.dstats[(size_t)i * a.D + lane - 32];
                m = st.x;
                iS = inv_sum(st.y);
            } else {
                merge_stats(a.stats_q + (size_t)(i * a.D + lane - 32) * a.NC, a.NC, m, iS);
            }
        }
    }
    // the test of draft t+1 in lane t: P_t(d) vs u * Q_{t+1}(d)
    const float mPt = __shfl(m, lane & 31, 64), iSPt = __shfl(iS, lane & 31, 64);
    const float mQt = __shfl(m, 32 + (lane & 31), 64), iSQt = __shfl(iS, 32 + (lane & 31), 64);
    bool reject = false, bad_tok = false;
    int d = -1;
    if (lane < n) {
        d = a.tokens[(size_t)i * a.D + lane];
        if (d < 0 || d >= a.V) {
            reject = true;
            bad_tok = true;
        } else {
            const float p = prob_of<LOGITS, T>(row_ptr<T>(a.target, q0 + lane, a.V), d, mPt, iSPt, a.invT);
            const float q = prob_of<LOGITS, T>(row_ptr<T>(a.draft, (long long)i * a.D + lane, a.V), d, mQt, iSQt, a.invT);
            const double u = (double)a.ua[(size_t)i * a.D + lane];
            reject = !(u * (double)q < (double)p);
            if (write && a.dbg_pq) {  // diagnostics: the values this test compared
                a.dbg_pq[(size_t)i * a.D + lane] = p;
                a.dbg_pq[((size_t)a.R + i) * a.D + lane] = q;
            }
        }
    }
    const uint64_t fails = __ballot(reject);
    const int acc = fails ? __builtin_ctzll(fails) : n;
    const int badflag = __shfl((int)bad_tok, acc & 63, 64) ? 4 : 0;
    if (write)
        for (int t = lane; t < a.b; t += 64) {
            if (t < acc) a.out_tokens[(size_t)i * a.b + t] = a.tokens[(size_t)i * a.D + t];
            else if (t > acc) a.out_tokens[(size_t)i * a.b + t] = -1;
        }
    // statistics of P_a (lane a) and Q_{a+1} (lane 32+a), gathered by every lane
    const float pm = __shfl(m, acc & 31, 64), piS = __shfl(iS, acc & 31, 64);
    const float qm = __shfl(m, 32 + (acc & 31), 64), qiS = __shfl(iS, 32 + (acc & 31), 64);
    if (lane == 0) {
        pl.a = acc;
        pl.n = n;
        pl.flag = acc < n ? badflag : 0;
        pl.mode = acc < n ? 0 : 1;
        pl.rowP = q0 + acc;
        pl.rowQ = acc < n ? i * a.D + acc : -1;
        pl.mP = pm;
        pl.iSP = piS;
        pl.mQ = acc < n ? qm : 0.0f;
        pl.iSQ = acc < n ? qiS : 0.0f;
        if (write) {
            a.plan[i] = pl;
            a.accept_len[i] = acc;
        }
    }
    return pl;
}


template <bool LOGITS>
__device__ inline uint64_t weight_xy(const ReqPlan& pl, int col, float x, float y, float invT);

// weight of token v in column col (see weight_xy), loading the values itself
template <bool LOGITS, typename T>
__device__ inline uint64_t weight_at(const AcceptArgs& a, const ReqPlan& pl, int col, int v) {
    const float x = load_x<T>(row_ptr<T>(a.target, pl.rowP, a.V), v);
    const float y = (pl.mode == 0 && col == 0) ? load_x<T>(row_ptr<T>(a.draft, pl.rowQ, a.V), v) : x;
    return weight_xy<LOGITS>(pl, col, x, y, a.invT);
}

// weight of one token from already loaded values x (target) and y (draft): column 0 is
// the residual (or bonus) weight, column 1 the fallback weight of P_a
template <bool LOGITS>
__device__ inline uint64_t weight_xy(const ReqPlan& pl, int col, float x, float y, float invT) {
    // the probability of prob_of, with the row's constants hoisted out of the token loop
    const float c = invT * kLog2e;
    const float pv = LOGITS ? __builtin_amdgcn_exp2f(__builtin_fmaf(x, c, -pl.mP * kLog2e)) * pl.iSP : x;
    if (pl.mode != 0 || col == 1) return weight_of(pv);
    const float qv = LOGITS ? __builtin_amdgcn_exp2f(__builtin_fmaf(y, c, -pl.mQ * kLog2e)) * pl.iSQ : y;
    float r = pv - qv;
    if (!(r > 0.0f)) r = 0.0f;
    return weight_of(r);
}

// Sum of one weight column over the contiguous range [lo, hi) of the vocabulary: 16-byte
// loads when the range is aligned, element loads otherwise.
template <bool LOGITS, typename T>
__device__ inline uint64_t range_sum(const AcceptArgs& a, const ReqPlan& pl, int col, int lo, int hi) {
    constexpr int VEC = 16 / sizeof(T);
    typedef T vec_t __attribute__((ext_vector_type(VEC)));
    const T* prow = row_ptr<T>(a.target, pl.rowP, a.V);
    const bool need_q = pl.mode == 0 && col == 0;
    const T* qrow = need_q ? row_ptr<T>(a.draft, pl.rowQ, a.V) : prow;
    uint64_t sum = 0;
    int v = lo;
    if ((a.V % VEC) == 0 && (lo % VEC) == 0) {
        for (; v + VEC <= hi; v += VEC) {
            const vec_t xp = *(const vec_t*)(prow + v);
            vec_t xq = xp;
            if (need_q) xq = *(const vec_t*)(qrow + v);
#pragma unroll
            for (int e = 0; e < VEC; e++) sum += weight_xy<LOGITS>(pl, col, to_f(xp[e]), to_f(xq[e]), a.invT);
        }
    }
    for (; v < hi; v++) sum += weight_xy<LOGITS>(pl, col, load_x<T>(prow, v), load_x<T>(qrow, v), a.invT);
    return sum;
}

// One thread's full, aligned range of kResPer tokens: every load is issued before any
// weight is computed (one memory round trip), and the values stay in registers for a
// later scan.
template <typename T>
struct RangeRegs {
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr int NV = kResPer / VEC;
    typedef T vec_t __attribute__((ext_vector_type(VEC)));
    vec_t xp[NV], xq[NV];
};

template <typename T>
__device__ inline bool range_is_full(const AcceptArgs& a, int lo, int hi) {
    return hi - lo == kResPer && (a.V % RangeRegs<T>::VEC) == 0 && (lo % RangeRegs<T>::VEC) == 0;
}

template <typename T>
__device__ inline void range_load(const AcceptArgs& a, const ReqPlan& pl, int col, int lo, RangeRegs<T>& g) {
    typedef typename RangeRegs<T>::vec_t vec_t;
    const vec_t* prow = (const vec_t*)(row_ptr<T>(a.target, pl.rowP, a.V) + lo);
    const bool need_q = pl.mode == 0 && col == 0;
    const vec_t* qrow = need_q ? (const vec_t*)(row_ptr<T>(a.draft, pl.rowQ, a.V) + lo) : prow;
#pragma unroll
    for (int k = 0; k < RangeRegs<T>::NV; k++) {
        g.xp[k] = prow[k];
        g.xq[k] = qrow[k];
    }
}

template <bool LOGITS, typename T>
__device__ inline uint64_t range_regs_sum(const AcceptArgs& a, const ReqPlan& pl, int col, const RangeRegs<T>& g) {
    uint64_t sum = 0;
#pragma unroll
    for (int k = 0; k < RangeRegs<T>::NV; k++)
#pragma unroll
        for (int e = 0; e < RangeRegs<T>::VEC; e++)
            sum += weight_xy<LOGITS>(pl, col, to_f(g.xp[k][e]), to_f(g.xq[k][e]), a.invT);
    return sum;
}

__device__ inline uint64_t wave_incl_scan_u64(uint64_t v, int lane) {
    for (int off = 1; off < 64; off <<= 1) {
        const uint64_t t = __shfl_up(v, off, 64);
        if (lane >= off) v += t;
    }
    return v;
}

__device__ inline uint64_t block_sum_u64(uint64_t v, uint64_t* red) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    uint64_t t = 0;
    for (int k = 0; k < kThreads / 64; k++) t += red[k];
    return t;
}

// ----------------------------------------------------------------------------------
// chunk sums: flat grid of (request, chunk); each workgroup takes the request's decision
// (first wave), then sums the integer residual (or bonus) weights of one vocabulary chunk
// ----------------------------------------------------------------------------------
// diagnostics: the fp32 probabilities of the draw's row pair over [lo, hi), as the weights
// of column 0 use them (the same expressions as weight_xy)
template <bool LOGITS, typename T>
__device__ inline void dbg_store_row(const AcceptArgs& a, const ReqPlan& pl, int i, int lo, int hi) {
    const float c = a.invT * kLog2e;
    const T* prow = row_ptr<T>(a.target, pl.rowP, a.V);
    for (int v = lo; v < hi; v++) {
        const float x = load_x<T>(prow, v);
        const float pv = LOGITS ? __builtin_amdgcn_exp2f(__builtin_fmaf(x, c, -pl.mP * kLog2e)) * pl.iSP : x;
        float qv = 0.0f;
        if (pl.mode == 0) {
            const float y = load_x<T>(row_ptr<T>(a.draft, pl.rowQ, a.V), v);
            qv = LOGITS ? __builtin_amdgcn_exp2f(__builtin_fmaf(y, c, -pl.mQ * kLog2e)) * pl.iSQ : y;
        }
        a.dbg_row[((size_t)i * 2 + 0) * a.V + v] = pv;
        a.dbg_row[((size_t)i * 2 + 1) * a.V + v] = qv;
    }
}

template <bool LOGITS, typename T, bool DBG = false>
__global__ __launch_bounds__(kThreads) void chunksum_kernel(AcceptArgs a) {
    __shared__ uint64_t red[kThreads / 64];
    __shared__ ReqPlan s_pl;
    const int i = blockIdx.x / a.NCR, c = blockIdx.x % a.NCR, tid = threadIdx.x;  // flat grid: (request, chunk)
    if (tid < 64) {
        const ReqPlan p0 = decide_req<LOGITS, T>(a, i, tid, c == 0);
        if (tid == 0) s_pl = p0;
    }
    __syncthreads();
    const ReqPlan pl = s_pl;
    if (pl.mode == 2) return;
    const int beg = c * kResChunk, end = min(a.V, beg + kResChunk);
    const int lo = min(end, beg + tid * kResPer), hi = min(end, lo + kResPer);
    uint64_t part;
    if (range_is_full<T>(a, lo, hi)) {
        RangeRegs<T> g;
        range_load<T>(a, pl, 0, lo, g);
        part = range_regs_sum<LOGITS, T>(a, pl, 0, g);
    } else {
        part = range_sum<LOGITS, T>(a, pl, 0, lo, hi);
    }
    if (DBG) dbg_store_row<LOGITS, T>(a, pl, i, lo, hi);
    if (a.tsum) a.tsum[((size_t)i * a.NCR + c) * kThreads + tid] = part;
    const uint64_t sr = block_sum_u64(part, red);
    if (tid == 0) a.csum[((size_t)i * a.NCR + c) * 2 + 0] = sr;
}

// ----------------------------------------------------------------------------------
// search of request i by one whole workgroup: Z = sum of the chunk sums, the threshold
// floor(m * Z / 2^24), the chunk holding it (wave scan), then the token inside that chunk
// (per-thread ranges, block scan, and the owning thread's scan of its loaded values).
// An empty residual falls back to the weights of P_a, summed here (rare). COH: the chunk
// sums and partial sums come from other workgroups of the running kernel.
// ----------------------------------------------------------------------------------
template <bool LOGITS, typename T, bool COH>
__device__ inline void search_req(const AcceptArgs& a, const int i, const ReqPlan& pl) {
    __shared__ uint64_t red[kThreads / 64];
    __shared__ uint64_t wsum[kThreads / 64];
    __shared__ int s_chunk, s_token;
    __shared__ uint64_t s_before;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int per = kResPer;
    // chunk sums: thread k < NCR keeps csum[k] in a register (wave 0 scans them below when
    // there are at most 64 chunks)
    uint64_t Z = 0, my_cs = 0;
    for (int k = tid; k < a.NCR; k += kThreads) {
        const uint64_t* src = a.csum + ((size_t)i * a.NCR + k) * 2;
        const uint64_t v = COH ? load_dev(src) : *src;
        if (k == tid) my_cs = v;
        Z += v;
    }
    Z = block_sum_u64(Z, red);
    int col = 0;
    int flag = pl.flag;
    if (Z == 0 && pl.mode == 0) {
        col = 1;
        flag |= 1;
        uint64_t zp = 0;
        for (int k = 0; k < a.NCR; k++) {
            const int beg = k * a.res_chunk, end = min(a.V, beg + a.res_chunk);
            const int lo = min(end, beg + tid * per), hi = min(end, lo + per);
            const uint64_t sk = block_sum_u64(range_sum<LOGITS, T>(a, pl, 1, lo, hi), red);
            if (tid == 0) a.csum[((size_t)i * a.NCR + k) * 2 + 1] = sk;
            zp += sk;
        }
        __syncthreads();
        Z = zp;
    }
    int token = -1;
    if (Z == 0) {
        flag |= 2;
    } else {
        const float u = a.us[i];
        uint32_t mu;
        if (!(u > 0.0f)) mu = 0;
        else if (u >= 1.0f) mu = (1u << 24) - 1;
        else mu = (uint32_t)(u * 16777216.0f);  // exact on the 2^-24 grid, truncates otherwise
        const uint64_t thr = (uint64_t)(((unsigned __int128)mu * Z) >> 24);
        // 1. the chunk holding thr: wave 0 scans the chunk sums 64 at a time
        if (w == 0) {
            uint64_t base = 0, before = 0;
            int found = -1;
            for (int c0 = 0; c0 < a.NCR && found < 0; c0 += 64) {
                const int k = c0 + lane;
                const uint64_t* src = a.csum + ((size_t)i * a.NCR + k) * 2 + col;
                const uint64_t v = k >= a.NCR ? 0 : (col == 0 && a.NCR <= 64) ? my_cs : COH ? load_dev(src) : *src;
                const uint64_t incl = base + wave_incl_scan_u64(v, lane);
                const bool hit = k < a.NCR && v > 0 && incl - v <= thr && thr < incl;
                const uint64_t m = __ballot(hit);
                if (m) {
                    const int src = __builtin_ctzll(m);
                    found = c0 + src;
                    before = __shfl(incl - v, src, 64);
                }
                base = __shfl(incl, 63, 64);
            }
            if (lane == 0) {
                s_chunk = found;
                s_before = before;
            }
        }
        __syncthreads();
        const int cs = s_chunk;
        if (cs >= 0 && col == 0 && a.tsum) {
            // 2. inside the chunk, from the chunk-sum pass's per-thread partial sums: wave 0
            //    finds the thread range holding thr (its 256 partials, 64 at a time), then
            //    the token among that range's kResPer tokens, one weight per lane
            if (w == 0) {
                const uint64_t rel = thr - s_before;
                const uint64_t* ts = a.tsum + ((size_t)i * a.NCR + cs) * kThreads;
                uint64_t v4[kThreads / 64];
#pragma unroll
                for (int k = 0; k < kThreads / 64; k++) v4[k] = COH ? load_dev(ts + k * 64 + lane) : ts[k * 64 + lane];
                uint64_t base = 0, before = 0;
                int found = -1;
#pragma unroll
                for (int k = 0; k < kThreads / 64; k++) {
                    if (found >= 0) break;
                    const uint64_t incl = base + wave_incl_scan_u64(v4[k], lane);
                    const uint64_t m = __ballot(v4[k] > 0 && incl - v4[k] <= rel && rel < incl);
                    if (m) {
                        const int src = __builtin_ctzll(m);
                        found = k * 64 + src;
                        before = __shfl(incl - v4[k], src, 64);
                    }
                    base = __shfl(incl, 63, 64);
                }
                int tok = -1;
                if (found >= 0) {
                    static_assert(kResPer <= 64, "one token per lane");
                    const int beg = cs * kResChunk, end = min(a.V, beg + kResChunk);
                    const int lo = min(end, beg + found * kResPer), hi = min(end, lo + kResPer);
                    const int v = lo + lane;
                    const uint64_t wv = lane < kResPer && v < hi ? weight_at<LOGITS, T>(a, pl, 0, v) : 0;
                    const uint64_t incl = before + wave_incl_scan_u64(wv, lane);
                    const uint64_t m = __ballot(wv > 0 && incl - wv <= rel && rel < incl);
                    if (m) tok = lo + __builtin_ctzll(m);
                }
                if (lane == 0) s_token = tok;
            }
            __syncthreads();
            token = s_token;
        } else if (cs >= 0) {
            // 2. inside the chunk: per-thread contiguous ranges, block exclusive scan
            const int beg = cs * kResChunk, end = min(a.V, beg + kResChunk);
            const int lo = min(end, beg + tid * per), hi = min(end, lo + per);
            const bool full = range_is_full<T>(a, lo, hi);
            RangeRegs<T> g;
            uint64_t loc;
            if (full) {
                range_load<T>(a, pl, col, lo, g);
                loc = range_regs_sum<LOGITS, T>(a, pl, col, g);
            } else {
                loc = range_sum<LOGITS, T>(a, pl, col, lo, hi);
            }
            const uint64_t incl = wave_incl_scan_u64(loc, lane);
            if (lane == 63) wsum[w] = incl;
            if (tid == 0) s_token = -1;
            __syncthreads();
            uint64_t wbase = 0;
            for (int k = 0; k < w; k++) wbase += wsum[k];
            const uint64_t rel = thr - s_before;
            const uint64_t excl = wbase + incl - loc;
            if (loc > 0 && excl <= rel && rel < excl + loc) {
                // this thread's range holds the token; a full range scans the values it
                // already holds
                uint64_t cum = s_before + excl;
                if (full) {
                    int found = -1;
#pragma unroll
                    for (int k = 0; k < RangeRegs<T>::NV; k++)
#pragma unroll
                        for (int e = 0; e < RangeRegs<T>::VEC; e++) {
                            const uint64_t wv = weight_xy<LOGITS>(pl, col, to_f(g.xp[k][e]), to_f(g.xq[k][e]), a.invT);
                            if (found < 0 && cum + wv > thr) found = lo + k * RangeRegs<T>::VEC + e;
                            cum += wv;
                        }
                    s_token = found;
                } else {
                    for (int v = lo; v < hi; v++) {
                        const uint64_t wv = weight_at<LOGITS, T>(a, pl, col, v);
                        if (cum + wv > thr) {
                            s_token = v;
                            break;
                        }
                        cum += wv;
                    }
                }
            }
            __syncthreads();
            token = s_token;
        }
    }
    if (tid == 0) {
        a.out_tokens[(size_t)i * a.b + pl.a] = token;
        if (a.flags) a.flags[i] = flag;
    }
}

// search: one workgroup per request (probability mode)
template <bool LOGITS, typename T>
__global__ __launch_bounds__(kThreads) void search_kernel(AcceptArgs a) {
    const ReqPlan pl = a.plan[blockIdx.x];
    if (pl.mode == 2) return;
    search_req<LOGITS, T, false>(a, blockIdx.x, pl);
}

// ----------------------------------------------------------------------------------
// draw (logits mode): flat grid of (request, chunk). The first wave takes the request's
// decision (the chunk-0 workgroup writes its outputs). The workgroup sums the residual
// (or bonus) weights of its chunk, stores the sum and its threads' partial sums
// device-coherently and counts itself; the request's last chunk workgroup runs the
// search.
// ----------------------------------------------------------------------------------
template <typename T, bool DBG = false>
__global__ __launch_bounds__(kThreads) void draw_kernel(AcceptArgs a) {
    __shared__ uint64_t red[kThreads / 64];
    __shared__ ReqPlan s_pl;
    __shared__ int s_last;
    const int i = blockIdx.x / a.NCR, c = blockIdx.x % a.NCR, tid = threadIdx.x;  // flat grid: (request, chunk)
    if (tid < 64) {
        const ReqPlan p0 = decide_req<true, T>(a, i, tid, c == 0);
        if (tid == 0) s_pl = p0;
    }
    __syncthreads();
    const ReqPlan pl = s_pl;
    if (pl.mode == 2) return;
    const int beg = c * kResChunk, end = min(a.V, beg + kResChunk);
    const int lo = min(end, beg + tid * kResPer), hi = min(end, lo + kResPer);
    uint64_t part;
    if (range_is_full<T>(a, lo, hi)) {
        RangeRegs<T> g;
        range_load<T>(a, pl, 0, lo, g);
        part = range_regs_sum<true, T>(a, pl, 0, g);
    } else {
        part = range_sum<true, T>(a, pl, 0, lo, hi);
    }
    if (DBG) dbg_store_row<true, T>(a, pl, i, lo, hi);
    if (a.tsum) store_dev(a.tsum + ((size_t)i * a.NCR + c) * kThreads + tid, part);
    const uint64_t sr = block_sum_u64(part, red);
    if (tid == 0) store_dev(a.csum + ((size_t)i * a.NCR + c) * 2, sr);
    wait_stores();
    __syncthreads();
    if (tid == 0) s_last = arrive(a.cnt + cnt_draw(i)) + 1 == (uint32_t)a.NCR;
    __syncthreads();
    if (!s_last) return;
    search_req<true, T, true>(a, i, pl);
}

// ----------------------------------------------------------------------------------
// Draft-row statistics (the drafter's side of the round): per draft row the softmax
// (max, sum) that acceptance would compute itself -- the same chunks, the same merge --
// and the confidence max_v Q_t(v) = 1 / sum that the budget takes as c_t.
// ----------------------------------------------------------------------------------
struct DStatsArgs {
    const void* logits;  // [rows, V]
    float2* part;        // [rows][NC]
    float2* stats;       // [rows] (max, sum)
    float* conf;         // [rows] or NULL
    int rows, V, NC, stats_chunk;
    float invT;
};

template <typename T>
__global__ __launch_bounds__(kThreads) void dstats_chunk_kernel(DStatsArgs a) {
    __shared__ float red[kThreads / 64];
    const int r = blockIdx.x / a.NC, c = blockIdx.x % a.NC;
    const T* row = row_ptr<T>(a.logits, r, a.V);
    const int beg = c * a.stats_chunk;
    const float2 st = chunk_stats<T>(row, beg, min(a.V, beg + a.stats_chunk), a.V, a.stats_chunk, a.invT, red);
    if (threadIdx.x == 0) a.part[(size_t)r * a.NC + c] = st;
}

__global__ __launch_bounds__(256) void dstats_merge_kernel(DStatsArgs a) {
    const int r = blockIdx.x * 256 + threadIdx.x;
    if (r >= a.rows) return;
    float m, S;
    merge_stats_ms(a.part + (size_t)r * a.NC, a.NC, m, S);
    a.stats[r] = make_float2(m, S);
    if (a.conf) a.conf[r] = inv_sum(S);  // max_v of exp(x - m) / S is exp(0) / S
}

// ----------------------------------------------------------------------------------
// Greedy verification (temperature 0): rejection sampling with one-hot target and draft
// rows. Draft t is accepted iff it is the argmax of P_{t-1}; the extra token is the argmax
// of P_a. Argmax: largest stored value (lowest index on ties, NaN skipped), so only the
// kept target rows are read and no arithmetic decides anything.
// ----------------------------------------------------------------------------------
struct ArgBest {
    float v;
    int idx;  // < 0: no non-NaN entry
};

// the better of two candidates: a valid one, then the larger value, then the lower index
__device__ inline ArgBest arg_better(ArgBest x, ArgBest y) {
    if (y.idx < 0) return x;
    if (x.idx < 0) return y;
    if (y.v > x.v || (y.v == x.v && y.idx < x.idx)) return y;
    return x;
}

__device__ inline ArgBest wave_arg_best(ArgBest x) {
    for (int off = 32; off > 0; off >>= 1) {
        ArgBest y;
        y.v = __shfl_xor(x.v, off, 64);
        y.idx = __shfl_xor(x.idx, off, 64);
        x = arg_better(x, y);
    }
    return x;
}

// flat grid of (target row slot, chunk): (max, argmax) of one chunk of a kept target row,
// stored as (value, index bits) in the statistics slot
template <typename T>
__global__ __launch_bounds__(kThreads) void argmax_kernel(AcceptArgs a) {
    constexpr int VEC = 16 / sizeof(T);
    typedef T vec_t __attribute__((ext_vector_type(VEC)));
    __shared__ float s_v[kThreads / 64];
    __shared__ int s_i[kThreads / 64];
    const int slot = blockIdx.x / a.NC, c = blockIdx.x % a.NC;
    if (slot >= a.qo[a.R]) return;
    const T* row = row_ptr<T>(a.target, slot, a.V);
    const int beg = c * a.stats_chunk, end = min(a.V, beg + a.stats_chunk);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    // each thread visits its elements in increasing index order: a strict > keeps the
    // lowest index among equal values
    ArgBest best{0.0f, -1};
    if ((a.V % VEC) == 0 && (end - beg) == a.stats_chunk) {
        const vec_t* rv = (const vec_t*)(row + beg);
        vec_t v[kStatsLoads];
#pragma unroll
        for (int k = 0; k < kStatsLoads; k++) v[k] = stream_load(rv + tid + k * kThreads);
#pragma unroll
        for (int k = 0; k < kStatsLoads; k++)
#pragma unroll
            for (int e = 0; e < VEC; e++) {
                const float x = to_f(v[k][e]);
                if (x == x && (best.idx < 0 || x > best.v)) {
                    best.v = x;
                    best.idx = beg + (tid + k * kThreads) * VEC + e;
                }
            }
    } else {
        for (int k = 0; k < kStatsLoads; k++)
            for (int e = 0; e < VEC; e++) {
                const int vi = beg + (tid + k * kThreads) * VEC + e;
                if (vi >= end) continue;
                const float x = load_x<T>(row, vi);
                if (x == x && (best.idx < 0 || x > best.v)) {
                    best.v = x;
                    best.idx = vi;
                }
            }
    }
    best = wave_arg_best(best);
    if (lane == 0) {
        s_v[w] = best.v;
        s_i[w] = best.idx;
    }
    __syncthreads();
    if (tid == 0) {
        ArgBest b = ArgBest{s_v[0], s_i[0]};
        for (int k = 1; k < kThreads / 64; k++) b = arg_better(b, ArgBest{s_v[k], s_i[k]});
        a.stats_t[(size_t)slot * a.NC + c] = make_float2(b.v, __int_as_float(b.idx));
    }
}

// one wavefront per request: lane r merges the chunk results of P_r, lane t tests draft
// t+1 against the argmax of P_t, a ballot finds the first mismatch
__global__ __launch_bounds__(64) void decide_greedy_kernel(AcceptArgs a) {
    const int i = blockIdx.x, lane = threadIdx.x;
    const int q0 = a.qo[i];
    const int n = a.qo[i + 1] - q0 - 1;
    const int K = a.qo[a.R];
    if (n < 0 || n > a.D || q0 < 0 || q0 + n + 1 > K || K > a.R * a.b) {  // malformed packing
        if (lane == 0) {
            a.accept_len[i] = 0;
            if (a.flags) a.flags[i] = 2;
        }
        for (int t = lane; t < a.b; t += 64) a.out_tokens[(size_t)i * a.b + t] = -1;
        return;
    }
    ArgBest rb{0.0f, -1};
    if (lane <= n) {
        const float2* st = a.stats_t + (size_t)(q0 + lane) * a.NC;
        for (int c = 0; c < a.NC; c++) {
            const float2 v = st[c];
            rb = arg_better(rb, ArgBest{v.x, __float_as_int(v.y)});
        }
    }
    const int am = rb.idx;  // argmax of P_lane
    bool reject = false, bad_tok = false;
    if (lane < n) {
        const int d = a.tokens[(size_t)i * a.D + lane];
        if (d < 0 || d >= a.V) {
            reject = true;
            bad_tok = true;
        } else {
            reject = d != am;
        }
    }
    const uint64_t fails = __ballot(reject);
    const int acc = fails ? __builtin_ctzll(fails) : n;
    const int token = __shfl(am, acc, 64);
    const int flag = (token < 0 ? 2 : 0) | (__shfl((int)bad_tok, acc & 63, 64) ? 4 : 0);
    for (int t = lane; t < a.b; t += 64) {
        int v = -1;
        if (t < acc) v = a.tokens[(size_t)i * a.D + t];
        else if (t == acc) v = token;
        a.out_tokens[(size_t)i * a.b + t] = v;
    }
    if (lane == 0) {
        a.accept_len[i] = acc;
        if (a.flags) a.flags[i] = flag;
    }
}

}  // namespace

hipError_t launch_accept(const sv_accept_desc& d, const AcceptPlan& p, const void* target,
                         const void* draft, const float* draft_stats, const int32_t* draft_tokens,
                         const int32_t* qo_indptr, const float* u_accept, const float* u_sample,
                         int32_t* accept_len, int32_t* out_tokens, int32_t* flags, void* ws,
                         hipStream_t stream, float* dbg_pq, float* dbg_row) {
    AcceptArgs a{};
    a.target = target;
    a.draft = draft;
    a.tokens = draft_tokens;
    a.qo = qo_indptr;
    a.ua = u_accept;
    a.us = u_sample;
    a.accept_len = accept_len;
    a.out_tokens = out_tokens;
    a.flags = flags;
    a.dstats = (const float2*)draft_stats;
    a.dbg_pq = dbg_pq;
    a.dbg_row = dbg_row;
    char* w = (char*)ws;
    a.stats_t = (float2*)(w + p.off_stats_t);
    a.stats_q = (float2*)(w + p.off_stats_q);
    a.plan = (ReqPlan*)(w + p.off_plan);
    a.csum = (uint64_t*)(w + p.off_csum);
    a.tsum = p.off_tsum ? (uint64_t*)(w + p.off_tsum) : nullptr;
    a.cnt = (uint32_t*)(w + p.off_cnt);
    a.R = d.num_reqs;
    a.b = d.block;
    a.D = d.block - 1;
    a.V = d.vocab;
    a.NC = p.stats_chunks;
    a.stats_chunk = p.stats_chunk;
    a.NCR = p.res_chunks;
    a.res_chunk = p.res_chunk;
    a.invT = d.kind == SV_LOGITS && d.temperature > 0.0f ? 1.0f / d.temperature : 1.0f;
    const bool logits = d.kind == SV_LOGITS;
    const bool bf = d.dtype == SV_BF16;
    if (d.temperature == 0.0f) {  // greedy verification
        const dim3 g((unsigned)((long long)d.num_reqs * d.block * p.stats_chunks));
        if (bf) hipLaunchKernelGGL(argmax_kernel<uint16_t>, g, dim3(kThreads), 0, stream, a);
        else hipLaunchKernelGGL(argmax_kernel<float>, g, dim3(kThreads), 0, stream, a);
        hipLaunchKernelGGL(decide_greedy_kernel, dim3(d.num_reqs), dim3(64), 0, stream, a);
        return hipGetLastError();
    }
    const dim3 gres((unsigned)((long long)p.res_chunks * d.num_reqs));
    if (logits) {
        const long long slots = (long long)d.num_reqs * d.block +
                                (draft_stats ? 0LL : (long long)d.num_reqs * (d.block > 1 ? d.block - 1 : 0));
        const dim3 g((unsigned)(slots * p.stats_chunks));
        if (bf) hipLaunchKernelGGL(rowstats_kernel<uint16_t>, g, dim3(kThreads), 0, stream, a);
        else hipLaunchKernelGGL(rowstats_kernel<float>, g, dim3(kThreads), 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (bf && dbg_row) hipLaunchKernelGGL((draw_kernel<uint16_t, true>), gres, dim3(kThreads), 0, stream, a);
        else if (bf) hipLaunchKernelGGL((draw_kernel<uint16_t>), gres, dim3(kThreads), 0, stream, a);
        else if (dbg_row) hipLaunchKernelGGL((draw_kernel<float, true>), gres, dim3(kThreads), 0, stream, a);
        else hipLaunchKernelGGL((draw_kernel<float>), gres, dim3(kThreads), 0, stream, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((chunksum_kernel<false, float>), gres, dim3(kThreads), 0, stream, a);
    hipLaunchKernelGGL((search_kernel<false, float>), dim3(d.num_reqs), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_draft_stats(const sv_draft_stats_desc& d, const void* logits, float* stats, float* conf, void* ws,
                              hipStream_t stream) {
    DStatsArgs a{};
    const int esz = d.dtype == SV_BF16 ? 2 : 4;
    a.logits = logits;
    a.part = (float2*)ws;
    a.stats = (float2*)stats;
    a.conf = conf;
    a.rows = d.num_reqs * d.drafts;
    a.V = d.vocab;
    a.stats_chunk = kThreads * kStatsLoads * (16 / esz);  // the chunks of sv_spec_accept
    a.NC = (d.vocab + a.stats_chunk - 1) / a.stats_chunk;
    a.invT = 1.0f / d.temperature;
    const dim3 g((unsigned)((long long)a.rows * a.NC));
    if (d.dtype == SV_BF16) hipLaunchKernelGGL(dstats_chunk_kernel<uint16_t>, g, dim3(kThreads), 0, stream, a);
    else hipLaunchKernelGGL(dstats_chunk_kernel<float>, g, dim3(kThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(dstats_merge_kernel, dim3((unsigned)((a.rows + 255) / 256)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace sv
