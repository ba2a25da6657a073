// Verify attention over a paged KV cache (AngelSpec Sec. 4.1: every kept block
// position is evaluated by the target model; Sec. 4.2: one dense packed batch).
//
// bf16 path (MFMA). A workgroup owns one (request i, kv-head h, split s) work item:
// the G*k_i query rows of that kv-head group against tokens [s*split, (s+1)*split)
// of the request's context. Query rows go on the N side of the MFMA and KV tokens
// on the M side, so S^T = K Q^T puts all scores of one query row in one lane pair:
// the online-softmax max/sum is lane-local plus one cross-half swap. The P^T
// fragment is then already in the B-operand layout of O^T = V^T P^T; V is staged
// transposed in LDS to serve the A operand. K and V tiles of 64 tokens are
// gathered through the page table into double-buffered LDS while the previous
// tile is multiplied. Work items whose split lies past the request's length exit
// at once; requests with more than one split write fp32 partials merged by a
// second kernel (log-sum-exp weights).
//
// fp32 path (vector ALU): one wavefront per (query row, head), 64 keys per step.
#include "sv_internal.h"

namespace sv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kTile = 64;  // KV tokens per pipeline step

struct AttnArgs {
    const void* q;
    const void* kc;
    const void* vc;
    const int32_t* page_table;
    const int32_t* qo;
    const int32_t* kv_lens;
    void* out;
    float* lse;
    float* part_o;    // [max_splits, total_q_max, Hq, d]
    float* part_lse;  // [max_splits, total_q_max, Hq]  (log2 domain)
    int R, total_q, Hq, Hkv, G, block;
    int log2P, maxp, num_pages, max_kv_len;
    int split, max_splits;
    float scale_log2;  // sm_scale * log2(e)
    float scale;       // sm_scale
};

__device__ inline float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// round-to-nearest-even fp32 -> bf16 bits
__device__ inline uint16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x7FFFFFu)) return 0x7FC0;
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// ---------------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------------
template <int HD>
struct Lds {
    static constexpr int kStride = HD + 8;       // K rows: HD bf16 + 16 B pad
    static constexpr int vStride = kTile + 8;    // V^T rows: 64 tokens + 16 B pad
    uint16_t k[2][kTile * kStride];
    uint16_t vt[2][HD * vStride];
};

template <int HD, int NW>
__global__ __launch_bounds__(NW * 64) void attn_bf16_kernel(AttnArgs a) {
    constexpr int NT = NW * 64;
    constexpr int CPR = HD / 8;                   // 16-byte chunks per token row
    constexpr int CHUNKS = kTile * CPR;           // per tile, per tensor
    constexpr int CPT = (CHUNKS + NT - 1) / NT;   // chunks per thread
    constexpr int KK = HD / 16;                   // MFMA k-steps over the head dim
    constexpr int DT = HD / 32;                   // output d-tiles
    __shared__ Lds<HD> lds;

    const int s = blockIdx.x, h = blockIdx.y, i = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int q0 = a.qo[i];
    const int k_i = a.qo[i + 1] - q0;
    int kv_len = a.kv_lens[i];
    if (kv_len > a.max_kv_len) kv_len = a.max_kv_len;
    const int L = kv_len - k_i;
    if (k_i <= 0 || k_i > a.block || L < 0 || q0 < 0 || q0 + k_i > a.total_q) return;
    const int tok_begin = s * a.split;
    if (tok_begin >= kv_len) return;
    const int tok_end = min(kv_len, tok_begin + a.split);
    const int nsplit = (kv_len + a.split - 1) / a.split;
    const int M = a.G * k_i;

    // this lane's query row (N index of the MFMA) and its half (K-slice selector)
    const int r = w * 32 + (lane & 31);
    const int half = lane >> 5;
    const bool row_ok = r < M;
    const int jq = row_ok ? r / a.G : 0;
    const int head = h * a.G + (row_ok ? r % a.G : 0);
    const int limit = L + jq;  // last visible key of this row (inclusive)

    const uint16_t* __restrict__ qp = (const uint16_t*)a.q;
    const uint16_t* __restrict__ kcp = (const uint16_t*)a.kc;
    const uint16_t* __restrict__ vcp = (const uint16_t*)a.vc;
    const int32_t* __restrict__ pt = a.page_table + (size_t)i * a.maxp;

    bf16x8 qf[KK];
    {
        const uint16_t* src = qp + ((size_t)(q0 + jq) * a.Hq + head) * HD;
#pragma unroll
        for (int kk = 0; kk < KK; kk++) {
            u16x8 v = row_ok ? *(const u16x8*)(src + kk * 16 + half * 8) : u16x8{0, 0, 0, 0, 0, 0, 0, 0};
            qf[kk] = __builtin_bit_cast(bf16x8, v);
        }
    }

    f32x16 o[DT];
#pragma unroll
    for (int t = 0; t < DT; t++) o[t] = f32x16{};
    float m_run = -1e30f, l_run = 0.0f;

    // global -> register staging of one tile (K and V), zeros past the split end
    u16x8 kreg[CPT], vreg[CPT];
    auto load_tile = [&](int tb) {
#pragma unroll
        for (int c = 0; c < CPT; c++) {
            const int chunk = tid + c * NT;
            u16x8 kv = {0, 0, 0, 0, 0, 0, 0, 0}, vv = {0, 0, 0, 0, 0, 0, 0, 0};
            if (chunk < CHUNKS) {
                const int tok = tb + chunk / CPR;
                const int dc = (chunk % CPR) * 8;
                if (tok < tok_end) {
                    const int slot = tok >> a.log2P;
                    const int pg = slot < a.maxp ? pt[slot] : -1;
                    if (pg >= 0 && pg < a.num_pages) {
                        const size_t off = (((size_t)pg * a.Hkv + h) << a.log2P | (size_t)(tok & ((1 << a.log2P) - 1))) * HD + dc;
                        kv = *(const u16x8*)(kcp + off);
                        vv = *(const u16x8*)(vcp + off);
                    }
                }
            }
            kreg[c] = kv;
            vreg[c] = vv;
        }
    };
    auto store_tile = [&](int buf) {
#pragma unroll
        for (int c = 0; c < CPT; c++) {
            const int chunk = tid + c * NT;
            if (chunk < CHUNKS) {
                const int t = chunk / CPR;
                const int dc = (chunk % CPR) * 8;
                *(u16x8*)&lds.k[buf][t * Lds<HD>::kStride + dc] = kreg[c];
#pragma unroll
                for (int e = 0; e < 8; e++) lds.vt[buf][(dc + e) * Lds<HD>::vStride + t] = vreg[c][e];
            }
        }
    };

    const int ntiles = (tok_end - tok_begin + kTile - 1) / kTile;
    load_tile(tok_begin);
    store_tile(0);
    __syncthreads();

    for (int it = 0; it < ntiles; it++) {
        const int buf = it & 1;
        const int tb = tok_begin + it * kTile;
        if (it + 1 < ntiles) load_tile(tb + kTile);

        if (w * 32 < M) {
            // S^T = K Q^T for two 32-token halves of the tile
            f32x16 sacc[2];
#pragma unroll
            for (int tt = 0; tt < 2; tt++) {
                f32x16 acc = f32x16{};
                const uint16_t* krow = &lds.k[buf][(tt * 32 + (lane & 31)) * Lds<HD>::kStride + half * 8];
#pragma unroll
                for (int kk = 0; kk < KK; kk++) {
                    const bf16x8 af = __builtin_bit_cast(bf16x8, *(const u16x8*)(krow + kk * 16));
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, qf[kk], acc, 0, 0, 0);
                }
                sacc[tt] = acc;
            }
            // scale, causal/tail mask (register e of half tt holds token 32tt + 8(e/4) + 4*half + e%4)
            const bool need_mask = (tb + kTile - 1 > L) || (tb + kTile > tok_end) || !row_ok;
            float mx = -INFINITY;
#pragma unroll
            for (int tt = 0; tt < 2; tt++) {
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    float z = sacc[tt][e] * a.scale_log2;
                    if (need_mask) {
                        const int tok = tb + tt * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                        if (!row_ok || tok > limit || tok >= tok_end) z = -INFINITY;
                    }
                    sacc[tt][e] = z;
                    mx = fmaxf(mx, z);
                }
            }
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            const float m_new = fmaxf(m_run, mx);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            float psum = 0.0f;
#pragma unroll
            for (int tt = 0; tt < 2; tt++)
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    const float p = __builtin_amdgcn_exp2f(sacc[tt][e] - m_new);
                    sacc[tt][e] = p;
                    psum += p;
                }
            l_run = l_run * alpha + psum;
            m_run = m_new;
#pragma unroll
            for (int t = 0; t < DT; t++) o[t] *= alpha;

            // O^T += V^T P^T over four 16-token k-chunks
#pragma unroll
            for (int c = 0; c < 4; c++) {
                bf16x8 pb;
#pragma unroll
                for (int e = 0; e < 8; e++) pb[e] = (__bf16)sacc[c >> 1][8 * (c & 1) + e];
#pragma unroll
                for (int t = 0; t < DT; t++) {
                    const uint16_t* vrow = &lds.vt[buf][(t * 32 + (lane & 31)) * Lds<HD>::vStride + 16 * c + 4 * half];
                    const uint64_t lo = *(const uint64_t*)vrow;
                    const uint64_t hi = *(const uint64_t*)(vrow + 8);
                    u16x8 vv;
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        vv[e] = (uint16_t)(lo >> (16 * e));
                        vv[4 + e] = (uint16_t)(hi >> (16 * e));
                    }
                    o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vv), pb, o[t], 0, 0, 0);
                }
            }
        }

        if (it + 1 < ntiles) store_tile(buf ^ 1);
        __syncthreads();
    }

    if (!row_ok) return;
    const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
    const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
    const float lse2 = l_tot > 0.0f ? m_run + __log2f(l_tot) : -INFINITY;
    const size_t orow = (size_t)(q0 + jq) * a.Hq + head;
    if (nsplit == 1) {
        uint16_t* op = (uint16_t*)a.out + orow * HD;
#pragma unroll
        for (int t = 0; t < DT; t++)
#pragma unroll
            for (int g = 0; g < 4; g++) {
                const int dd = t * 32 + 8 * g + 4 * half;
                uint64_t pk = 0;
#pragma unroll
                for (int e = 0; e < 4; e++) pk |= (uint64_t)f2bf(o[t][4 * g + e] * inv) << (16 * e);
                *(uint64_t*)(op + dd) = pk;
            }
        if (a.lse && half == 0) a.lse[orow] = lse2 * kLn2;
    } else {
        float* pp = a.part_o + ((size_t)s * a.total_q * a.Hq + orow) * HD;
#pragma unroll
        for (int t = 0; t < DT; t++)
#pragma unroll
            for (int g = 0; g < 4; g++) {
                const int dd = t * 32 + 8 * g + 4 * half;
                f32x4 v = {o[t][4 * g] * inv, o[t][4 * g + 1] * inv, o[t][4 * g + 2] * inv, o[t][4 * g + 3] * inv};
                *(f32x4*)(pp + dd) = v;
            }
        if (half == 0) a.part_lse[(size_t)s * a.total_q * a.Hq + orow] = lse2;
    }
}

// merge split partials: one wavefront per (row, head); lanes over d
template <int HD, bool BF16OUT>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
    const int unit = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int K = a.qo[a.R];
    if (K > a.total_q) return;
    const int row = unit / a.Hq, head = unit % a.Hq;
    if (row >= K) return;
    // request of this row
    int lo = 0, hi = a.R - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.qo[mid] <= row) lo = mid; else hi = mid - 1;
    }
    const int i = lo;
    int kv_len = a.kv_lens[i];
    if (kv_len > a.max_kv_len) kv_len = a.max_kv_len;
    const int k_i = a.qo[i + 1] - a.qo[i];
    if (kv_len - k_i < 0 || k_i > a.block) return;
    const int nsplit = (kv_len + a.split - 1) / a.split;
    if (nsplit <= 1) return;
    const size_t orow = (size_t)row * a.Hq + head;
    const size_t sstride = (size_t)a.total_q * a.Hq;
    float mx = -INFINITY;
    for (int s = 0; s < nsplit; s++) mx = fmaxf(mx, a.part_lse[s * sstride + orow]);
    constexpr int PER = HD / 64 > 0 ? HD / 64 : 1;
    float acc[PER];
#pragma unroll
    for (int e = 0; e < PER; e++) acc[e] = 0.0f;
    float wsum = 0.0f;
    for (int s = 0; s < nsplit; s++) {
        const float l2 = a.part_lse[s * sstride + orow];
        const float wgt = l2 == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(l2 - mx);
        wsum += wgt;
        const float* src = a.part_o + (s * sstride + orow) * HD;
#pragma unroll
        for (int e = 0; e < PER; e++) {
            const int dd = lane + 64 * e;
            if (dd < HD) acc[e] += wgt * src[dd];
        }
    }
    const float inv = wsum > 0.0f ? 1.0f / wsum : 0.0f;
#pragma unroll
    for (int e = 0; e < PER; e++) {
        const int dd = lane + 64 * e;
        if (dd < HD) {
            if (BF16OUT) ((uint16_t*)a.out)[orow * HD + dd] = f2bf(acc[e] * inv);
            else ((float*)a.out)[orow * HD + dd] = acc[e] * inv;
        }
    }
    if (a.lse && lane == 0) a.lse[orow] = wsum > 0.0f ? (mx + __log2f(wsum)) * kLn2 : -INFINITY;
}

// ---------------------------------------------------------------------------------
// fp32 vector kernel: one wavefront per (query row, head); HD <= 256, HD % 4 == 0
// ---------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void attn_f32_kernel(AttnArgs a, int HD) {
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int unit = blockIdx.x * 4 + wv;
    const int K = a.qo[a.R];
    if (K > a.total_q) return;
    const int row = unit / a.Hq, head = unit % a.Hq;
    if (row >= K) return;
    int lo = 0, hi = a.R - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.qo[mid] <= row) lo = mid; else hi = mid - 1;
    }
    const int i = lo;
    const int k_i = a.qo[i + 1] - a.qo[i];
    int kv_len = a.kv_lens[i];
    if (kv_len > a.max_kv_len) kv_len = a.max_kv_len;
    const int L = kv_len - k_i;
    if (L < 0 || k_i > a.block) return;
    const int limit = L + (row - a.qo[i]);
    const int kvh = head / a.G;
    const float* qp = (const float*)a.q + ((size_t)row * a.Hq + head) * HD;  // wave-uniform
    const float* kcp = (const float*)a.kc;
    const float* vcp = (const float*)a.vc;
    const int32_t* pt = a.page_table + (size_t)i * a.maxp;
    const int P = 1 << a.log2P;
    float o[4] = {0.f, 0.f, 0.f, 0.f};
    float m = -INFINITY, l = 0.0f;
    for (int base = 0; base <= limit; base += 64) {
        const int sk = base + lane;
        float z = -INFINITY;
        size_t off = 0;
        bool ok = false;
        if (sk <= limit) {
            const int slot = sk >> a.log2P;
            const int pg = slot < a.maxp ? pt[slot] : -1;
            if (pg >= 0 && pg < a.num_pages) {
                off = (((size_t)pg * a.Hkv + kvh) * P + (sk & (P - 1))) * HD;
                float dot = 0.0f;
                for (int e = 0; e < HD; e += 4) {
                    const f32x4 kv4 = *(const f32x4*)(kcp + off + e);
                    dot += qp[e] * kv4[0] + qp[e + 1] * kv4[1] + qp[e + 2] * kv4[2] + qp[e + 3] * kv4[3];
                }
                z = dot * a.scale;
                ok = true;
            }
        }
        float mx = z;
        for (int x = 32; x > 0; x >>= 1) mx = fmaxf(mx, __shfl_xor(mx, x, 64));
        const float m_new = fmaxf(m, mx);
        if (m_new == -INFINITY) continue;
        const float alpha = m == -INFINITY ? 0.0f : expf(m - m_new);
        const float p = ok ? expf(z - m_new) : 0.0f;
        float ps = p;
        for (int x = 32; x > 0; x >>= 1) ps += __shfl_xor(ps, x, 64);
        l = l * alpha + ps;
        m = m_new;
        for (int e = 0; e < 4; e++) o[e] *= alpha;
        const int cnt = min(64, limit - base + 1);
        for (int jj = 0; jj < cnt; jj++) {
            const float pj = __shfl(p, jj, 64);
            const int okj = __shfl((int)ok, jj, 64);
            if (!okj) continue;
            const size_t offj = __shfl((unsigned long long)off, jj, 64);
            for (int e = 0; e < 4; e++) {
                const int dd = lane + 64 * e;
                if (dd < HD) o[e] += pj * vcp[offj + dd];
            }
        }
    }
    float* op = (float*)a.out + ((size_t)row * a.Hq + head) * HD;
    const float inv = l > 0.0f ? 1.0f / l : 0.0f;
    for (int e = 0; e < 4; e++) {
        const int dd = lane + 64 * e;
        if (dd < HD) op[dd] = o[e] * inv;
    }
    if (a.lse && lane == 0) a.lse[(size_t)row * a.Hq + head] = l > 0.0f ? m + logf(l) : -INFINITY;
}

int ilog2(int x) {
    int r = 0;
    while ((1 << r) < x) r++;
    return r;
}

}  // namespace

AttnPlan plan_attn(const sv_attn_desc& d) {
    AttnPlan p{};
    const int maxM = (d.num_q_heads / d.num_kv_heads) * d.block;
    p.waves = maxM <= 64 ? 2 : (maxM <= 128 ? 4 : 8);
    if (d.dtype == SV_F32) {
        p.kv_split = 0;
        p.max_splits = 1;
        return p;
    }
    int split = d.kv_split;
    if (split <= 0) {
        // aim for ~2048 work items over the worst case (every request at max_kv_len)
        const long long work = (long long)d.num_reqs * d.num_kv_heads;
        long long want = (long long)d.max_kv_len * work / 2048;
        if (want < 1024) want = 1024;
        split = (int)(((want + 63) / 64) * 64);
    }
    if (split > d.max_kv_len) split = ((d.max_kv_len + 63) / 64) * 64;
    if (split < 64) split = 64;
    p.kv_split = split;
    p.max_splits = (d.max_kv_len + split - 1) / split;
    if (p.max_splits < 1) p.max_splits = 1;
    if (p.max_splits > 1) {
        p.part_o_bytes = (size_t)p.max_splits * d.total_q_max * d.num_q_heads * d.head_dim * sizeof(float);
        p.part_lse_bytes = (size_t)p.max_splits * d.total_q_max * d.num_q_heads * sizeof(float);
    }
    return p;
}

hipError_t launch_attn(const sv_attn_desc& d, const AttnPlan& plan, const void* q,
                       const void* k_cache, const void* v_cache, const int32_t* page_table,
                       const int32_t* qo_indptr, const int32_t* kv_lens, void* out, float* lse,
                       void* ws, hipStream_t stream) {
    AttnArgs a{};
    a.q = q;
    a.kc = k_cache;
    a.vc = v_cache;
    a.page_table = page_table;
    a.qo = qo_indptr;
    a.kv_lens = kv_lens;
    a.out = out;
    a.lse = lse;
    a.part_o = plan.part_o_bytes ? (float*)ws : nullptr;
    a.part_lse = plan.part_o_bytes ? (float*)((char*)ws + plan.part_o_bytes) : nullptr;
    a.R = d.num_reqs;
    a.total_q = d.total_q_max;
    a.Hq = d.num_q_heads;
    a.Hkv = d.num_kv_heads;
    a.G = d.num_q_heads / d.num_kv_heads;
    a.block = d.block;
    a.log2P = ilog2(d.page_size);
    a.maxp = d.max_pages_per_req;
    a.num_pages = d.num_pages;
    a.max_kv_len = d.max_kv_len;
    a.split = plan.kv_split;
    a.max_splits = plan.max_splits;
    a.scale = d.sm_scale > 0.0f ? d.sm_scale : 1.0f / sqrtf((float)d.head_dim);
    a.scale_log2 = a.scale * kLog2e;

    if (d.dtype == SV_F32) {
        const int units = d.total_q_max * d.num_q_heads;
        hipLaunchKernelGGL(attn_f32_kernel, dim3((units + 3) / 4), dim3(256), 0, stream, a, d.head_dim);
        return hipGetLastError();
    }
    const dim3 grid(plan.max_splits, d.num_kv_heads, d.num_reqs);
#define SV_LAUNCH_ATTN(HDV, NWV) \
    hipLaunchKernelGGL((attn_bf16_kernel<HDV, NWV>), grid, dim3(NWV * 64), 0, stream, a)
    if (d.head_dim == 128) {
        if (plan.waves == 2) SV_LAUNCH_ATTN(128, 2);
        else if (plan.waves == 4) SV_LAUNCH_ATTN(128, 4);
        else SV_LAUNCH_ATTN(128, 8);
    } else {
        if (plan.waves == 2) SV_LAUNCH_ATTN(64, 2);
        else if (plan.waves == 4) SV_LAUNCH_ATTN(64, 4);
        else SV_LAUNCH_ATTN(64, 8);
    }
#undef SV_LAUNCH_ATTN
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || plan.max_splits <= 1) return e;
    const int units = d.total_q_max * d.num_q_heads;
    if (d.head_dim == 128)
        hipLaunchKernelGGL((attn_merge_kernel<128, true>), dim3((units + 3) / 4), dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL((attn_merge_kernel<64, true>), dim3((units + 3) / 4), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace sv
