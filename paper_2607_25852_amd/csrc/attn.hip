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
// fp32 path (vector ALU): one workgroup per (query row, head); its four waves take
// interleaved 64-key tiles and merge their softmax states at the end.
#include <atomic>

#include "attn_plan.h"
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
static_assert(kTile == kAttnTile, "the work plan counts tiles of the kernel's size");

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
    int split, max_splits, nrb;  // nrb: row blocks (16 rows per wave) per (request, kv-head)
    int max_items;               // R * max_splits * Hkv * nrb (capped at INT_MAX): the longest work list
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
// ---------------------------------------------------------------------------------
// LDS tile layout: a 64-token tile of K and of V, each [token][HD] bf16, rows of HD*2
// bytes with their 16-byte chunks XOR-swizzled: logical chunk c of token t sits at
// position c ^ swz(t). swz swaps the two 2-bit fields of t % 16 so that (a) the 16
// rows read together by one quarter-wave of the K-operand loads hit 16 different chunk
// positions and (b) the 4 rows x 4 chunks read by one half-wave of the transpose reads
// (two 16-lane groups) do too.
// ---------------------------------------------------------------------------------
__device__ __host__ inline int swz(int t) { return ((t & 3) << 2) | ((t >> 2) & 3); }

template <int HD, int NBUF>
struct LdsRing {
    static constexpr int kTileBytes = kTile * HD * 2;  // one tensor
    static constexpr int kMaxSlots = 1024;              // page-table entries of one split
    uint16_t kv[NBUF][2][kTile * HD];                   // [buffer][K=0/V=1][token*HD + d]
    int32_t pid[kMaxSlots];
};

// Asynchronous 16-byte-per-lane copy global -> LDS: lane l's 16 bytes land at
// lds_base + 16*l. Issued from inline assembly so the compiler does not drain it
// before every LDS read; completion is awaited explicitly with wait_vm<N>(). The
// loads carry the non-temporal hint: every K/V byte is read by one workgroup once,
// so keeping it in L2 and the last-level cache only evicts lines that are reused.
__device__ inline void dma16(const void* gptr, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(gptr), "s"(lds_base)
                 : "memory", "m0");
}
// Same copy with a wave-uniform 64-bit base in SGPRs and a 32-bit per-lane byte offset.
__device__ inline void dma16s(uint32_t voff, const void* sbase, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(sbase),
                 "s"(lds_base)
                 : "memory", "m0");
}
template <int N>
__device__ inline void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// One work item (request i, kv-head h, split s, up to (NW/HALVES)*32 query rows from row0
// of the kv-head group). NBUF-deep LDS ring:
// tile t is multiplied while tiles t+1 .. t+NBUF-1 stream in. HALVES == 2: wave w owns
// query rows 32*(w/2) .. +31 of the row block and token half w%2 of every tile (so a
// 64-row group keeps all four SIMDs busy, two waves each); the two halves of a row group
// merge their softmax states at the end. HALVES == 1: wave w owns rows 32*w .. +31 over
// the whole tile (256 rows per workgroup). Every early return is uniform over the
// workgroup.
template <int HD, int NW, int NBUF, bool ONEPAGE, int HALVES>
__device__ __forceinline__ void attn_item(const AttnArgs& a, LdsRing<HD, NBUF>& lds, int i, int h, int s, int row0) {
    constexpr int CPR = HD / 8;             // 16-byte chunks per token row
    constexpr int TPS = 1024 / (HD * 2);    // tokens per 1 KB DMA segment
    constexpr int NSEG = kTile / TPS;       // segments per tensor per tile
    constexpr int IPW = 2 * NSEG / NW;      // DMA instructions per wave per tile
    static_assert(IPW * NW == 2 * NSEG, "DMA split");
    constexpr int KK = HD / 16;             // MFMA k-steps over the head dim
    constexpr int DT = HD / 32;             // output d-tiles
    constexpr int PF = NBUF - 1;            // prefetch distance in tiles

    // The thread id passes through an empty asm statement, so the per-lane values derived
    // from it (LDS and DMA offsets) are recomputed per item instead of being hoisted out
    // of the persistent item loop, where the invariants of both wave mappings would stay
    // live together (252 VGPRs instead of about 220, leaving no room for the operand
    // prefetch in compute_tile).
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, w = tid >> 6;
    const int q0 = a.qo[i];
    const int k_i = a.qo[i + 1] - q0;
    int kv_len = a.kv_lens[i];
    if (kv_len > a.max_kv_len) kv_len = a.max_kv_len;
    const int L = kv_len - k_i;
    // (bitwise or: both descriptor loads are issued before the test)
    if ((k_i <= 0) | (k_i > a.block) | (L < 0) | (q0 < 0) | (q0 + k_i > a.total_q)) return;
    const int tok_begin = s * a.split;
    if (tok_begin >= kv_len) return;
    const int tok_end = min(kv_len, tok_begin + a.split);
    const int nsplit = (kv_len + a.split - 1) / a.split;
    constexpr int RB = (NW / HALVES) * 32;    // query rows this mapping covers
    const int M = min(a.G * k_i - row0, RB);  // rows of this item
    if (M <= 0) return;

    // page ids of this split -> LDS (the host keeps a split within 1024 pages). The first
    // page id of each thread is loaded before the query fragments and stored after them,
    // so the two round trips overlap.
    const int slot0 = tok_begin >> a.log2P;
    const int nslots = ((tok_end - 1) >> a.log2P) - slot0 + 1;
    const int32_t* __restrict__ pt = a.page_table + (size_t)i * a.maxp;
    int pg0 = -1;
    if (tid < nslots && slot0 + tid < a.maxp) pg0 = pt[slot0 + tid];

    // this lane's query row (N index of the MFMA) and its half (K-slice selector)
    // row group; token half of each tile (HALVES == 2), else the whole tile
    const int rg = w / HALVES, th = HALVES == 2 ? (w & 1) : 0;
    const int r = rg * 32 + (lane & 31);
    const int half = lane >> 5;
    const bool row_ok = r < M;
    const int rr = row0 + (row_ok ? r : 0);  // row within the request's kv-head group
    const int jq = rr / a.G;
    const int head = h * a.G + rr % a.G;
    const int limit = L + jq;  // last visible key of this row (inclusive)
    const int last_key = min(limit, tok_end - 1);  // ... and of this split

    // Per-lane element offsets of the V^T transpose reads inside a tile's V buffer: read
    // (qh, d-tile t) of 16-token k-chunk c lies at 16c*HD + vofs[qh][t] (for half-tile waves
    // c counts from their own half, whose offset vofs includes). The swizzle sees only the
    // token's position mod 16, which c does not change, so these 2*DT values serve every
    // chunk of every tile and each read costs one add of the buffer base.
    int vofs[2][DT];
    {
        const int g = lane >> 4, jl = lane & 15;
#pragma unroll
        for (int qh = 0; qh < 2; qh++) {
            const int tl = 8 * qh + 4 * (g >> 1) + (jl >> 2);  // token mod 16
#pragma unroll
            for (int t = 0; t < DT; t++) {
                const int dd = 32 * t + 16 * (g & 1) + 4 * (jl & 3);
                vofs[qh][t] = (HALVES == 2 ? th * 32 * HD : 0) + tl * HD +
                              (((dd >> 3) ^ (swz(tl) & (CPR - 1))) << 3) + (dd & 7);
            }
        }
    }
    const uint16_t* __restrict__ qp = (const uint16_t*)a.q;
    const uint16_t* __restrict__ kcp = (const uint16_t*)a.kc;
    const uint16_t* __restrict__ vcp = (const uint16_t*)a.vc;
    bf16x8 qf[KK];
    {
        const uint16_t* src = qp + ((size_t)(q0 + jq) * a.Hq + head) * HD;
#pragma unroll
        for (int kk = 0; kk < KK; kk++) {
            u16x8 v = row_ok ? *(const u16x8*)(src + kk * 16 + half * 8) : u16x8{0, 0, 0, 0, 0, 0, 0, 0};
            qf[kk] = __builtin_bit_cast(bf16x8, v);
        }
    }
    if (tid < nslots) lds.pid[tid] = (pg0 >= 0 && pg0 < a.num_pages) ? pg0 : -1;
    for (int e = tid + NW * 64; e < nslots; e += NW * 64) {
        const int slot = slot0 + e;
        const int pg = slot < a.maxp ? pt[slot] : -1;
        lds.pid[e] = (pg >= 0 && pg < a.num_pages) ? pg : -1;
    }
    // the query fragments must have landed before the DMA ring starts: a wait the
    // compiler sees (vmcnt(0)) keeps it from re-checking them inside the loop, where
    // a vmcnt(0) would also drain the ring
    __builtin_amdgcn_s_waitcnt(0x0F70);
    f32x16 o[DT];
#pragma unroll
    for (int t = 0; t < DT; t++) o[t] = f32x16{};
    float m_run = -1e30f, l_run = 0.0f;

    const size_t head_off = (size_t)h << a.log2P;
    const int pmask = (1 << a.log2P) - 1;
    const uint32_t lds_ring = (uint32_t)(uintptr_t)&lds.kv[0][0][0];
    __syncthreads();  // page ids visible

    // DMA of one tile: wave w issues segments w*IPW .. w*IPW+IPW-1 of the 2*NSEG
    // (K segments first, then V). Lane l of a segment moves token row t = seg*TPS + l/CPR,
    // position l%CPR, fetching logical chunk (l%CPR) ^ swz(t); the per-lane byte offset of
    // that chunk inside the tile is loop-invariant.
    // ONEPAGE (page size >= 64): a 64-token tile lies inside one page, so each tile needs
    // one wave-uniform base address; an invalid page reads page 0 (always present).
    // Otherwise every lane looks its page up; tokens past the split end or on an invalid
    // page read the first element of the cache. Either way such tokens are masked out of
    // the scores and zeroed in the V operand.
    uint32_t voff[IPW], ldsoff[IPW];
    int tk[IPW];
#pragma unroll
    for (int k = 0; k < IPW; k++) {
        const int n = w * IPW + k;
        const int seg = n % NSEG;
        const int t = seg * TPS + lane / CPR;
        tk[k] = t;
        voff[k] = (uint32_t)(t * HD + (((lane % CPR) ^ (swz(t) & (CPR - 1))) << 3)) * 2u;
        ldsoff[k] = (uint32_t)__builtin_amdgcn_readfirstlane((n / NSEG) * LdsRing<HD, NBUF>::kTileBytes + seg * 1024);
    }
    const int my_tensor = __builtin_amdgcn_readfirstlane((w * IPW) / NSEG);  // a wave moves one tensor
    const uint16_t* cbase = my_tensor ? vcp : kcp;
    auto issue_tile = [&](int tile, int buf) {
        const int tb = tok_begin + tile * kTile;
        const uint32_t lbuf = lds_ring + (uint32_t)(buf * 2 * LdsRing<HD, NBUF>::kTileBytes);
        if constexpr (ONEPAGE) {
            const int pg = __builtin_amdgcn_readfirstlane(lds.pid[(tb >> a.log2P) - slot0]);
            const uint16_t* base = pg >= 0
                ? cbase + ((((size_t)pg * a.Hkv) << a.log2P) + head_off + (size_t)(tb & pmask)) * HD
                : cbase + (size_t)(tb & pmask) * HD;
#pragma unroll
            for (int k = 0; k < IPW; k++) dma16s(voff[k], base, lbuf + ldsoff[k]);
        } else {
#pragma unroll
            for (int k = 0; k < IPW; k++) {
                const int tok = tb + tk[k];
                const int pg = lds.pid[min((tok >> a.log2P) - slot0, nslots - 1)];
                const uint16_t* src = (tok < tok_end && pg >= 0)
                    ? cbase + ((((size_t)pg * a.Hkv) << a.log2P) + head_off + (size_t)(tok & pmask)) * HD
                          + (voff[k] / 2 - tk[k] * HD)
                    : cbase;
                dma16(src, lbuf + ldsoff[k]);
            }
        }
    };

    constexpr int NSB = 2 / HALVES;  // 32-token halves of a tile handled by this wave
    auto compute_tile = [&](int buf, int tb) {
        if (rg * 32 >= M) return;
        const uint16_t* kt = lds.kv[buf][0];
        const uint16_t* vt = lds.kv[buf][1];
        // S^T = K Q^T for each 32-token half this wave owns (unscaled), as two independent
        // accumulation chains: the two halves (whole-tile waves), or the even and odd
        // k-steps of one half. Each K fragment is read from LDS KPD MFMAs before the MFMA
        // that consumes it; the scheduling barriers keep that order, so the LDS latency
        // runs under the matrix pipe instead of stalling every MFMA.
        f32x16 sacc[NSB];
        {
            const int sw = swz(lane & 31) & (CPR - 1);  // swz depends on t % 16 only
            const uint16_t* krow0 = kt + ((HALVES == 2 ? th : 0) * 32 + (lane & 31)) * HD;
            constexpr int NF = NSB * KK;  // K fragments (= MFMAs) per tile
            constexpr int KPD = 4;
            // fragment j: whole-tile waves alternate the token halves (j % 2) at k-step j / 2;
            // half-tile waves take k-step j of their half
            auto kaddr = [&](int j) {
                if constexpr (NSB == 2) return krow0 + (j & 1) * 32 * HD + (((2 * (j >> 1) + half) ^ sw) << 3);
                else return krow0 + (((2 * j + half) ^ sw) << 3);
            };
            bf16x8 kb[KPD + 1];
            f32x16 c0 = f32x16{}, c1 = f32x16{};
#pragma unroll
            for (int j = 0; j < KPD; j++) kb[j] = __builtin_bit_cast(bf16x8, *(const u16x8*)kaddr(j));
#pragma unroll
            for (int j = 0; j < NF; j++) {
                if (j + KPD < NF) kb[(j + KPD) % (KPD + 1)] = __builtin_bit_cast(bf16x8, *(const u16x8*)kaddr(j + KPD));
                __builtin_amdgcn_sched_barrier(0);
                const bf16x8 bq = NSB == 2 ? qf[j >> 1] : qf[j];
                if (j & 1) c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb[j % (KPD + 1)], bq, c1, 0, 0, 0);
                else c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb[j % (KPD + 1)], bq, c0, 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (NSB == 2) {
                sacc[0] = c0;
                sacc[1] = c1;
            } else {
                sacc[0] = c0 + c1;
            }
        }
        if constexpr (NSB == 2) {
            // Causal/tail mask on the raw scores: register e of half hh holds token
            // tb + 32hh + 4*half + (8(e/4) + e%4), masked when that token is past the row's last
            // visible key or the split end. Only halves reaching past L (the first row's limit)
            // or the split end need it, a wave-uniform test. Padding rows (r >= M) are not
            // masked: their query is zero, and their output column is neither written nor
            // mixed into the other columns.
    #pragma unroll
            for (int sb = 0; sb < NSB; sb++) {
                const int tb_h = tb + (HALVES == 2 ? th : sb) * 32;
                if (tb_h + 31 > L || tb_h + 32 > tok_end) {
                    const int dlim = last_key - tb_h - 4 * half;  // mask where 8(e/4) + e%4 > dlim
    #pragma unroll
                    for (int e = 0; e < 16; e++)
                        if (8 * (e >> 2) + (e & 3) > dlim) sacc[sb][e] = -INFINITY;
                }
            }
            // One online-softmax step per tile over the owned halves: the row max (lane-local,
            // then across the lane halves: the row's other 16 scores sit in lane l ^ 32, and
            // v_permlane32_swap with both operands = mx returns the lower half's values in one
            // result and the upper half's in the other), then a lazy rescale: the running max
            // moves only when a score exceeds it by more than 8 (log2 units), so p = 2^(z - m)
            // <= 256 stays exact in fp32 and bf16, and most tiles skip the accumulator rescale.
            float mx = fmaxf(fmaxf(sacc[0][0], sacc[0][1]), sacc[0][2]);
    #pragma unroll
            for (int e = 3; e < 15; e += 2) mx = fmaxf(fmaxf(mx, sacc[0][e]), sacc[0][e + 1]);
            mx = fmaxf(mx, sacc[0][15]);
            if constexpr (NSB == 2) {
    #pragma unroll
                for (int e = 0; e < 16; e += 2) mx = fmaxf(fmaxf(mx, sacc[1][e]), sacc[1][e + 1]);
            }
            {
                const auto sw2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
                mx = fmaxf(__uint_as_float(sw2[0]), __uint_as_float(sw2[1]));
            }
            const float mxs = mx * a.scale_log2;  // max in scaled log2 units (-inf: all masked)
            if (__any(mxs > m_run + 8.0f)) {
                const float m_new = fmaxf(m_run, mxs);
                const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
                l_run *= alpha;
    #pragma unroll
                for (int t = 0; t < DT; t++) o[t] *= alpha;
                m_run = m_new;
            }
            const float nm = -m_run;

            // O^T += V^T P^T. MFMA J of the tile: half J / NJ (whole-tile waves; else this
            // wave's half), 16-token k-chunk (J % NJ) / DT of that half, d-tile J % DT. The V^T
            // operand comes from two transpose reads: in 16-lane group g = lane/16, input lane
            // jl addresses token 16c + 8q + 4(g/2) + jl/4 at dims 32t + 16(g%2) + 4(jl%4) .. +3,
            // and output lane jl receives dim 32t + 16(g%2) + jl of tokens 16c + 8q + 4(g/2) +
            // 0..3. The operands are read VPD MFMAs ahead; the first VPD are in flight while the
            // exponents of the first half are computed.
            const int g = lane >> 4, jl = lane & 15;
            constexpr int NJ = 2 * DT;    // PV MFMAs per 32-token half
            constexpr int NT = NSB * NJ;  // PV MFMAs per tile for this wave
            constexpr int VPD = 4;
            auto vread = [&](int J) {
                const int c = 2 * (J / NJ) + (J % NJ) / DT, t = J % DT;  // (whole-tile waves)
                i16x4 vq[2];
    #pragma unroll
                for (int qh = 0; qh < 2; qh++) {
                    const uint16_t* addr = vt + 16 * c * HD + vofs[qh][t];
                    vq[qh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)addr);
                }
                return __builtin_shufflevector(vq[0], vq[1], 0, 1, 2, 3, 4, 5, 6, 7);
            };
            i16x8 vb[VPD + 1];
    #pragma unroll
            for (int j = 0; j < VPD; j++) vb[j] = vread(j);
            __builtin_amdgcn_sched_barrier(0);
            // p = 2^(z * scale * log2e - m) of the first half, its row sum, and the bf16 P^T
            // fragments (already in the B-operand layout)
            float ps0 = 0.0f, ps1 = 0.0f;
    #pragma unroll
            for (int e = 0; e < 16; e++) {
                sacc[0][e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[0][e], a.scale_log2, nm));
                ps0 += sacc[0][e];
            }
            bf16x8 pb[NSB][2];
    #pragma unroll
            for (int cc = 0; cc < 2; cc++)
    #pragma unroll
                for (int e = 0; e < 8; e++) pb[0][cc][e] = (__bf16)sacc[0][8 * cc + e];
            __builtin_amdgcn_sched_barrier(0);
            // PV MFMAs. Whole-tile waves compute the second half's exponents between the first
            // half's MFMAs (16 / NJ per MFMA), so the vector ALU works under the matrix pipe.
    #pragma unroll
            for (int J = 0; J < NT; J++) {
                if (J + VPD < NT) vb[(J + VPD) % (VPD + 1)] = vread(J + VPD);
                __builtin_amdgcn_sched_barrier(0);
                const int t = J % DT;
                o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vb[J % (VPD + 1)]),
                                                                pb[J / NJ][(J % NJ) / DT], o[t], 0, 0, 0);
                if constexpr (NSB == 2) {
                    if (J < NJ) {
                        constexpr int EPM = 16 / NJ;
    #pragma unroll
                        for (int x = 0; x < EPM; x++) {
                            const int e = EPM * J + x;
                            sacc[1][e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[1][e], a.scale_log2, nm));
                            ps1 += sacc[1][e];
                        }
                        if (J == NJ - 1) {
    #pragma unroll
                            for (int cc = 0; cc < 2; cc++)
    #pragma unroll
                                for (int e = 0; e < 8; e++) pb[1][cc][e] = (__bf16)sacc[1][8 * cc + e];
                        }
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            l_run += ps0 + ps1;
        } else {
            // Half-tile waves: one online-softmax step per tile on the wave's half.
            const int g = lane >> 4, jl = lane & 15;
            const int hh = th;
            const int tb_h = tb + hh * 32;
            if (tb_h + 31 > L || tb_h + 32 > tok_end) {
                const int dlim = last_key - tb_h - 4 * half;  // mask where 8(e/4) + e%4 > dlim
#pragma unroll
                for (int e = 0; e < 16; e++)
                    if (8 * (e >> 2) + (e & 3) > dlim) sacc[0][e] = -INFINITY;
            }
            float mx = fmaxf(fmaxf(sacc[0][0], sacc[0][1]), sacc[0][2]);
#pragma unroll
            for (int e = 3; e < 15; e += 2) mx = fmaxf(fmaxf(mx, sacc[0][e]), sacc[0][e + 1]);
            mx = fmaxf(mx, sacc[0][15]);
            {
                const auto sw2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
                mx = fmaxf(__uint_as_float(sw2[0]), __uint_as_float(sw2[1]));
            }
            const float mxs = mx * a.scale_log2;
            if (__any(mxs > m_run + 8.0f)) {
                const float m_new = fmaxf(m_run, mxs);
                const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
                l_run *= alpha;
#pragma unroll
                for (int t = 0; t < DT; t++) o[t] *= alpha;
                m_run = m_new;
            }
            constexpr int NJ = 2 * DT;
            constexpr int VPD = 4;
            auto vread = [&](int j) {
                const int c = j / DT, t = j % DT;  // chunk within the wave's half
                i16x4 vq[2];
#pragma unroll
                for (int qh = 0; qh < 2; qh++) {
                    const uint16_t* addr = vt + 16 * c * HD + vofs[qh][t];
                    vq[qh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)addr);
                }
                return __builtin_shufflevector(vq[0], vq[1], 0, 1, 2, 3, 4, 5, 6, 7);
            };
            i16x8 vb[VPD + 1];
#pragma unroll
            for (int j = 0; j < VPD; j++) vb[j] = vread(j);
            __builtin_amdgcn_sched_barrier(0);
            const float nm = -m_run;
            float psum = 0.0f;
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[0][e], a.scale_log2, nm));
                sacc[0][e] = p;
                psum += p;
            }
            l_run += psum;
            bf16x8 pb[2];
#pragma unroll
            for (int cc = 0; cc < 2; cc++)
#pragma unroll
                for (int e = 0; e < 8; e++) pb[cc][e] = (__bf16)sacc[0][8 * cc + e];
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int j = 0; j < NJ; j++) {
                if (j + VPD < NJ) vb[(j + VPD) % (VPD + 1)] = vread(j + VPD);
                __builtin_amdgcn_sched_barrier(0);
                const int t = j % DT;
                o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vb[j % (VPD + 1)]), pb[j / DT],
                                                                o[t], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };

    // pipeline: before multiplying tile t, wait until its DMA (and only its) is done,
    // barrier (tile t visible to all waves; tile t-1 no longer read), then refill the
    // buffer of tile t-1 with tile t+PF.
    const int ntiles = (tok_end - tok_begin + kTile - 1) / kTile;
#pragma unroll
    for (int t = 0; t < PF; t++)
        if (t < ntiles) issue_tile(t, t);
    for (int t = 0; t < ntiles; t++) {
        const int newer = min(PF - 1, ntiles - 1 - t);  // tiles issued after t
        if constexpr (PF >= 3) {
            if (newer >= 2) wait_vm<2 * IPW>();
            else if (newer == 1) wait_vm<IPW>();
            else wait_vm<0>();
        } else {
            if (newer >= 1) wait_vm<IPW>();
            else wait_vm<0>();
        }
        // the last tile may reach past the split end: the lanes that copied those V rows
        // (foreign data, possibly non-finite) zero them, so P = 0 there contributes exactly 0
        if (t == ntiles - 1 && tok_begin + (t + 1) * kTile > tok_end && my_tensor == 1) {
            const int tb = tok_begin + t * kTile;
            char* vbuf = (char*)&lds.kv[0][0][0] + (t % NBUF) * 2 * LdsRing<HD, NBUF>::kTileBytes;
#pragma unroll
            for (int k = 0; k < IPW; k++)
                if (tb + tk[k] >= tok_end) *(u16x8*)(vbuf + ldsoff[k] + 16 * lane) = u16x8{};
        }
        __syncthreads();
        if (t + PF < ntiles) issue_tile(t + PF, (t + PF) % NBUF);
        compute_tile(t % NBUF, tok_begin + t * kTile);
    }

    // HALVES == 2: merge the token halves of each row group. The odd wave parks O in the
    // ring and (m, l) in the page-id area (both free now), the even wave combines and
    // writes. Both waves hold the same (row, dim) elements in the same lanes and registers.
    float l_tot = l_run + __shfl_xor(l_run, 32, 64);
    const bool grp_ok = rg * 32 < M;
    if constexpr (HALVES == 2) {
        static_assert((NW / 2) * 64 * 16 * DT * sizeof(float) <= sizeof(lds.kv), "park O");
        static_assert((NW / 2) * 96 * sizeof(float) <= sizeof(lds.pid), "park m, l");
        __syncthreads();
        float* park = (float*)&lds.kv[0][0][0] + (size_t)rg * (64 * 16 * DT);
        float* park_ml = (float*)&lds.pid[0] + rg * 96;
        if (grp_ok && th == 1) {
#pragma unroll
            for (int t = 0; t < DT; t++)
#pragma unroll
                for (int e = 0; e < 16; e++) park[(t * 16 + e) * 64 + lane] = o[t][e];
            park_ml[lane] = m_run;
            if (lane < 32) park_ml[64 + lane] = l_tot;  // rows in lanes 0..31
        }
        __syncthreads();
        if (!grp_ok || th == 1 || !row_ok) return;
        const float m2 = park_ml[lane];
        const float l2 = park_ml[64 + (lane & 31)];
        const float mm = fmaxf(m_run, m2);
        const float a1 = __builtin_amdgcn_exp2f(m_run - mm), a2 = __builtin_amdgcn_exp2f(m2 - mm);
#pragma unroll
        for (int t = 0; t < DT; t++)
#pragma unroll
            for (int e = 0; e < 16; e++) o[t][e] = o[t][e] * a1 + park[(t * 16 + e) * 64 + lane] * a2;
        l_tot = l_tot * a1 + l2 * a2;
        m_run = mm;
    } else {
        if (!grp_ok || !row_ok) return;
    }
    const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
    const float lse2 = l_tot > 0.0f ? m_run + __log2f(l_tot) : -INFINITY;
    const size_t orow = (size_t)(q0 + jq) * a.Hq + head;
    if (nsplit == 1) {
        uint16_t* op = (uint16_t*)a.out + orow * HD;
#pragma unroll
        for (int t = 0; t < DT; t++)
#pragma unroll
            for (int g2 = 0; g2 < 4; g2++) {
                const int dd = t * 32 + 8 * g2 + 4 * half;
                uint64_t pk = 0;
#pragma unroll
                for (int e = 0; e < 4; e++) pk |= (uint64_t)f2bf(o[t][4 * g2 + e] * inv) << (16 * e);
                *(uint64_t*)(op + dd) = pk;
            }
        if (a.lse && half == 0) a.lse[orow] = lse2 * kLn2;
    } else {
        float* pp = a.part_o + ((size_t)s * a.total_q * a.Hq + orow) * HD;
#pragma unroll
        for (int t = 0; t < DT; t++)
#pragma unroll
            for (int g2 = 0; g2 < 4; g2++) {
                const int dd = t * 32 + 8 * g2 + 4 * half;
                f32x4 v = {o[t][4 * g2] * inv, o[t][4 * g2 + 1] * inv, o[t][4 * g2 + 2] * inv, o[t][4 * g2 + 3] * inv};
                *(f32x4*)(pp + dd) = v;
            }
        if (half == 0) a.part_lse[(size_t)s * a.total_q * a.Hq + orow] = lse2;
    }
}

// Work list of the persistent kernel (attn_plan.h), built by one workgroup.
__global__ __launch_bounds__(1024) void attn_plan_kernel(AttnArgs a, int32_t* groups, int32_t* ctr) {
    __shared__ int cursor[kPlanBuckets];
    __shared__ int wsum[1024 / 64];
    AttnPlanArgs pa{a.R, a.block, a.total_q, a.max_kv_len, a.split, a.Hkv, a.nrb, groups, ctr};
    build_attn_plan<1024>(pa, [&](int i, int& q0, int& k_i, int& kv) {
        q0 = a.qo[i];
        k_i = a.qo[i + 1] - q0;
        kv = a.kv_lens[i];
    }, cursor, wsum);
}

template <int HD, int NW, int NBUF, bool ONEPAGE, bool WIDE>
__global__ __launch_bounds__(NW * 64, 1) void attn_bf16_kernel(AttnArgs a, const int32_t* __restrict__ groups,
                                                               int32_t* __restrict__ ctr) {
    __shared__ __attribute__((aligned(16))) LdsRing<HD, NBUF> lds;
    __shared__ int s_item;
    // A work list that was never built (a run on a workspace without a plan) holds arbitrary
    // values: its length is capped by the longest possible list, a negative claim ends the
    // loop and items naming a request or split that does not exist are skipped, so every
    // access stays in bounds (the results are then unspecified).
    const int nitems = min(ctr[0], a.max_items);
    const int per_group = a.Hkv * a.nrb;
    for (;;) {
        if (threadIdx.x == 0) s_item = atomicAdd(&ctr[1], 1);
        __syncthreads();
        const int item = s_item;
        __syncthreads();
        if (item < 0 || item >= nitems) break;
        const uint32_t gv = (uint32_t)groups[item / per_group];  // request << 16 | split
        const int within = item % per_group;
        const int i = (int)(gv >> 16), h = within / a.nrb, s = (int)(gv & 0xFFFFu);
        if (i >= a.R || s >= a.max_splits) continue;
        const int row0 = (within % a.nrb) * (WIDE ? 2 * NW * 16 : NW * 16);
        if (WIDE && a.G * (a.qo[i + 1] - a.qo[i]) - row0 > NW * 16)
            attn_item<HD, NW, NBUF, ONEPAGE, 1>(a, lds, i, h, s, row0);
        else
            attn_item<HD, NW, NBUF, ONEPAGE, 2>(a, lds, i, h, s, row0);
    }
    // the last workgroup to finish leaves the counters as the plan left them, so the
    // next call on the same plan (another layer of the round) starts clean: every
    // workgroup has made its last claim before it counts itself here
    if (threadIdx.x == 0 && atomicAdd(&ctr[2], 1) == (int)gridDim.x - 1) {
        ctr[1] = 0;
        ctr[2] = 0;
    }
}


// merge split partials: grid (row chunk, kv-head, request), one thread per (query row of
// the group, 4-dim slice); every split's lse and partial are loaded before any math (one
// round of loads for up to 8 splits). Requests with a single split were written
// directly by the main kernel and exit here.
template <int HD, bool BF16OUT>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
    constexpr int SL = HD / 4;  // 4-dim slices per row
    const int h = blockIdx.y, i = blockIdx.z;
    const int q0 = a.qo[i], k_i = a.qo[i + 1] - q0;
    int kv_len = a.kv_lens[i];
    if (kv_len > a.max_kv_len) kv_len = a.max_kv_len;
    if (k_i <= 0 || k_i > a.block || kv_len - k_i < 0 || q0 < 0 || q0 + k_i > a.total_q) return;
    const int nsplit = (kv_len + a.split - 1) / a.split;
    if (nsplit <= 1) return;
    const int u = blockIdx.x * 256 + threadIdx.x;
    if (u >= a.G * k_i * SL) return;
    const int r = u / SL, sl = u % SL;
    const size_t orow = (size_t)(q0 + r / a.G) * a.Hq + h * a.G + r % a.G;
    const size_t sstride = (size_t)a.total_q * a.Hq;
    float mx = -INFINITY, wsum = 0.0f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < nsplit; s0 += 8) {
        float lw[8];
        f32x4 v[8];
#pragma unroll
        for (int k = 0; k < 8; k++) {
            const bool ok = s0 + k < nsplit;
            lw[k] = ok ? a.part_lse[(s0 + k) * sstride + orow] : -INFINITY;
            v[k] = ok ? *(const f32x4*)(a.part_o + ((s0 + k) * sstride + orow) * HD + sl * 4) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        float bm = mx;
#pragma unroll
        for (int k = 0; k < 8; k++) bm = fmaxf(bm, lw[k]);
        if (bm == -INFINITY) continue;
        const float sc = mx == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(mx - bm);
        wsum *= sc;
        acc *= sc;
#pragma unroll
        for (int k = 0; k < 8; k++) {
            const float wgt = lw[k] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(lw[k] - bm);
            wsum += wgt;
            acc += wgt * v[k];
        }
        mx = bm;
    }
    const float inv = wsum > 0.0f ? 1.0f / wsum : 0.0f;
    if (BF16OUT) {
        uint64_t pk = 0;
#pragma unroll
        for (int e = 0; e < 4; e++) pk |= (uint64_t)f2bf(acc[e] * inv) << (16 * e);
        *(uint64_t*)((uint16_t*)a.out + orow * HD + sl * 4) = pk;
    } else {
        *(f32x4*)((float*)a.out + orow * HD + sl * 4) = acc * inv;
    }
    if (a.lse && sl == 0) a.lse[orow] = wsum > 0.0f ? (mx + __log2f(wsum)) * kLn2 : -INFINITY;
}

// ---------------------------------------------------------------------------------
// fp32 vector kernel: one workgroup of four waves per (query row, head); HD <= 256, HD % 4 == 0
// ---------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void attn_f32_kernel(AttnArgs a, int HD) {
    // one workgroup per (row, head); wave wv takes the 64-key tiles wv, wv + 4, ... and the
    // four waves' softmax states are merged at the end
    __shared__ float s_o[4][4][64];
    __shared__ float s_ml[4][2];
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int unit = blockIdx.x;
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
    for (int base = 64 * wv; base <= limit; base += 256) {
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
#pragma unroll 4
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
        // P V, keys in order for every output element. The key index is uniform, so each
        // key's p, mask bit and V row offset are broadcast with readlane (no LDS traffic), and
        // the V loads of 32 keys are issued before their products. Keys outside the mask or
        // on an invalid page are skipped, never multiplied.
        const int cnt = min(64, limit - base + 1);
        const uint32_t okmask_lo = (uint32_t)__ballot(ok), okmask_hi = (uint32_t)(__ballot(ok) >> 32);
        const uint32_t off_lo = (uint32_t)off, off_hi = (uint32_t)(off >> 32);
#pragma unroll
        for (int e = 0; e < 4; e++) {
            if (64 * e >= HD) break;
            const int dd = lane + 64 * e;
            const bool dok = dd < HD;
            for (int j0 = 0; j0 < cnt; j0 += 32) {
                float vv[32];
#pragma unroll
                for (int u = 0; u < 32; u++) {
                    const int jj = j0 + u;
                    const bool okj = jj < cnt && (((jj < 32 ? okmask_lo >> jj : okmask_hi >> (jj - 32)) & 1u) != 0);
                    const size_t offj = ((size_t)(uint32_t)__builtin_amdgcn_readlane((int)off_hi, jj & 63) << 32) |
                                        (uint32_t)__builtin_amdgcn_readlane((int)off_lo, jj & 63);
                    vv[u] = (okj && dok) ? vcp[offj + dd] : 0.0f;
                }
#pragma unroll
                for (int u = 0; u < 32; u++) {
                    const int jj = j0 + u;
                    const bool okj = jj < cnt && (((jj < 32 ? okmask_lo >> jj : okmask_hi >> (jj - 32)) & 1u) != 0);
                    if (okj) o[e] += __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, p), jj & 63)) * vv[u];
                }
            }
        }
    }
    // merge the four waves' (m, l, o): weights exp(m_w - M) over M = max m_w
#pragma unroll
    for (int e = 0; e < 4; e++) s_o[wv][e][lane] = o[e];
    if (lane == 0) {
        s_ml[wv][0] = m;
        s_ml[wv][1] = l;
    }
    __syncthreads();
    if (wv != 0) return;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; w++) M = fmaxf(M, s_ml[w][0]);
    float lt = 0.0f, ot[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < 4; w++) {
        const float mw = s_ml[w][0];
        const float wt = mw == -INFINITY ? 0.0f : expf(mw - M);
        lt += s_ml[w][1] * wt;
#pragma unroll
        for (int e = 0; e < 4; e++) ot[e] += s_o[w][e][lane] * wt;
    }
    float* op = (float*)a.out + ((size_t)row * a.Hq + head) * HD;
    const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
    for (int e = 0; e < 4; e++) {
        const int dd = lane + 64 * e;
        if (dd < HD) op[dd] = ot[e] * inv;
    }
    if (a.lse && lane == 0) a.lse[(size_t)row * a.Hq + head] = lt > 0.0f ? M + logf(lt) : -INFINITY;
}

int ilog2(int x) {
    int r = 0;
    while ((1 << r) < x) r++;
    return r;
}

}  // namespace


hipError_t launch_attn(const sv_attn_desc& d, const AttnPlan& plan, const void* q,
                       const void* k_cache, const void* v_cache, const int32_t* page_table,
                       const int32_t* qo_indptr, const int32_t* kv_lens, void* out, float* lse,
                       void* ws, hipStream_t stream, int phases) {
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
    {
        const long long mi = (long long)d.num_reqs * plan.max_splits * d.num_kv_heads * plan.row_blocks;
        a.max_items = mi > 0x7FFFFFFFLL ? 0x7FFFFFFF : (int)mi;
    }
    a.scale = d.sm_scale > 0.0f ? d.sm_scale : 1.0f / sqrtf((float)d.head_dim);
    a.scale_log2 = a.scale * kLog2e;

    if (d.dtype == SV_F32) {  // no work plan: one workgroup per (row, head)
        if (!(phases & kAttnRun)) return hipSuccess;
        const int units = d.total_q_max * d.num_q_heads;
        hipLaunchKernelGGL(attn_f32_kernel, dim3(units), dim3(256), 0, stream, a, d.head_dim);
        return hipGetLastError();
    }
    a.nrb = plan.row_blocks;
    // persistent grid: one workgroup per compute unit of the current device
    static std::atomic<int> cu_count[64];  // zero-initialised (static storage)
    int dev = 0;
    hipError_t e0 = hipGetDevice(&dev);
    if (e0 != hipSuccess) return e0;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    int ncu = cu_count[dev].load(std::memory_order_relaxed);
    if (ncu == 0) {
        int n = 0;
        e0 = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
        if (e0 != hipSuccess) return e0;
        ncu = n > 0 ? n : 1;
        cu_count[dev].store(ncu, std::memory_order_relaxed);
    }
    char* wsb = (char*)ws;
    int32_t* groups = (int32_t*)(wsb + plan.off_groups);
    int32_t* ctr = (int32_t*)(wsb + plan.off_ctr);
    if (phases & kAttnPlan) hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(1024), 0, stream, a, groups, ctr);
    if (!(phases & kAttnRun)) return hipGetLastError();
    const dim3 grid(ncu);
#define SV_LAUNCH_ATTN(HDV, ONEP, HALV) \
    hipLaunchKernelGGL((attn_bf16_kernel<HDV, 8, 4, ONEP, HALV == 1>), grid, dim3(8 * 64), 0, stream, a, groups, ctr)
    const bool onepage = d.page_size >= kTile;
    if (plan.halves == 2) {
        if (d.head_dim == 128) {
            if (onepage) SV_LAUNCH_ATTN(128, true, 2);
            else SV_LAUNCH_ATTN(128, false, 2);
        } else {
            if (onepage) SV_LAUNCH_ATTN(64, true, 2);
            else SV_LAUNCH_ATTN(64, false, 2);
        }
    } else {
        if (d.head_dim == 128) {
            if (onepage) SV_LAUNCH_ATTN(128, true, 1);
            else SV_LAUNCH_ATTN(128, false, 1);
        } else {
            if (onepage) SV_LAUNCH_ATTN(64, true, 1);
            else SV_LAUNCH_ATTN(64, false, 1);
        }
    }
#undef SV_LAUNCH_ATTN
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || plan.max_splits <= 1) return e;
    const int rows_per_group = (d.num_q_heads / d.num_kv_heads) * d.block;
    const dim3 mgrid((rows_per_group * (d.head_dim / 4) + 255) / 256, d.num_kv_heads, d.num_reqs);
    if (d.head_dim == 128)
        hipLaunchKernelGGL((attn_merge_kernel<128, true>), mgrid, dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL((attn_merge_kernel<64, true>), mgrid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace sv
