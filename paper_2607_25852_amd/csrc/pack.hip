// The dense verify batch of the kept prefixes (AngelSpec Sec. 4.2, packing) and the
// append of their keys and values to the paged cache. Both are plain data movement:
// integer index arithmetic and 16-byte copies, no floating point.
#include "sv_internal.h"

namespace sv {
namespace {

struct PackArgs {
    const int32_t* block_tokens;  // [R, b]
    const int32_t* ctx;           // [R]
    const int32_t* qo;            // [R+1]
    int32_t* tokens;              // [total_max]
    int32_t* positions;           // [total_max]
    int32_t* kv_lens;             // [R]
    int R, b, total_max;
};

// one thread per (request, block position)
__global__ __launch_bounds__(256) void pack_kernel(PackArgs a) {
    const long long e = (long long)blockIdx.x * 256 + threadIdx.x;
    if (e >= (long long)a.R * a.b) return;
    const int i = (int)(e / a.b), j = (int)(e % a.b);
    const int q0 = a.qo[i], k_i = a.qo[i + 1] - q0;
    const int L = a.ctx[i];
    const bool ok = k_i >= 1 && k_i <= a.b && q0 >= 0 && q0 + k_i <= a.total_max;
    if (j == 0) a.kv_lens[i] = ok ? L + k_i : L;
    if (!ok || j >= k_i) return;
    a.tokens[q0 + j] = a.block_tokens[(size_t)i * a.b + j];
    a.positions[q0 + j] = L + j;
}

struct AppendArgs {
    const char* k_new;  // [total_max, Hkv, d]
    const char* v_new;
    const int32_t* page_table;  // [R, maxp]
    const int32_t* qo;
    const int32_t* ctx;
    char* kc;  // [num_pages, Hkv, P, d]
    char* vc;
    int R, total_max, block, Hkv, log2P, maxp, num_pages;
    int row_bytes;  // d * element size, a multiple of 16
};

// grid (request * block position, kv-head); the threads copy the 16-byte chunks of the
// K row, then of the V row
__global__ __launch_bounds__(128) void append_kernel(AppendArgs a) {
    const int e = blockIdx.x, h = blockIdx.y;
    const int i = e / a.block, j = e % a.block;
    const int q0 = a.qo[i], k_i = a.qo[i + 1] - q0;
    if (k_i < 1 || k_i > a.block || j >= k_i || q0 < 0 || q0 + k_i > a.total_max) return;
    const long long s = (long long)a.ctx[i] + j;  // position of the row in the sequence
    if (a.ctx[i] < 0) return;
    const long long col = s >> a.log2P;
    if (col >= a.maxp) return;
    const int pg = a.page_table[(size_t)i * a.maxp + col];
    if (pg < 0 || pg >= a.num_pages) return;
    const int slot = (int)(s & ((1 << a.log2P) - 1));
    const size_t src = ((size_t)(q0 + j) * a.Hkv + h) * a.row_bytes;
    const size_t dst = ((((size_t)pg * a.Hkv + h) << a.log2P) + slot) * a.row_bytes;
    const int chunks = a.row_bytes / 16;
    for (int c = threadIdx.x; c < 2 * chunks; c += blockDim.x) {
        const bool v = c >= chunks;
        const int cc = v ? c - chunks : c;
        const uint4 x = *(const uint4*)((v ? a.v_new : a.k_new) + src + cc * 16);
        *(uint4*)((v ? a.vc : a.kc) + dst + cc * 16) = x;
    }
}

int ilog2i(int x) {
    int r = 0;
    while ((1 << r) < x) r++;
    return r;
}

}  // namespace

hipError_t launch_pack(const sv_pack_desc& d, const int32_t* block_tokens, const int32_t* ctx_lens,
                       const int32_t* qo_indptr, int32_t* tokens, int32_t* positions, int32_t* kv_lens,
                       hipStream_t stream) {
    PackArgs a{block_tokens, ctx_lens, qo_indptr, tokens, positions, kv_lens, d.num_reqs, d.block, d.total_max};
    const long long n = (long long)d.num_reqs * d.block;
    hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_append(const sv_append_desc& d, const void* k_new, const void* v_new, const int32_t* page_table,
                         const int32_t* qo_indptr, const int32_t* ctx_lens, void* k_cache, void* v_cache,
                         hipStream_t stream) {
    AppendArgs a{};
    a.k_new = (const char*)k_new;
    a.v_new = (const char*)v_new;
    a.page_table = page_table;
    a.qo = qo_indptr;
    a.ctx = ctx_lens;
    a.kc = (char*)k_cache;
    a.vc = (char*)v_cache;
    a.R = d.num_reqs;
    a.total_max = d.total_max;
    a.block = d.block;
    a.Hkv = d.num_kv_heads;
    a.log2P = ilog2i(d.page_size);
    a.maxp = d.max_pages_per_req;
    a.num_pages = d.num_pages;
    a.row_bytes = d.head_dim * (d.dtype == SV_F32 ? 4 : 2);
    hipLaunchKernelGGL(append_kernel, dim3((unsigned)((long long)d.num_reqs * d.block), d.num_kv_heads), dim3(128), 0,
                       stream, a);
    return hipGetLastError();
}

}  // namespace sv
