/*
 * specverify.h -- C ABI of libspecverify: the data-parallel core of one
 * speculative-decoding draft-verify round on an AMD Instinct MI355X (gfx950).
 *
 * The round (AngelSpec, Sec. 4 "Real-World Deployment: D-cut", and the
 * rejection-sampling verification of Sec. 1) has three steps, one call each,
 * and two data-movement calls between the budget and the attention:
 *
 *   sv_alloc_budget  D-cut verification budget: prefix confidence scores, a
 *                    global top-K over every request's draft positions, the
 *                    budget ratio chosen against a profiled cost, and the dense
 *                    packing of the kept positions (qo_indptr).
 *   sv_pack_verify   the dense verify batch (tokens, positions, key counts) of
 *                    the kept prefixes, the target model's input;
 *   sv_append_kv     the kept positions' keys and values into the paged cache;
 *   sv_verify_attn   attention of every kept position over its request's paged
 *                    KV cache: causal inside the block, full over the context,
 *                    grouped-query heads.
 *   sv_spec_accept   speculative acceptance: softmax of the target logits, the
 *                    per-position test u < min(1, p/q), the first-rejection
 *                    cut, and the extra token drawn from the normalised residual
 *                    max(p - q, 0), or from p when the whole block survives.
 *
 * On the drafter's side, sv_draft_stats gives each draft row its softmax
 * normaliser and the confidence c_t the budget takes; sv_spec_accept_stats is the
 * acceptance that uses those normalisers instead of re-reading the draft rows.
 *
 * Conventions shared by every entry point
 *   - All array pointers are caller-owned DEVICE memory unless marked "host".
 *     The library allocates nothing and keeps no state between calls (apart from
 *     the fixed device scratch of sv_spec_accept_noalloc); each call only enqueues
 *     kernels on `stream` (a hipStream_t; NULL = the default stream) and returns
 *     without waiting for them.
 *   - Descriptors are host structs, read during the call only.
 *   - Alignment: the floating-point data arrays (q, caches, out, logits) and the
 *     workspaces must be 16-byte aligned; int32 and fp32 index / scalar arrays
 *     4-byte aligned. Misaligned pointers are rejected with SV_ERR_INVALID_ARG.
 *   - Host-side argument checks run before anything is enqueued. On failure the
 *     call returns a non-zero sv_status, enqueues nothing, and sv_last_error()
 *     (thread-local) describes the reason. A failed launch returns SV_ERR_HIP.
 *   - Device data is not validated beyond what keeps every memory access in
 *     bounds (page ids, row ranges and token ids are range-checked by the
 *     kernels); out-of-range values give unspecified but finite-memory results.
 *   - "b" (block) is the number of verify positions per request: the certain
 *     token that ends the committed context plus D = b - 1 draft tokens.
 *     Position 0 is the certain token; drafts are positions 1..D.
 *   - Uniform random numbers are inputs (the caller's generator), fp32 in [0,1).
 *   - Calls on different streams may run concurrently (no shared state); calls
 *     sharing a workspace buffer must be ordered by the caller.
 */
#ifndef SPECVERIFY_H
#define SPECVERIFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SV_ABI_VERSION 1

typedef enum {
    SV_OK = 0,
    SV_ERR_INVALID_ARG = 1, /* a descriptor field or pointer is invalid */
    SV_ERR_UNSUPPORTED = 2, /* valid request outside what the kernels implement */
    SV_ERR_WORKSPACE = 3,   /* workspace missing or smaller than the size query */
    SV_ERR_HIP = 4          /* a HIP launch failed (see sv_last_error) */
} sv_status;

typedef enum { SV_F32 = 0, SV_BF16 = 1 } sv_dtype;
typedef enum { SV_LOGITS = 0, SV_PROBS = 1 } sv_input_kind;
typedef enum { SV_BUDGET_FIXED = 0, SV_BUDGET_COST = 1 } sv_budget_mode;

#define SV_MAX_BLOCK 16            /* b <= 16 verify positions per request */
#define SV_MAX_RATIOS 8
#define SV_MAX_BUDGET_REQS 4096    /* R for sv_alloc_budget */
#define SV_MAX_BUDGET_POSITIONS 8192 /* R * b for sv_alloc_budget */
#define SV_MAX_VOCAB (1 << 22)

/* ------------------------------------------------------------------------- */
/* D-cut budget (Sec. 4.2, eqs. dcut-score, dcut-expected-advance,            */
/* dcut-budget, dcut-batch-utility, dcut-select, and "Packing and correctness")*/
/* ------------------------------------------------------------------------- */
typedef struct {
    int32_t num_reqs;     /* R >= 1 (the paper's B, active requests)            */
    int32_t block;        /* b in [1, 16]                                        */
    int32_t mode;         /* sv_budget_mode                                       */
    int32_t fixed_budget; /* FIXED: K with R <= K <= R*b                          */
    int32_t num_ratios;   /* COST: 1..8 candidate ratios                          */
    int32_t ratio_permille[SV_MAX_RATIOS]; /* COST: strictly ascending, (0, 1000] */
    uint32_t cost[SV_MAX_RATIOS]; /* COST: profiled step cost C(R, rho_j) > 0,
                                     any integer time unit                      */
} sv_budget_desc;

/*
 * sv_alloc_budget -- choose how many draft positions of each request to verify.
 *
 *   scores   s[i][0] = 1, s[i][t] = s[i][t-1] * c[i][t], an fp32 product taken
 *            left to right (eq. dcut-score); a confidence is clamped to [0,1]
 *            first and NaN counts as 0, which keeps scores non-increasing.
 *   order    all R*b positions ranked by score (higher first), ties to the
 *            shallower position (Sec. 4.2), then to the lower request index;
 *            taking the first K in this order keeps a contiguous prefix of
 *            every request's block.
 *   budget   FIXED: K = fixed_budget.  COST: for each ratio rho_j,
 *            K_j = max(R, ceil(rho_j * R * b)) (eq. dcut-budget); utility
 *            U_j = sum of the top-K_j scores, each as floor(s * 2^40) in
 *            uint64 (eq. dcut-batch-utility, in fixed point); the chosen ratio
 *            maximises U_j / C_j, compared exactly as U_a*C_b vs U_b*C_a in
 *            128 bits, ties to the smaller ratio (eq. dcut-select).
 *   packing  n_i = kept positions of request i minus 1 (drafts kept),
 *            qo_indptr = exclusive prefix sum of n_i + 1: the rows of request i
 *            in the dense verify batch are qo_indptr[i] .. qo_indptr[i+1]-1.
 *
 * conf       [R, b-1] fp32, c[i][t] for drafts t = 1..b-1 (may be NULL if b = 1)
 * keep       [R] int32 out: n_i in [0, b-1]
 * qo_indptr  [R+1] int32 out
 * sel        [2] int32 out: {K, index of the chosen ratio or -1 in FIXED mode}
 * scores     [R, b] fp32 out, or NULL
 * utility    [num_ratios] uint64 out (COST) or [1] (FIXED: U of the fixed K), or NULL
 * Limits: R <= 4096, R*b <= 8192. One workgroup; no workspace.
 */
sv_status sv_alloc_budget(const sv_budget_desc* desc, const float* conf, int32_t* keep,
                          int32_t* qo_indptr, int32_t* sel, float* scores, uint64_t* utility,
                          void* stream);

/* ------------------------------------------------------------------------- */
/* The dense verify batch of the kept prefixes (Sec. 4.2, "Packing and        */
/* correctness") and the cache append of their keys and values                */
/* ------------------------------------------------------------------------- */
typedef struct {
    int32_t num_reqs;  /* R >= 1                                               */
    int32_t block;     /* b in [1, 16]                                          */
    int32_t total_max; /* rows allocated in tokens / positions (>= qo_indptr[R]) */
} sv_pack_desc;

/*
 * sv_pack_verify -- the dense verify batch of the kept block prefixes: for request
 * i with k_i = qo_indptr[i+1]-qo_indptr[i] kept positions and committed context
 * L_i = ctx_lens[i], row r = qo_indptr[i] + j (0 <= j < k_i) gets
 *     tokens[r] = block_tokens[i][j]   (position 0: the certain token, then drafts)
 *     positions[r] = L_i + j           (absolute position in the sequence)
 * and kv_lens[i] = L_i + k_i, the key count sv_verify_attn reads once the kept
 * positions' keys and values are in the cache (sv_append_kv).
 * A request with k_i outside [1, b], or with rows outside [0, total_max), gets no
 * rows and kv_lens[i] = L_i.
 * block_tokens [R, b] int32; ctx_lens [R] int32 >= 0; qo_indptr [R+1] int32
 * tokens, positions [total_max] int32 out (rows that no request owns are untouched);
 * kv_lens [R] int32 out. All pointers are device memory owned by the caller; the
 * call is asynchronous on `stream` and allocates nothing.
 */
sv_status sv_pack_verify(const sv_pack_desc* desc, const int32_t* block_tokens, const int32_t* ctx_lens,
                         const int32_t* qo_indptr, int32_t* tokens, int32_t* positions, int32_t* kv_lens,
                         void* stream);

typedef struct {
    int32_t num_reqs;          /* R >= 1                                        */
    int32_t total_max;         /* rows allocated in k_new / v_new               */
    int32_t block;             /* max k_i (<= 16)                               */
    int32_t num_kv_heads;      /* Hkv                                           */
    int32_t head_dim;          /* d; d * element size a multiple of 16 bytes    */
    int32_t page_size;         /* P, a power of two in [1, 4096]                */
    int32_t max_pages_per_req; /* columns of page_table                          */
    int32_t num_pages;         /* pages in each cache                            */
    int32_t dtype;             /* sv_dtype of the rows and the caches            */
} sv_append_desc;

/*
 * sv_append_kv -- write the keys and values of the packed verify rows into the paged
 * cache (the step between the target's projection and sv_verify_attn): row
 * r = qo_indptr[i] + j of k_new / v_new, for every kv-head, goes to position
 * s = ctx_lens[i] + j of request i, i.e. page page_table[i][s / P], slot s % P.
 * A row whose page id is outside [0, num_pages) or whose page column is outside
 * [0, max_pages_per_req) is skipped, and so is every row of a request with k_i
 * outside [1, block], rows outside [0, total_max) or ctx_lens[i] < 0; nothing else
 * in the caches is written. Two requests that map a position to the same page slot
 * race (the caller owns the page table). Device memory owned by the caller;
 * asynchronous on `stream`; allocates nothing.
 * k_new, v_new [total_max, Hkv, d]; k_cache, v_cache [num_pages, Hkv, P, d]
 * page_table [R, max_pages_per_req] int32; qo_indptr [R+1]; ctx_lens [R] int32
 */
sv_status sv_append_kv(const sv_append_desc* desc, const void* k_new, const void* v_new,
                       const int32_t* page_table, const int32_t* qo_indptr, const int32_t* ctx_lens,
                       void* k_cache, void* v_cache, void* stream);

/* ------------------------------------------------------------------------- */
/* Verify attention (every kept position is evaluated by the target model,    */
/* Sec. 4.1; the dense packed batch of Sec. 4.2).                             */
/* ------------------------------------------------------------------------- */
typedef struct {
    int32_t num_reqs;          /* R in [1, 65535]                                   */
    int32_t total_q_max;       /* rows in q / out / lse: qo_indptr[R] <= it <= R*block,
                                  and total_q_max * num_q_heads < 2^31                */
    int32_t block;             /* max k_i (<= 16)                                   */
    int32_t num_q_heads;       /* Hq                                               */
    int32_t num_kv_heads;      /* Hkv, Hq % Hkv == 0; G = Hq / Hkv                   */
    int32_t head_dim;          /* d: bf16 64 or 128; fp32 any multiple of 4 <= 256  */
    int32_t page_size;         /* P tokens per page, a power of two in [1, 4096]    */
    int32_t max_pages_per_req; /* columns of page_table                              */
    int32_t num_pages;         /* pages in each cache                                */
    int32_t max_kv_len;        /* upper bound of kv_lens[i], <= 2^22                  */
    int32_t dtype;             /* sv_dtype of q, caches and out                       */
    float sm_scale;            /* logit scale; 0 means 1/sqrt(d)                      */
    int32_t kv_split;          /* tokens per split-KV work item (multiple of 64), 0 = auto */
} sv_attn_desc;

/*
 * sv_verify_attn -- for request i with k_i = qo_indptr[i+1]-qo_indptr[i] rows
 * and committed context L_i = kv_lens[i] - k_i, query row j (0 <= j < k_i) of
 * head h attends to keys s = 0 .. L_i + j of kv-head floor(h / G):
 *     z_s = sm_scale * <q, K_s>,  lse = ln sum_s exp(z_s),  o = sum_s exp(z_s - lse) V_s.
 * Key s of request i sits in page page_table[i][s / P], slot s % P. The block's
 * own keys and values (positions L_i .. L_i + k_i - 1) must already be in the
 * cache; pages and slots past kv_lens[i] are never read.
 *
 * q          [total_q_max, Hq, d]  (rows packed by qo_indptr)
 * k_cache, v_cache [num_pages, Hkv, P, d]
 * page_table [R, max_pages_per_req] int32
 * qo_indptr  [R+1] int32 (1 <= k_i <= block), kv_lens [R] int32 (k_i <= kv_lens[i] <= max_kv_len)
 * out        [total_q_max, Hq, d] same dtype as q;  lse [total_q_max, Hq] fp32 or NULL
 * ws         scratch of at least sv_verify_attn_workspace_size(desc) bytes (bf16:
 *            the work list of the persistent kernel and the partial results of
 *            split-KV work items; fp32: none), device memory, overwritten by every call.
 * bf16 runs on MFMA with fp32 accumulation; fp32 runs on vector ALUs in fp32.
 */
sv_status sv_verify_attn(const sv_attn_desc* desc, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* page_table, const int32_t* qo_indptr,
                         const int32_t* kv_lens, void* out, float* lse, void* ws, size_t ws_bytes,
                         void* stream);
size_t sv_verify_attn_workspace_size(const sv_attn_desc* desc);

/*
 * sv_verify_attn_plan and sv_verify_attn_run -- sv_verify_attn in two parts: the bf16
 * path's work plan (which (request, kv-head, split, row block) items exist, largest
 * first) depends only on the descriptor, qo_indptr and kv_lens, so a round builds it once
 * and every attention layer of that round runs on it, as serving engines plan a batch
 * once per step (Sec. 4.2: one packed verify batch per round, evaluated by every layer
 * of the target model).
 *   sv_verify_attn_plan  writes the plan into ws (sv_verify_attn_workspace_size(desc)
 *                        bytes); the fp32 path has no plan and the call enqueues nothing.
 *   sv_verify_attn_run   sv_verify_attn's arguments and results, using the plan that ws
 *                        holds: it must have been built (by sv_verify_attn_plan or
 *                        sv_prepare_round) for the same descriptor, qo_indptr and
 *                        kv_lens. Each run leaves the plan as it found it (its work
 *                        counter is reset by the last workgroup to finish), so runs on
 *                        one plan may follow each other on the stream; runs on one
 *                        workspace must not overlap. On a workspace that holds no plan,
 *                        or a plan built for other inputs, the results are unspecified
 *                        but every memory access stays in bounds.
 * Results equal sv_verify_attn's bit for bit. Errors as for sv_verify_attn.
 */
sv_status sv_verify_attn_plan(const sv_attn_desc* desc, const int32_t* qo_indptr, const int32_t* kv_lens,
                              void* ws, size_t ws_bytes, void* stream);
sv_status sv_verify_attn_run(const sv_attn_desc* desc, const void* q, const void* k_cache,
                             const void* v_cache, const int32_t* page_table, const int32_t* qo_indptr,
                             const int32_t* kv_lens, void* out, float* lse, void* ws, size_t ws_bytes,
                             void* stream);

/*
 * sv_prepare_round -- the round's set-up in one launch on one workgroup: sv_alloc_budget
 * (D-cut, Sec. 4.2), then sv_pack_verify on the budget's own qo_indptr (the packing of
 * Sec. 4.2), then, when adesc is not NULL, sv_verify_attn_plan over the key counts just
 * packed, into attn_ws. Arguments and results as in those calls (bdesc and pdesc must
 * agree on num_reqs and block, as must adesc); the outputs equal theirs bit for bit.
 * Limits are those of sv_alloc_budget (R <= 4096, R*b <= 8192). Each small call costs a
 * launch and its gap whatever it does, so the round's three set-up steps share one.
 */
sv_status sv_prepare_round(const sv_budget_desc* bdesc, const float* conf, int32_t* keep, int32_t* qo_indptr,
                           int32_t* sel, float* scores, uint64_t* utility, const sv_pack_desc* pdesc,
                           const int32_t* block_tokens, const int32_t* ctx_lens, int32_t* tokens,
                           int32_t* positions, int32_t* kv_lens, const sv_attn_desc* adesc, void* attn_ws,
                           size_t attn_ws_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Speculative acceptance (rejection-sampling verification, Sec. 1; the       */
/* acceptance probability of eq. mtp-acceptance-tv)                           */
/* ------------------------------------------------------------------------- */
typedef struct {
    int32_t num_reqs;   /* R >= 1                                            */
    int32_t block;      /* b in [1, 16]                                        */
    int32_t vocab;      /* V in [1, 2^22]                                      */
    int32_t kind;       /* sv_input_kind: LOGITS (fp32 or bf16) or PROBS (fp32) */
    int32_t dtype;      /* sv_dtype of target and draft                         */
    float temperature;  /* T > 0: rejection sampling, LOGITS p = softmax(l / T);
                           T == 0: greedy verification (either kind)            */
} sv_accept_desc;

/*
 * sv_spec_accept -- for request i with n_i = qo_indptr[i+1]-qo_indptr[i]-1 drafts:
 *   P_r = target row qo_indptr[i]+r (r = 0..n_i): the target distribution of
 *         block position r+1;  Q_t = draft row (i, t-1): the draft distribution
 *         of draft t (t = 1..n_i), d_t = draft_tokens[i][t-1].
 *   1. draft t is accepted iff u_accept[i][t-1] * Q_t(d_t) < P_{t-1}(d_t),
 *      evaluated exactly (fp64 product of fp32 values);
 *   2. a_i = (first rejected t) - 1, or n_i when none is rejected;
 *   3. extra token: after a rejection from r = max(P_{a_i} - Q_{a_i+1}, 0)
 *      (fp32 difference), else from r = P_{n_i}; drawn by the inverse CDF of the
 *      integer weights w(v) = floor(min(r(v),1) * 2^40): the smallest v whose
 *      running sum of w exceeds floor(m * Z / 2^24), m = floor(u_sample[i] * 2^24),
 *      Z = sum w. An empty residual (Z = 0) falls back to P_{a_i} (flag bit 0);
 *      if that is empty too the token is -1 (flag bit 1);
 *   4. out_tokens[i] = d_1 .. d_{a_i}, token, then -1; accept_len[i] = a_i.
 *   A draft token outside [0, V) is rejected (flag bit 2).
 * In LOGITS mode the probabilities are softmax(logits / T) computed in fp32 on
 * the GPU (row max and sum of exponentials per row, read once).
 * temperature == 0 selects greedy verification (the T -> 0 limit; the paper also
 * evaluates T = 0): draft t is accepted iff d_t is the argmax of P_{t-1}, and the
 * extra token is the argmax of P_{a_i}. Argmax = the largest stored value (logit or
 * probability), lowest index on ties, NaN entries skipped; a row with no non-NaN
 * entry gives token -1 (flag bit 1). Only the kept target rows are read; draft,
 * u_accept and u_sample may be NULL.
 *
 * target      [qo_indptr[R], V] rows packed by qo_indptr (fp32 or bf16)
 * draft       [R, b-1, V] (fp32 or bf16); only rows t-1 < n_i are read
 * draft_tokens, u_accept [R, b-1] (int32, fp32); u_sample [R] fp32
 * qo_indptr   [R+1] int32 with 0 <= n_i <= b-1
 * accept_len  [R] int32 out; out_tokens [R, b] int32 out; flags [R] int32 out or NULL
 * ws          scratch of at least sv_spec_accept_workspace_size(desc) bytes.
 */
sv_status sv_spec_accept(const sv_accept_desc* desc, const void* target, const void* draft,
                         const int32_t* draft_tokens, const int32_t* qo_indptr,
                         const float* u_accept, const float* u_sample, int32_t* accept_len,
                         int32_t* out_tokens, int32_t* flags, void* ws, size_t ws_bytes,
                         void* stream);
size_t sv_spec_accept_workspace_size(const sv_accept_desc* desc);

/*
 * sv_spec_accept_noalloc -- sv_spec_accept without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments, kernels, results and errors as
 * sv_spec_accept, minus ws / ws_bytes; the library allocates nothing.
 * The workspace is a fixed 16 MiB device array inside the library, one per GPU, held from
 * the first call on that GPU until the process ends. Shapes whose
 * sv_spec_accept_workspace_size exceeds 16 MiB are rejected with SV_ERR_UNSUPPORTED
 * (c64_b16-like rounds need about 2.3 MiB). Every call on a GPU uses that GPU's array and
 * leaves its contents behind: calls that overlap on one GPU (different streams or host
 * threads without ordering) race and give undefined results; order them, or use
 * sv_spec_accept with separate workspaces. The array belongs to the device of `stream`
 * (NULL: the current device).
 */
sv_status sv_spec_accept_noalloc(const sv_accept_desc* desc, const void* target, const void* draft,
                                 const int32_t* draft_tokens, const int32_t* qo_indptr, const float* u_accept,
                                 const float* u_sample, int32_t* accept_len, int32_t* out_tokens, int32_t* flags,
                                 void* stream);

/*
 * sv_spec_accept_debug -- sv_spec_accept (LOGITS, temperature > 0) that also exports the
 * fp32 values its decisions were taken on, so that a reference implementation of the
 * acceptance rule (Sec. 1) applied to exactly those values can replay them:
 *   dbg_pq  [2, R, b-1] fp32 out: [0][i][t-1] = P_{t-1}(d_t), [1][i][t-1] = Q_t(d_t) as
 *           compared by the test of draft t (t = 1..n_i); other entries untouched;
 *   dbg_row [R, 2, V] fp32 out: [i][0] = P_{a_i}(v), [i][1] = Q_{a_i+1}(v) (0 for a bonus
 *           draw) as the residual weights of the draw use them; untouched for a malformed
 *           request.
 * The results are those of sv_spec_accept. A diagnostics call for tests: the export
 * writes 8*R*V bytes more and is slower. Device memory owned by the caller.
 */
sv_status sv_spec_accept_debug(const sv_accept_desc* desc, const void* target, const void* draft,
                               const int32_t* draft_tokens, const int32_t* qo_indptr, const float* u_accept,
                               const float* u_sample, int32_t* accept_len, int32_t* out_tokens, int32_t* flags,
                               float* dbg_pq, float* dbg_row, void* ws, size_t ws_bytes, void* stream);

/*
 * sv_spec_accept_stats -- sv_spec_accept (LOGITS, temperature > 0) with the draft rows'
 * softmax statistics supplied by the drafter (sv_draft_stats, same temperature and
 * dtype): draft_stats [R, b-1, 2] fp32 holds (m, S) per draft row, m = max_v l(v)/T and
 * S = sum_v 2^((l(v)/T - m) log2 e). The draft rows are then read only at the drafted
 * token and, after a rejection, the one residual row; the kept target rows are still
 * streamed once. With statistics from sv_draft_stats the results equal those of
 * sv_spec_accept bit for bit (the same chunks and the same merge). The confidence
 * c_t of the budget is the same pass's max_v Q_t(v) (Sec. 4.2), so the drafter's one
 * pass over its rows serves both. Other arguments, workspace and errors as
 * sv_spec_accept; draft_stats is device memory, 8-byte aligned, NULL only when b == 1.
 */
sv_status sv_spec_accept_stats(const sv_accept_desc* desc, const void* target, const void* draft,
                               const float* draft_stats, const int32_t* draft_tokens, const int32_t* qo_indptr,
                               const float* u_accept, const float* u_sample, int32_t* accept_len,
                               int32_t* out_tokens, int32_t* flags, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Draft-row statistics (the drafter's side of the round: the confidences c_t */
/* of Sec. 4.2 and the normalisers acceptance needs)                          */
/* ------------------------------------------------------------------------- */
typedef struct {
    int32_t num_reqs;   /* R >= 1                                   */
    int32_t drafts;     /* rows per request (b - 1 of the round) >= 1 */
    int32_t vocab;      /* V in [1, 2^22]                           */
    int32_t dtype;      /* sv_dtype of the logits                   */
    float temperature;  /* T > 0, as in the acceptance call          */
} sv_draft_stats_desc;

/*
 * sv_draft_stats -- for every draft row r of draft_logits [R, drafts, V]:
 *   stats[r] = (m, S), m = max_v l(v)/T, S = sum_v 2^((l(v)/T - m) log2 e) (fp32, in
 *   the chunks and merge order of sv_spec_accept);
 *   conf[r] = max_v softmax(l/T)(v) = 1/S (0 for a row without a finite entry), the
 *   token-level confidence c_t of Sec. 4.2 that sv_alloc_budget takes.
 * stats [R*drafts, 2] fp32 out (8-byte aligned); conf [R*drafts] fp32 out or NULL;
 * ws scratch of sv_draft_stats_workspace_size(desc) bytes, overwritten. Device memory
 * owned by the caller; asynchronous on `stream`; the library allocates nothing.
 */
size_t sv_draft_stats_workspace_size(const sv_draft_stats_desc* desc);
sv_status sv_draft_stats(const sv_draft_stats_desc* desc, const void* draft_logits, float* stats, float* conf,
                         void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* status                                                                      */
/* ------------------------------------------------------------------------- */
const char* sv_status_string(int32_t status); /* static string, never NULL        */
const char* sv_last_error(void);              /* thread-local, "" when none        */
int32_t sv_abi_version(void);                 /* SV_ABI_VERSION                    */

#ifdef __cplusplus
}
#endif
#endif /* SPECVERIFY_H */
