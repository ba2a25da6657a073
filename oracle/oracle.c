/*
 * oracle.c -- plain, slow, obviously-correct CPU reference for the three steps of
 * one draft-verify round (AngelSpec, "Real-World Deployment: D-cut", Sec. 4, and the
 * rejection-sampling verification it relies on, Sec. 1 and Sec. 2.3).
 *
 * THIS IS TEST INFRASTRUCTURE. Only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark may load it. It shares no code, header, table or
 * helper with the GPU library; the two meet only in the seeded input generator.
 *
 * Precision: floating point is fp64 except where the method fixes fp32 values
 * (prefix scores and probabilities, which are the fp32 quantities the kernels
 * exchange). Decisions use exact arithmetic:
 *   - the acceptance test  u < min(1, p/q)  is evaluated as the exact fp64
 *     product  u*q < p  (two 24-bit significands multiply exactly in fp64);
 *   - the extra-token draw is an inverse CDF over integer weights
 *     w(v) = floor(r(v) * 2^40), so the sum is exact and order-free;
 *   - batch utility U is a sum of floor(s * 2^40) in uint64, and the
 *     runtime-aware ratio choice compares U_a*C_b against U_b*C_a in 128 bits.
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -fopenmp -shared -fPIC.
 *
 * Parity pins (tests/test_oracle_*.py): brute-force optimality of the budget,
 * its invariants and tie rules, the exact output-distribution identity of
 * accept-then-residual sampling enumerated over the uniform grid, Monte-Carlo
 * overlap/accepted-length closed forms, and closed-form attention cases.
 */
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_EINVAL 1

/* ------------------------------------------------------------------ */
/* small helpers                                                        */
/* ------------------------------------------------------------------ */

static float bf16_to_float(uint16_t h) {
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* element v of row `row` of a [rows, V] matrix stored as fp32 (dtype 0) or bf16 (dtype 1) */
static float load_elem(const void* base, int dtype, int64_t row, int V, int v) {
    if (dtype == 0) return ((const float*)base)[row * (int64_t)V + v];
    return bf16_to_float(((const uint16_t*)base)[row * (int64_t)V + v]);
}

/* Confidence sanitising: the prefix-product argument (scores non-increasing,
 * Sec. 4.2 after eq. dcut-expected-advance) needs c in [0,1]; NaN counts as 0. */
static float clamp_conf(float c) {
    if (!(c > 0.0f)) return 0.0f; /* NaN, negative, -0 */
    if (c > 1.0f) return 1.0f;
    return c;
}

/* ------------------------------------------------------------------ */
/* Step 1 of D-cut: prefix scores, eq. dcut-score                       */
/*   s_{i,0} = 1,  s_{i,k} = prod_{t=1..k} c_{i,t}, taken left to right  */
/*   in fp32 (the association order is fixed so the value is unique).   */
/* conf: [R, b-1] fp32;  scores: [R, b] fp32                            */
/* ------------------------------------------------------------------ */
void oracle_prefix_scores(int R, int b, const float* conf, float* scores) {
    for (int i = 0; i < R; i++) {
        float s = 1.0f;
        scores[(int64_t)i * b] = s;
        for (int t = 1; t < b; t++) {
            s = s * clamp_conf(conf[(int64_t)i * (b - 1) + (t - 1)]);
            scores[(int64_t)i * b + t] = s;
        }
    }
}

/* candidate (request i, depth t) with its score */
typedef struct {
    float s;
    int t;
    int i;
} cand_t;

/* Global order of Sec. 4.2: higher score first; ties go to the shallower depth
 * (this is what keeps every request's kept set a contiguous prefix); remaining
 * ties (equal score and depth in two requests) go to the lower request index. */
static int cand_cmp(const void* a, const void* b) {
    const cand_t* x = (const cand_t*)a;
    const cand_t* y = (const cand_t*)b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    if (x->t != y->t) return x->t < y->t ? -1 : 1;
    if (x->i != y->i) return x->i < y->i ? -1 : 1;
    return 0;
}

/* fixed-point value of a score in units of 2^-40 (scores lie in [0,1]) */
static uint64_t score_fixed(float s) { return (uint64_t)((double)s * 1099511627776.0); }

/*
 * D-cut budget selection (Sec. 4.2).
 *   eq. dcut-budget:        K_rho = max(R, ceil(rho * R * b)),  b = D+1 positions
 *   eq. dcut-batch-utility: U(rho) = sum_i  Ahat_i(n_i^rho) = sum of the top-K_rho scores
 *   eq. dcut-select:        rho* = argmax_rho U(rho) / C(rho)   (ties -> the smaller ratio)
 *   packing:                n_i = (#kept positions of request i) - 1, qo_indptr = exclusive
 *                           scan of n_i + 1
 * mode 0 = fixed budget K (no ratio search, sel[1] = -1, utility[0] = U_K).
 * ratio_pm: ratios in permille (250 = 0.25), strictly ascending, in (0, 1000].
 * cost: C(R, rho_j), positive integers (any time unit).
 * Outputs: keep [R], qo_indptr [R+1], sel[2] = {K*, index of rho* or -1},
 *          scores [R,b] (nullable), utility [nratios] or [1] (nullable).
 */
int oracle_budget(int R, int b, int mode, int fixed_K, int nratios, const int* ratio_pm,
                  const uint32_t* cost, const float* conf, int* keep, int* qo_indptr, int* sel,
                  float* scores_out, uint64_t* utility_out) {
    if (R < 1 || b < 1) return ORC_EINVAL;
    const int N = R * b;
    float* scores = (float*)malloc(sizeof(float) * (size_t)N);
    cand_t* cand = (cand_t*)malloc(sizeof(cand_t) * (size_t)N);
    if (!scores || !cand) {
        free(scores);
        free(cand);
        return ORC_EINVAL;
    }
    oracle_prefix_scores(R, b, conf, scores);

    /* global top-K over all R*b candidates: sort in the order above */
    for (int i = 0; i < R; i++)
        for (int t = 0; t < b; t++) {
            cand_t c = {scores[i * b + t], t, i};
            cand[i * b + t] = c;
        }
    qsort(cand, (size_t)N, sizeof(cand_t), cand_cmp);

    int Kstar;
    int best = -1;
    if (mode == 0) {
        if (fixed_K < R || fixed_K > N) {
            free(scores);
            free(cand);
            return ORC_EINVAL;
        }
        Kstar = fixed_K;
        if (utility_out) {
            uint64_t U = 0;
            for (int k = 0; k < Kstar; k++) U += score_fixed(cand[k].s);
            utility_out[0] = U;
        }
    } else {
        if (nratios < 1 || nratios > 8) {
            free(scores);
            free(cand);
            return ORC_EINVAL;
        }
        uint64_t U[8];
        int Kr[8];
        for (int j = 0; j < nratios; j++) {
            /* ceil(rho * R * b) with rho = pm / 1000, in integers */
            int64_t num = (int64_t)ratio_pm[j] * R * b;
            int Kj = (int)((num + 999) / 1000);
            if (Kj < R) Kj = R;
            if (Kj > N) Kj = N;
            Kr[j] = Kj;
            uint64_t u = 0;
            for (int k = 0; k < Kj; k++) u += score_fixed(cand[k].s);
            U[j] = u;
            if (utility_out) utility_out[j] = u;
        }
        best = 0;
        for (int j = 1; j < nratios; j++) {
            unsigned __int128 lhs = (unsigned __int128)U[j] * cost[best];
            unsigned __int128 rhs = (unsigned __int128)U[best] * cost[j];
            if (lhs > rhs) best = j;
        }
        Kstar = Kr[best];
    }

    for (int i = 0; i < R; i++) keep[i] = -1;
    for (int k = 0; k < Kstar; k++) keep[cand[k].i] += 1;
    qo_indptr[0] = 0;
    for (int i = 0; i < R; i++) qo_indptr[i + 1] = qo_indptr[i] + keep[i] + 1;
    sel[0] = Kstar;
    sel[1] = best;
    if (scores_out) memcpy(scores_out, scores, sizeof(float) * (size_t)N);
    free(scores);
    free(cand);
    return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Speculative acceptance (rejection-sampling verification, Sec. 1;     */
/* overlap identity eq. mtp-acceptance-tv).                             */
/* ------------------------------------------------------------------ */

/* integer sampling weight of a probability-like value r: floor(r * 2^40), with
 * r clamped to [0, 1] and NaN treated as 0 */
static uint64_t weight_of(float r) {
    if (!(r > 0.0f)) return 0;
    if (r > 1.0f) r = 1.0f;
    return (uint64_t)((double)r * 1099511627776.0);
}

/* one probability row: either given (kind 1) or softmax(logits / T) (kind 0) */
typedef struct {
    const void* base;
    int dtype;
    int kind;
    int V;
    float temperature;
    int64_t row;
    double m;   /* max of x (logits mode) */
    double S;   /* sum of exp(x - m)   (logits mode) */
} prow_t;

static float logit_scaled(const prow_t* pr, int v) {
    float l = load_elem(pr->base, pr->dtype, pr->row, pr->V, v);
    return l / pr->temperature;
}

static void prow_init(prow_t* pr) {
    if (pr->kind == 1) return;
    double m = -INFINITY;
    for (int v = 0; v < pr->V; v++) {
        double x = (double)logit_scaled(pr, v);
        if (x > m) m = x;
    }
    double S = 0.0;
    for (int v = 0; v < pr->V; v++) S += exp((double)logit_scaled(pr, v) - m);
    pr->m = m;
    pr->S = S;
}

/* fp32 probability of token v in this row */
static float prow_prob(const prow_t* pr, int v) {
    if (pr->kind == 1) return load_elem(pr->base, pr->dtype, pr->row, pr->V, v);
    double e = exp((double)logit_scaled(pr, v) - pr->m);
    return (float)(e / pr->S);
}

/*
 * Acceptance for R requests.  Request i keeps n_i = qo_indptr[i+1]-qo_indptr[i]-1 drafts.
 *   target [K, V]:  packed rows; row qo_indptr[i]+r is the target distribution P_r
 *                   for block position r+1 (r = 0..n_i; P_0 follows the certain token).
 *   draft  [R, b-1, V]: row (i, t-1) is the draft distribution Q_t of draft t.
 *   draft_tokens [R, b-1]: d_t.   u_accept [R, b-1], u_sample [R]: uniforms in [0,1).
 * Steps per request:
 *   1. accept draft t (t = 1..n_i) iff  u_t * Q_t(d_t) < P_{t-1}(d_t)  (exact fp64);
 *   2. a_i = (first rejected t) - 1, or n_i if none is rejected;
 *   3. extra token from r = max(P_{a}-Q_{a+1}, 0) after a rejection, else from P_{n_i}
 *      (the bonus); r is formed in fp32, sampled by the integer inverse CDF
 *      token = min { v : sum_{v'<=v} w(v') > floor(m_u * Z / 2^24) },
 *      m_u = u_sample * 2^24, Z = sum w;  if Z = 0 after a rejection, P_a is used
 *      instead (flag bit 0); if that is zero too, token = -1 (flag bit 1);
 *   4. out_tokens[i] = d_1..d_{a_i}, token, -1 ...;  accept_len[i] = a_i.
 *   A draft token outside [0, V) is rejected and sets flag bit 2.
 * kind 0 = logits (p = softmax(l / T), fp64 internally, rounded to fp32),
 * kind 1 = probabilities given as fp32 rows.  dtype 0 = fp32, 1 = bf16 (logits only).
 * diag_p/diag_q [R, b-1] (nullable): P_{t-1}(d_t) and Q_t(d_t) as used by the test.
 * diag_cdf [R, 4] (nullable): (thr, cumulative weight before the token, the token's
 * weight, Z) as doubles, so a caller can see how far the draw is from a CDF step.
 */
int oracle_accept(int R, int b, int V, int kind, int dtype, float temperature, const void* target,
                  const void* draft, const int* draft_tokens, const int* qo_indptr,
                  const float* u_accept, const float* u_sample, int* accept_len, int* out_tokens,
                  int* flags, double* diag_p, double* diag_q, double* diag_cdf) {
    if (R < 1 || b < 1 || V < 1) return ORC_EINVAL;
    if (kind == 1 && dtype != 0) return ORC_EINVAL;
    if (kind == 0 && !(temperature > 0.0f)) return ORC_EINVAL;
    const int D = b - 1;
    for (int i = 0; i < R; i++) {
        int n = qo_indptr[i + 1] - qo_indptr[i] - 1;
        if (n < 0 || n > D) return ORC_EINVAL;
    }
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < R; i++) {
        const int n = qo_indptr[i + 1] - qo_indptr[i] - 1;
        int flag = 0;
        prow_t P[17], Q[17];
        if (n > 16) {
            bad = 1;
            continue;
        }
        for (int r = 0; r <= n; r++) {
            prow_t pr = {target, dtype, kind, V, temperature, (int64_t)qo_indptr[i] + r, 0.0, 0.0};
            prow_init(&pr);
            P[r] = pr;
        }
        for (int t = 1; t <= n; t++) {
            prow_t qr = {draft, dtype, kind, V, temperature, (int64_t)i * D + (t - 1), 0.0, 0.0};
            prow_init(&qr);
            Q[t] = qr;
        }
        /* steps 1-2: accept test and first-rejection cut */
        int a = n;
        for (int t = 1; t <= n; t++) {
            int d = draft_tokens[(int64_t)i * D + (t - 1)];
            double pv = 0.0, qv = 0.0;
            int acc = 0;
            if (d < 0 || d >= V) {
                flag |= 4;
            } else {
                pv = (double)prow_prob(&P[t - 1], d);
                qv = (double)prow_prob(&Q[t], d);
                acc = ((double)u_accept[(int64_t)i * D + (t - 1)] * qv < pv);
            }
            if (diag_p) diag_p[(int64_t)i * D + (t - 1)] = pv;
            if (diag_q) diag_q[(int64_t)i * D + (t - 1)] = qv;
            if (!acc) {
                a = t - 1;
                break;
            }
        }
        /* step 3: residual (after a rejection) or bonus distribution, integer CDF */
        uint64_t* w = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)V);
        uint64_t Z = 0;
        for (int v = 0; v < V; v++) {
            float r;
            if (a < n) {
                float pv = prow_prob(&P[a], v);
                float qv = prow_prob(&Q[a + 1], v);
                r = pv - qv; /* fp32 subtraction */
                if (!(r > 0.0f)) r = 0.0f;
            } else {
                r = prow_prob(&P[n], v);
            }
            w[v] = weight_of(r);
            Z += w[v];
        }
        if (Z == 0 && a < n) {
            flag |= 1;
            for (int v = 0; v < V; v++) {
                w[v] = weight_of(prow_prob(&P[a], v));
                Z += w[v];
            }
        }
        int token = -1;
        double c_before = 0.0, thr_d = 0.0, w_tok = 0.0;
        if (Z == 0) {
            flag |= 2;
        } else {
            float us = u_sample[i];
            uint64_t mu;
            if (!(us > 0.0f)) mu = 0;
            else if (us >= 1.0f) mu = (1u << 24) - 1;
            else mu = (uint64_t)((double)us * 16777216.0);
            uint64_t thr = (uint64_t)(((unsigned __int128)mu * Z) >> 24);
            uint64_t cum = 0;
            for (int v = 0; v < V; v++) {
                if (cum + w[v] > thr) {
                    token = v;
                    break;
                }
                cum += w[v];
            }
            c_before = (double)cum;
            thr_d = (double)thr;
            if (token >= 0) w_tok = (double)w[token];
        }
        if (diag_cdf) {
            diag_cdf[(int64_t)i * 4 + 0] = thr_d;
            diag_cdf[(int64_t)i * 4 + 1] = c_before;
            diag_cdf[(int64_t)i * 4 + 2] = w_tok;
            diag_cdf[(int64_t)i * 4 + 3] = (double)Z;
        }
        free(w);
        /* step 4: commit */
        for (int k = 0; k < b; k++) out_tokens[(int64_t)i * b + k] = -1;
        for (int t = 1; t <= a; t++)
            out_tokens[(int64_t)i * b + (t - 1)] = draft_tokens[(int64_t)i * D + (t - 1)];
        out_tokens[(int64_t)i * b + a] = token;
        accept_len[i] = a;
        if (flags) flags[i] = flag;
    }
    return bad ? ORC_EINVAL : ORC_OK;
}

/*
 * Greedy verification (temperature 0): the limit of the rule above when both the target
 * and the draft distributions are one-hot at their argmax (the paper evaluates T = 0).
 *   argmax of a row: the largest stored value (logits or probabilities; the softmax is
 *   monotone, so T plays no part), lowest index on ties, NaN entries skipped; -1 when
 *   every entry is NaN.
 *   1. accept draft t (t = 1..n_i) iff d_t == argmax P_{t-1};
 *   2. a_i = (first rejected t) - 1, or n_i;
 *   3. extra token = argmax P_{a_i} (the residual of two one-hot rows after a rejection,
 *      the bonus otherwise); -1 sets flag bit 1;
 *   4. commit as above.  A draft token outside [0, V) is rejected (flag bit 2).
 * Only the target rows are read.
 */
static int row_argmax(const void* base, int dtype, int64_t row, int V) {
    int best = -1;
    float bv = 0.0f;
    for (int v = 0; v < V; v++) {
        float x = load_elem(base, dtype, row, V, v);
        if (x != x) continue; /* NaN */
        if (best < 0 || x > bv) {
            best = v;
            bv = x;
        }
    }
    return best;
}

int oracle_accept_greedy(int R, int b, int V, int dtype, const void* target, const int* draft_tokens,
                         const int* qo_indptr, int* accept_len, int* out_tokens, int* flags) {
    if (R < 1 || b < 1 || V < 1) return ORC_EINVAL;
    const int D = b - 1;
    for (int i = 0; i < R; i++) {
        int n = qo_indptr[i + 1] - qo_indptr[i] - 1;
        if (n < 0 || n > D) return ORC_EINVAL;
    }
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < R; i++) {
        const int n = qo_indptr[i + 1] - qo_indptr[i] - 1;
        int flag = 0;
        int a = n;
        for (int t = 1; t <= n; t++) {
            int d = draft_tokens[(int64_t)i * D + (t - 1)];
            int acc = 0;
            if (d < 0 || d >= V) flag |= 4;
            else acc = (d == row_argmax(target, dtype, (int64_t)qo_indptr[i] + (t - 1), V));
            if (!acc) {
                a = t - 1;
                break;
            }
        }
        int token = row_argmax(target, dtype, (int64_t)qo_indptr[i] + a, V);
        if (token < 0) flag |= 2;
        for (int k = 0; k < b; k++) out_tokens[(int64_t)i * b + k] = -1;
        for (int t = 1; t <= a; t++) out_tokens[(int64_t)i * b + (t - 1)] = draft_tokens[(int64_t)i * D + (t - 1)];
        out_tokens[(int64_t)i * b + a] = token;
        accept_len[i] = a;
        if (flags) flags[i] = flag;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Verify attention (every kept position is evaluated by the target,   */
/* Sec. 4.1; packed batch of Sec. 4.2).  Plain definition, fp64:        */
/*   query row j of request i, head h sees keys s = 0 .. L_i + j,        */
/*   L_i = kv_len_i - k_i;  key s lives in page page_table[i][s / P],    */
/*   slot s % P, kv-head h / (Hq / Hkv);                                  */
/*   z_s = scale * <q, K_s>,  lse = log sum_s exp z_s,                    */
/*   o = sum_s exp(z_s - lse) V_s.                                        */
/* q [K, Hq, d]; caches [num_pages, Hkv, P, d]; dtype 0 fp32, 1 bf16.     */
/* nsel < 0: every (row, head); else the listed (sel_rows[k], sel_heads[k]). */
/* out [n, d] fp64 and lse [n] fp64 in the order of the units.           */
/* ------------------------------------------------------------------ */
int oracle_attn(int R, int Hq, int Hkv, int d, int P, int maxp, int num_pages, int dtype,
                const void* q, const void* kc, const void* vc, const int* page_table,
                const int* qo_indptr, const int* kv_lens, double scale, int nsel,
                const int* sel_rows, const int* sel_heads, double* out, double* lse) {
    if (R < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || d < 1 || P < 1) return ORC_EINVAL;
    const int G = Hq / Hkv;
    const int K = qo_indptr[R];
    const int nunits = nsel < 0 ? K * Hq : nsel;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 4)
    for (int u = 0; u < nunits; u++) {
        int row = nsel < 0 ? u / Hq : sel_rows[u];
        int h = nsel < 0 ? u % Hq : sel_heads[u];
        int i = 0;
        while (i < R && !(qo_indptr[i] <= row && row < qo_indptr[i + 1])) i++;
        if (i == R || h < 0 || h >= Hq) {
            bad = 1;
            continue;
        }
        int j = row - qo_indptr[i];
        int k_i = qo_indptr[i + 1] - qo_indptr[i];
        int L = kv_lens[i] - k_i;
        int last = L + j; /* inclusive */
        if (L < 0 || (last + P) / P > maxp) {
            bad = 1;
            continue;
        }
        int kvh = h / G;
        double* qd = (double*)malloc(sizeof(double) * (size_t)d);
        double* z = (double*)malloc(sizeof(double) * (size_t)(last + 1));
        for (int e = 0; e < d; e++)
            qd[e] = dtype == 0 ? (double)((const float*)q)[((int64_t)row * Hq + h) * d + e]
                               : (double)bf16_to_float(((const uint16_t*)q)[((int64_t)row * Hq + h) * d + e]);
        double mx = -INFINITY;
        for (int s = 0; s <= last; s++) {
            int pg = page_table[(int64_t)i * maxp + s / P];
            if (pg < 0 || pg >= num_pages) {
                bad = 1;
                z[s] = -INFINITY;
                continue;
            }
            int64_t off = (((int64_t)pg * Hkv + kvh) * P + (s % P)) * d;
            double dot = 0.0;
            for (int e = 0; e < d; e++) {
                double kv = dtype == 0 ? (double)((const float*)kc)[off + e]
                                       : (double)bf16_to_float(((const uint16_t*)kc)[off + e]);
                dot += qd[e] * kv;
            }
            z[s] = scale * dot;
            if (z[s] > mx) mx = z[s];
        }
        double den = 0.0;
        for (int s = 0; s <= last; s++) den += exp(z[s] - mx);
        double l = mx + log(den);
        double* o = out + (int64_t)u * d;
        for (int e = 0; e < d; e++) o[e] = 0.0;
        for (int s = 0; s <= last; s++) {
            int pg = page_table[(int64_t)i * maxp + s / P];
            if (pg < 0 || pg >= num_pages) continue;
            double wgt = exp(z[s] - l);
            int64_t off = (((int64_t)pg * Hkv + kvh) * P + (s % P)) * d;
            for (int e = 0; e < d; e++) {
                double vv = dtype == 0 ? (double)((const float*)vc)[off + e]
                                       : (double)bf16_to_float(((const uint16_t*)vc)[off + e]);
                o[e] += wgt * vv;
            }
        }
        lse[u] = l;
        free(qd);
        free(z);
    }
    return bad ? ORC_EINVAL : ORC_OK;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the parallel loops above (the host baseline times 1 and all). n < 1
 * leaves the setting unchanged. Returns the setting in force afterwards. */
int oracle_set_num_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
    return omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}
