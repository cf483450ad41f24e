/*
 * resispec_oracle.c -- plain fp64 CPU oracle for the ResiSpec verification step.
 *
 * TEST INFRASTRUCTURE ONLY (see resispec_oracle.h).  Slow and literal on purpose:
 * every distribution is a full array of doubles, every sum is a sequential loop
 * in vocabulary order, and no step is fused, blocked or reordered.
 *
 * Paper sections followed:
 *   - softmax with temperature: Preliminary (target/draft distributions), and the
 *     decoding configuration of the Reproducibility appendix (temperature, nucleus 1.0);
 *   - standard residual, Eq. (1), and the multi-candidate recurrence, Eq. (2);
 *   - Algorithm 1 (ResiSpec Sampling and Verification) with its GetProxy function,
 *     read together with the Step 1-3 description that follows it;
 *   - tree walk: Preliminary, "Multi-candidate Tree-structured Verification".
 */
#include "resispec_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* bf16 bit pattern -> value.  A bf16 is the upper half of an IEEE binary32, so the
 * widening is exact. */
static double bf16_to_double(uint16_t h) {
    uint32_t bits = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static double logit_at(const void* logits, int32_t dtype, int64_t j) {
    if (dtype == OR_BF16) return bf16_to_double(((const uint16_t*)logits)[j]);
    return (double)((const float*)logits)[j];
}

/* Preliminary: p = softmax(l / T), written as exp((l_j - max l) / T) / sum. */
int32_t or_softmax(const void* logits, int32_t dtype, int64_t V, float temperature, double* out) {
    if (!logits || !out || V <= 0 || !(temperature > 0.0f)) return OR_BAD_ARG;
    if (dtype != OR_F32 && dtype != OR_BF16) return OR_BAD_ARG;
    const double T = (double)temperature;
    double m = -INFINITY;
    for (int64_t j = 0; j < V; ++j) {
        double l = logit_at(logits, dtype, j);
        if (l > m) m = l;
    }
    if (m == -INFINITY) {
        for (int64_t j = 0; j < V; ++j) out[j] = 0.0;
        return OR_UNDERFLOW;
    }
    double total = 0.0;
    for (int64_t j = 0; j < V; ++j) {
        double e = exp((logit_at(logits, dtype, j) - m) / T);
        out[j] = e;
        total += e;
    }
    for (int64_t j = 0; j < V; ++j) out[j] /= total;
    return OR_OK;
}

/* Algorithm 1, function GetProxy(p, q, x0), applied to the current residual R
 * (in the role of p) and the current draft D (in the role of q):
 *   budget      Z = D(x0) - R(x0)
 *   projection  r_j = min(Z * D_j, R_j) for j != x0, r_x0 = 0
 *   deficit     Delta = Z - sum_j r_j
 *   redistribution: Delta is spread over the remaining capacity R_j - r_j of the
 *               tokens j != x0, in proportion to that capacity (one-shot fill,
 *               x0 keeps r_x0 = 0 as the projection step fixed it)
 *   proxy       K = R - r + s, then K(x0) = D(x0); the slack s is what the last
 *               assignment adds, so it is non-zero only at x0 where r is zero
 *               (disjoint supports, Definition 1). */
int32_t or_get_proxy(const double* R, const double* D, int64_t V, int64_t x0,
                     double* r, double* s, double* K, or_proxy_info* info) {
    if (!R || !D || !r || !s || !K || V <= 0 || x0 < 0 || x0 >= V) return OR_BAD_ARG;
    const double Z = D[x0] - R[x0];
    if (!(Z > 0.0)) return OR_BAD_ARG;

    /* Step 1: budgeting and initial projection. */
    for (int64_t j = 0; j < V; ++j) {
        if (j == x0) { r[j] = 0.0; continue; }
        const double want = Z * D[j];
        r[j] = (want < R[j]) ? want : R[j];
    }
    double M = 0.0;
    for (int64_t j = 0; j < V; ++j) M += r[j];
    const double delta = Z - M;

    /* Step 2: capacity-aware redistribution of the deficit. */
    double C = 0.0;
    for (int64_t j = 0; j < V; ++j) {
        const double cap = (j == x0) ? 0.0 : (R[j] - r[j]);
        C += cap;
    }
    if (C > 0.0) {
        for (int64_t j = 0; j < V; ++j) {
            if (j == x0) continue;
            const double cap = R[j] - r[j];
            r[j] += delta * cap / C;
        }
    }

    /* Step 3: proxy formulation with the local alignment at x0. */
    for (int64_t j = 0; j < V; ++j) K[j] = R[j] - r[j];
    K[x0] = D[x0];
    for (int64_t j = 0; j < V; ++j) s[j] = K[j] - (R[j] - r[j]);

    if (info) {
        info->Z = Z;
        info->M = M;
        info->delta = delta;
        info->C = C;
    }
    return OR_OK;
}

/* R_next = norm(max(R - K, 0)): Algorithm 1's residual update with K the proxy,
 * and Eq. (1)/(2) with K the draft. */
int32_t or_residual_update(const double* R, const double* K, int64_t V, double* R_next) {
    if (!R || !K || !R_next || V <= 0) return OR_BAD_ARG;
    double total = 0.0;
    for (int64_t j = 0; j < V; ++j) {
        const double d = R[j] - K[j];
        R_next[j] = (d > 0.0) ? d : 0.0;
        total += R_next[j];
    }
    if (!(total > 0.0)) {
        for (int64_t j = 0; j < V; ++j) R_next[j] = 0.0;
        return OR_UNDERFLOW;
    }
    for (int64_t j = 0; j < V; ++j) R_next[j] /= total;
    return OR_OK;
}

/* Without-replacement candidates: the rejected id leaves the draft, which is
 * renormalised before the next sibling is verified (EAGLE integration paragraph
 * of the Reproducibility appendix: the draft is updated after each rejection). */
int32_t or_draft_remove(double* D, int64_t V, int64_t x) {
    if (!D || V <= 0 || x < 0 || x >= V) return OR_BAD_ARG;
    D[x] = 0.0;
    double total = 0.0;
    for (int64_t j = 0; j < V; ++j) total += D[j];
    if (!(total > 0.0)) {
        for (int64_t j = 0; j < V; ++j) D[j] = 0.0;
        return OR_UNDERFLOW;
    }
    for (int64_t j = 0; j < V; ++j) D[j] /= total;
    return OR_OK;
}

/* Algorithm 1's final step, x ~ R, realised as an inverse-CDF draw over the
 * vocabulary in ascending id order with one uniform. */
int32_t or_invcdf(const double* R, int64_t V, double u, int32_t* token, double* margin) {
    if (!R || !token || !margin || V <= 0) return OR_BAD_ARG;
    if (!(u >= 0.0 && u < 1.0)) return OR_BAD_UNIFORM;
    double total = 0.0;
    for (int64_t j = 0; j < V; ++j) total += R[j];
    if (!(total > 0.0)) return OR_UNDERFLOW;
    const double t = u * total;
    double c = 0.0;
    for (int64_t j = 0; j < V; ++j) {
        const double before = c;
        c += R[j];
        if (c > t) {
            const double lo = t - before, hi = c - t;
            *token = (int32_t)j;
            *margin = ((lo < hi) ? lo : hi) / total;
            return OR_OK;
        }
    }
    /* Not reachable for u < 1 with a sequential total; kept as the documented fallback. */
    for (int64_t j = V - 1; j >= 0; --j) {
        if (R[j] > 0.0) { *token = (int32_t)j; *margin = 0.0; return OR_OK; }
    }
    return OR_UNDERFLOW;
}

static void result_init(or_node_result* res) {
    res->kind = OR_KIND_FAULT;
    res->accepted_index = -1;
    res->token = -1;
    res->status = OR_OK;
    res->n_tests = 0;
    res->flagged = 0;
    res->min_accept_margin = 1e300;
    res->sample_margin = 1e300;
}

/* Algorithm 1 (mode RESISPEC) / Eq. (2) (mode SPECINFER) for one node. */
int32_t or_verify_node(const double* p, const double* q, int64_t V,
                       const int32_t* cand, const float* ua, int32_t b, float ur,
                       int32_t mode, int32_t without_replacement,
                       or_node_result* res, double* final_R) {
    if (!p || !res || V <= 0 || b < 0) return OR_BAD_ARG;
    if (b > 0 && (!q || !cand || !ua)) return OR_BAD_ARG;
    if (mode != OR_MODE_RESISPEC && mode != OR_MODE_SPECINFER) return OR_BAD_ARG;
    result_init(res);
    if (final_R) memset(final_R, 0, (size_t)V * sizeof(double));

    const size_t bytes = (size_t)V * sizeof(double);
    double* R  = (double*)malloc(bytes);
    double* D  = (double*)malloc(bytes);
    double* Rn = (double*)malloc(bytes);
    double* r  = (double*)malloc(bytes);
    double* s  = (double*)malloc(bytes);
    double* K  = (double*)malloc(bytes);
    if (!R || !D || !Rn || !r || !s || !K) {
        free(R); free(D); free(Rn); free(r); free(s); free(K);
        return OR_BAD_ARG;
    }
    memcpy(R, p, bytes);                 /* residual R <- P */
    if (b > 0) memcpy(D, q, bytes);      /* draft D <- Q */

    int32_t st = OR_OK;
    for (int32_t i = 0; i < b; ++i) {
        const int32_t x = cand[i];
        if (x < 0 || (int64_t)x >= V) { st = OR_BAD_TOKEN; goto done; }
        const double u = (double)ua[i];
        if (!(u >= 0.0 && u < 1.0)) { st = OR_BAD_UNIFORM; goto done; }
        if (!(D[x] > 0.0)) { st = OR_ZERO_DRAFT; goto done; }

        const double ratio = R[x] / D[x];
        const double margin = fabs(u - ratio);
        if (margin < res->min_accept_margin) res->min_accept_margin = margin;
        if (margin < OR_FLAG_WINDOW) res->flagged = 1;
        res->n_tests += 1;

        if (u < ratio) {                   /* accept x_i */
            res->kind = OR_KIND_ACCEPT;
            res->accepted_index = i;
            res->token = x;
            goto done;
        }
        if (mode == OR_MODE_SPECINFER) {   /* Eq. (2): K is the draft itself */
            st = or_residual_update(R, D, V, Rn);
        } else {                           /* Algorithm 1: K = GetProxy(R, D, x_i) */
            or_proxy_info info;
            st = or_get_proxy(R, D, V, x, r, s, K, &info);
            if (st == OR_OK) st = or_residual_update(R, K, V, Rn);
        }
        if (st != OR_OK) goto done;
        { double* t = R; R = Rn; Rn = t; }
        if (without_replacement) (void)or_draft_remove(D, V, x);
    }

    /* All candidates rejected (or none): draw from the current residual. */
    {
        const double u = (double)ur;
        int32_t tok = -1;
        double margin = 0.0;
        st = or_invcdf(R, V, u, &tok, &margin);
        if (st != OR_OK) goto done;
        res->kind = (b > 0) ? OR_KIND_RESAMPLE : OR_KIND_BONUS;
        res->token = tok;
        res->sample_margin = margin;
        if (margin < OR_FLAG_WINDOW) res->flagged = 1;
        if (final_R) memcpy(final_R, R, bytes);
    }

done:
    res->status = st;
    if (st != OR_OK) {
        res->kind = OR_KIND_FAULT;
        res->accepted_index = -1;
        res->token = -1;
    }
    free(R); free(D); free(Rn); free(r); free(s); free(K);
    return OR_OK;
}

int32_t or_verify_node_batch(const double* p, const double* q, int64_t V,
                             const int32_t* cand, const float* ua, const float* ur,
                             int32_t b, int64_t n_trials, int32_t mode,
                             int32_t without_replacement, int32_t* out_token,
                             int32_t* out_accepted_index) {
    if (!p || !ur || !out_token || n_trials < 0 || b < 0) return OR_BAD_ARG;
    for (int64_t t = 0; t < n_trials; ++t) {
        or_node_result res;
        int32_t rc = or_verify_node(p, q, V, cand ? cand + t * b : NULL, ua ? ua + t * b : NULL,
                                    b, ur[t], mode, without_replacement, &res, NULL);
        if (rc != OR_OK) return rc;
        out_token[t] = (res.status == OR_OK) ? res.token : -1;
        if (out_accepted_index) out_accepted_index[t] = res.accepted_index;
    }
    return OR_OK;
}

/* Exact enumeration: every candidate value x is drawn with probability D(x)
 * (the current draft), accepted with probability min(1, R(x)/D(x)) because the
 * uniform is U[0,1) and the test is strict, and otherwise the node continues with
 * the updated residual (and, without replacement, the updated draft). */
static int32_t enum_rec(const double* R, const double* D, int32_t V, int32_t level, int32_t k,
                        int32_t mode, int32_t worep, double weight, double* out) {
    if (level == k) {
        for (int32_t j = 0; j < V; ++j) out[j] += weight * R[j];
        return OR_OK;
    }
    double dsum = 0.0;
    for (int32_t j = 0; j < V; ++j) dsum += D[j];
    if (!(dsum > 0.0)) {       /* no candidate left to draw: final draw from R */
        for (int32_t j = 0; j < V; ++j) out[j] += weight * R[j];
        return OR_OK;
    }
    const size_t bytes = (size_t)V * sizeof(double);
    double* Rn = (double*)malloc(bytes);
    double* Dn = (double*)malloc(bytes);
    double* r = (double*)malloc(bytes);
    double* s = (double*)malloc(bytes);
    double* K = (double*)malloc(bytes);
    int32_t st = OR_OK;
    if (!Rn || !Dn || !r || !s || !K) { st = OR_BAD_ARG; goto out_free; }
    for (int32_t x = 0; x < V; ++x) {
        if (!(D[x] > 0.0)) continue;
        const double wx = weight * D[x];
        const double ratio = R[x] / D[x];
        const double acc = (ratio < 1.0) ? ratio : 1.0;
        out[x] += wx * acc;
        if (acc >= 1.0) continue;
        const double wrej = wx * (1.0 - acc);
        if (mode == OR_MODE_SPECINFER) {
            st = or_residual_update(R, D, V, Rn);
        } else {
            st = or_get_proxy(R, D, V, x, r, s, K, NULL);
            if (st == OR_OK) st = or_residual_update(R, K, V, Rn);
        }
        if (st != OR_OK) goto out_free;
        memcpy(Dn, D, bytes);
        if (worep) (void)or_draft_remove(Dn, V, x);
        st = enum_rec(Rn, Dn, V, level + 1, k, mode, worep, wrej, out);
        if (st != OR_OK) goto out_free;
    }
out_free:
    free(Rn); free(Dn); free(r); free(s); free(K);
    return st;
}

int32_t or_enumerate(const double* p, const double* q, int32_t V, int32_t k,
                     int32_t mode, int32_t without_replacement, double* out) {
    if (!p || !q || !out || V <= 0 || k < 0) return OR_BAD_ARG;
    if (mode != OR_MODE_RESISPEC && mode != OR_MODE_SPECINFER) return OR_BAD_ARG;
    for (int32_t j = 0; j < V; ++j) out[j] = 0.0;
    return enum_rec(p, q, V, 0, k, mode, without_replacement, 1.0, out);
}

/* ---------------------------------------------------------------- trees ---- */

static const void* row_ptr(const void* base, int32_t dtype, int64_t row, int64_t V) {
    if (dtype == OR_BF16) return (const void*)((const uint16_t*)base + row * V);
    return (const void*)((const float*)base + row * V);
}

/* A tree row is valid when node 0 is the root (parent -1) and every other node's
 * parent precedes it (topological numbering, e.g. breadth-first). */
static int tree_is_valid(const int32_t* parent, int32_t N) {
    if (N <= 0 || parent[0] != -1) return 0;
    for (int32_t n = 1; n < N; ++n)
        if (parent[n] < 0 || parent[n] >= n) return 0;
    return 1;
}

/* Children of node n in ascending node index. */
static int32_t children_of(const int32_t* parent, int32_t N, int32_t n, int32_t* kids) {
    int32_t c = 0;
    for (int32_t m = n + 1; m < N; ++m)
        if (parent[m] == n) kids[c++] = m;
    return c;
}

/* Evaluate node n of sequence b on its own (its outcome does not depend on how
 * the walk reached it: each node owns its uniforms). */
static int32_t eval_node(const void* target, const void* draft, int32_t dtype,
                         const int32_t* node_token, const int32_t* parent,
                         const float* u_accept, const float* u_resample,
                         int32_t b, int32_t N, int64_t V, float T, int32_t mode, int32_t worep,
                         int32_t bonus, int32_t n, int32_t* kids, double* p, double* q,
                         int32_t* cand, float* ua, or_node_result* res, int32_t* child,
                         double* final_R) {
    const int64_t row = (int64_t)b * N + n;
    const int32_t* par = parent + (int64_t)b * N;
    result_init(res);
    *child = -1;
    if (final_R) memset(final_R, 0, (size_t)V * sizeof(double));
    if (!tree_is_valid(par, N)) { res->status = OR_BAD_TREE; return OR_OK; }
    const int32_t nk = children_of(par, N, n, kids);
    if (nk == 0 && !bonus) { res->kind = OR_KIND_NONE; return OR_OK; }
    int32_t st = or_softmax(row_ptr(target, dtype, row, V), dtype, V, T, p);
    if (st != OR_OK) { res->status = st; res->kind = OR_KIND_FAULT; return OR_OK; }
    if (nk > 0) {
        st = or_softmax(row_ptr(draft, dtype, row, V), dtype, V, T, q);
        if (st != OR_OK) { res->status = st; res->kind = OR_KIND_FAULT; return OR_OK; }
        for (int32_t i = 0; i < nk; ++i) {
            cand[i] = node_token[(int64_t)b * N + kids[i]];
            ua[i] = u_accept[(int64_t)b * N + kids[i]];
        }
    }
    int32_t rc = or_verify_node(p, q, V, cand, ua, nk, u_resample[row], mode, worep, res, final_R);
    if (rc != OR_OK) return rc;
    if (res->status == OR_OK && res->kind == OR_KIND_ACCEPT) *child = kids[res->accepted_index];
    return OR_OK;
}

int32_t or_verify_tree_walk(const void* target, const void* draft, int32_t dtype,
                            const int32_t* node_token, const int32_t* parent,
                            const float* u_accept, const float* u_resample,
                            int32_t B, int32_t N, int64_t V, int32_t max_depth,
                            float temperature, int32_t mode, int32_t without_replacement,
                            int32_t bonus, int32_t* out_tokens, int32_t* out_len,
                            int32_t* out_status, int32_t* out_flagged) {
    if (!target || !draft || !node_token || !parent || !u_accept || !u_resample) return OR_BAD_ARG;
    if (!out_tokens || !out_len || !out_status || !out_flagged) return OR_BAD_ARG;
    if (B < 0 || N <= 0 || V <= 0 || max_depth < 0) return OR_BAD_ARG;
    const int64_t W = (int64_t)max_depth + 1;
    double* p = (double*)malloc((size_t)V * sizeof(double));
    double* q = (double*)malloc((size_t)V * sizeof(double));
    int32_t* kids = (int32_t*)malloc((size_t)N * sizeof(int32_t));
    int32_t* cand = (int32_t*)malloc((size_t)N * sizeof(int32_t));
    float* ua = (float*)malloc((size_t)N * sizeof(float));
    if (!p || !q || !kids || !cand || !ua) {
        free(p); free(q); free(kids); free(cand); free(ua);
        return OR_BAD_ARG;
    }
    for (int32_t b = 0; b < B; ++b) {
        int32_t* tok = out_tokens + (int64_t)b * W;
        for (int64_t i = 0; i < W; ++i) tok[i] = -1;
        int32_t len = 0, status = OR_OK, flagged = 0, n = 0;
        for (;;) {
            or_node_result res;
            int32_t child = -1;
            int32_t rc = eval_node(target, draft, dtype, node_token, parent, u_accept, u_resample,
                                   b, N, V, temperature, mode, without_replacement, bonus, n,
                                   kids, p, q, cand, ua, &res, &child, NULL);
            if (rc != OR_OK) { free(p); free(q); free(kids); free(cand); free(ua); return rc; }
            if (res.flagged) flagged = 1;
            if (res.status != OR_OK) { status = res.status; break; }
            if (res.kind == OR_KIND_ACCEPT) {
                if (len >= max_depth) { status = OR_DEPTH_EXCEEDED; break; }
                tok[len++] = res.token;
                n = child;
                continue;
            }
            if (res.kind == OR_KIND_RESAMPLE || res.kind == OR_KIND_BONUS) tok[len] = res.token;
            break;
        }
        if (status != OR_OK) {
            for (int64_t i = 0; i < W; ++i) tok[i] = -1;
            len = -1;
        }
        out_len[b] = len;
        out_status[b] = status;
        out_flagged[b] = flagged;
    }
    free(p); free(q); free(kids); free(cand); free(ua);
    return OR_OK;
}

int32_t or_verify_tree_nodes(const void* target, const void* draft, int32_t dtype,
                             const int32_t* node_token, const int32_t* parent,
                             const float* u_accept, const float* u_resample,
                             int32_t B, int32_t N, int64_t V, float temperature,
                             int32_t mode, int32_t without_replacement, int32_t bonus,
                             const int64_t* rows, int64_t n_rows,
                             int32_t* out_child, int32_t* out_token, int32_t* out_status,
                             int32_t* out_flagged, double* out_margin, double* out_final_R) {
    if (!target || !draft || !node_token || !parent || !u_accept || !u_resample || !rows) return OR_BAD_ARG;
    if (!out_child || !out_token || !out_status || !out_flagged) return OR_BAD_ARG;
    if (B < 0 || N <= 0 || V <= 0 || n_rows < 0) return OR_BAD_ARG;
    double* p = (double*)malloc((size_t)V * sizeof(double));
    double* q = (double*)malloc((size_t)V * sizeof(double));
    int32_t* kids = (int32_t*)malloc((size_t)N * sizeof(int32_t));
    int32_t* cand = (int32_t*)malloc((size_t)N * sizeof(int32_t));
    float* ua = (float*)malloc((size_t)N * sizeof(float));
    if (!p || !q || !kids || !cand || !ua) {
        free(p); free(q); free(kids); free(cand); free(ua);
        return OR_BAD_ARG;
    }
    int32_t rc = OR_OK;
    for (int64_t i = 0; i < n_rows; ++i) {
        const int64_t row = rows[i];
        if (row < 0 || row >= (int64_t)B * N) { rc = OR_BAD_ARG; break; }
        const int32_t b = (int32_t)(row / N), n = (int32_t)(row % N);
        or_node_result res;
        int32_t child = -1;
        rc = eval_node(target, draft, dtype, node_token, parent, u_accept, u_resample, b, N, V,
                       temperature, mode, without_replacement, bonus, n, kids, p, q, cand, ua,
                       &res, &child, out_final_R ? out_final_R + i * V : NULL);
        if (rc != OR_OK) break;
        out_child[i] = child;
        out_token[i] = res.token;
        out_status[i] = res.status;
        out_flagged[i] = res.flagged;
        if (out_margin) {
            out_margin[i] = (res.min_accept_margin < res.sample_margin) ? res.min_accept_margin
                                                                        : res.sample_margin;
        }
    }
    free(p); free(q); free(kids); free(cand); free(ua);
    return rc;
}

/* ------------------------------------------------------------------------------------
 * The draft step: Philox4x32-10 uniforms and candidate draws.
 * ---------------------------------------------------------------------------------- */

void or_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {              /* key schedule: add the Weyl constants */
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

float or_u01(uint32_t w) { return (float)(w >> 8) * (1.0f / 16777216.0f); }

void or_node_uniforms(uint64_t seed, uint64_t offset, int32_t b, int32_t n, float* ua,
                      float* ur, float* uc) {
    const uint32_t ctr[4] = {(uint32_t)n, (uint32_t)b, (uint32_t)offset, (uint32_t)(offset >> 32)};
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    or_philox4x32_10(ctr, key, w);
    if (ua) *ua = or_u01(w[0]);
    if (ur) *ur = or_u01(w[1]);
    if (uc) *uc = or_u01(w[2]);
}

int32_t or_sample_candidates(const void* draft, int32_t dtype, int64_t V, float temperature,
                             int32_t k, int32_t without_replacement, const float* uc,
                             int32_t* tokens, double* margins) {
    if (!draft || V <= 0 || k < 0 || (k > 0 && (!uc || !tokens || !margins))) return OR_BAD_ARG;
    double* D = (double*)malloc((size_t)V * sizeof(double));
    if (!D) return OR_BAD_ARG;
    int32_t st = or_softmax(draft, dtype, V, temperature, D);
    for (int32_t i = 0; i < k; ++i) {
        tokens[i] = -1;
        margins[i] = 0.0;
    }
    if (st == OR_OK) {
        for (int32_t i = 0; i < k; ++i) {
            int32_t tok = -1;
            double margin = 0.0;
            st = or_invcdf(D, V, (double)uc[i], &tok, &margin);
            if (st != OR_OK) break;
            tokens[i] = tok;
            margins[i] = margin;
            if (without_replacement && i + 1 < k) {
                st = or_draft_remove(D, V, tok);
                if (st != OR_OK) break;
            }
        }
    }
    free(D);
    return st;
}

int32_t or_draft_tree(const void* draft, int32_t dtype, const int32_t* parent, int32_t B,
                      int32_t N, int64_t V, float temperature, int32_t without_replacement,
                      uint64_t seed, uint64_t offset, int32_t* node_token, float* u_accept,
                      float* u_resample, int32_t* flagged, double* margin) {
    if (!draft || !parent || !node_token || !u_accept || !u_resample || !flagged || !margin ||
        B < 0 || N <= 0 || V <= 0)
        return OR_BAD_ARG;
    int32_t* kids = (int32_t*)malloc((size_t)N * sizeof(int32_t));
    int32_t* toks = (int32_t*)malloc((size_t)N * sizeof(int32_t));
    float* uc = (float*)malloc((size_t)N * sizeof(float));
    double* mg = (double*)malloc((size_t)N * sizeof(double));
    if (!kids || !toks || !uc || !mg) {
        free(kids); free(toks); free(uc); free(mg);
        return OR_BAD_ARG;
    }
    int32_t status = OR_OK;
    for (int32_t b = 0; b < B; ++b) {
        const int32_t* par = parent + (int64_t)b * N;
        int32_t* nt = node_token + (int64_t)b * N;
        for (int32_t n = 0; n < N; ++n) {
            or_node_uniforms(seed, offset, b, n, &u_accept[(int64_t)b * N + n],
                             &u_resample[(int64_t)b * N + n], NULL);
            nt[n] = -1;
            flagged[(int64_t)b * N + n] = 0;
            margin[(int64_t)b * N + n] = 1e300;
        }
        if (!tree_is_valid(par, N)) {
            status = OR_BAD_TREE;
            continue;
        }
        for (int32_t n = 0; n < N; ++n) {
            const int32_t k = children_of(par, N, n, kids);
            if (k == 0) continue;
            for (int32_t i = 0; i < k; ++i) or_node_uniforms(seed, offset, b, kids[i], NULL, NULL, &uc[i]);
            const void* row = row_ptr(draft, dtype, (int64_t)b * N + n, V);
            const int32_t st = or_sample_candidates(row, dtype, V, temperature, k, without_replacement,
                                                    uc, toks, mg);
            for (int32_t i = 0; i < k; ++i) {
                nt[kids[i]] = (st == OR_OK) ? toks[i] : -1;
                margin[(int64_t)b * N + kids[i]] = mg[i];
                flagged[(int64_t)b * N + kids[i]] = (st == OR_OK && mg[i] < OR_FLAG_WINDOW) ? 1 : 0;
            }
        }
    }
    free(kids); free(toks); free(uc); free(mg);
    return status;
}
