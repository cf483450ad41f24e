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
 *   - Algorithm 1 (ResiSpec Sampling and Verification), with the proxy it subtracts
 *     built from Definition 1 (proxy mechanism), its probability and local-alignment
 *     constraints and Proposition 1 (global mass identity);
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

/* The proxy of Definition 1 for the residual R (in the place of the target) and the
 * draft D once the candidate x0 has been rejected (Algorithm 1 calls it with the
 * current pair; reading A-4).  Definition 1 writes the proxy as k = R - r + s:
 *
 *  - s, the slack, is fixed by the local-alignment constraint k(x0) = D(x0).  No mass
 *    can be reserved at x0 (R is exhausted there, r(x0) = 0), so s(x0) = D(x0) - R(x0);
 *    the algorithm's budget Z is exactly this gap, and by Proposition 1 (sum s = Z) the
 *    slack has no mass anywhere else.
 *  - r, the reserved mass, is the residual the proxy leaves behind (R' = r / Z).  Its
 *    ideal shape is the draft scaled to the budget, Z * D, which the target cannot
 *    always hold: r <= R caps it, and the mass the cap removes is given back to the
 *    tokens that still have headroom R_j - min(Z D_j, R_j), in proportion to that
 *    headroom (reading A-2; x0 has neither a share of the shape nor headroom), so that
 *    r sums to Z.
 *
 * The four sums the construction rests on are returned in info: Z, the capped shape's
 * mass M, the missing mass Z - M and the total headroom C. */
int32_t or_get_proxy(const double* R, const double* D, int64_t V, int64_t x0,
                     double* r, double* s, double* K, or_proxy_info* info) {
    if (!R || !D || !r || !s || !K || V <= 0 || x0 < 0 || x0 >= V) return OR_BAD_ARG;
    const double Z = D[x0] - R[x0];
    if (!(Z > 0.0)) return OR_BAD_ARG;

    /* the capped shape (kept in r for now) and its mass */
    double M = 0.0;
    for (int64_t j = 0; j < V; ++j) {
        r[j] = (j == x0) ? 0.0 : fmin(Z * D[j], R[j]);
        M += r[j];
    }
    /* headroom left under the cap, and the share of it the missing mass fills */
    double C = 0.0;
    for (int64_t j = 0; j < V; ++j) C += (j == x0) ? 0.0 : R[j] - r[j];
    const double missing = Z - M;
    const double fill = (C > 0.0) ? missing / C : 0.0;
    for (int64_t j = 0; j < V; ++j)
        if (j != x0) r[j] += fill * (R[j] - r[j]);

    /* the proxy: away from x0 there is no slack and K = R - r; at x0 the alignment
     * constraint fixes K(x0) = D(x0), which is R(x0) - r(x0) plus the slack Z */
    for (int64_t j = 0; j < V; ++j) {
        s[j] = (j == x0) ? Z : 0.0;
        K[j] = (j == x0) ? D[x0] : R[j] - r[j];
    }

    if (info) {
        info->Z = Z;
        info->M = M;
        info->delta = missing;
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

/* Scratch rows of one node's verification. */
typedef struct {
    double *R, *D, *Rn, *r, *s, *K;
} node_rows;

static int node_rows_alloc(node_rows* w, int64_t V) {
    const size_t bytes = (size_t)V * sizeof(double);
    w->R = (double*)malloc(bytes);
    w->D = (double*)malloc(bytes);
    w->Rn = (double*)malloc(bytes);
    w->r = (double*)malloc(bytes);
    w->s = (double*)malloc(bytes);
    w->K = (double*)malloc(bytes);
    return w->R && w->D && w->Rn && w->r && w->s && w->K;
}

static void node_rows_free(node_rows* w) {
    free(w->R); free(w->D); free(w->Rn); free(w->r); free(w->s); free(w->K);
}

/* The state after candidate x is rejected.  The residual loses what was subtracted for
 * the test, norm(max(R - K, 0)): K is the draft itself in the standard recurrence
 * (Eq. 2) and the proxy of Definition 1 in ResiSpec (Algorithm 1).  Without
 * replacement x also leaves the draft (reading A-6). */
static int32_t reject_candidate(node_rows* w, int64_t V, int32_t x, int32_t mode, int32_t worep) {
    const double* K = w->D;
    if (mode == OR_MODE_RESISPEC) {
        const int32_t st = or_get_proxy(w->R, w->D, V, x, w->r, w->s, w->K, NULL);
        if (st != OR_OK) return st;
        K = w->K;
    }
    const int32_t st = or_residual_update(w->R, K, V, w->Rn);
    if (st != OR_OK) return st;
    double* t = w->R;
    w->R = w->Rn;
    w->Rn = t;
    if (worep) (void)or_draft_remove(w->D, V, x);
    return OR_OK;
}

/* The checks every tested candidate passes before its ratio is formed. */
static int32_t candidate_fault(const node_rows* w, int64_t V, int32_t x, double u) {
    if (x < 0 || (int64_t)x >= V) return OR_BAD_TOKEN;
    if (!(u >= 0.0 && u < 1.0)) return OR_BAD_UNIFORM;
    if (!(w->D[x] > 0.0)) return OR_ZERO_DRAFT;
    return OR_OK;
}

/* One node (mode RESISPEC: Algorithm 1; mode SPECINFER: Eq. 2).  Candidate i is
 * accepted when its uniform falls strictly below R(x_i) / D(x_i) for the residual and
 * draft left by the candidates before it; the first accepted candidate ends the node.
 * When none is accepted (or there is none), the node's token is the inverse-CDF draw
 * from the last residual. */
int32_t or_verify_node(const double* p, const double* q, int64_t V,
                       const int32_t* cand, const float* ua, int32_t b, float ur,
                       int32_t mode, int32_t without_replacement,
                       or_node_result* res, double* final_R) {
    if (!p || !res || V <= 0 || b < 0) return OR_BAD_ARG;
    if (b > 0 && (!q || !cand || !ua)) return OR_BAD_ARG;
    if (mode != OR_MODE_RESISPEC && mode != OR_MODE_SPECINFER) return OR_BAD_ARG;
    result_init(res);
    if (final_R) memset(final_R, 0, (size_t)V * sizeof(double));

    node_rows w;
    if (!node_rows_alloc(&w, V)) {
        node_rows_free(&w);
        return OR_BAD_ARG;
    }
    const size_t bytes = (size_t)V * sizeof(double);
    memcpy(w.R, p, bytes);
    if (b > 0) memcpy(w.D, q, bytes);

    int32_t st = OR_OK;
    int32_t accepted = -1;
    for (int32_t i = 0; i < b && accepted < 0 && st == OR_OK; ++i) {
        const int32_t x = cand[i];
        const double u = (double)ua[i];
        st = candidate_fault(&w, V, x, u);
        if (st != OR_OK) break;
        const double ratio = w.R[x] / w.D[x];
        const double margin = fabs(u - ratio);
        if (margin < res->min_accept_margin) res->min_accept_margin = margin;
        if (margin < OR_FLAG_WINDOW) res->flagged = 1;
        res->n_tests += 1;
        if (u < ratio) accepted = i;
        else st = reject_candidate(&w, V, x, mode, without_replacement);
    }

    if (st == OR_OK && accepted >= 0) {
        res->kind = OR_KIND_ACCEPT;
        res->accepted_index = accepted;
        res->token = cand[accepted];
    } else if (st == OR_OK) {
        int32_t tok = -1;
        double margin = 0.0;
        st = or_invcdf(w.R, V, (double)ur, &tok, &margin);
        if (st == OR_OK) {
            res->kind = (b > 0) ? OR_KIND_RESAMPLE : OR_KIND_BONUS;
            res->token = tok;
            res->sample_margin = margin;
            if (margin < OR_FLAG_WINDOW) res->flagged = 1;
            if (final_R) memcpy(final_R, w.R, bytes);
        }
    }
    res->status = st;
    if (st != OR_OK) {
        res->kind = OR_KIND_FAULT;
        res->accepted_index = -1;
        res->token = -1;
    }
    node_rows_free(&w);
    return OR_OK;
}

/* Whether a claimed outcome of one node is admissible: every decision the claim implies
 * must be the oracle's own, except that a decision inside the flag window may go either
 * way.  The claim fixes the path through the node: candidates before claim_index are
 * rejected and claim_index is accepted, or (claim_index < 0) every candidate is
 * rejected and claim_token is drawn.  An accept test is within the window when
 * |u - ratio| < OR_FLAG_WINDOW; a draw may return any token j with R_j > 0 whose
 * interval [C_{j-1}, C_j) of the cumulative residual comes within
 * OR_FLAG_WINDOW * sum(R) of u * sum(R).  *verdict: 1 if every decision agrees outside
 * the window, 2 if the claim is admissible only through decisions inside it, 0 if it is
 * not admissible (a fault on the claimed path included). */
int32_t or_check_node_outcome(const double* p, const double* q, int64_t V,
                              const int32_t* cand, const float* ua, int32_t b, float ur,
                              int32_t mode, int32_t without_replacement,
                              int32_t claim_index, int32_t claim_token, int32_t* verdict) {
    if (!p || !verdict || V <= 0 || b < 0 || claim_index >= b) return OR_BAD_ARG;
    if (b > 0 && (!q || !cand || !ua)) return OR_BAD_ARG;
    if (mode != OR_MODE_RESISPEC && mode != OR_MODE_SPECINFER) return OR_BAD_ARG;
    *verdict = 0;
    node_rows w;
    if (!node_rows_alloc(&w, V)) {
        node_rows_free(&w);
        return OR_BAD_ARG;
    }
    const size_t bytes = (size_t)V * sizeof(double);
    memcpy(w.R, p, bytes);
    if (b > 0) memcpy(w.D, q, bytes);

    int windowed = 0, ok = 1;
    const int32_t tested = (claim_index >= 0) ? claim_index + 1 : b;
    for (int32_t i = 0; i < tested && ok; ++i) {
        const int32_t x = cand[i];
        const double u = (double)ua[i];
        if (candidate_fault(&w, V, x, u) != OR_OK) { ok = 0; break; }
        const double ratio = w.R[x] / w.D[x];
        const int accept_claimed = (i == claim_index);
        const int accept_oracle = u < ratio;
        if (accept_claimed != accept_oracle) {
            if (fabs(u - ratio) < OR_FLAG_WINDOW) windowed = 1;
            else ok = 0;
        }
        if (ok && !accept_claimed && reject_candidate(&w, V, x, mode, without_replacement) != OR_OK)
            ok = 0;
    }
    if (ok && claim_index >= 0) {
        ok = (cand[claim_index] == claim_token);
    } else if (ok) {
        const double u = (double)ur;
        double total = 0.0;
        for (int64_t j = 0; j < V; ++j) total += w.R[j];
        if (!(u >= 0.0 && u < 1.0) || !(total > 0.0) || claim_token < 0 || (int64_t)claim_token >= V) {
            ok = 0;
        } else {
            int32_t tok = -1;
            double margin = 0.0;
            (void)or_invcdf(w.R, V, u, &tok, &margin);
            if (tok != claim_token) {
                double before = 0.0;
                for (int64_t j = 0; j < claim_token; ++j) before += w.R[j];
                const double after = before + w.R[claim_token];
                const double t = u * total, win = OR_FLAG_WINDOW * total;
                if (before <= t + win && after > t - win) windowed = 1;
                else ok = 0;
            }
        }
    }
    *verdict = ok ? (windowed ? 2 : 1) : 0;
    node_rows_free(&w);
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

/* Claimed outcomes of selected nodes (rows[i] = b * N + n), checked one by one with
 * or_check_node_outcome.  A claim is (child, token, status) as the node outcome arrays
 * of a verification hold them.  A claimed fault is admissible only when the oracle's
 * own evaluation of the node ends in the same fault; a claimed child must be a child of
 * the node (its position among the children in ascending index is the claimed
 * candidate).  out_verdict[i]: 1, 2 or 0 as for one node. */
int32_t or_check_tree_nodes(const void* target, const void* draft, int32_t dtype,
                            const int32_t* node_token, const int32_t* parent,
                            const float* u_accept, const float* u_resample,
                            int32_t B, int32_t N, int64_t V, float temperature,
                            int32_t mode, int32_t without_replacement, int32_t bonus,
                            const int64_t* rows, int64_t n_rows, const int32_t* claim_child,
                            const int32_t* claim_token, const int32_t* claim_status,
                            int32_t* out_verdict) {
    if (!target || !draft || !node_token || !parent || !u_accept || !u_resample || !rows) return OR_BAD_ARG;
    if (!claim_child || !claim_token || !claim_status || !out_verdict) return OR_BAD_ARG;
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
                       &res, &child, NULL);
        if (rc != OR_OK) break;
        int32_t verdict = 0;
        if (claim_status[i] != OR_OK || res.status != OR_OK) {
            /* faults are not decisions: the claim must name the oracle's own fault */
            verdict = (claim_status[i] == res.status && claim_child[i] == -1 && claim_token[i] == -1) ? 1 : 0;
        } else if (res.kind == OR_KIND_NONE) {
            verdict = (claim_child[i] == -1 && claim_token[i] == -1) ? 1 : 0;
        } else {
            const int32_t nk = children_of(parent + (int64_t)b * N, N, n, kids);
            int32_t idx = -1, known = (claim_child[i] == -1);
            for (int32_t c = 0; c < nk; ++c)
                if (kids[c] == claim_child[i]) { idx = c; known = 1; }
            if (known) {
                rc = or_check_node_outcome(p, nk > 0 ? q : NULL, V, cand, ua, nk,
                                           u_resample[row], mode, without_replacement, idx,
                                           claim_token[i], &verdict);
                if (rc != OR_OK) break;
            }
        }
        out_verdict[i] = verdict;
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

/* Whether claimed draws of k candidates from D = softmax(draft / T) are admissible: draw
 * i, from the draft left by the claimed draws before it (without replacement), must be
 * the inverse-CDF draw of uc[i], or a token whose interval [C_{j-1}, C_j) comes within
 * OR_FLAG_WINDOW * sum(D) of uc[i] * sum(D).  *verdict: 1 every draw exact, 2 admissible
 * only through a windowed draw, 0 not admissible. */
int32_t or_check_candidates(const void* draft, int32_t dtype, int64_t V, float temperature,
                            int32_t k, int32_t without_replacement, const float* uc,
                            const int32_t* claimed, int32_t* verdict) {
    if (!draft || !verdict || V <= 0 || k < 0 || (k > 0 && (!uc || !claimed))) return OR_BAD_ARG;
    *verdict = 0;
    double* D = (double*)malloc((size_t)V * sizeof(double));
    if (!D) return OR_BAD_ARG;
    int ok = (or_softmax(draft, dtype, V, temperature, D) == OR_OK);
    int windowed = 0;
    for (int32_t i = 0; i < k && ok; ++i) {
        const int32_t c = claimed[i];
        int32_t tok = -1;
        double margin = 0.0;
        if (c < 0 || (int64_t)c >= V || or_invcdf(D, V, (double)uc[i], &tok, &margin) != OR_OK) {
            ok = 0;
            break;
        }
        if (tok != c) {
            double total = 0.0, before = 0.0;
            for (int64_t j = 0; j < V; ++j) total += D[j];
            for (int64_t j = 0; j < c; ++j) before += D[j];
            const double t = (double)uc[i] * total, win = OR_FLAG_WINDOW * total;
            if (before <= t + win && before + D[c] > t - win) windowed = 1;
            else ok = 0;
        }
        if (ok && without_replacement && i + 1 < k && or_draft_remove(D, V, c) != OR_OK) ok = 0;
    }
    *verdict = ok ? (windowed ? 2 : 1) : 0;
    free(D);
    return OR_OK;
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
