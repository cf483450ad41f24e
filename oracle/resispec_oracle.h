/*
 * resispec_oracle.h -- plain fp64 CPU oracle for the ResiSpec verification step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link or
 * call this code: only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg use it.  It shares no header, helper, table or
 * constant with the GPU library; its status codes are defined here on their own.
 *
 * Every function follows the paper ("ResiSpec: Enhancing Multi-Candidate
 * Speculative Sampling via Residual Distribution Shaping") step by step in
 * double precision and materialises every intermediate the paper names
 * (r, Delta, capacity, s, K, the residual R), so that the GPU's closed-form
 * evaluation is checked against the literal procedure.
 *
 * Layout conventions: logits rows are contiguous over the vocabulary; a tree
 * batch is [B][N][V]; fp32 logits are `float`, bf16 logits are passed as
 * their raw 16-bit patterns (`uint16_t`) and widened exactly.
 */
#ifndef RESISPEC_ORACLE_H
#define RESISPEC_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes (per node / per sequence). */
#define OR_OK                 0
#define OR_BAD_TOKEN          1  /* candidate id outside [0, V) */
#define OR_ZERO_DRAFT         2  /* candidate whose current draft probability is 0 */
#define OR_UNDERFLOW          3  /* residual (or softmax) total is 0 */
#define OR_BAD_TREE           4  /* parent array is not a rooted topological tree */
#define OR_BAD_UNIFORM        5  /* a uniform outside [0, 1) */
#define OR_DEPTH_EXCEEDED     6  /* accepted path longer than max_depth */
#define OR_BAD_ARG           -1  /* invalid call (NULL, sizes) */

/* Modes. */
#define OR_MODE_RESISPEC   0     /* Algorithm 1 with GetProxy */
#define OR_MODE_SPECINFER  1     /* standard recurrence, Eq. (2) */

/* Logits element types. */
#define OR_F32   0
#define OR_BF16  1

/* Outcome kinds of one node. */
#define OR_KIND_ACCEPT    0   /* a candidate was accepted */
#define OR_KIND_RESAMPLE  1   /* every candidate rejected; token drawn from the final residual */
#define OR_KIND_BONUS     2   /* node without candidates; token drawn from p */
#define OR_KIND_NONE      3   /* node without candidates and bonus sampling off */
#define OR_KIND_FAULT     4

/* Flag window: a decision whose margin is below this is reported as flagged. */
#define OR_FLAG_WINDOW 1e-6

typedef struct {
    int32_t kind;            /* OR_KIND_* */
    int32_t accepted_index;  /* position in the candidate list, -1 if none */
    int32_t token;           /* accepted candidate id or sampled id, -1 if none */
    int32_t status;          /* OR_OK or a fault code */
    int32_t n_tests;         /* accept tests performed */
    int32_t flagged;         /* 1 if a decision margin fell inside the flag window */
    double  min_accept_margin; /* min |u - ratio| over the tests performed (1e300 if none) */
    double  sample_margin;     /* inverse-CDF margin / total (1e300 if no draw) */
} or_node_result;

typedef struct {
    double Z;        /* budget q(x0) - p(x0) */
    double M;        /* sum of the clipped projection before redistribution */
    double delta;    /* Z - M */
    double C;        /* remaining capacity sum over j != x0 */
} or_proxy_info;

/* softmax((l - max l) / T) in fp64.  Returns OR_OK, OR_UNDERFLOW (all -inf) or OR_BAD_ARG. */
int32_t or_softmax(const void* logits, int32_t dtype, int64_t V, float temperature, double* out);

/* The proxy K = R - r + s of Definition 1 after the rejection of x0 (Algorithm 1's
 * GetProxy, applied to the current residual R and draft D): writes r (reserved mass),
 * s (slack) and K.  Requires D[x0] > R[x0].  Returns OR_OK or OR_BAD_ARG. */
int32_t or_get_proxy(const double* R, const double* D, int64_t V, int64_t x0,
                     double* r, double* s, double* K, or_proxy_info* info);

/* R_next = norm(max(R - K, 0)).  Used with K = proxy (ResiSpec) or K = D (Eq. 2). */
int32_t or_residual_update(const double* R, const double* K, int64_t V, double* R_next);

/* Without-replacement draft update: D <- norm(D * 1[j != x]). */
int32_t or_draft_remove(double* D, int64_t V, int64_t x);

/* Inverse-CDF draw in ascending vocabulary order: smallest j with C_j > u * sum(R).
 * Writes the token and the margin min(t - C_{j-1}, C_j - t) / sum(R). */
int32_t or_invcdf(const double* R, int64_t V, double u, int32_t* token, double* margin);

/* One node: sequential accept/reject of b candidates, residual updates, final draw.
 * p, q: target and draft distributions.  cand[b], ua[b]: candidates and their uniforms.
 * ur: uniform of the final draw.  final_R (optional, V doubles) receives the
 * distribution the final draw used (zeros if a candidate was accepted). */
int32_t or_verify_node(const double* p, const double* q, int64_t V,
                       const int32_t* cand, const float* ua, int32_t b, float ur,
                       int32_t mode, int32_t without_replacement,
                       or_node_result* res, double* final_R);

/* Whether a claimed outcome of one node (claim_index >= 0: that candidate accepted and
 * claim_token its id; claim_index < 0: every candidate rejected and claim_token drawn)
 * is admissible when decisions inside the flag window may go either way.
 * *verdict: 1 every decision agrees outside the window, 2 admissible only through
 * decisions inside it, 0 not admissible. */
int32_t or_check_node_outcome(const double* p, const double* q, int64_t V,
                              const int32_t* cand, const float* ua, int32_t b, float ur,
                              int32_t mode, int32_t without_replacement,
                              int32_t claim_index, int32_t claim_token, int32_t* verdict);

/* Same node, many independent trials (statistics tests): cand[n][b], ua[n][b], ur[n]. */
int32_t or_verify_node_batch(const double* p, const double* q, int64_t V,
                             const int32_t* cand, const float* ua, const float* ur,
                             int32_t b, int64_t n_trials, int32_t mode,
                             int32_t without_replacement, int32_t* out_token,
                             int32_t* out_accepted_index);

/* Exact output distribution of one node with k candidates drawn from the current
 * draft (i.i.d. from q, or sequentially without replacement), by recursion over
 * every candidate value with analytic accept probabilities.  out[V]. */
int32_t or_enumerate(const double* p, const double* q, int32_t V, int32_t k,
                     int32_t mode, int32_t without_replacement, double* out);

/* Tree batch, sequential walk: per sequence, start at the root, verify the
 * children of the current node in ascending node index, descend on accept,
 * stop on a resample or at a leaf (bonus draw when bonus != 0).
 * Outputs per sequence: tokens[B][max_depth+1] (-1 padded), accepted length,
 * status, flagged, and the min margin seen on the walked path. */
int32_t or_verify_tree_walk(const void* target, const void* draft, int32_t dtype,
                            const int32_t* node_token, const int32_t* parent,
                            const float* u_accept, const float* u_resample,
                            int32_t B, int32_t N, int64_t V, int32_t max_depth,
                            float temperature, int32_t mode, int32_t without_replacement,
                            int32_t bonus, int32_t* out_tokens, int32_t* out_len,
                            int32_t* out_status, int32_t* out_flagged);

/* Tree batch, independent evaluation of selected nodes (rows[i] = b * N + n).
 * child[i]: accepted child node index or -1; token[i]: the node's emitted token
 * (accepted candidate's id, resampled id, bonus id, or -1); status/flagged per node;
 * margin: the smallest decision margin of the node (accept tests and the draw). */
int32_t or_verify_tree_nodes(const void* target, const void* draft, int32_t dtype,
                             const int32_t* node_token, const int32_t* parent,
                             const float* u_accept, const float* u_resample,
                             int32_t B, int32_t N, int64_t V, float temperature,
                             int32_t mode, int32_t without_replacement, int32_t bonus,
                             const int64_t* rows, int64_t n_rows,
                             int32_t* out_child, int32_t* out_token, int32_t* out_status,
                             int32_t* out_flagged, double* out_margin /* n_rows or NULL */,
                             double* out_final_R /* n_rows*V or NULL */);

/* Claimed (child, token, status) outcomes of selected nodes checked against the
 * oracle with or_check_node_outcome; out_verdict[n_rows] as there.  A claimed fault
 * must be the oracle's own fault of that node. */
int32_t or_check_tree_nodes(const void* target, const void* draft, int32_t dtype,
                            const int32_t* node_token, const int32_t* parent,
                            const float* u_accept, const float* u_resample,
                            int32_t B, int32_t N, int64_t V, float temperature,
                            int32_t mode, int32_t without_replacement, int32_t bonus,
                            const int64_t* rows, int64_t n_rows, const int32_t* claim_child,
                            const int32_t* claim_token, const int32_t* claim_status,
                            int32_t* out_verdict);

/* ---- the draft step: uniforms and candidate draws (run before verification) ---- */

/* Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as
 * 1, 2, 3", SC'11): ten rounds over the 4-word counter, each round two 32x32->64
 * multiplications and xors with the 2-word key, the key advanced by the Weyl
 * constants between rounds. */
void or_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Uniform in [0, 1) from a 32-bit word: its top 24 bits times 2^-24 (exact in fp32). */
float or_u01(uint32_t w);

/* The uniforms of node n of sequence b: Philox4x32-10 of counter
 * (n, b, offset low word, offset high word) under key (seed low word, seed high word);
 * word 0 -> u_accept, word 1 -> u_resample, word 2 -> uc, the uniform that draws node
 * n's own token from its parent's draft distribution. */
void or_node_uniforms(uint64_t seed, uint64_t offset, int32_t b, int32_t n, float* ua,
                      float* ur, float* uc);

/* k candidates from D = softmax(draft / T): candidate i is the inverse-CDF draw
 * (or_invcdf) of D with uniform uc[i]; without replacement D loses the drawn token and
 * is renormalised (or_draft_remove) before the next draw.  tokens[k], margins[k]. */
int32_t or_sample_candidates(const void* draft, int32_t dtype, int64_t V, float temperature,
                             int32_t k, int32_t without_replacement, const float* uc,
                             int32_t* tokens, double* margins);

/* Whether claimed draws claimed[k] of k candidates are admissible draws of
 * or_sample_candidates with uniforms uc[k]: each draw (from the draft left by the
 * claimed draws before it, without replacement) exact, or within the flag window of its
 * inverse-CDF boundary.  *verdict: 1 all exact, 2 admissible through a windowed draw,
 * 0 not admissible. */
int32_t or_check_candidates(const void* draft, int32_t dtype, int64_t V, float temperature,
                            int32_t k, int32_t without_replacement, const float* uc,
                            const int32_t* claimed, int32_t* verdict);

/* The draft step of a tree batch: for every node with children, its children's
 * tokens drawn from its draft row (children in ascending node index), and every
 * node's u_accept / u_resample.  node_token[.,0] = -1.  flagged[b][n] = 1 when node
 * n's draw margin is below OR_FLAG_WINDOW; margin[b][n] the margin (1e300 for the
 * root).  Returns OR_BAD_TREE for a malformed parent array, else OR_OK (per-row
 * underflow leaves that row's children at -1). */
int32_t or_draft_tree(const void* draft, int32_t dtype, const int32_t* parent, int32_t B,
                      int32_t N, int64_t V, float temperature, int32_t without_replacement,
                      uint64_t seed, uint64_t offset, int32_t* node_token, float* u_accept,
                      float* u_resample, int32_t* flagged, double* margin);

#ifdef __cplusplus
}
#endif
#endif /* RESISPEC_ORACLE_H */
