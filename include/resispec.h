/*
 * resispec.h -- C ABI of libresispec.so, the MI355X (gfx950) verification step of
 * ResiSpec multi-candidate speculative sampling.
 *
 * What it computes (paper: "ResiSpec: Enhancing Multi-Candidate Speculative
 * Sampling via Residual Distribution Shaping"):
 *   for every node of a batch of draft trees, the temperature softmax of the
 *   target and draft logits over the whole vocabulary (Preliminary), the
 *   sequential accept/reject of the node's candidates with acceptance
 *   min(1, R(x)/D(x)) against the current residual R (Eq. 2, Algorithm 1), the
 *   residual update after each rejection -- the standard norm(max(R - D, 0))
 *   (Eq. 1/2, mode RS_MODE_SPECINFER) or ResiSpec's proxy-shaped residual
 *   norm(max(R - GetProxy(R, D, x), 0)) (Algorithm 1, mode RS_MODE_RESISPEC) --
 *   and the inverse-CDF draw from the final residual when every candidate is
 *   rejected; then a walk from each root that follows accepted children and
 *   returns the accepted tokens (Preliminary, tree-structured verification).
 *
 * Conventions shared by every entry point:
 *   - All array arguments are DEVICE pointers owned by the caller unless stated
 *     otherwise.  The library never allocates, frees or keeps them.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *     stream).  Results are valid once the stream reaches the call.  No entry
 *     point synchronises the device.
 *   - Argument errors are returned synchronously as rs_status and nothing is
 *     launched.  Data faults found on the device (bad token ids, a candidate
 *     with zero draft probability, a malformed tree, out-of-range uniforms) are
 *     reported per row / per sequence in out_status (rs_seq_status); the outputs
 *     of such a row/sequence are -1.
 *   - Logits rows are contiguous over the vocabulary.  fp32 or bf16 (raw bf16,
 *     widened exactly to fp32 in the kernel).  Rows whose byte length is a
 *     multiple of 16 and whose base pointer is 16-byte aligned take the
 *     vectorised path; any other V or alignment is handled element by element.
 *   - Uniforms are fp32 in [0, 1).  The accept test is strict: u < ratio.
 *   - Thread safety: calls are stateless and re-entrant.
 */
#ifndef RESISPEC_H
#define RESISPEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RESISPEC_ABI_VERSION 3

/* Largest number of candidates (children) one node may have. */
#define RS_MAX_CANDIDATES 64
/* Largest supported vocabulary. */
#define RS_MAX_VOCAB (1 << 22)

typedef enum {
    RS_OK = 0,
    RS_ERR_INVALID_ARG = 1,  /* NULL pointer, non-positive size, T <= 0, unknown mode/dtype */
    RS_ERR_WORKSPACE = 2,    /* workspace NULL or smaller than resispec_workspace_bytes() */
    RS_ERR_UNSUPPORTED = 3,  /* size beyond RS_MAX_VOCAB / RS_MAX_CANDIDATES, or a row
                                group that cannot run on this device */
    RS_ERR_HIP = 4           /* a HIP launch error */
} rs_status;

/* Per-row / per-sequence device-side status (out_status). */
typedef enum {
    RS_SEQ_OK = 0,
    RS_SEQ_BAD_TOKEN = 1,        /* candidate id outside [0, V) */
    RS_SEQ_ZERO_DRAFT = 2,       /* a tested candidate has current draft probability 0 */
    RS_SEQ_UNDERFLOW = 3,        /* softmax or residual total is 0 (e.g. an all -inf row) */
    RS_SEQ_BAD_TREE = 4,         /* parent[.,0] != -1 or parent[n] not in [0, n) */
    RS_SEQ_BAD_UNIFORM = 5,      /* a used uniform outside [0, 1) */
    RS_SEQ_DEPTH_EXCEEDED = 6,   /* accepted path longer than max_depth */
    RS_SEQ_TOO_MANY_CHILDREN = 7, /* a node with more than RS_MAX_CANDIDATES children */
    RS_SEQ_GROUP_TIMEOUT = 8,    /* row groups: a workgroup did not receive the others'
                                    slot totals of a pass within 20 ms */
    RS_SEQ_DEFERRED = 9          /* node outcomes of resispec_decide_nodes only: the node
                                    rejected its one candidate, or is a leaf, and its draw
                                    is left to the walk (resispec_walk_draw), which makes it
                                    only where a walk ends */
} rs_seq_status;

typedef enum { RS_MODE_RESISPEC = 0, RS_MODE_SPECINFER = 1 } rs_mode;
typedef enum { RS_F32 = 0, RS_BF16 = 1 } rs_dtype;

typedef struct {
    int32_t mode;                /* rs_mode */
    int32_t logits_dtype;        /* rs_dtype, same for target and draft */
    float   temperature;         /* > 0; softmax((l - max l) / T) for target and draft alike */
    int32_t without_replacement; /* 1: candidates of a node were drawn without replacement;
                                    each rejected id leaves the draft, which is renormalised
                                    before the next sibling is tested */
    int32_t bonus;               /* tree only: 1 = a walk that ends at a leaf draws one more
                                    token from that leaf's target distribution */
} rs_params;

/*
 * Flat verify: row b of the target/draft logits is one position with k candidates
 * (Eq. 2 / Algorithm 1 on a single node per row).
 *   target_logits, draft_logits : [B][V] fp32 or bf16 (prm->logits_dtype)
 *   cand_ids                    : [B][k] int32, verified in column order
 *   u_accept                    : [B][k] fp32, column i is the uniform of candidate i
 *   u_resample                  : [B]    fp32, uniform of the final draw
 *   out_token                   : [B] int32  accepted candidate id, or the id drawn
 *                                 from the final residual when all k are rejected
 *   out_accepted_len            : [B] int32  1 if a candidate was accepted, else 0
 *   out_status                  : [B] int32  rs_seq_status; may be NULL
 * k = 0 draws directly from the target distribution.  B = 0 is a no-op.
 */
rs_status resispec_verify(const void* target_logits, const void* draft_logits,
                          const int32_t* cand_ids, const float* u_accept,
                          const float* u_resample, int32_t B, int32_t V, int32_t k,
                          const rs_params* prm, int32_t* out_token,
                          int32_t* out_accepted_len, int32_t* out_status, void* stream);

/*
 * Tree verify over B sequences of N nodes each (node 0 = root): Algorithm 1 at every node
 * (accept test Eq. 2; residual update Eq. 1/2 or GetProxy by prm->mode), then the walk
 * down the accepted children of the tree-structured verification (§Preliminary).
 *   target_logits, draft_logits : [B][N][V]; row n is the target / draft distribution
 *                                 over the tokens that follow node n (the distribution
 *                                 node n's children were drawn from).  Draft rows of
 *                                 leaf nodes are never read.
 *   node_token                  : [B][N] int32 token of each node (entry 0 ignored)
 *   parent                      : [B][N] int32 parent node, parent[.,0] = -1 and
 *                                 parent[.,n] in [0, n) (topological numbering)
 *   u_accept                    : [B][N] fp32, entry n is used when node n is tested
 *   u_resample                  : [B][N] fp32, entry n is used when node n draws from its
 *                                 final residual (all children rejected) or its bonus
 *   max_depth                   : >= depth of the deepest node; out_tokens row width is
 *                                 max_depth + 1
 *   out_tokens                  : [B][max_depth+1] int32 accepted draft tokens followed by
 *                                 the drawn token, padded with -1
 *   out_accepted_len            : [B] int32 number of accepted draft tokens (-1 on a fault)
 *   out_status                  : [B] int32 rs_seq_status; may be NULL
 *   workspace                   : device buffer of at least resispec_workspace_bytes(B, N)
 *                                 bytes (per-node outcomes); contents on entry are ignored
 * Children of a node are tested in ascending node index.  Every node's outcome is
 * computed independently (each node owns its uniforms), then a walk from the root
 * follows accepted children; the result equals the sequential walk.
 */
rs_status resispec_verify_tree(const void* target_logits, const void* draft_logits,
                               const int32_t* node_token, const int32_t* parent,
                               const float* u_accept, const float* u_resample,
                               int32_t B, int32_t N, int32_t V, int32_t max_depth,
                               const rs_params* prm, int32_t* out_tokens,
                               int32_t* out_accepted_len, int32_t* out_status,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * The all-nodes schedule of resispec_verify_tree with deferred draws (same arguments, same
 * results, bit for bit).  A node's draw from its final residual, and a leaf's bonus draw,
 * matter only where a walk ends (§Preliminary, tree-structured verification: the walk
 * draws once, at the node where it stops), so they are made there.  Two launches:
 *   - every node row with children takes pass 1 (the softmax statistics of Preliminary)
 *     and its tests (Eq. 2, Algorithm 1); a row with several candidates also takes the
 *     rejection passes its later tests need, and draws at once if it rejects them all; a
 *     row with one candidate that it rejects keeps its pass-1 slot totals in the
 *     workspace instead of drawing (no rejection pass re-reads its logits); a leaf's row,
 *     which serves only its bonus draw, is not read;
 *   - one workgroup per sequence walks the decisions and, where the walk ends at such a
 *     row, takes it up again: the residual pass of its rejection (Eq. 1/2 or GetProxy)
 *     over that row alone, or a leaf's pass 1, then the inverse-CDF draw, with the same
 *     arithmetic on the same values as resispec_verify_tree.
 *   workspace : device buffer of at least resispec_deferred_workspace_bytes(B, N) bytes,
 *               16-byte aligned (node outcomes, then 2 KiB of slot totals per node row);
 *               contents on entry are ignored.  Calls that overlap on one workspace race.
 * Errors and statuses as resispec_verify_tree.
 */
rs_status resispec_verify_tree_deferred(const void* target_logits, const void* draft_logits,
                                        const int32_t* node_token, const int32_t* parent,
                                        const float* u_accept, const float* u_resample,
                                        int32_t B, int32_t N, int32_t V, int32_t max_depth,
                                        const rs_params* prm, int32_t* out_tokens,
                                        int32_t* out_accepted_len, int32_t* out_status,
                                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * The two launches of resispec_verify_tree_deferred, for callers that schedule them
 * separately (same kernels, same results):
 *   resispec_decide_nodes: every node's tests into `workspace`; node outcomes (see
 *     resispec_node_outcomes, which reads this workspace too) are the accepted child,
 *     the drawn token of a row with several candidates that rejected them all, a fault,
 *     or RS_SEQ_DEFERRED;
 *   resispec_walk_draw: the walk from each root over those outcomes, with the deferred
 *     draw where a walk ends (same inputs, and the workspace written by
 *     resispec_decide_nodes with the same B and N, earlier on the same stream); it
 *     records the outcome of each node it draws for in the workspace.
 * resispec_walk over such a workspace draws nothing: a walk that ends at a deferred node
 * reports RS_SEQ_DEFERRED as its status.
 */
rs_status resispec_decide_nodes(const void* target_logits, const void* draft_logits,
                                const int32_t* node_token, const int32_t* parent,
                                const float* u_accept, const float* u_resample,
                                int32_t B, int32_t N, int32_t V, const rs_params* prm,
                                void* workspace, size_t workspace_bytes, void* stream);

rs_status resispec_walk_draw(const void* target_logits, const void* draft_logits,
                             const int32_t* node_token, const int32_t* parent,
                             const float* u_accept, const float* u_resample,
                             int32_t B, int32_t N, int32_t V, int32_t max_depth,
                             const rs_params* prm, void* workspace, size_t workspace_bytes,
                             int32_t* out_tokens, int32_t* out_accepted_len,
                             int32_t* out_status, void* stream);

/* Workspace bytes resispec_verify_tree_deferred needs for B sequences of N nodes (0 if
 * B <= 0 or N <= 0). */
size_t resispec_deferred_workspace_bytes(int32_t B, int32_t N);

/*
 * resispec_verify_tree without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, kernels and results as resispec_verify_tree; the
 * per-node outcomes go to a static device array of the library (one per GPU, held until
 * the process ends) sized for RS_NOALLOC_MAX_ROWS node rows (768 KiB).  The call
 * allocates nothing and nothing needs clearing: every call writes all B * N outcomes
 * before its walk reads them.  All calls on one GPU share that array, so calls that
 * overlap on one GPU (on different streams, or from different threads) race; calls
 * ordered on one stream do not.
 * RS_ERR_UNSUPPORTED when B * N > RS_NOALLOC_MAX_ROWS; RS_ERR_HIP if the array's device
 * address cannot be found; otherwise the errors of resispec_verify_tree.
 */
#define RS_NOALLOC_MAX_ROWS 65536
rs_status resispec_verify_tree_noalloc(const void* target_logits, const void* draft_logits,
                                       const int32_t* node_token, const int32_t* parent,
                                       const float* u_accept, const float* u_resample,
                                       int32_t B, int32_t N, int32_t V, int32_t max_depth,
                                       const rs_params* prm, int32_t* out_tokens,
                                       int32_t* out_accepted_len, int32_t* out_status,
                                       void* stream);

/*
 * Path-only schedule of resispec_verify_tree (same arguments without the workspace, same
 * results): one workgroup per sequence walks its tree from the root and verifies only
 * the nodes the walk reaches, one after another (Preliminary, tree-structured
 * verification: a node is verified only after its parent accepted it).  It reads the
 * rows of about accepted_len + 1 nodes per sequence instead of all N, and runs
 * B workgroups.  Per-node outcomes are the same functions of the node's rows and
 * uniforms as in the all-nodes schedule, so the tokens, lengths and statuses are
 * identical, faults included: both report only what the walk meets (a malformed
 * parent array is met at the root, whose row checks the whole array).
 */
rs_status resispec_verify_tree_path(const void* target_logits, const void* draft_logits,
                                    const int32_t* node_token, const int32_t* parent,
                                    const float* u_accept, const float* u_resample,
                                    int32_t B, int32_t N, int32_t V, int32_t max_depth,
                                    const rs_params* prm, int32_t* out_tokens,
                                    int32_t* out_accepted_len, int32_t* out_status, void* stream);

/*
 * The path-only schedule (§Preliminary walk, Algorithm 1 at each node it reaches) with row
 * groups, for batches too small to fill the device with one workgroup per sequence (same
 * results as resispec_verify_tree_path and resispec_verify_tree, bit for bit). Each
 * sequence gets `group_size` 512-thread workgroups that verify every row of its walk
 * together: each sweeps its share of the row's slots in every pass, and after a pass they
 * exchange their slots' totals through `workspace` (64-bit words tagged with the pass, so
 * a reader waits for the words of the current pass and no fence is needed).  The group
 * forms only when all its workgroups have started within 20 us of the first; otherwise
 * the first to give up waiting does the sequence alone (same results).  Every wait is
 * bounded: a workgroup that does not receive the others' totals within 20 ms reports
 * RS_SEQ_GROUP_TIMEOUT.
 *   group_size      : 0 = automatic (as many members as the device holds at once, up to
 *                     16 and to one per 4 slots of a row; 1 when that is under 2 or
 *                     workspace is NULL), 1 = one workgroup per sequence,
 *                     2..16 = that many (RS_ERR_UNSUPPORTED if B * group_size workgroups
 *                     cannot be resident at once or if a row has fewer slots than
 *                     members)
 *   workspace       : device buffer of at least resispec_path_workspace_bytes(B, V) bytes,
 *                     16-byte aligned, caller-owned; its counters and exchange words are
 *                     zeroed by the call itself (on `stream`) before the verification
 *                     kernel, and its residual rows need no initial contents; NULL allowed
 *                     when group_size is 0 or 1 (the later rejection passes then re-derive
 *                     the residual from the logits: same results; they also do so when B *
 *                     group_size exceeds the device's compute units, where the cache's
 *                     traffic costs more than it saves).  Calls that overlap on one
 *                     workspace race.
 * Other arguments, outputs and statuses as resispec_verify_tree_path.
 */
rs_status resispec_verify_tree_path_group(const void* target_logits, const void* draft_logits,
                                          const int32_t* node_token, const int32_t* parent,
                                          const float* u_accept, const float* u_resample,
                                          int32_t B, int32_t N, int32_t V, int32_t max_depth,
                                          const rs_params* prm, int32_t* out_tokens,
                                          int32_t* out_accepted_len, int32_t* out_status,
                                          int32_t group_size, void* workspace,
                                          size_t workspace_bytes, void* stream);

/*
 * resispec_verify_tree (Algorithm 1 at every node, §Preliminary walk) with row groups, for
 * batches of few rows (same results, bit for bit): every node row gets `group_size`
 * 512-thread workgroups that verify it together, exchanging slot totals through the
 * workspace with bounded waits like the path schedule's row groups (a group that does not
 * form within 20 us is done by one of its workgroups alone; RS_SEQ_GROUP_TIMEOUT after 20
 * ms without the others' totals), then the walk runs as in resispec_verify_tree.
 *   group_size : 0 = automatic (at most one workgroup per CU for B * N rows, up to 8
 *                members per row, one per 8 slots of a row and one per 40 KiB of a row's
 *                logits, none below 160 KiB; 1 = the ordinary one-workgroup row kernel
 *                when that is under 2),
 *                1 = the ordinary kernel,
 *                2..16 = that many (RS_ERR_UNSUPPORTED if B * N * group_size workgroups
 *                cannot be resident at once or a row has fewer slots than members)
 *   workspace  : device buffer of at least resispec_tree_group_workspace_bytes(B, N)
 *                bytes, 16-byte aligned, caller-owned (node outcomes, then one group
 *                state per row; its counters are zeroed by the call itself on `stream`).
 *                Calls that overlap on one workspace race.
 * Other arguments, outputs and statuses as resispec_verify_tree.
 */
rs_status resispec_verify_tree_group(const void* target_logits, const void* draft_logits,
                                     const int32_t* node_token, const int32_t* parent,
                                     const float* u_accept, const float* u_resample, int32_t B,
                                     int32_t N, int32_t V, int32_t max_depth, const rs_params* prm,
                                     int32_t* out_tokens, int32_t* out_accepted_len,
                                     int32_t* out_status, int32_t group_size, void* workspace,
                                     size_t workspace_bytes, void* stream);

/* Workspace bytes resispec_verify_tree_group needs (0 if B <= 0 or N <= 0). */
size_t resispec_tree_group_workspace_bytes(int32_t B, int32_t N);

/* The group size resispec_verify_tree_group chooses with group_size = 0 for B * N rows
 * of V elements (16-byte aligned rows assumed), on the current device; -1 for invalid
 * arguments.  Host only: launches nothing. */
int32_t resispec_tree_group_size(int32_t B, int32_t N, int32_t V, const rs_params* prm);

/* Testing hook: the time limits of row groups in later launches of this process, in
 * ticks of the device's 100 MHz wall clock; UINT64_MAX restores a default.
 *   barrier_ticks   : every wait of a formed group for its members' totals (default
 *                     2,000,000 = 20 ms); a small limit makes groups report
 *                     RS_SEQ_GROUP_TIMEOUT instead of waiting, which is how the tests
 *                     exercise that path
 *   formation_ticks : the wait for a group's workgroups to start (default 2,000 = 20 us);
 *                     0 makes nearly every group fall back to one workgroup
 * Not for concurrent use with launches on other threads.  Always RS_OK. */
rs_status resispec_debug_set_group_waits(uint64_t barrier_ticks, uint64_t formation_ticks);

/* Workspace bytes resispec_verify_tree_path_group needs for B sequences of V-element rows
 * (0 if B <= 0, V <= 0 or V > RS_MAX_VOCAB): one row-group state per sequence, then two
 * fp32 rows per sequence (V rounded up to a multiple of 1024 each), in which the ResiSpec
 * rejection passes after a row's second rejection keep the residual of the previous pass
 * and the draft's masses instead of re-deriving them from the logits through the chain
 * of earlier proxies (Algorithm 1 loop: each rejection updates R from the current R and
 * D). */
size_t resispec_path_workspace_bytes(int32_t B, int32_t V);

/* The group size resispec_verify_tree_path_group chooses with group_size = 0 for B
 * sequences of V-element rows (16-byte aligned rows assumed), on the current device;
 * -1 for invalid arguments.  Host only: launches nothing. */
int32_t resispec_path_group_size(int32_t B, int32_t V, const rs_params* prm);

/*
 * The draft step that precedes verification (Preliminary: candidates are drawn from the
 * draft distribution; Algorithm 1 draws x_i ~ D and r_i ~ Uniform(0, 1)), on the device:
 *   - every node's uniforms: Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11) of
 *     counter (n, b, offset low word, offset high word) under key (seed low word, seed
 *     high word); word 0 -> u_accept[b][n], word 1 -> u_resample[b][n], word 2 -> the
 *     uniform that draws node n's own token; a word w maps to (w >> 8) * 2^-24;
 *   - every node's children's tokens, drawn from softmax(draft[b][n] / T) by inverse CDF
 *     in ascending vocabulary order, children in ascending node index; with
 *     prm->without_replacement each draw removes its token (and renormalises) before the
 *     next.
 *   draft_logits : [B][N][V] (prm->logits_dtype); draft rows of leaves are not read
 *   parent       : [B][N] int32, as for resispec_verify_tree
 *   node_token   : [B][N] int32 out; entry 0 = -1.  A node whose draft row has no usable
 *                  mass, or which has more than RS_MAX_CANDIDATES children, leaves its
 *                  children at -1; a malformed tree sets every entry of the sequence to -1.
 *   u_accept, u_resample : [B][N] fp32 out
 *   out_status   : [B] int32 out (RS_SEQ_OK or RS_SEQ_BAD_TREE), may be NULL
 * prm->mode and prm->bonus are ignored.  The outputs feed resispec_verify_tree directly.
 */
rs_status resispec_draft_candidates(const void* draft_logits, const int32_t* parent,
                                    int32_t B, int32_t N, int32_t V, const rs_params* prm,
                                    uint64_t seed, uint64_t offset, int32_t* node_token,
                                    float* u_accept, float* u_resample, int32_t* out_status,
                                    void* stream);

/*
 * The two stages of resispec_verify_tree, for callers that schedule them separately
 * (same kernels, same results): Algorithm 1 at every node, then the walk of §Preliminary.
 *   resispec_verify_nodes: every node's own outcome (accepted child or drawn token) into
 *     `workspace`, from the same inputs as resispec_verify_tree;
 *   resispec_walk: the walk from each root over the outcomes in `workspace` (written by
 *     resispec_verify_nodes with the same B and N, earlier on the same stream).
 * The workspace layout is private to the library.
 */
rs_status resispec_verify_nodes(const void* target_logits, const void* draft_logits,
                                const int32_t* node_token, const int32_t* parent,
                                const float* u_accept, const float* u_resample,
                                int32_t B, int32_t N, int32_t V, const rs_params* prm,
                                void* workspace, size_t workspace_bytes, void* stream);

rs_status resispec_walk(const int32_t* node_token, int32_t B, int32_t N, int32_t max_depth,
                        const void* workspace, size_t workspace_bytes, int32_t* out_tokens,
                        int32_t* out_accepted_len, int32_t* out_status, void* stream);

/*
 * Every node's own outcome as resispec_verify_nodes left it in `workspace` (the same
 * B and N, earlier on the same stream), copied into caller arrays (device-to-device,
 * stream-ordered, asynchronous): the outcome of Algorithm 1 at each node, as the debug
 * entry below reports it.  The workspace of resispec_decide_nodes (and resispec_walk_draw)
 * is read the same way; there, nodes whose draw was deferred and not made report
 * RS_SEQ_DEFERRED.
 *   node_child, node_token_out, node_status : [B][N] int32 device out, as in
 *                 resispec_verify_tree_debug
 * RS_ERR_INVALID_ARG for B < 0, N <= 0 or NULL outputs (B > 0); RS_ERR_WORKSPACE for a
 * missing or short workspace.
 */
rs_status resispec_node_outcomes(const void* workspace, size_t workspace_bytes, int32_t B,
                                 int32_t N, int32_t* node_child, int32_t* node_token_out,
                                 int32_t* node_status, void* stream);

/* Workspace bytes resispec_verify_tree needs for B sequences of N nodes. */
size_t resispec_workspace_bytes(int32_t B, int32_t N);

/*
 * Host-side check of a tree batch (HOST pointers, synchronous, no device work).
 * Returns RS_OK when every sequence has parent[.,0] = -1, parent[.,n] in [0, n),
 * at most RS_MAX_CANDIDATES children per node and every node_token (n >= 1) in
 * [0, V); RS_ERR_INVALID_ARG otherwise.  If first_bad is not NULL it receives the
 * flat index b*N+n of the first offending entry (or -1).
 */
rs_status resispec_validate_tree_host(const int32_t* parent, const int32_t* node_token,
                                      int32_t B, int32_t N, int32_t V, int64_t* first_bad);

/*
 * Same as resispec_verify_tree, and also writes each node's own outcome (testing and
 * debugging; not the timed path):
 *   node_child  : [B][N] int32 accepted child node index, -1 if none
 *   node_token_out : [B][N] int32 token the node emits (accepted candidate, drawn token,
 *                 or -1)
 *   node_status : [B][N] int32 rs_seq_status of the node
 *   residual_out: [B][N][V] fp32 or NULL; for nodes that drew a token, the normalised
 *                 distribution of the draw (final residual, or the target for a bonus);
 *                 other rows are zero.  Costs one more pass over the logits.
 */
rs_status resispec_verify_tree_debug(const void* target_logits, const void* draft_logits,
                                     const int32_t* node_token, const int32_t* parent,
                                     const float* u_accept, const float* u_resample,
                                     int32_t B, int32_t N, int32_t V, int32_t max_depth,
                                     const rs_params* prm, int32_t* out_tokens,
                                     int32_t* out_accepted_len, int32_t* out_status,
                                     void* workspace, size_t workspace_bytes,
                                     int32_t* node_child, int32_t* node_token_out,
                                     int32_t* node_status, float* residual_out, void* stream);

/* Static description of a status code. */
const char* resispec_status_string(int32_t status);

/* RESISPEC_ABI_VERSION of the loaded library. */
int32_t resispec_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* RESISPEC_H */
