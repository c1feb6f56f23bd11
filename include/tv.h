/*
 * tv.h -- batched verification of speculative token trees on MI355X (gfx950).
 *
 * Traversal Verification (arXiv 2505.12398, Sec. 3.1, Algorithm 3) and the
 * top-down token-level baseline (Sec. 2.2: recursive rejection sampling,
 * Algorithm 2, applied layer by layer) for a batch of independent trees.
 *
 * Problem statement (Alg. 3 REQUIRE; Def. de_tree and Def. def2 in Sec. 3.3):
 * a tree of drafted tokens rooted at the prefix X_0, the draft model's
 * next-token distribution at every node that has children, the target model's
 * next-token distribution at every node; the output is an accepted chain
 * X^tau = (X_0, ..., X_tau) from the root plus one extra token Y, distributed
 * exactly as the target model would have generated them.
 *
 * Conventions shared by both verifiers (the paper leaves them open):
 *   - nodes are numbered so that parents[i] < i; node 0 is the root;
 *   - children are ordered by ascending node index (Alg. 3 takes "the first
 *     leaf" in this order, i.e. post-order DFS, App. E);
 *   - row i of a logits tensor is the next-token distribution after the path
 *     root..i; a child's acceptance ratio uses its parent's rows;
 *   - the distributions are softmax(logits / T) with the same temperature T
 *     for target and draft;
 *   - uniforms[b][i] (i >= 1) is the uniform that tests node i, accepted iff
 *     u < theta; uniforms[b][0] draws Y by inverse CDF in ascending token
 *     order (the smallest y with u * W < C(y), C the running sum, W its total).
 *
 * Memory and streams. Every pointer is a device pointer. The caller owns all
 * buffers, including a device workspace of tv_workspace_size() bytes that the
 * call uses as scratch (the partial sums of every vocabulary pass and one
 * batch descriptor per group; its contents need no initialisation and are
 * meaningless afterwards). The library
 * allocates nothing, keeps no state between calls and never synchronises the
 * host: work is enqueued on `stream` and the call returns. Inputs are
 * read-only. Outputs are written for every tree, including trees whose status
 * is not TV_TREE_OK (they get -1 sentinels). Calls that write the same output
 * buffers or share a workspace must be ordered by the caller.
 *
 * Execution. One call enqueues a small initialisation kernel and one
 * cooperative launch of at most as many workgroups as the device holds at
 * once, in groups that each verify one tree at a time (several workgroups per
 * tree; three per tree at 256 trees on MI355X). The members of a group
 * exchange partial sums through the workspace and wait for each other at
 * every vocabulary pass; a group with no tree left lends its workgroups to
 * running groups. The launch waits until the whole grid can be resident.
 * Every wait inside the kernel is bounded: a call that makes no progress for
 * 4 seconds gives up and reports TV_TREE_ABORTED for the trees it did not
 * finish.
 *
 * Errors. Argument problems the host can see (null pointers, sizes, enums,
 * temperature, misaligned pointers) return a tv_status_t other than TV_OK and
 * enqueue nothing. Problems in the data (a bad tree, non-finite logits) are
 * reported per tree in status[b]. A failed kernel launch returns TV_ERR_HIP.
 */
#ifndef TV_H
#define TV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum tv_status {
  TV_OK = 0,
  TV_ERR_INVALID_ARG = 1,  /* null pointer, negative size, unknown enum, T <= 0 or not finite */
  TV_ERR_UNSUPPORTED = 2,  /* size or temperature beyond the limits below, or target and draft
                              pointers whose addresses differ modulo 16 bytes */
  TV_ERR_WORKSPACE = 3,    /* workspace NULL, smaller than tv_workspace_size() or not
                              256-byte aligned */
  TV_ERR_HIP = 4           /* the kernel launch failed (hipGetLastError) */
} tv_status_t;

typedef enum tv_dtype {
  TV_DTYPE_BF16 = 0,       /* bfloat16 logits (uint16 bit patterns) */
  TV_DTYPE_F32 = 1         /* float32 logits */
} tv_dtype_t;

/*
 * How the children of a node were drawn from its draft distribution
 * (Def. de_tree allows both). The draft update after a rejection must match:
 *   WITHOUT_REPLACEMENT -- siblings drawn one after another without
 *     replacement; a rejected token's draft probability is set to zero and the
 *     rest renormalised (Eq. e2; the blue lines of Algorithm 2). Siblings must
 *     carry distinct tokens (else status TV_TREE_DUP_SIBLING).
 *   WITH_REPLACEMENT -- siblings drawn i.i.d.; the draft distribution stays as
 *     it is after a rejection.
 */
typedef enum tv_sibling_mode {
  TV_SIBLINGS_WITHOUT_REPLACEMENT = 0,
  TV_SIBLINGS_WITH_REPLACEMENT = 1
} tv_sibling_mode_t;

/* Per-tree status written to status[b]. */
enum {
  TV_TREE_OK = 0,
  TV_TREE_BAD_PARENT = 1,  /* parents[b][0] != -1, or parents[b][i] outside [0, i) */
  TV_TREE_BAD_TOKEN = 2,   /* tokens[b][i] outside [0, vocab) for some i >= 1 */
  TV_TREE_DUP_SIBLING = 3, /* two siblings share a token in WITHOUT_REPLACEMENT mode */
  TV_TREE_NONFINITE = 4,   /* a row the verifier read holds NaN or +inf or no finite value,
                              or a drafted token has draft logit -inf */
  TV_TREE_DEGENERATE = 5,  /* a residual distribution the algorithm samples from has zero
                              mass in floating point (impossible in exact arithmetic) */
  TV_TREE_ABORTED = 6      /* not verified: the call gave up after its wait limit (see
                              Execution above) */
};

/* Values written to node_state[b][i]. */
enum {
  TV_NODE_UNTESTED = 0,    /* never compared against its uniform */
  TV_NODE_ACCEPTED = 1,    /* the accepted node (Traversal Verification marks only the
                              last node of X^tau; the token-level verifier marks every
                              accepted node on the path). A root accepted with tau = 0
                              is marked too. */
  TV_NODE_REJECTED = 2,    /* tested and rejected */
  TV_NODE_PRUNED = 3       /* discarded untested because its parent's acceptance rate
                              had dropped to exactly 0 (Sec. 3.2 example) */
};

/* Limits of this implementation. */
#define TV_MAX_BATCH (1 << 20)     /* trees per call */
#define TV_MAX_NODES 1024          /* num_nodes = N + 1 (root included) */
#define TV_MAX_VOCAB (1 << 20)          /* bf16 logits */
#define TV_MAX_VOCAB_F32 (1 << 19)      /* fp32 logits */
#define TV_MIN_TEMPERATURE 1.0e-3f
#define TV_MAX_TEMPERATURE 1.0e3f
#define TV_NUM_COUNTERS 4
#define TV_MAX_LMHEAD_ROWS (1 << 18)    /* rows of one tv_lmhead_stats call (its grid of
                                           128 x 128 tiles then stays below 2^24 workgroups) */
#define TV_MAX_HIDDEN (1 << 16)         /* hidden size of tv_lmhead_stats */

/*
 * Bytes of device workspace tv_verify / tv_verify_tokenlevel need for these
 * sizes (valid for either dtype; at most about 2.5 MiB, about 2.0 MiB for 256
 * trees). Returns 0 for invalid sizes (batch < 1, vocab < 2 or
 * beyond the limits below); a batch of 0 needs no workspace.
 */
size_t tv_workspace_size(int32_t batch, int32_t num_nodes, int32_t vocab);

/*
 * Traversal Verification, Algorithm 3 (Sec. 3.1) with Eq. (e1)-(e3), on
 * `batch` independent trees of `num_nodes` = N + 1 nodes each.
 *
 * Inputs (device, row-major, contiguous):
 *   parents        int32 [batch][num_nodes]   parents[b][0] = -1, 0 <= parents[b][i] < i
 *   tokens         int32 [batch][num_nodes]   drafted token of node i (tokens[b][0] unused)
 *   target_logits  dtype [batch][num_nodes][vocab]   target model logits per node
 *   draft_logits   dtype [batch][num_nodes][vocab]   draft model logits per node; rows of
 *                  nodes without children are never read
 *   dtype          TV_DTYPE_BF16 or TV_DTYPE_F32 (both logits tensors)
 *   temperature    T, applied to both models; finite, in [TV_MIN_TEMPERATURE, TV_MAX_TEMPERATURE]
 *   vocab          2 .. TV_MAX_VOCAB (bf16) or TV_MAX_VOCAB_F32 (fp32)
 *   uniforms       float32 [batch][num_nodes], each in [0, 1)
 *   mode           tv_sibling_mode_t
 * Outputs (device):
 *   accept_len     int32 [batch]   tau, the depth of the accepted node (0: root only)
 *   accepted_node  int32 [batch]   index of the last node of X^tau (its ancestors are the path)
 *   bonus_token    int32 [batch]   Y
 *   status         int32 [batch]   TV_TREE_*
 *   node_state     int8  [batch][num_nodes] or NULL   TV_NODE_*
 *   node_theta     float [batch][num_nodes] or NULL   acceptance probability the node was
 *                  tested with; 0 for pruned nodes, -1 for untested nodes.
 *                  When NULL, tv_verify applies early rejection: a node's rate never
 *                  rises under Eq. (e3) (S <= p by Eq. e1), so when the last child of a
 *                  non-root node j is rejected while u[j] >= p(j), j is rejected without
 *                  its update (one pass over j's rows fewer). Every other output is the
 *                  same either way; only j's exact theta is then never computed.
 *   p_init         float [batch][num_nodes] or NULL   Alg. 3 initial chain rates p^ini.
 *                  Asking for them makes the verifier read the rows of every node that
 *                  has children, which the traversal itself may not need.
 *   counters       int32 [batch][TV_NUM_COUNTERS] or NULL:
 *                  [0] nodes whose target and draft rows were read for the traversal,
 *                  [1] residual updates executed (Eq. e1-e3; one pass over both rows of
 *                      the parent; without the ones early rejection skips),
 *                  [2] 1 if the accepted node has no children (its target row is read for Y),
 *                  [3] nodes tested against their uniform
 *   workspace      device buffer of at least tv_workspace_size() bytes, 256-byte aligned
 *   stream         HIP stream the work is enqueued on (NULL: the default stream)
 * Returns a tv_status_t.
 */
int tv_verify(int32_t batch, int32_t num_nodes, int32_t vocab,
              const int32_t* parents, const int32_t* tokens,
              const void* target_logits, const void* draft_logits, int32_t dtype,
              float temperature, const float* uniforms, int32_t mode,
              int32_t* accept_len, int32_t* accepted_node, int32_t* bonus_token,
              int32_t* status, int8_t* node_state, float* node_theta, float* p_init,
              int32_t* counters, void* workspace, size_t workspace_bytes,
              hipStream_t stream);

/*
 * tv_verify without a caller workspace, for callers that cannot allocate
 * device memory or cannot pass a workspace: code that is being captured into
 * a HIP graph, serving loops and harnesses that forbid allocation. Same
 * arguments, outputs and per-tree statuses as tv_verify, minus workspace and
 * workspace_bytes. The call allocates nothing: it uses a device scratch array
 * of 3 MiB that the library holds on every device it runs on until the
 * process ends (its address is looked up once per device, on the first call
 * there). That covers every size the limits below allow; a size needing more
 * would return TV_ERR_UNSUPPORTED. Every call on one device shares that
 * device's scratch, and each call clears what it needs: calls on one device
 * must not overlap (calls on different streams of one device race; order them,
 * e.g. on one stream). Calls on different devices are independent.
 */
int tv_verify_noalloc(int32_t batch, int32_t num_nodes, int32_t vocab,
                      const int32_t* parents, const int32_t* tokens,
                      const void* target_logits, const void* draft_logits, int32_t dtype,
                      float temperature, const float* uniforms, int32_t mode,
                      int32_t* accept_len, int32_t* accepted_node, int32_t* bonus_token,
                      int32_t* status, int8_t* node_state, float* node_theta, float* p_init,
                      int32_t* counters, hipStream_t stream);

/*
 * tv_verify with the row statistics given by the caller, so that the verifier
 * reads a node's logits only for its residual updates (Eq. e1-e3) and for Y,
 * never to normalise them. The distributions of the problem statement
 * (Alg. 3 REQUIRE) are softmax(logits / T) per row; for row (b, i):
 *   target_max[b][i] = max_x target_logits[b][i][x]          float [batch][num_nodes]
 *   target_sum[b][i] = sum_x exp((target_logits[b][i][x] - target_max[b][i]) / T)
 *                                                              double [batch][num_nodes]
 * and the same for the draft rows (draft_max, draft_sum). tv_lmhead_stats
 * produces them with the logits; any producer may be used. Only the entries
 * of nodes that have children are read. A non-finite maximum, or a sum that is
 * not finite and positive, at a row the traversal consults gives
 * TV_TREE_NONFINITE. Every other argument, output and status is that of
 * tv_verify; the results equal tv_verify's up to the rounding of the sums.
 * All four pointers are required (else TV_ERR_INVALID_ARG).
 */
int tv_verify_stats(int32_t batch, int32_t num_nodes, int32_t vocab,
                    const int32_t* parents, const int32_t* tokens,
                    const void* target_logits, const void* draft_logits, int32_t dtype,
                    float temperature, const float* uniforms, int32_t mode,
                    const float* target_max, const double* target_sum,
                    const float* draft_max, const double* draft_sum,
                    int32_t* accept_len, int32_t* accepted_node, int32_t* bonus_token,
                    int32_t* status, int8_t* node_state, float* node_theta, float* p_init,
                    int32_t* counters, void* workspace, size_t workspace_bytes,
                    hipStream_t stream);

/*
 * LM head with fused row statistics: the model layer whose outputs the
 * verifier reads. For rows = the tree nodes of a batch (M), hidden size K and
 * vocabulary N:
 *   logits[m][n] = bf16( sum_k hidden[m][k] * weight[n][k] )   (fp32 accumulation,
 *                                                              round to nearest even)
 *   row_max[m]   = max_n logits[m][n]
 *   row_sum[m]   = sum_n exp((logits[m][n] - row_max[m]) / T)  (of the rounded logits)
 * which are the inputs tv_verify_stats takes (one call for the target model,
 * one for the draft model). hidden bf16 [rows][hidden_size], weight bf16
 * [vocab][hidden_size] (the usual [out][in] layout of a linear layer), both
 * 16-byte aligned and contiguous, hidden_size a multiple of 8; logits bf16
 * [rows][vocab]; row_max float [rows]; row_sum double [rows]. The matrix
 * products run on the bf16 matrix cores (MFMA); the statistics are formed in
 * the same kernel from the rounded logits it holds, so they cost no pass over
 * the logits. A NaN or infinite logit makes its row's sum NaN or infinite.
 * workspace: device buffer of tv_lmhead_workspace_size(rows, vocab) bytes,
 * 256-byte aligned (a maximum and a sum per row and 256-column tile).
 * Returns a tv_status_t; argument errors launch nothing.
 */
size_t tv_lmhead_workspace_size(int32_t rows, int32_t vocab);
int tv_lmhead_stats(int32_t rows, int32_t hidden_size, int32_t vocab, const void* hidden,
                    const void* weight, float temperature, void* logits, float* row_max,
                    double* row_sum, void* workspace, size_t workspace_bytes,
                    hipStream_t stream);

/*
 * Token-level tree verification (Sec. 2.2): starting at the root, the children
 * of the current node are tested in index order with recursive rejection
 * sampling (Algorithm 2; without replacement per `mode`); an accepted child
 * becomes the current node; Y is drawn from the target at an accepted leaf or
 * from the residual once every child of the current node is rejected.
 * Same arguments and layouts as tv_verify; p_init, if not NULL, is filled with -1.
 */
int tv_verify_tokenlevel(int32_t batch, int32_t num_nodes, int32_t vocab,
                         const int32_t* parents, const int32_t* tokens,
                         const void* target_logits, const void* draft_logits, int32_t dtype,
                         float temperature, const float* uniforms, int32_t mode,
                         int32_t* accept_len, int32_t* accepted_node, int32_t* bonus_token,
                         int32_t* status, int8_t* node_state, float* node_theta,
                         float* p_init, int32_t* counters, void* workspace,
                         size_t workspace_bytes, hipStream_t stream);

/*
 * Draft-tree token sampler: the step that builds the trees tv_verify checks.
 * A draft tree (Def. de_tree, Sec. 3.3) gives the children of every node
 * tokens drawn from the draft model's distribution at that node,
 * softmax(draft_logits[b][j] / temperature), with or without replacement.
 * The children of a node are drawn in ascending node index, child c by the
 * inverse CDF in ascending token order at uniforms[b][c]
 * (y = min{y : u*W < C(y)}, W the row's total weight). Without replacement,
 * each drawn token is removed before the next sibling's draw (the draft step
 * of Eq. (e2)), so siblings never repeat. Uniforms come from the caller, like
 * tv_verify's.
 *
 * Inputs (device, row-major, contiguous): parents int32 [batch][num_nodes]
 * (parents[b][0] = -1, 0 <= parents[b][i] < i); draft_logits dtype
 * [batch][num_nodes][vocab] (rows of nodes without children are not read);
 * uniforms float32 [batch][num_nodes], each in [0, 1) (u[b][0] unused);
 * temperature, vocab and mode as for tv_verify.
 * Outputs (device): tokens int32 [batch][num_nodes] (tokens[b][0] = -1; every
 * token -1 for a tree whose status is not TV_TREE_OK); status int32 [batch]:
 * TV_TREE_OK, TV_TREE_BAD_PARENT, TV_TREE_NONFINITE (a row with children has
 * NaN, +inf or no finite entry) or TV_TREE_DEGENERATE (without replacement, a
 * node has more children than tokens of positive probability); the largest
 * code found when there are several. No workspace; nothing is allocated.
 * Returns a tv_status_t; argument errors launch nothing.
 */
int tv_draft_tokens(int32_t batch, int32_t num_nodes, int32_t vocab, const int32_t* parents,
                    const void* draft_logits, int32_t dtype, float temperature,
                    const float* uniforms, int32_t mode, int32_t* tokens, int32_t* status,
                    hipStream_t stream);

/* path_len codes of tv_commit_paths besides a length */
#define TV_COMMIT_OVERFLOW (-1)       /* the chain is longer than max_len */
#define TV_COMMIT_INCONSISTENT (-2)   /* accepted_node out of range or a link not pointing back */

/*
 * Accepted-path commit: the step after verification. For every tree, the
 * output of Def. def2 (Sec. 3.3), the accepted chain X^tau and the token Y,
 * laid out for the next decoding cycle:
 *   path_nodes  int32 [batch][max_len]      nodes of X^tau after the root, from the root
 *                                           down (the drafted positions whose cache
 *                                           entries are kept), then -1
 *   path_tokens int32 [batch][max_len + 1]  their drafted tokens, then Y, then -1
 *   path_len    int32 [batch]               tokens committed, tau + 1; 0 for a tree whose
 *                                           status is not TV_TREE_OK; TV_COMMIT_OVERFLOW or
 *                                           TV_COMMIT_INCONSISTENT (rows then all -1)
 * Inputs (device): parents and tokens as for tv_verify; accepted_node,
 * bonus_token and status as tv_verify or tv_verify_tokenlevel wrote them.
 * max_len in 0 .. TV_MAX_NODES (path_nodes may be NULL when it is 0). No
 * workspace; nothing is allocated. Returns a tv_status_t; argument errors
 * launch nothing.
 */
int tv_commit_paths(int32_t batch, int32_t num_nodes, const int32_t* parents,
                    const int32_t* tokens, const int32_t* accepted_node,
                    const int32_t* bonus_token, const int32_t* status, int32_t max_len,
                    int32_t* path_nodes, int32_t* path_tokens, int32_t* path_len,
                    hipStream_t stream);

/* Static, human-readable name of a tv_status_t value ("unknown status" otherwise). */
const char* tv_status_string(int code);

#ifdef __cplusplus
}
#endif

#endif /* TV_H */
