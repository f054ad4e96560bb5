/*
 * treespark.h -- C ABI of the TreeSpark draft-tree step on MI355X (gfx950).
 *
 * The library computes one speculative-decoding round's draft tree and its
 * verification, as described in "TreeSpark" (arXiv 2609.22098):
 *   ts_expand      parent-conditioned expansion of a frontier of parents
 *                  (§1 Eq. 1; §3.2 item 1; §3.3 residual-proposal equation;
 *                  §3.4 Eq. 3; §5.6 per-node work)
 *   ts_build_tree  best-first expansion of whole trees under (N, K, theta)
 *                  (§3.2 Algorithm 1; §3.5)
 *   ts_verify      greedy exact-match or recursive-rejection verification
 *                  (§3.2 item 3; §3.3 and Proposition 1)
 *   ts_tree_mask   the tree attention mask and position ids of the target's
 *                  verification pass (§3.2 item 3; §5)
 *
 * Conventions shared by every call
 *   - Model tensors are DEVICE pointers owned by the caller, row-major:
 *       U  [R][D][V]  drafter base logits; row d of request q gives the logits
 *                     of the children of a depth-d parent (the LM-shifted
 *                     block semantics of §3.1)
 *       E  [V][r]     W1 of the Markov head: row x = W1[x]
 *       W2 [V][r]     W2 of the Markov head: row v = W2[v], so the transition
 *                     bias is B(x, v) = <W1[x], W2[v]> (§3.1); as an r x V
 *                     matrix W this is W2 transposed
 *     All three share one dtype (TS_F32 or TS_BF16) and start at 16-byte
 *     aligned addresses (TS_EINVAL otherwise).  Accumulation is fp32.
 *   - The library never frees, retains or writes caller tensors other than
 *     the documented outputs.  It allocates no device memory: scratch comes
 *     from the caller's workspace (sizes from the *_workspace_size calls).
 *   - Randomness is Philox4x32-10 keyed by `seed`, counter
 *     (c0, path lo32, path hi32, request<<12 | depth<<4 | tag), where a node
 *     is named by its structural path id: 4 bits per level, digit = sibling
 *     index - 1, level d at bits [4d, 4d+4).  Per-token draws use c0 = y>>2
 *     and word y&3; per-stage draws use c0 = j and word 0; sequential
 *     sibling draws use c0 = j and words 0..2; tags are 1 (expand, Gumbel),
 *     2 (accept), 3 (bonus), 4 (expand, sequential).  A uniform is
 *     u = ((w>>9) + 0.5) * 2^-23.
 *   - Every call returns TS_OK (0) or a negative ts_status.  On an error
 *     detected on the host nothing is launched and no output is written;
 *     ts_last_error() (per thread) describes it.  No exception crosses the ABI.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 */
#ifndef TREESPARK_H
#define TREESPARK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TS_OK = 0,
  TS_EINVAL = -1,        /* bad argument (null pointer, size out of range, ...) */
  TS_EUNSUPPORTED = -2,  /* valid but beyond the library's limits (below) */
  TS_EHIP = -3,          /* a HIP runtime call failed */
  TS_ENOSPACE = -4,      /* workspace smaller than the *_workspace_size result */
  TS_EINTERNAL = -5      /* an internal consistency check failed */
} ts_status;

typedef enum { TS_F32 = 0, TS_BF16 = 1 } ts_dtype;

/* How the k sibling draws of a parent at T > 0 are realised.  Both give k
 * draws without replacement from q_T in draw order, i.e. the residual
 * proposals q_T^(j) of §3.3; they differ in which random words decide them.
 *   TS_SAMPLER_GUMBEL      the k largest of z / T - log(-log u_y), one word
 *                          per (parent, token y) (tag 1, c0 = y >> 2).
 *   TS_SAMPLER_SEQUENTIAL  the draws one after another, as §3.3 states them:
 *                          draw j picks a 4096-token segment, a 64-token
 *                          block in it and a token in it, each in proportion
 *                          to its remaining q_T mass (the first index whose
 *                          cumulative mass exceeds u * total), from words
 *                          0, 1, 2 of one Philox call (tag 4, c0 = j).
 * The sampler does not matter at T = 0. */
typedef enum { TS_SAMPLER_GUMBEL = 0, TS_SAMPLER_SEQUENTIAL = 1 } ts_sampler;

/* Limits of the library: K <= TS_MAX_K siblings, D <= TS_MAX_D (the path id
 * holds 4 bits per level), R < 2^20 requests, V <= TS_MAX_V; the rank r is
 * one of 32, 64, 128, 256 for bf16 and one of 16, 32, 64 for fp32. */
#define TS_MAX_K 16
#define TS_MAX_D 16
#define TS_MAX_R (1 << 20)
#define TS_MAX_RANK 256
#define TS_MAX_V (256 * 4096) /* 256 chunks of at most 4096 tokens per parent */

/* Drafter outputs of one round (device pointers, see above). */
typedef struct {
  const void* U;
  const void* E;
  const void* W2;
  int32_t R, D, V, r;
  int32_t dtype; /* ts_dtype of U, E and W2 */
} ts_drafter;

/* Calibrated edge acceptance p-hat = sigmoid(a * logit(q0) + b), §3.4 Eq. 3.
 * The paper's deployed values are a = 0.67, b = -0.46. */
typedef struct {
  float a, b;
} ts_calib;

/* One frontier parent (device array element, 24 bytes). */
typedef struct {
  int32_t token;    /* parent token x_p, 0 <= token < V */
  int32_t depth;    /* 0 <= depth < D; its children use U row `depth` */
  int32_t request;  /* 0 <= request < R */
  float log_surv;   /* log S(parent): log of the path survival (§3.5) */
  uint64_t path;    /* structural path id of the parent */
} ts_parent;

/* Outputs of ts_expand, DEVICE pointers, [P][k] row-major unless noted.
 * Children are in draw order: at T = 0 the top-k tokens of q0 by (q0 desc,
 * id asc); at T > 0 the k draws without replacement from q_T (ts_sampler).
 * Slot j (1-based) of parent p creates child j; its key is the heap priority
 * of Algorithm 1: at T = 0 the child's own log survival, at T > 0 the
 * admissible pre-draw bound log S(p) + log p-hat(max q0 over tokens not drawn
 * before j) of §3.2.  Optional pointers may be NULL. */
typedef struct {
  int32_t* child_token;    /* [P][k] required */
  float* child_log_q0;     /* [P][k] required: log q0(child | parent) */
  float* child_log_qT;     /* [P][k] optional: log qT(child | parent); NaN at T = 0 */
  float* child_log_surv;   /* [P][k] required: log S(child) = log S(p) + log p-hat */
  float* slot_key;         /* [P][k] required */
  int32_t* rank_token;     /* [P][k] optional: top-k tokens by q0 */
  float* rank_log_q0;      /* [P][k] optional: their log q0 */
  float* lse0;             /* [P] optional: log-sum-exp of the logits z */
  float* lseT;             /* [P] optional: log-sum-exp of z / T; NaN at T = 0 */
  int32_t* diag;           /* [P] optional: candidate runs whose recomputed maximum differed
                              from the streaming pass (always 0 unless the device misbehaves) */
  void** events;           /* optional: 3 caller-created hipEvent_t, recorded on `stream`
                              before pass 1, between the passes and after pass 2 (timing) */
} ts_expand_out;

/* Bytes of device workspace ts_expand needs for P parents (0 if P == 0),
 * for either sampler. */
size_t ts_expand_workspace_size(const ts_drafter* d, int32_t P, int32_t k, float T);

/*
 * ts_expand: evaluate P frontier parents.  For each parent p with token x,
 * depth d and request q, the logits are z[y] = U[q][d][y] + <E[x], W2[y]>
 * (§1 Eq. 1); q0 = softmax(z), qT = softmax(z / T).  Each of the k children
 * gets log q0, log qT, log p-hat and log S(child) = log S(p) + log p-hat
 * (Eq. 3; §3.5).  parents is a DEVICE array of P ts_parent.
 * sampler is a ts_sampler (used at T > 0).
 * Asynchronous on `stream`.  Arguments checked on the host: null pointers,
 * sizes, k in [1, min(V, TS_MAX_K)], T >= 0 and finite, sampler, workspace
 * size.
 * Parent fields are checked on the device: a parent with a token, depth or
 * request out of range gets child_token -1 and NaN values, and nothing out
 * of bounds is read.
 * U may hold -inf (masked tokens).  With fewer than k finite logits in a
 * parent's row, the sequential draws after the last finite token are empty
 * (child_token -1; log q0, log qT, log S and slot key -inf), while the greedy
 * order and the Gumbel draws continue with -inf tokens by id.  No input
 * value makes a kernel read outside the arrays it was given.
 * Performance note: parents that share (request, depth) should be adjacent.
 */
int32_t ts_expand(const ts_drafter* d, const ts_parent* parents, int32_t P, ts_calib calib,
                  int32_t k, float T, uint64_t seed, int32_t sampler, const ts_expand_out* out,
                  void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of the per-GPU scratch array ts_expand_noalloc works in. */
#define TS_NOALLOC_SCRATCH_BYTES (32u << 20)

/*
 * ts_expand_noalloc: ts_expand without a workspace argument, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation.  It calls no allocator.  Its
 * scratch is a file-scope device array of TS_NOALLOC_SCRATCH_BYTES bytes, one
 * copy on each GPU the library runs on, held until the process ends.
 *   - The launch needs what ts_expand's plan for it needs (a function of P, V,
 *     r, the sampler and the device's compute units; about 24 MB for 2048
 *     parents at V = 151936 with sequential draws).  A launch that needs more
 *     returns TS_EUNSUPPORTED before anything is launched.
 *   - Every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents (nothing in it needs to start at zero).  Calls that
 *     overlap in time on one GPU (other streams, other threads) race and give
 *     undefined results; calls ordered on one stream do not.
 * Arguments, outputs, checks and errors otherwise as ts_expand.
 */
int32_t ts_expand_noalloc(const ts_drafter* d, const ts_parent* parents, int32_t P, ts_calib calib,
                          int32_t k, float T, uint64_t seed, int32_t sampler, const ts_expand_out* out,
                          void* stream);

/* A draft tree per request, HOST memory, capacity `cap` = N + 1 rows per
 * request ([R][cap] row-major), node 0 = the root (anchor token, depth 0).
 * Nodes are in creation order, which is the pop order of Algorithm 1. */
typedef struct {
  int32_t R, cap;
  int32_t* n;          /* [R] materialised nodes, root excluded */
  int32_t* token;      /* [R][cap] */
  int32_t* parent;     /* [R][cap], -1 for the root */
  int32_t* depth;      /* [R][cap] */
  int32_t* rank;       /* [R][cap] sibling draw index (1-based), 0 for the root */
  uint64_t* path;      /* [R][cap] structural path id */
  float* log_surv;     /* [R][cap] log S(node) */
  float* log_q0;       /* [R][cap] log q0(token | parent), 0 for the root */
  float* log_qT;       /* [R][cap] log qT(token | parent), NaN at T = 0 and for the root */
  float* key;          /* [R][cap] key of the slot whose pop created the node */
  int32_t* evals;      /* [R] optional (may be NULL): parents evaluated for the request */
} ts_tree;

/* Limits of the device-resident waves of ts_build_tree (larger trees use
 * the host-driven waves). */
#define TS_DEVICE_WAVES_MAX_N 512
#define TS_DEVICE_WAVES_MAX_CHILDREN 1024

size_t ts_build_tree_workspace_size(const ts_drafter* d, int32_t N, int32_t K, float T);

/*
 * ts_build_tree: grow one tree per request by best-first expansion
 * (§3.2 Algorithm 1): pop the slot with the largest key (ties: shallower
 * child, then smaller child path id), stop when the popped key is below
 * log(theta[q]) (theta = 0 never stops, the fixed-budget case of §3.2) or
 * when N nodes exist; a node at depth D gets no slot; a node re-offers a
 * slot for its next child until it has K children.  The result equals the
 * sequential heap of Algorithm 1; it is computed in breadth waves, each one
 * expansion over all requests' pending parents.
 * budget > 0 adds one node budget shared by all requests (§4, per-request
 * budget allocation by greedy water-filling): the trees then hold the best
 * `budget` nodes of all requests together in the order (key desc, request
 * asc, child depth asc, child path asc), each request still at most N nodes
 * and stopped by its own theta.  Under one marginal price this is the theta
 * rule with theta_q raised to the key of the last node taken.  budget <= 0:
 * no shared budget.
 * Where the waves run: with budget <= 0, 1 <= N <= TS_DEVICE_WAVES_MAX_N and
 * max(1, N - 1) * K <= TS_DEVICE_WAVES_MAX_CHILDREN the waves and the tree
 * assembly run on the device (a control kernel per wave keeps each request's
 * best N slots and writes the next frontier; the host only reads each wave's
 * size, one wave ahead of the GPU); otherwise the host keeps the slots and
 * launches each wave.  Both give the same trees.
 * anchor [R], theta [R] are HOST arrays.  out is a HOST tree: out->cap must
 * be >= N + 1 and out->R == d->R; rows past n[q] are written with token and
 * parent -1, depth and rank 0, path 0 and NaN values.  device_out (may be
 * NULL) is a tree with the same R and cap whose arrays are DEVICE memory: it
 * receives the same tree (for ts_tree_mask without a host round trip).
 * sampler is a ts_sampler (used at T > 0).  Synchronises `stream`.
 */
int32_t ts_build_tree(const ts_drafter* d, const int32_t* anchor, const float* theta, int32_t N,
                      int32_t budget, int32_t K, ts_calib calib, float T, uint64_t seed,
                      int32_t sampler, ts_tree* out, const ts_tree* device_out, void* workspace,
                      size_t workspace_bytes, void* stream);

size_t ts_verify_workspace_size(const ts_drafter* d, int32_t cap, float T);

/*
 * ts_verify: accept a root path of each request's tree and emit one bonus
 * (correction) token.  target is a DEVICE array [R][cap][V] of dtype
 * target_dtype: row i of request q holds the target model's next-token
 * logits after the root path of node i.
 *   T == 0: exact match (§3.2 item 3): from the root, descend to the child
 *           whose token is the target argmax (ties: smallest id); the bonus
 *           is the argmax at the node where no child matches.
 *   T  > 0: recursive rejection (§3.3): at each visited node the target
 *           residual starts at p = softmax(row / T); siblings are tried in
 *           draw order with q_j = qT restricted to tokens not drawn before j
 *           and renormalised (qT is recomputed from U, E, W2); child j is
 *           accepted iff u < p_j(x_j) / q_j(x_j), else
 *           p_{j+1} = norm(max(p_j - q_j, 0)); the bonus is a Gumbel-max draw
 *           from the final residual.
 * tree is the HOST tree from ts_build_tree (tree->R == d->R, tree->cap ==
 * cap of target).  path_nodes [R][TS_MAX_D], path_len [R], bonus [R] are
 * HOST outputs (node indices into the tree).  Synchronises `stream`.
 */
int32_t ts_verify(const ts_drafter* d, const ts_tree* tree, const void* target,
                  int32_t target_dtype, float T, uint64_t seed, int32_t* path_nodes,
                  int32_t* path_len, int32_t* bonus, void* workspace, size_t workspace_bytes,
                  void* stream);

/* ------------------------------------------------------------------ serving
 * Load-aware tree shaping (§4): a deployment measures a price ladder
 * theta*(bs, T) once (Algorithm 2) and looks up each round's price from the
 * active batch size and the temperature.  A rung with theta < 0 is the chain
 * sentinel: the round runs the chain (K = 1, N = the block length b). */
typedef struct {
  int32_t bs_max;  /* the rung covers batches of at most bs_max requests */
  float T;         /* sampling temperature of the rung */
  float theta;     /* price; < 0 selects the chain */
} ts_ladder_rung;

typedef struct {
  float theta;    /* price for ts_build_tree (0 for the chain: no stop) */
  int32_t K;      /* sibling cap */
  int32_t N;      /* node cap */
  int32_t chain;  /* 1 if the chain sentinel was selected */
} ts_round_policy;

/*
 * ts_ladder_lookup: the policy of one round.  Among the rungs, take the
 * tabulated temperature nearest to T (ties: the lower one); among its rungs,
 * the one with the smallest bs_max >= bs (if bs exceeds them all, the one
 * with the largest bs_max).  A price >= 0 gives {theta, K, N, 0}; the chain
 * sentinel gives {0, 1, block_len, 1}.  rungs is a HOST array of n rungs.
 * Errors: NULL pointers, n < 1, bs < 1, T < 0 or not finite, K outside
 * [1, TS_MAX_K], N < 0, block_len outside [1, TS_MAX_D].
 */
int32_t ts_ladder_lookup(const ts_ladder_rung* rungs, int32_t n, int32_t bs, float T, int32_t K,
                         int32_t N, int32_t block_len, ts_round_policy* out);

/*
 * ts_ladder_default: the paper's measured A100 ladder with the interpolation
 * it states (Table 2; §4 scheduler simulation): at T = 0, theta = 0.02 for
 * bs <= 4, 0.05 for bs <= 8 and 0.15 above; at T = 0.5 and T = 1, theta = 0.05
 * for bs <= 8 and the chain above.  It is specific to that deployment: a new
 * one measures its own ladder.  Writes at most cap rungs to the HOST array
 * rungs and returns the number of rungs of the ladder (7).
 */
int32_t ts_ladder_default(ts_ladder_rung* rungs, int32_t cap);

/* Largest tree (rows per request) the mask builder accepts. */
#define TS_MAX_CAP 4096

/* Words per mask row of a tree with cap rows: ceil(cap / 32) (0 if cap < 1). */
int32_t ts_tree_mask_words(int32_t cap);

/*
 * ts_tree_mask: the tree attention mask and position ids of the target's
 * verification forward over the flattened trees (§3.2 item 3: one target
 * pass with a tree attention mask and per-depth position ids; §5: an
 * ancestor bitmask per row).  Row i of request q (node 0 = the anchor) sees
 * exactly the nodes on its root path, itself included: bit (j & 31) of word
 * (j >> 5) of row i is set iff node j is i or an ancestor of i.
 * pos[q][i] = pos_offset[q] + depth(i), the depth counted along the parent
 * chain (pos_offset NULL reads as 0).  Rows i > n[q] are all zero and get
 * pos -1.
 *   parent [R][cap], n [R], pos_offset [R]: DEVICE inputs in the ts_tree
 *       layout (parent[q][0] = -1 and 0 <= parent[q][i] < i for i >= 1);
 *   mask [R][cap][ts_tree_mask_words(cap)] (uint32), pos [R][cap]: DEVICE
 *       outputs, fully written.
 * A parent chain that breaks the ordering rule stops at the break (nothing
 * outside the arrays is read); n[q] < 0 gives an empty tree and
 * n[q] >= cap is read as cap - 1.  Asynchronous on `stream`.  Host checks:
 * null pointers, R >= 0, 1 <= cap <= TS_MAX_CAP.
 */
int32_t ts_tree_mask(const int32_t* parent, const int32_t* n, int32_t R, int32_t cap,
                     const int32_t* pos_offset, uint32_t* mask, int32_t* pos, void* stream);

/*
 * Calibration of the edge-acceptance estimate (§3.4 Eq. 3): the labels a
 * greedy (T = 0) round produces, and the two-scalar Platt fit
 * p-hat = sigmoid(a logit q0 + b).  In a greedy round the verifier shows, for
 * every materialised node, whether its token is the target's greedy choice
 * at its parent; the fit uses the edges whose ancestors were all accepted
 * (the population that path-survival products condition on).  A deployment
 * fits the two scalars once per drafter-target pair.
 */

/* Bytes of device workspace ts_calib_labels needs for R requests of capacity cap. */
size_t ts_calib_labels_workspace_size(int32_t R, int32_t cap);

/*
 * ts_calib_labels: tree is a HOST tree (ts_build_tree's out) of R requests
 * and capacity cap; target is a DEVICE array [R][cap][V] of target_dtype
 * (row i: the target's next-token logits after node i's root path).  For
 * every request q and node 1 <= i <= n[q] it writes, to DEVICE arrays
 * [R][cap]:
 *   x[q][i]   = logit q0 = log q0 - log(1 - q0) of the node (from
 *               tree->log_q0; +inf where q0 == 1);
 *   y[q][i]   = 1 if the node's token is the argmax (smallest id on ties) of
 *               the target row of its parent, else 0;
 *   sel[q][i] = 1 if every edge on the root path of its parent has y = 1.
 * Row 0 and rows past n[q] get x NaN, y -1, sel 0.  Host checks: null
 * pointers, R >= 1, the tree's shape (0 <= n < cap, parents before
 * children, tokens in [0, V)), target_dtype, workspace size.  Synchronises
 * `stream`.
 */
int32_t ts_calib_labels(const ts_tree* tree, const void* target, int32_t target_dtype, int32_t V, float* x,
                        int32_t* y, int32_t* sel, void* workspace, size_t workspace_bytes, void* stream);

/*
 * ts_calib_fit: the maximum-likelihood (a, b) of y ~ Bernoulli(sigmoid(a x +
 * b)) over the samples i < n with sel[i] = 1, y[i] in {0, 1} and x[i]
 * finite (x, y, sel: DEVICE arrays in the ts_calib_labels layout, flattened).
 * Newton's method from (0, 0); a step that raises the negative
 * log-likelihood is halved until it does not; at most max_iter steps,
 * stopping when a step moves both scalars by less than tol.  Sums are fp64
 * in a fixed order.  out: DEVICE float[4] = {a, b, mean negative
 * log-likelihood, steps}; a, b and the likelihood are NaN when no sample
 * takes part or the curvature is singular (a single input value), and a
 * separable sample keeps growing until max_iter.  Asynchronous on
 * `stream`.  Host checks: null pointers, n >= 0, max_iter >= 1, tol > 0.
 */
int32_t ts_calib_fit(const float* x, const int32_t* y, const int32_t* sel, int32_t n, int32_t max_iter,
                     double tol, float* out, void* stream);

/*
 * ts_verify_set_mode: how ts_verify runs its T > 0 levels on the calling
 * thread.  TS_VERIFY_AUTO (the default): in one launch per level whenever
 * every workgroup of the level can be resident at once (the workgroups of an
 * item wait for one another between the walk's steps), else through the
 * per-stage launches.  TS_VERIFY_STAGED: always through the per-stage
 * launches, which never wait on other workgroups; for callers that keep
 * other kernels running on the device during ts_verify (a level's one launch
 * assumes its workgroups get the whole device, and otherwise waits up to
 * about a tenth of a second per step before it runs the level again per
 * stage).  Both give results within the same rounding of the walk.
 * Errors: an unknown mode.
 */
#define TS_VERIFY_AUTO 0
#define TS_VERIFY_STAGED 1
int32_t ts_verify_set_mode(int32_t mode);

/*
 * ts_verify_level_counts: how the T > 0 levels of ts_verify calls on the
 * calling thread ran.  *fused: levels run in one launch, each workgroup
 * holding its chunk of the target and draft rows in registers (when every
 * workgroup of the level can be resident at once); *fallbacks: of those, the
 * levels run again through the per-stage launches because a wait between
 * workgroups ran out; *staged: levels run through the per-stage launches from
 * the start (pass A, one launch per stage, resolve).  The counts are the
 * thread's totals since its first call (ts_release_thread_state keeps them).
 * Errors: NULL pointers.
 */
int32_t ts_verify_level_counts(int64_t* fused, int64_t* fallbacks, int64_t* staged);

/* Description of the last error on the calling thread ("" if none). */
const char* ts_last_error(void);

/*
 * ts_release_thread_state: free what the library keeps for the calling host
 * thread between calls: a page-locked staging buffer (the small transfers of
 * ts_build_tree, ts_verify and ts_calib_labels, which kernels also read and
 * write directly).  It first waits for the current device
 * (hipDeviceSynchronize).  Call it before
 * the thread or the process ends, while the HIP runtime is still up: the
 * library frees nothing from thread-exit or process-exit handlers, since those
 * may run after the runtime (or a profiler attached to it) has been torn down.
 * A later call that needs the buffer allocates it again.
 * Returns TS_OK, or TS_EHIP if a HIP call fails.
 */
int32_t ts_release_thread_state(void);

/* Library version string. */
const char* ts_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TREESPARK_H */
