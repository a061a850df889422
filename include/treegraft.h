/*
 * treegraft.h - C ABI of libtreegraft.so, the MI355X (gfx950) hot path of
 * tree-based speculative decoding with a shared, multi-drafter draft tree
 * (TreeGraft: Adaptive Multi-Drafter Grafting for Tree-Based Speculative
 * Decoding).
 *
 * Four calls:
 *   tg_tree_verify_attention  target-side tree attention of a draft tree
 *                             against a prefix KV cache (Alg. 3 mask; Sec. 3.1)
 *   tg_tree_expand_topk       one standard expansion step (Sec. 3.1; Alg. 1)
 *   tg_tree_rescore_graft     one middle-drafter step: expanded pool,
 *                             rescoring, reselection, non-destructive graft
 *                             (Sec. 3.2; Alg. 2, middle branch)
 *   tg_tree_accept            greedy (temperature 0) acceptance of the longest
 *                             draft path matching the target (Sec. 3.2,
 *                             "Distribution preservation"; App. E)
 *
 * Conventions shared by every call
 *   - Every pointer argument is DEVICE memory owned by the caller, except the
 *     tg_tree struct itself, which is a host struct holding device pointers.
 *     The library never allocates per call; scratch memory is the caller's
 *     `workspace`, sized by the matching *_workspace() query (any contents;
 *     one call at a time per workspace).
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream).  The returned tg_status reports host-side argument checks and
 *     the kernel launch only.
 *   - Data errors that only the device can see are OR-ed into `*d_err` (a
 *     device uint32, optional: NULL disables reporting).  Each bit has a
 *     documented safe fallback, so kernels always complete.  Read it after
 *     synchronising the stream.
 *   - Arrays are dense, row-major, with the shapes written next to each
 *     argument.  Node ids are dense per tree and topological: a node's parent
 *     id is smaller than its own.  The root is implicit: id -1, cumulative
 *     score 0, depth 0.
 *   - Scores are natural logs: an edge score p(u) of the paper is stored as
 *     logp = log p(u), a path score s(v) = prod p(u) as cum = log s(v).
 *     logp = fl(x - lse) and cum = fl(cum_parent + logp) are single IEEE fp32
 *     operations (x = the token's fp32 logit, lse = the row's log-sum-exp).
 *   - Rankings: a logits row's top-k tokens are ordered by (logit desc,
 *     token asc); node rankings use (cum desc, depth asc, id asc), the key
 *     Alg. 3 fixes for pruning.  -0.0 ranks equal to +0.0.
 *   - Apart from the optional benchmark trace (tg_trace_*, process-global
 *     and not thread-safe, off by default), the library holds no mutable
 *     global state: with tracing off every call is reentrant.
 */
#ifndef TREEGRAFT_H
#define TREEGRAFT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TG_OK = 0,
  TG_ERR_INVALID_ARG = 1,  /* NULL pointer, negative size, inconsistent shapes */
  TG_ERR_UNSUPPORTED = 2,  /* valid but outside the supported limits below   */
  TG_ERR_WORKSPACE = 3,    /* workspace NULL or smaller than the query says   */
  TG_ERR_HIP = 4           /* a HIP runtime call or kernel launch failed      */
} tg_status;

typedef enum { TG_F32 = 0, TG_BF16 = 1 } tg_dtype;

/* Device error word bits and the fallback each one triggers. */
#define TG_DERR_BAD_PARENT 1u  /* parent[i] >= i or < -1: read as -1            */
#define TG_DERR_CAPACITY 2u    /* append would exceed tree cap: that tree is    *
                                * left unchanged; accept: an acceptable node    *
                                * deeper than max_depth was ignored             */
#define TG_DERR_NONFINITE 4u   /* NaN or +inf logit: read as -inf               */
#define TG_DERR_BAD_PREFIX 8u  /* prefix_len < 0 or prefix_len + N > S_max:     *
                                * that sequence's outputs are written as zeros  */
#define TG_DERR_BAD_NODE 16u   /* frontier id outside [-1, n_nodes), strong-    *
                                * logits rows < n_nodes + 1, or a tree larger   *
                                * than a kernel limit: that tree is unchanged   */

#define TG_NO_NODE (-2)        /* padding of frontier outputs (-1 is the root) */

/* Variant flags of tg_tree_rescore_graft (0 = the method of Sec. 3.2).  The
 * first two are the Sec. 5.3 ablations. */
#define TG_POOL_NEWONLY 1u     /* w/o EG: pool C = N_k, the previous step's
                                  new nodes (ids >= new_from[b]; -1 = root) */
#define TG_GRAFT_OVERWRITE 2u  /* w/o ND: grafting under a frontier node
                                  first removes its existing subtrees       */
#define TG_GRAFT_DEDUP 4u      /* skip a new child whose token an existing
                                  child of the same parent already carries  */

/* Limits (TG_ERR_UNSUPPORTED outside them). */
#define TG_MAX_TOPK 64         /* K of expand, M of rescore                     */
#define TG_MAX_CAP 4096        /* tree capacity (nodes per tree, root excluded) */
#define TG_MAX_EXPAND_CHILDREN 8192 /* F * K of one expand call                */
#define TG_MAX_VERIFY_NODES 1024    /* N of one verify call                    */
#define TG_MAX_NGRAM 16             /* n_max of the n-gram drafter             */
#define TG_MAX_NGRAM_FRONTIER 1024  /* F of one n-gram expansion               */
#define TG_NOALLOC_SCRATCH_BYTES (32u << 20) /* scratch of the no-allocation call */

/*
 * Caller-owned draft tree, structure of arrays, one row of `cap` slots per
 * batch element (Sec. 3.1: each non-root node stores its token, its edge
 * score and its path score; Sec. 3.2: the middle drafter's visited set P).
 * Slots [0, n_nodes[b]) are live.  `visited` and `root_visited` hold P_k
 * membership (1 = entered a middle-drafter pool before).
 */
typedef struct {
  int32_t *parent;        /* [B, cap] parent id, -1 = root                   */
  int32_t *token;         /* [B, cap] token id                               */
  int32_t *depth;         /* [B, cap] depth (root 0); must equal the length  *
                           * of the parent chain                             */
  float *logp;            /* [B, cap] fp32 log edge score                    */
  float *cum;             /* [B, cap] fp32 log path score                    */
  uint8_t *visited;       /* [B, cap] 0/1                                    */
  uint8_t *root_visited;  /* [B]      0/1                                    */
  int32_t *n_nodes;       /* [B]      live node count, updated by appends    */
  int32_t cap;            /* slots per batch element, <= TG_MAX_CAP          */
} tg_tree;

const char *tg_status_str(tg_status s);

/*
 * Start a new drafting turn: every tree becomes the lone root (n_nodes = 0,
 * root unvisited; Alg. 1/2 initialise T_1 = {r} and P_1 = empty).  Slots are
 * not cleared.  A kernel, not a memset, so the call can sit in a captured
 * HIP graph.
 */
tg_status tg_tree_reset(const tg_tree *tree, int B, void *stream);

/* ------------------------------------------------------------------------ */
/* Tree-verify attention (Alg. 3 mask; Sec. 3.1 root = verified prefix).     */
/*
 * For batch b, tree node i and query head h (KV head g = h / (Hq / Hkv)):
 * node i attends to the prefix cache positions [0, L_b) and to the tree slots
 * L_b + a for every a on its root-to-node path (its ancestors and itself), i.e.
 * mask(i, j) = 1 iff j is the root (the prefix), an ancestor of i, or i.
 *   out = softmax(sm_scale * q K^T) V over those keys.
 *
 * q          [B, N, Hq, D]       dtype
 * k_cache    [B, Hkv, S_max, D]  dtype; prefix at [0, L_b), the N tree nodes'
 * v_cache    [B, Hkv, S_max, D]  keys/values at [L_b, L_b + N)
 * parent     [B, N] int32, parent[i] in [-1, i-1]; -1 = hangs under the prefix
 * prefix_len [B] int32 (device), L_b >= 0 and L_b + N <= S_max
 * out        [B, N, Hq, D]       dtype (fp32 accumulation inside)
 * D in {64, 128}; Hq % Hkv == 0; 1 <= N <= TG_MAX_VERIFY_NODES;
 * sm_scale finite and >= 0; q, k_cache, v_cache and out 16-byte aligned
 * (else TG_ERR_INVALID_ARG).
 * dtype TG_BF16 runs the MFMA kernel; TG_F32 runs an fp32 VALU kernel.
 * Device errors: BAD_PARENT (that parent read as -1), BAD_PREFIX (zeros).
 */
size_t tg_verify_attention_workspace(int B, int N, int Hq, int Hkv, int D,
                                     int S_max, tg_dtype dtype);

tg_status tg_tree_verify_attention(const void *q, const void *k_cache,
                                   const void *v_cache, const int32_t *parent,
                                   const int32_t *prefix_len, void *out, int B,
                                   int N, int Hq, int Hkv, int D, int S_max,
                                   float sm_scale, tg_dtype dtype,
                                   void *workspace, size_t ws_bytes,
                                   uint32_t *d_err, void *stream);

/*
 * tg_tree_verify_attention without a workspace, for callers that cannot
 * allocate (code under HIP graph capture, serving loops, harnesses that
 * forbid allocation).  Same arguments, results and device errors as
 * tg_tree_verify_attention, same kernels; the split-prefix partials go to a
 * scratch array of TG_NOALLOC_SCRATCH_BYTES that the library keeps in every
 * device's memory from its first use until the process ends.  The call uses
 * the scratch of the current device (the stream must belong to it); its
 * first call on a device looks the array's address up, later calls allocate
 * nothing and call no allocating routine.
 * Limits: a shape whose workspace query exceeds TG_NOALLOC_SCRATCH_BYTES is
 * rejected with TG_ERR_WORKSPACE before anything is launched.
 * Calls on one device share the scratch: two calls that overlap in time on
 * one GPU (different streams, or host threads) race and may corrupt each
 * other's output; calls ordered on one stream do not.  The scratch needs no
 * clearing (every call writes all of the partials it reads).
 */
tg_status tg_tree_verify_attention_noalloc(const void *q, const void *k_cache,
                                           const void *v_cache, const int32_t *parent,
                                           const int32_t *prefix_len, void *out, int B, int N,
                                           int Hq, int Hkv, int D, int S_max, float sm_scale,
                                           tg_dtype dtype, uint32_t *d_err, void *stream);

/* ------------------------------------------------------------------------ */
/* One expansion step (Sec. 3.1; Alg. 1).                                   */
/*
 * For tree b and each live frontier row f < F_b (F_b = n_frontier[b], or F
 * when n_frontier is NULL), row logits[b, f, :] are the drafter's next-token
 * logits at frontier node v = frontier[b, f] (-1 = root):
 *   lse_f = log sum_t exp(x_t)                      (fp32, exported in row_lse)
 *   top-K tokens y_j of the row, j = 0..K-1         (logit desc, token asc)
 *   child (f, j): id n_b + f*K + j, parent v, token y_j, depth depth(v)+1,
 *                 logp = fl(x_{y_j} - lse_f), cum = fl(cum(v) + logp),
 *                 visited 0.
 * All F_b*K children are attached (n_nodes[b] += F_b*K).  next_frontier[b]
 * receives the ids of the best min(N, F_b*K) new children by (cum desc,
 * depth asc, id asc), best first, padded with TG_NO_NODE; n_next[b] their
 * count.  A row whose logits are all -inf has lse -inf and gives logp -inf.
 *
 * logits        [B, F, V] fp32
 * frontier      [B, F] int32, ids in [-1, n_nodes[b])
 * n_frontier    [B] int32 or NULL
 * row_lse       [B, F] fp32 out (rows f >= F_b untouched)
 * next_frontier [B, N] int32 out;  n_next [B] int32 out
 * 1 <= K <= min(V, TG_MAX_TOPK); 1 <= N; F*K <= TG_MAX_EXPAND_CHILDREN.
 * Device errors: NONFINITE; BAD_NODE or CAPACITY leave tree b unchanged
 * (n_next[b] = 0, row_lse still written).
 */
size_t tg_expand_topk_workspace(int B, int F, int V, int K, int N);

tg_status tg_tree_expand_topk(const tg_tree *tree, const float *logits,
                              const int32_t *frontier,
                              const int32_t *n_frontier, int B, int F, int V,
                              int K, int N, float *row_lse,
                              int32_t *next_frontier, int32_t *n_next,
                              void *workspace, size_t ws_bytes,
                              uint32_t *d_err, void *stream);

/* ------------------------------------------------------------------------ */
/* One middle-drafter step (Sec. 3.2 candidate-pool equation; Alg. 2).      */
/*
 * strong_logits[b, r, :] are the middle drafter's next-token logits at the
 * root (r = 0) and at node r-1 (r >= 1); rows of nodes the drafter ran on in
 * an earlier step are its cached logits.  For tree b:
 *   1. pool C = {v < n_b : !visited[v]}, plus the root while !root_visited.
 *   2. for each non-root v in C: logp[v] = fl(x - lse) with x the logit of
 *      token[v] in row parent[v]+1 and lse that row's log-sum-exp; then, in
 *      parent-before-child order, cum[v] = fl(cum[parent] + logp[v]).
 *   3. graft frontier F = the best min(W, |C|) of C by (cum desc, depth asc,
 *      id asc) (root: id -1, cum 0, depth 0).
 *   4. non-destructive graft: for frontier rank f and each of the top-M
 *      tokens (rank j) of row F[f]+1, attach a NEW child with id
 *      n_b + f*M + j, parent F[f], logp = fl(x - lse), cum = fl(cum(F[f]) +
 *      logp), depth depth(F[f]) + 1, visited 0.  No existing node's parent,
 *      token or depth is written.
 *   5. P <- P u C: visited[v] = 1 for v in C, root_visited = 1 if the root
 *      is in C; n_b += |F|*M.
 * Variants (flags, any combination):
 *   TG_POOL_NEWONLY: step 1 uses C = {v : new_from[b] <= v < n_b} (the root
 *      when new_from[b] == -1); new_from [B] int32 device, read only with
 *      this flag (BAD_NODE when outside [-1, n_b], then clamped).
 *   TG_GRAFT_OVERWRITE: between steps 3 and 4 every node with a strict
 *      ancestor in F is removed (a frontier node inside a removed subtree
 *      leaves F) and the survivors are renumbered densely in id order, all
 *      their fields moved; F and the new children use the new ids; the
 *      children of surviving slot f are n_b' + f*M + j.
 *   TG_GRAFT_DEDUP: a (slot, rank) whose token an existing child of F[f]
 *      carries is not attached; the attached children take dense ids in
 *      (slot, rank) order.  (After an overwrite a frontier node has no
 *      children, so nothing is skipped.)
 *   The capacity check is the upper bound n_b + |F|*M in every variant.
 * row_lse[b, r] is written for the rows the step reads: v+1 and parent(v)+1
 * for v in C (other rows untouched).  graft_frontier[b] = F (ids, -1 = root),
 * padded with TG_NO_NODE; n_graft[b] = |F|.
 * The grafted children are N_{k+1}, the pool of a following small step (Sec.
 * 3.2, small steps use C = N_k).  When next_frontier is non-NULL it receives
 * their best min(N, |F|*M) ids by (cum desc, depth asc, id asc), padded with
 * TG_NO_NODE, and n_next[b] their count: the frontier to hand to
 * tg_tree_expand_topk for that small step.
 *
 * strong_logits  [B, R, V] fp32, R >= n_nodes[b] + 1 for every b
 * row_lse        [B, R] fp32 out;  graft_frontier [B, W] int32 out;
 * n_graft        [B] int32 out
 * next_frontier  [B, N] int32 out or NULL;  n_next [B] int32 out (NULL iff
 *                next_frontier is NULL);  N >= 1 when next_frontier is used
 * 1 <= M <= min(V, TG_MAX_TOPK); 1 <= W; cap <= TG_MAX_CAP; flags within
 * the three bits above (TG_ERR_UNSUPPORTED otherwise, or when the step's LDS
 * layout for this cap, M and flags exceeds 160 KiB: the graft variants need
 * 20 bytes per slot more, so they stop at cap 2048 for small M).
 * Device errors: NONFINITE; BAD_NODE (R too small) or CAPACITY
 * (n_b + |F|*M > cap) leave tree b unchanged with n_graft[b] = 0 and
 * n_next[b] = 0.
 */
size_t tg_rescore_graft_workspace(int B, int R, int V, int W, int M, int cap);

tg_status tg_tree_rescore_graft(const tg_tree *tree, const float *strong_logits,
                                int B, int R, int V, int W, int M,
                                uint32_t flags, const int32_t *new_from, float *row_lse,
                                int32_t *graft_frontier, int32_t *n_graft,
                                int32_t *next_frontier, int32_t *n_next, int N,
                                void *workspace, size_t ws_bytes,
                                uint32_t *d_err, void *stream);

/* ------------------------------------------------------------------------ */
/* The n-gram small drafter (App. C.1, the small drafter's implementation): a
 * training-free lookup that proposes children from the target's prefill.  */
/*
 * tg_ngram_cache builds the prefill cache of B sequences:
 *   cand_tok[b, i, :], cand_logp[b, i, :] = the top-m tokens of logits row
 *     (b, i) (the target's logits after x_<=i) by (logit desc, token asc) and
 *     their log-probabilities fl(x - lse), lse as in tg_tree_expand_topk;
 *     every row 0 <= i < L is cached;
 *   fallback_pos[b] = the last position i < ctx_len[b] of the most frequent
 *     token of context[b, :ctx_len[b]] (ties to the smallest token id), -1
 *     for an empty context.
 * logits [B, L, V] fp32; context [B, L] int32 (tokens in [0, V), others are
 * skipped and raise BAD_NODE); ctx_len [B] int32 device; cand_tok [B, L, m]
 * int32 out; cand_logp [B, L, m] fp32 out; fallback_pos [B] int32 out.
 * 1 <= m <= min(V, TG_MAX_TOPK).  Device errors: NONFINITE, BAD_NODE.
 *
 * tg_tree_expand_ngram is one small-drafter step (Alg. 1 with the n-gram
 * drafter).  For frontier node v (slot f) of tree b the prefix is
 * context[b, :ctx_len[b]] followed by the tokens on v's root path; its
 * matched position j is the latest end position in the context of its
 * longest suffix of length n_max, n_max - 1, ..., 1 found there (the root's
 * own prefix matches at ctx_len - 1), else fallback_pos[b] (BAD_NODE and
 * ctx_len - 1 when that is not a context position).  v gets the K children
 * (ids n_b + f*K + k) token = cand_tok[b, j, k], logp = cand_logp[b, j, k],
 * cum = fl(cum(v) + logp), depth(v) + 1, visited 0; next_frontier / n_next
 * as in tg_tree_expand_topk; match_pos[b, f] = j (-1 padded; may be NULL).
 * 1 <= K <= m; 1 <= n_max <= TG_MAX_NGRAM; F <= TG_MAX_NGRAM_FRONTIER;
 * F*K <= TG_MAX_EXPAND_CHILDREN; cap <= TG_MAX_CAP.
 * Device errors: BAD_NODE (frontier id out of range: tree b unchanged);
 * BAD_PREFIX (ctx_len outside [1, L]: unchanged); CAPACITY (unchanged).
 */
size_t tg_ngram_cache_workspace(int B, int L, int V, int m);

tg_status tg_ngram_cache(const float *logits, const int32_t *context, const int32_t *ctx_len,
                         int B, int L, int V, int m, int32_t *cand_tok, float *cand_logp,
                         int32_t *fallback_pos, void *workspace, size_t ws_bytes,
                         uint32_t *d_err, void *stream);

tg_status tg_tree_expand_ngram(const tg_tree *tree, const int32_t *frontier,
                               const int32_t *n_frontier, const int32_t *context,
                               const int32_t *ctx_len, const int32_t *cand_tok,
                               const float *cand_logp, const int32_t *fallback_pos, int B,
                               int F, int L, int m, int K, int N, int n_max,
                               int32_t *match_pos, int32_t *next_frontier, int32_t *n_next,
                               uint32_t *d_err, void *stream);

/* ------------------------------------------------------------------------ */
/* Greedy acceptance (temperature 0; Sec. 3.2; App. E).                     */
/*
 * greedy[b, 0] is the target's arg-max token after the prefix (the root),
 * greedy[b, 1+i] its arg-max after node i.  A node is acceptable iff every
 * node u on its root path has token[u] == greedy[b, parent[u]+1].  The
 * accepted node is the deepest acceptable node of depth <= max_depth (ties
 * to the smallest id); accept_len[b] = its depth (number of accepted draft
 * tokens, 0 if none), accept_path[b] = its root path (node ids, root first,
 * padded with -1), bonus[b] = greedy[b, accepted+1] (greedy[b, 0] if none).
 *
 * parent, token [B, cap] int32; n_nodes [B] int32 (<= cap, <= TG_MAX_CAP)
 * greedy        [B, cap + 1] int32
 * accept_len [B], accept_path [B, max_depth], bonus [B]  int32 out
 * Device errors: BAD_PARENT (read as -1); CAPACITY (an acceptable node
 * deeper than max_depth was ignored); BAD_NODE (n_nodes > cap: tree treated
 * as empty).
 */
tg_status tg_tree_accept(const int32_t *parent, const int32_t *token,
                         const int32_t *n_nodes, const int32_t *greedy, int B,
                         int cap, int max_depth, int32_t *accept_len,
                         int32_t *accept_path, int32_t *bonus, uint32_t *d_err,
                         void *stream);

/*
 * tg_tree_accept_logits: the same acceptance straight from the target's
 * logits.  greedy[b, r] = arg-max of logits[b, r] (ties to the smallest
 * token id; NaN and +inf read as -inf, NONFINITE) for r <= n_nodes[b], -1
 * for the other rows; then tg_tree_accept on that greedy array.
 *
 * logits  [B, R, V] fp32 (row 0 = after the prefix, 1+i = after node i);
 *         R >= n_nodes[b] + 1, else BAD_NODE and the missing rows read -1
 *         (nothing below them is acceptable)
 * greedy  [B, cap + 1] int32 out; the other arguments as tg_tree_accept.
 */
tg_status tg_tree_accept_logits(const int32_t *parent, const int32_t *token,
                                const int32_t *n_nodes, const float *logits, int B, int cap,
                                int R, int V, int max_depth, int32_t *greedy,
                                int32_t *accept_len, int32_t *accept_path, int32_t *bonus,
                                uint32_t *d_err, void *stream);

/* ------------------------------------------------------------------------ */
/* Final pruning and the verification buffers (Alg. 3, global score-based
 * pruning with ancestor closure).                                          */
/*
 * tg_tree_global_prune keeps at most B_ver non-root nodes of each tree b:
 * the non-root nodes are ranked by (cum desc, depth asc, id asc); in rank
 * order each node is kept together with its not-yet-kept ancestors when the
 * kept set (root included) stays within M = B_ver + 1, until it holds M
 * nodes; a tree with n_nodes <= B_ver keeps everything.  Depths are
 * recomputed from `parent` (root depth 0).  The kept nodes are re-indexed by
 * (depth, original id), which puts parents before children.  Verify index 0
 * is the root and verify index j + 1 is kept node j.  Outputs for tree b
 * (nk = n_keep[b] kept non-root nodes, nl = n_leaves[b]):
 *   kept[b, j]          original node id of kept node j         [B, B_ver]
 *   vparent[b, j]       its parent as a kept-node index, -1 = root [B, B_ver]
 *   vtoken[b, j]        its token                               [B, B_ver]
 *   position_ids[b, u]  depth of verify row u (root 0)          [B, B_ver + 1]
 *   mask[b, u, w]       bit v of word w = v / 32 is set iff verify node v
 *                       is the root, an ancestor of u or u itself
 *                                               [B, B_ver + 1, ceil((B_ver + 1) / 32)]
 *   retrieval[b, r, c]  the root-to-leaf path of the r-th leaf (leaves in
 *                       verify order), as verify indices with the root at
 *                       column 0, padded with -1          [B, B_ver + 1, max_path]
 *   n_keep[b], n_leaves[b]                                      [B]
 * Entries past nk, past nl and past a path are -1 (mask words 0).  Errors
 * (device word): n_nodes outside [0, cap] -> TG_DERR_BAD_NODE (nothing
 * kept); a parent outside [-1, v-1] -> TG_DERR_BAD_PARENT (read as the root);
 * a root-to-leaf path longer than max_path -> TG_DERR_CAPACITY (that tree's
 * retrieval rows are all -1).  When the ranking puts every parent before its
 * children (always so for trees this library grows: cum never increases
 * along a path and ties go to the smaller depth) the kept set is the first
 * B_ver ranked nodes; other inputs take the literal loop on one thread
 * (O(n * depth)).  Host checks: 1 <= B_ver <= TG_MAX_CAP, 1 <= max_path,
 * tree cap <= TG_MAX_CAP, every pointer non-NULL except d_err / stream.
 */
tg_status tg_tree_global_prune(const tg_tree *tree, int B, int B_ver, int max_path,
                               int32_t *kept, int32_t *vparent, int32_t *vtoken,
                               int32_t *position_ids, uint32_t *mask, int32_t *retrieval,
                               int32_t *n_keep, int32_t *n_leaves, uint32_t *d_err,
                               void *stream);

/*
 * tg_kv_compact: the cache update after acceptance.  The verified tokens
 * extend the prefix (Sec. 3.1: the draft tree's root is the verified
 * prefix).  For sequence b with L = prefix_len[b] and n = n_path[b], the K
 * and V rows at cache positions L + path[b, j] move to L + j for j < n, in
 * every KV head, and new_prefix_len[b] = L + n.  path[b, .] holds tree slots
 * of the verify layout (slot a lives at cache row L + a): the root's slot 0
 * first when it carries a token, then the accepted nodes, parents first.
 * It must be strictly increasing with path[b, j] >= j and
 * L + path[b, j] < S_max; otherwise sequence b is left untouched,
 * new_prefix_len[b] = L and TG_DERR_BAD_NODE is raised.  k_cache, v_cache
 * [B, Hkv, S_max, D] in `dtype`, updated in place; path [B, max_path];
 * prefix_len, n_path, new_prefix_len [B] device int32 (new_prefix_len must
 * not alias prefix_len).  Host checks: D in {64, 128}, 0 <= max_path,
 * positive sizes.
 */
tg_status tg_kv_compact(void *k_cache, void *v_cache, const int32_t *prefix_len,
                        const int32_t *path, const int32_t *n_path, int B, int Hkv, int S_max,
                        int D, int max_path, tg_dtype dtype, int32_t *new_prefix_len,
                        uint32_t *d_err, void *stream);

/* ------------------------------------------------------------------------ */
/* Scheduler observations and margin predictor (App. B.2: the candidate tree
 * signals and the reselection preview frontier; App. B.4: the margin
 * predictor; Sec. 4.3 runtime scheduling).                                 */
/*
 * tg_tree_signals computes, for each tree b with current frontier
 * frontier[b, 0:Fb] (node ids, -1 = root; Fb = n_frontier[b], or F when
 * n_frontier is NULL), the ten pre-action signals into signals[b, 0:10] in
 * this order: depth_before, leaf_ratio_before, pre_reselect_depth_delta,
 * pre_reselect_cands, max_depth_before, collapse_debt,
 * pre_reselect_past_ratio, pre_reselect_overlap, pre_reselect_score,
 * finite_score_ratio_before.  The preview frontier is Top_W of the nodes
 * (root included) whose depth lies within `lookback` below a frontier
 * depth, ranked by (cum desc, depth asc, id asc).  Scores are the stored
 * log-domain cum (root 0); "finite" means cum > -inf; depths are the
 * stored ones (root 0).  An empty mean is NaN.
 * When params is not NULL it holds the predictor's 3,265 weights, row-major
 * W1[64,17], b1[64], W2[32,64], b2[32], W3[1,32], b3[1] (fp32), and
 * context[b, 0:11] the runtime context (4) and scheduling history (7); the
 * input is context followed by depth_before, leaf_ratio_before,
 * collapse_debt, pre_reselect_past_ratio, pre_reselect_overlap,
 * pre_reselect_score, and margin[b] / action[b] (1 = call the middle
 * drafter iff margin > 0) are written.  Errors: n_nodes outside [0, cap] or
 * a frontier id outside [-1, n_nodes) -> TG_DERR_BAD_NODE and NaN signals.
 * Host checks: F, W >= 1, lookback >= 0, cap <= TG_MAX_CAP; context, margin
 * and action are required with params.
 */
tg_status tg_tree_signals(const tg_tree *tree, const int32_t *frontier, const int32_t *n_frontier,
                          int B, int F, int W, int lookback, const float *context,
                          const float *params, float *signals, float *margin, int32_t *action,
                          uint32_t *d_err, void *stream);

/* ------------------------------------------------------------------------ */
/* Kernel timing (benchmarks and profiling; not part of the hot path).      */
/*
 * tg_trace_begin(capacity) creates `capacity` HIP event pairs and turns
 * tracing on: from then on every kernel the library launches is bracketed by
 * hipEventRecord(start) / hipEventRecord(stop) on the stream it is launched
 * on, so each record is the device time of one kernel including its
 * dispatch (a few microseconds more than a profiler's kernel time).
 * Launches beyond `capacity` are not recorded.  Meant for eager launches:
 * event records captured into a HIP graph cannot be timed.
 * tg_trace_read waits for the recorded events and writes at most
 * max_records records in launch order (kernel names are static strings
 * owned by the library) without ending the trace.  tg_trace_end does the
 * same once, then frees the events and turns tracing off.  Tracing state is process-global
 * and not thread-safe; while it is off (the default) no event is created or
 * recorded.  Errors: TG_ERR_INVALID_ARG when tracing is not on (read, end)
 * or already on (begin), or capacity <= 0; TG_ERR_HIP when an event fails.
 */
typedef struct {
  const char *kernel;
  float ms;
} tg_trace_record;

tg_status tg_trace_begin(int capacity);
tg_status tg_trace_read(tg_trace_record *out, int max_records, int *n_records);
tg_status tg_trace_end(tg_trace_record *out, int max_records, int *n_records);

#ifdef __cplusplus
}
#endif

#endif /* TREEGRAFT_H */
