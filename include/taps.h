/* taps.h -- C ABI of the TAPS draft-tree verification hot path on MI355X (gfx950).
 *
 * One decoding round of TAPS (Target-Aware Prefix Tree Selection, arXiv 2606.00487):
 *   taps_select       per-position top-K of the drafter marginals (Sec. 4.1, Stage 1),
 *                     sibling-softmax edge probabilities q_cond (Eq. 1), reach
 *                     probabilities q_reach (Eq. 2), utility (Eq. 3) and the greedy
 *                     budgeted prefix-closed selection of Alg. 1.
 *   tree_verify_attn  tree-masked verification attention: every selected node attends
 *                     to the cached context and to its own ancestors (Sec. 4.1 Stage 3,
 *                     Sec. 4.3: verification needs a connected subtree at the root).
 *                     tree_verify_attn_paged: the same over a paged KV cache.
 *   accept_walk       greedy (temperature 0) acceptance of the longest matching root
 *                     path (Sec. 1: one prefix path is committed per round; Limitations).
 *   kv_commit         the round's state update: the accepted path's tree K/V rows move
 *                     to the rows right after the context, and the emitted tokens
 *                     (kv_commit_paged: the same on a paged cache).
 *   verify_layer      one attention layer of the target over the tree: projections,
 *                     per-head RMSNorm, rotary positions by tree depth, tree attention,
 *                     output projection (the verification forward's layer slice).
 *
 * Conventions shared by every call:
 *   - Pointers are DEVICE memory owned by the caller unless marked [host].
 *   - Calls validate their arguments on the host, then enqueue kernels on `stream`.
 *     They never synchronize, never allocate, and keep no state between calls.
 *   - Invalid arguments return an error before anything is enqueued.  A failed kernel
 *     launch returns TAPS_ERR_HIP.  Kernels never trap: pathological data (NaN, +-inf,
 *     empty rows) produces the defined outputs documented per call.
 *   - Workspace sizes are pure functions of the host-side sizes.  A workspace may be
 *     reused by consecutive calls on one stream; concurrent calls need their own.
 */
#ifndef TAPS_H
#define TAPS_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TAPS_OK = 0,
  TAPS_ERR_INVALID_ARG = -1,  /* null pointer, size out of range, misaligned buffer */
  TAPS_ERR_UNSUPPORTED = -2,  /* valid request this build does not implement      */
  TAPS_ERR_WORKSPACE = -3,    /* workspace missing or smaller than required        */
  TAPS_ERR_HIP = -4           /* a kernel launch failed (hipGetLastError)          */
} taps_status;

typedef enum { TAPS_BF16 = 0, TAPS_FP32 = 1 } taps_dtype;
typedef enum { TAPS_LOGITS = 0, TAPS_PROBS = 1 } taps_kind;
typedef enum {
  TAPS_SCORER_SIBLING = 0,
  TAPS_SCORER_MARGINAL = 1,
  TAPS_SCORER_LEARNED = 2
} taps_scorer;

/* Limits of this build. */
#define TAPS_MAX_BLOCK 32    /* draft positions D (tree depth)              */
#define TAPS_MAX_K 16        /* candidates per position                     */
#define TAPS_MAX_BUDGET 512  /* N_max, root included                        */

/* [host] Weights of the learned-scorer hook (Sec. 4.2, "Scorer design"): a per-edge MLP
 * whose trained weights are not published, so the caller brings its own.  DEVICE fp32
 * arrays owned by the caller:
 *   emb         [vocab][emb_dim] token embeddings
 *   W1          [hidden][2*emb_dim + 3] first layer over the edge features, in this
 *               order: parent token embedding, child token embedding, child depth,
 *               child log-probability, positional entropy of the child's row
 *   b1, w2      [hidden]; b2 the output bias
 *   root_token  [batch] int32 token at each request's current position (the root's
 *               token, the parent token of depth-1 children); outside [0, vocab): a
 *               zero embedding
 *   emb_dim     1..32;  hidden  1..64 */
typedef struct {
  const float *emb, *W1, *b1, *w2;
  float b2;
  const int32_t *root_token;
  int32_t emb_dim, hidden;
} taps_scorer_mlp;

/* [host] Selection parameters (Sec. 4.1 Stage 1 and 3; Eq. 3; Alg. 1).
 *   batch    requests B >= 0 (0: nothing is enqueued)
 *   block    draft positions D, 1..TAPS_MAX_BLOCK; row i of a request's marginals is the
 *            distribution of the token at tree depth i+1 (the root, depth 0, is the
 *            current position and carries no drafted token)
 *   vocab    V >= K
 *   K        candidates per position, 1..TAPS_MAX_K
 *   budget   N_max, 1..TAPS_MAX_BUDGET; the root counts toward it
 *   dtype    TAPS_BF16 or TAPS_FP32 marginals
 *   kind     TAPS_LOGITS: the edge logit of a child is beta * (its drafter logit);
 *            TAPS_PROBS: the marginals are probabilities, used as the sibling weights
 *            directly (beta must be 1)
 *   lambda1  > 0, finite: per-node cost in Eq. 3
 *   lambda2  >= 0, finite: per-depth cost in Eq. 3 (negative values: UNSUPPORTED)
 *   tau      minimum utility; a node is added only while its utility is > tau (not NaN)
 *   beta     >= 0, finite scorer temperature for LOGITS
 *   scorer   TAPS_SCORER_SIBLING (0; the default of a zeroed struct): q_cond is the
 *            sibling softmax over the K candidates, below.  TAPS_SCORER_MARGINAL: the
 *            scoring ablation of Sec. 5 (the scorer removed, selection by the drafter's
 *            marginal confidence): q_cond is the candidate's full-vocabulary marginal,
 *            below; LOGITS then needs beta = 1.  TAPS_SCORER_LEARNED: the learned
 *            scorer's MLP (mlp) gives each edge a logit, normalised over the parent's
 *            candidate children by a sibling softmax; LOGITS only; block * K * K must
 *            not exceed 7168 (its q_cond table lives in LDS)
 *   mlp      [host] weights, read only with TAPS_SCORER_LEARNED */
typedef struct {
  int32_t batch, block, vocab, K, budget;
  int32_t dtype, kind;
  double lambda1, lambda2, tau, beta;
  int32_t scorer;
  const taps_scorer_mlp *mlp;
} taps_select_params;

/* Selected subtree S per request, breadth first: nodes ordered by depth, then by rank
 * path (the ranks of the tokens from the root down), so a parent always precedes its
 * children.  Arrays are [batch][budget] unless noted; slots n..budget-1 hold
 * parent = token = depth = rank = -1 and q_reach = 0.
 *   parent    index of the parent node within the request; -1 at the root (index 0)
 *   token     vocabulary id; -1 at the root
 *   depth     0 at the root
 *   rank      rank of the token in its position's top-K; -1 at the root
 *   q_reach   Eq. 2 reach probability, fp64; 1.0 at the root
 *   n_nodes   [batch] number of selected nodes n, 1 <= n <= budget
 *   topk_idx  [batch][block][K] top-K vocabulary ids per position: value descending,
 *             then index ascending; -0 equals +0; NaN ranks below -inf
 *   topk_val  [batch][block][K] their marginal values widened to float (exact), or NULL */
typedef struct {
  int32_t *parent;
  int32_t *token;
  int32_t *depth;
  int32_t *rank;
  double *q_reach;
  int32_t *n_nodes;
  int32_t *topk_idx;
  float *topk_val;
} taps_tree;

/* Bytes of scratch taps_select needs (per-chunk top-K candidates; with the marginal scorer
 * on logits also one 64-bit normaliser partial per chunk, with the learned scorer two). */
size_t taps_select_workspace_bytes(const taps_select_params *p);

/* Host-only check of the parameters, no device access (the first step of taps_select). */
taps_status taps_select_validate(const taps_select_params *p);

/* Target-aware selection (Sec. 4.1-4.3, Eq. 1-3, Alg. 1) for `batch` requests.
 *   marginals  [batch][block][vocab] bf16 or fp32, row-major, 16-byte aligned base
 *   out        device arrays described at taps_tree ([host] struct)
 * Edge probability of a rank-r child of any depth-i node (sibling softmax, Eq. 1):
 *   LOGITS  e_r = EXP(beta * (x_r - x_0)), PROBS  e_r = x_r if x_r > 0 else 0;
 *   Z = e_0 + e_1 + ... (in rank order); q_cond = e_r / Z, or 0 when Z is 0 or not finite.
 * Learned scorer: features of an edge into row i (the parent token's embedding, the child
 *   token's, i+1, the child's log-probability (x_v - M) - LOG(Z), the row's entropy
 *   LOG(Z) - S / Z with S = 2^-42 * sum of rint(2^42 * t_j (x_j - M)), t_j = EXP(x_j - M),
 *   terms with t_j = 0 counting 0); a_k = relu(b1[k] + sum_j W1[k][j] f_j) (NaN -> 0),
 *   logit = b2 + sum_k w2[k] a_k, fp64 with sums in index order; q_cond = EXP(l_r - max l)
 *   / (sum over the K siblings in rank order), NaN logits ignored in the max.  LOG is the
 *   shared fp64 logarithm (frexp reduction to [sqrt(1/2), sqrt(2)), 2 atanh series to s^27).
 * Marginal scorer: LOGITS  q_cond = EXP(x_r - M) / Z, M the row maximum, Z = 2^-42 *
 *   sum over the whole row of rint(2^42 * EXP(x_j - M)) (an exact integer sum; NaN
 *   entries count 0), 0 when Z is 0; PROBS  q_cond = min(x_r, 1) if x_r > 0 else 0.
 * EXP is the shared fp64 exponential (Cody-Waite reduction, degree-13 Taylor, no FMA).
 * q_reach multiplies q_cond along the path (Eq. 2); utility = q_reach / (lambda1 +
 * lambda2 * depth) (Eq. 3); all in IEEE fp64.  Ties in the greedy argmax of Alg. 1 go to
 * the shallower node, then to the lexicographically smaller rank path. */
taps_status taps_select(const void *marginals, const taps_select_params *p,
                        const taps_tree *out, void *ws, size_t ws_bytes,
                        hipStream_t stream);

/* taps_select for callers that cannot allocate: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, results and errors as
 * taps_select, without the workspace: the selection's scratch is a static device array of
 * TAPS_SELECT_SCRATCH_BYTES per GPU, which the library holds until the process ends (the
 * first call on a device looks up its address).  The call allocates nothing.
 *   - Parameters whose taps_select_workspace_bytes exceed TAPS_SELECT_SCRATCH_BYTES return
 *     TAPS_ERR_WORKSPACE before anything is enqueued.
 *   - The array is shared by every call on the same GPU and keeps the last call's
 *     contents (no call reads what another left): calls that may overlap in time on one
 *     GPU (other streams, other host threads) race and must be serialized by the caller.
 *   - The device is the one current on the calling thread; `stream` must belong to it. */
#define TAPS_SELECT_SCRATCH_BYTES (8u << 20)
taps_status taps_select_noalloc(const void *marginals, const taps_select_params *p,
                                const taps_tree *out, hipStream_t stream);

/* Bytes of scratch tree_verify_attn needs (split-KV partial outputs). */
size_t tree_verify_attn_workspace_bytes(int32_t batch, int32_t budget, int32_t Hq,
                                        int32_t Hkv, int32_t head_dim, int32_t max_ctx,
                                        int32_t dtype);

/* Host-only check of the attention sizes, no device access. */
taps_status tree_verify_attn_validate(int32_t batch, int32_t budget, int32_t Hq,
                                      int32_t Hkv, int32_t head_dim, int32_t max_ctx,
                                      int32_t dtype, float scale);

/* Tree-masked verification attention for `batch` requests.
 *   Q_tree       [batch][budget][Hq][head_dim] queries of the tree nodes (tree order)
 *   K_cache,
 *   V_cache      [rows][Hkv][head_dim]; request b owns rows kv_offset[b] ..
 *                kv_offset[b] + ctx_len[b] + budget - 1: its context first, then one
 *                reserved row per tree node i at kv_offset[b] + ctx_len[b] + i
 *   kv_offset    [batch] int64 first cache row of each request
 *   ctx_len      [batch] context rows; values outside [0, max_ctx] are clamped to it
 *   tree_parent  [batch][budget] parent index per node (taps_tree.parent); a node whose
 *                parent is not in [0, i) sees only the context and itself
 *   n_nodes      [batch] nodes to compute; clamped to [0, budget]
 *   head_dim     64 or 128; Hq a multiple of Hkv; query head h reads KV head h/(Hq/Hkv)
 *   max_ctx      [host] upper bound of ctx_len, sizes the grid
 *   dtype        TAPS_BF16 (fp32 accumulation, output rounded to nearest even) or TAPS_FP32
 *   scale        softmax scale, finite and > 0 (usually 1/sqrt(head_dim))
 *   O            [batch][budget][Hq][head_dim] same dtype as Q; rows i >= n are not written
 * O[b,i,h] = softmax_j(scale * Q[b,i,h] . K[j,g]) V[j,g] over the context rows and the
 * ancestor-or-self tree rows of node i, g = h / (Hq/Hkv). */
taps_status tree_verify_attn(const void *Q_tree, const void *K_cache, const void *V_cache,
                             const int64_t *kv_offset, const int32_t *ctx_len,
                             const int32_t *tree_parent, const int32_t *n_nodes,
                             int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                             int32_t head_dim, int32_t max_ctx, int32_t dtype, float scale,
                             void *O, void *ws, size_t ws_bytes, hipStream_t stream);

/* tree_verify_attn that also times its main attention kernel: `ev_begin` and `ev_end` are
 * set to the start and the end of that kernel's execution (hipExtLaunchKernel events; the
 * split combine that follows is not included), so hipEventElapsedTime gives the kernel's
 * own duration.  Either event may be NULL; both must have been created.  For profiling
 * callers. */
taps_status tree_verify_attn_timed(const void *Q_tree, const void *K_cache, const void *V_cache,
                                   const int64_t *kv_offset, const int32_t *ctx_len,
                                   const int32_t *tree_parent, const int32_t *n_nodes,
                                   int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                                   int32_t head_dim, int32_t max_ctx, int32_t dtype,
                                   float scale, void *O, void *ws, size_t ws_bytes,
                                   hipStream_t stream, hipEvent_t ev_begin, hipEvent_t ev_end);

/* Bytes of scratch tree_verify_attn_paged needs for these sizes and page size (0 when
 * they are not supported). */
size_t tree_verify_attn_paged_workspace_bytes(int32_t batch, int32_t budget, int32_t Hq,
                                              int32_t Hkv, int32_t head_dim, int32_t max_ctx,
                                              int32_t page_rows);

/* tree_verify_attn over a paged KV cache, for batched serving (the Limitations leave the
 * cache layout to the serving system; pages let requests grow without moving rows).  Same
 * result as tree_verify_attn with request b's logical cache row r (its context rows
 * 0 .. ctx-1, then node i at row ctx + i) stored at
 *   K_pages[block_table[b][r / page_rows]][r % page_rows] (and V_pages alike).
 *   K_pages,
 *   V_pages      [num_pages][page_rows][Hkv][head_dim] bf16 pools, 16-byte aligned
 *   num_pages    pages in each pool (>= 1; num_pages * page_rows below 2^32, else
 *                TAPS_ERR_UNSUPPORTED)
 *   page_rows    rows per page: a power of two from 32 to 4096
 *   block_table  [batch][max_pages] int32 page ids, row b covering request b's rows in
 *                order; max_pages * page_rows must be at least max_ctx + budget.  Entries
 *                the request's rows do not reach are not read for keys; ids outside
 *                [0, num_pages) are clamped into it (never a read outside the pools; the
 *                result is then meaningless)
 *   the other arguments as for tree_verify_attn (no kv_offset); head_dim 128 and TAPS_BF16
 *   only (other sizes and types: TAPS_ERR_UNSUPPORTED)
 *   ws           tree_verify_attn_paged_workspace_bytes(...) bytes, 16-byte aligned */
taps_status tree_verify_attn_paged(const void *Q_tree, const void *K_pages, const void *V_pages,
                                   int32_t num_pages, int32_t page_rows,
                                   const int32_t *block_table, int32_t max_pages,
                                   const int32_t *ctx_len, const int32_t *tree_parent,
                                   const int32_t *n_nodes, int32_t batch, int32_t budget,
                                   int32_t Hq, int32_t Hkv, int32_t head_dim, int32_t max_ctx,
                                   int32_t dtype, float scale, void *O, void *ws,
                                   size_t ws_bytes, hipStream_t stream);

/* tree_verify_attn_paged that also times its main attention kernel, as
 * tree_verify_attn_timed does.  For profiling callers. */
taps_status tree_verify_attn_paged_timed(const void *Q_tree, const void *K_pages,
                                         const void *V_pages, int32_t num_pages,
                                         int32_t page_rows, const int32_t *block_table,
                                         int32_t max_pages, const int32_t *ctx_len,
                                         const int32_t *tree_parent, const int32_t *n_nodes,
                                         int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                                         int32_t head_dim, int32_t max_ctx, int32_t dtype,
                                         float scale, void *O, void *ws, size_t ws_bytes,
                                         hipStream_t stream, hipEvent_t ev_begin,
                                         hipEvent_t ev_end);

/* Greedy acceptance walk (temperature 0).
 *   tree           [host] struct; parent, token and n_nodes are read
 *   target_tokens  [batch][budget] target model's greedy token after each node
 *   path           [batch][block+1] accepted node indices from the root, -1 padded
 *   path_len       [batch] accepted nodes including the root (1 .. block+1)
 *   bonus          [batch] target token after the last accepted node
 * A node is accepted when its token equals the target token after its parent and its
 * parent is accepted; the root always is. */
taps_status accept_walk(const taps_tree *tree, int32_t batch, int32_t budget,
                        int32_t block, const int32_t *target_tokens, int32_t *path,
                        int32_t *path_len, int32_t *bonus, hipStream_t stream);

/* KV commit of the accepted path: the round's state update after accept_walk (Sec. 1:
 * each decoding round commits only one prefix path; the paper leaves the update itself
 * to the serving system).
 *   K_cache,
 *   V_cache      [rows][Hkv][head_dim] in the layout of tree_verify_attn, updated in place:
 *                for request b the rows of the m committed path nodes, kv_offset[b] +
 *                ctx + path[b][j], move to rows kv_offset[b] + ctx + j (j = 0 .. m-1, the
 *                root's row stays); no other row is written.  ctx = ctx_len[b] clamped to
 *                [0, max_ctx].
 *   kv_offset,
 *   ctx_len      as for tree_verify_attn (not written)
 *   tree         [host] struct; token is read ([batch][budget], node tokens)
 *   path,
 *   path_len,
 *   bonus        accept_walk's outputs.  The committed path is the root followed by the
 *                entries path[b][1 .. path_len[b]-1] up to (not including) the first one
 *                that is not larger than the previous entry or not below budget; m is its
 *                length (1 .. block+1)
 *   new_ctx_len  [batch] ctx + m; must not be the ctx_len array (other workgroups of the
 *                same request may still read ctx_len)
 *   committed    [batch][block+1] the tokens the round emits: the drafted tokens of the
 *                m-1 accepted nodes in path order, then the bonus token, then -1
 *   n_committed  [batch] m (tokens emitted)
 *   dtype        TAPS_BF16 or TAPS_FP32 (element size of the cache)
 * K_cache and V_cache must be 16-byte aligned.  Calls that touch the same cache rows must
 * not overlap in time. */
taps_status kv_commit(void *K_cache, void *V_cache, const int64_t *kv_offset,
                      const int32_t *ctx_len, const taps_tree *tree, const int32_t *path,
                      const int32_t *path_len, const int32_t *bonus, int32_t batch,
                      int32_t budget, int32_t block, int32_t Hkv, int32_t head_dim,
                      int32_t max_ctx, int32_t dtype, int32_t *new_ctx_len,
                      int32_t *committed, int32_t *n_committed, hipStream_t stream);

/* kv_commit for a paged KV cache (the layout of tree_verify_attn_paged): the same update
 * in logical rows, request b's logical row r being row r % page_rows of page
 * block_table[b][r / page_rows] of K_pages and V_pages ([num_pages][page_rows][Hkv]
 * [head_dim], 16-byte aligned).  The rows of the m committed path nodes, logical rows
 * ctx + path[b][j], move to logical rows ctx + j; no other row is written.  page_rows is a
 * power of two from 32 to 4096 and max_pages * page_rows >= max_ctx + budget; page ids
 * outside [0, num_pages) are clamped into it.  A request's rows must sit in pages of its
 * own (pages shared with another request of the same call race).  The other arguments and
 * outputs as for kv_commit. */
taps_status kv_commit_paged(void *K_pages, void *V_pages, int32_t num_pages, int32_t page_rows,
                            const int32_t *block_table, int32_t max_pages,
                            const int32_t *ctx_len, const taps_tree *tree, const int32_t *path,
                            const int32_t *path_len, const int32_t *bonus, int32_t batch,
                            int32_t budget, int32_t block, int32_t Hkv, int32_t head_dim,
                            int32_t max_ctx, int32_t dtype, int32_t *new_ctx_len,
                            int32_t *committed, int32_t *n_committed, hipStream_t stream);

/* [host] Weights of one attention layer of the target, a Qwen3-style block.  DEVICE bf16
 * arrays owned by the caller, row-major [out][in], 16-byte aligned:
 *   Wq [Hq*head_dim][hidden], Wk and Wv [Hkv*head_dim][hidden], Wo [hidden][Hq*head_dim]
 *   q_norm, k_norm [head_dim] per-head RMSNorm weights of the queries and keys
 *   rope_theta  rotary base, finite and > 1 (Qwen3: 1e6)
 *   norm_eps    RMSNorm epsilon, finite and >= 0 (Qwen3: 1e-6)
 *   hidden      model width, a multiple of 64, at most 16384 */
typedef struct {
  const void *Wq, *Wk, *Wv, *Wo, *q_norm, *k_norm;
  double rope_theta;
  float norm_eps;
  int32_t hidden;
} taps_layer_weights;

/* Bytes of scratch verify_layer needs (projection partials, Q, O, attention partials);
 * 0 for sizes verify_layer rejects. */
size_t verify_layer_workspace_bytes(int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                                    int32_t head_dim, int32_t hidden, int32_t max_ctx);

/* One attention layer of the target over the selected trees: the layer slice of the
 * verification forward (Sec. 4.1, the verification stage, and Sec. 4.3 run the target once
 * over the tree with tree attention).  bf16 storage, fp32 accumulation.
 *   X          [batch][budget][hidden] bf16 hidden states of the tree nodes (tree order),
 *              16-byte aligned
 *   w          the layer's weights (above)
 *   K_cache,
 *   V_cache    as for tree_verify_attn (bf16); the key and value of node i < n_nodes[b]
 *              are written to row kv_offset[b] + ctx_len[b] + i, no other row is written
 *   kv_offset, ctx_len, max_ctx, scale: as for tree_verify_attn
 *   tree       parent, depth and n_nodes of the selected trees (taps_tree; other fields
 *              are not read)
 *   head_dim   128
 *   Y          [batch][budget][hidden] bf16, 16-byte aligned; rows i >= n_nodes[b] are not
 *              defined
 *   ws         verify_layer_workspace_bytes(...) bytes, 256-byte aligned
 * Steps: q, k, v = X W^T per node; RMSNorm of each query and key head; rotary embedding
 * at position ctx_len[b] + depth (the root right after the context, siblings at one
 * position; pairs (j, j + head_dim/2) turn by pos * rope_theta^(-2j/head_dim)); Q, K and
 * V rounded to bf16; tree attention as tree_verify_attn; O rounded to bf16; Y = O Wo^T
 * rounded to bf16. */
taps_status verify_layer(const void *X, const taps_layer_weights *w, void *K_cache,
                         void *V_cache, const int64_t *kv_offset, const int32_t *ctx_len,
                         const taps_tree *tree, int32_t batch, int32_t budget, int32_t Hq,
                         int32_t Hkv, int32_t head_dim, int32_t max_ctx, float scale, void *Y,
                         void *ws, size_t ws_bytes, hipStream_t stream);

/* Bytes of scratch verify_layer_paged needs (0 when the sizes are not supported). */
size_t verify_layer_paged_workspace_bytes(int32_t batch, int32_t budget, int32_t Hq,
                                          int32_t Hkv, int32_t head_dim, int32_t hidden,
                                          int32_t max_ctx, int32_t page_rows);

/* verify_layer over a paged KV cache, for batched serving (Sec. 4.1 Stage 3 and Sec. 4.3
 * for the layer's tree attention; the Limitations leave cache management to the serving
 * system), in the layout of tree_verify_attn_paged: node i's key and value go to logical
 * row ctx + i of request b, i.e. row (ctx + i) % page_rows of page
 * block_table[b][(ctx + i) / page_rows]; the attention reads the pages.  K_pages, V_pages,
 * num_pages, page_rows, block_table and max_pages as for tree_verify_attn_paged (same
 * validation and errors); the other arguments as for verify_layer (no kv_offset).  Only
 * the nodes' rows of the pools are written. */
taps_status verify_layer_paged(const void *X, const taps_layer_weights *w, void *K_pages,
                               void *V_pages, int32_t num_pages, int32_t page_rows,
                               const int32_t *block_table, int32_t max_pages,
                               const int32_t *ctx_len, const taps_tree *tree, int32_t batch,
                               int32_t budget, int32_t Hq, int32_t Hkv, int32_t head_dim,
                               int32_t max_ctx, float scale, void *Y, void *ws, size_t ws_bytes,
                               hipStream_t stream);

/* Human-readable name of a status code (static string). */
const char *taps_status_string(int32_t status);

/* Host evaluation of the shared fp64 exponential used on the device, for testing the
 * definition against other implementations without a GPU. */
double taps_spec_exp_host(double t);

#ifdef __cplusplus
}
#endif
#endif /* TAPS_H */
