/*
 * treeverify.h -- C ABI of the tree-verification hot path on MI355X (gfx950).
 *
 * Two calls make up one verification step of parallel tree drafting
 * speculative decoding:
 *
 *   tv_tree_verify_attention  every draft-tree node's query attends to its
 *                             sequence's KV cache and to its own ancestors and
 *                             itself in the tree (Sec. 2.2: the tree-causal mask
 *                             M[v,u] = 0 iff u is an ancestor of v or v itself,
 *                             the prefix being visible to all nodes, and the
 *                             masked attention softmax(Q_v K^T / sqrt(d) + M_v) V;
 *                             App. E: the ancestor relation is built inside the
 *                             kernel, no dense per-request mask exists).
 *   tv_tree_accept            the target's greedy prediction (argmax) at every
 *                             node, then the deepest fully accepted root-to-node
 *                             path: a node is accepted when its token equals the
 *                             prediction at its parent and its parent is accepted
 *                             (Sec. 2.4, greedy rule; App. E).
 *
 * Conventions shared by both calls
 *   - Every tensor pointer is caller-owned DEVICE memory, row-major and
 *     contiguous, 16-byte aligned.  The library never allocates or frees.
 *   - Calls are asynchronous on `stream` (0 = the null stream) and never
 *     synchronise the host.  They keep no global mutable state (apart from
 *     tv_tree_accept_noalloc, which shares a static scratch array per GPU);
 *     concurrent calls are safe when they use distinct workspaces.
 *   - The workspace is caller-owned device memory of at least the size the
 *     matching *_workspace() query returns.  It must be zero-filled once
 *     before its first use; the kernels leave it ready for the next call.
 *     Do not modify it between calls.
 *   - Node 0 of every sequence is the root (the token already sampled by the
 *     previous step, App. E); parent[b,0] = -1 and 0 <= parent[b,i] < i for
 *     i >= 1 (children follow their parent, as in Alg. 1).
 *   - Return value: TV_OK or a negative tv_status for errors the host can
 *     detect (null pointers, bad sizes, unsupported shapes, misalignment,
 *     a workspace that is too small, launch failures).  Nothing is launched
 *     when an error is returned.
 *   - Errors found on the device do not stop the host: a sequence whose
 *     parent array breaks the rule above gets NaN in all its attention output
 *     rows, and accept_len[b] = -1 with path[b,:] = -1 from tv_tree_accept
 *     (also when its accepted path would need more than Dmax entries).
 */
#ifndef TREEVERIFY_H
#define TREEVERIFY_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { TV_BF16 = 0, TV_F32 = 1 } tv_dtype;

typedef enum {
  TV_OK = 0,
  TV_ERR_NULL = -1,         /* a required pointer is NULL */
  TV_ERR_SHAPE = -2,        /* a size is < 1 (or < 0 where 0 is allowed) or inconsistent */
  TV_ERR_DTYPE = -3,        /* unknown logits dtype */
  TV_ERR_UNSUPPORTED = -4,  /* D not in {64,128}, N above TV_MAX_NODES, ... */
  TV_ERR_WORKSPACE = -5,    /* workspace NULL or smaller than required */
  TV_ERR_LAUNCH = -6,       /* the HIP runtime rejected a launch */
  TV_ERR_ALIGN = -7,        /* a tensor pointer is not 16-byte aligned */
  TV_ERR_SCRATCH = -8       /* sizes exceed the static scratch of tv_tree_accept_noalloc */
} tv_status;

/* Largest tree (nodes per sequence, root included) either call accepts. */
#define TV_MAX_NODES 2048

/* Human-readable name of a status code (static storage, never NULL). */
const char* tv_status_string(int status);

/* ABI version, bumped on any incompatible change. */
int tv_version(void);

/*
 * Workspace bytes tv_tree_verify_attention needs for these sizes (0 when the
 * sizes are invalid).  Depends only on the arguments, never on kv_len.
 */
size_t tv_tree_verify_attention_workspace(int B, int N, int Hq, int Hkv, int D,
                                          int Lmax);

/*
 * Tree-masked grouped-query attention of all draft-tree nodes (Sec. 2.2).
 *
 *   q       [B, N, Hq, D]     bf16  queries of the tree nodes (post-RoPE)
 *   k_cache [B, Lmax, Hkv, D] bf16  cached prefix keys (post-RoPE)
 *   v_cache [B, Lmax, Hkv, D] bf16  cached prefix values
 *   k_tree  [B, N, Hkv, D]    bf16  keys of the tree nodes
 *   v_tree  [B, N, Hkv, D]    bf16  values of the tree nodes
 *   parent  [B, N]            int32 parent node index, -1 for the root
 *   kv_len  [B]               int32 valid cache length per sequence, in
 *                                   [0, Lmax]; NULL means Lmax for all.
 *                                   Cache rows >= kv_len[b] are never read.
 *   out     [B, N, Hq, D]     bf16  result, round-to-nearest-even
 *
 * Query head h uses KV head h / (Hq / Hkv).  Node i of sequence b sees cache
 * rows [0, kv_len[b]) and tree nodes on its root path, itself included.
 * Scores are scaled by `scale` (<= 0 selects 1/sqrt(D)); the softmax and all
 * accumulation run in fp32, products of bf16 operands on the matrix cores.
 * Requirements: Hq % Hkv == 0, D in {64, 128}, 1 <= N <= TV_MAX_NODES,
 * B >= 1, Lmax >= 0; visible keys and values must be finite.
 *
 * Tree-tail layout (the serving engine wrote the draft nodes' K/V into the
 * cache right after the context, App. E): pass k_tree = v_tree = NULL.  Node
 * i's key and value are then cache row kv_len[b] + i; kv_len is clamped to
 * [0, Lmax - N] (NULL: Lmax - N for all) and Lmax >= N is required
 * (TV_ERR_SHAPE otherwise).  Exactly one of them NULL is TV_ERR_NULL.
 */
int tv_tree_verify_attention(const void* q, const void* k_cache,
                             const void* v_cache, const void* k_tree,
                             const void* v_tree, const int32_t* parent,
                             const int32_t* kv_len, void* out, int B, int N,
                             int Hq, int Hkv, int D, int Lmax, float scale,
                             void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/*
 * The same attention over a paged cache (App. E: the verification kernel
 * reads the serving engine's paged KV cache).  Position t of sequence b is
 * row t % block_size of pool block block_table[b, t / block_size].
 *
 *   k_pool, v_pool [num_blocks, block_size, Hkv, D] bf16
 *   block_table    [B, max_blocks] int32; entries outside [0, num_blocks)
 *                  are clamped into it (no memory outside the pool is read;
 *                  that sequence's result is then meaningless)
 *   kv_len [B] in [0, max_blocks * block_size], NULL = max_blocks * block_size
 *
 * block_size is a power of two >= 32.  Everything else as in
 * tv_tree_verify_attention with Lmax = max_blocks * block_size, including
 * the workspace (tv_tree_verify_attention_workspace(B, N, Hq, Hkv, D,
 * max_blocks * block_size)); results are identical to the padded call on
 * the gathered cache.
 */
int tv_tree_verify_attention_paged(const void* q, const void* k_pool, const void* v_pool,
                                   const int32_t* block_table, int block_size, int max_blocks,
                                   int num_blocks, const void* k_tree, const void* v_tree,
                                   const int32_t* parent, const int32_t* kv_len, void* out,
                                   int B, int N, int Hq, int Hkv, int D, float scale,
                                   void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * Attention under the draft head's training mask (App. "Training Details"):
 * each of the A sampled anchors of a training example starts a block of S
 * positions (the anchor, then mask tokens).  Position j of block k attends to
 * the context rows t < anchors[b, k] (the verified prefix) and to positions
 * 0 .. j of its own block; never to later positions or to other blocks.
 *
 *   q            [B, A, S, Hq, D]  bf16  block queries (post-RoPE)
 *   k_ctx, v_ctx [B, L, Hkv, D]    bf16  context K/V of the example
 *   k_blk, v_blk [B, A, S, Hkv, D] bf16  K/V of the block positions
 *   anchors      [B, A]            int32 anchor positions, clamped to [0, L]
 *   out          [B, A, S, Hq, D]  bf16
 *
 * Scale, precision, GQA mapping and requirements as in
 * tv_tree_verify_attention with B*A sequences of S nodes (S <= TV_MAX_NODES,
 * B*A <= 2^24); it runs on the same kernels, each block as a chain tree whose
 * cache is its example's context cut at its anchor.  The workspace is
 * tv_block_causal_attention_workspace(B, A, S, Hq, Hkv, D, L) bytes,
 * zero-filled before first use like the verification workspace.  Forward
 * only.
 */
size_t tv_block_causal_attention_workspace(int B, int A, int S, int Hq, int Hkv, int D,
                                          int L);
int tv_block_causal_attention(const void* q, const void* k_ctx, const void* v_ctx,
                              const void* k_blk, const void* v_blk, const int32_t* anchors,
                              void* out, int B, int A, int S, int Hq, int Hkv, int D, int L,
                              float scale, void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

/*
 * Commit the accepted path (App. E): the keys and values of nodes
 * path[b, 0 .. accept_len[b]-1] (root first) of k_tree/v_tree are copied to
 * cache positions kv_len[b] .. kv_len[b] + accept_len[b] - 1 and kv_len[b]
 * grows by accept_len[b].  A sequence whose accept_len is < 1 or > Dmax,
 * whose path names a node outside [0, N), or whose commit would pass Lmax,
 * is left unchanged (cache and kv_len).  The tree buffers must not overlap
 * the cache.
 *
 * Tree-tail layout (k_tree = v_tree = NULL, as in tv_tree_verify_attention):
 * node i's K/V are cache row kv_len[b] + i, and the commit moves row
 * kv_len[b] + path[b, j] to row kv_len[b] + j in place (path must be a
 * root-to-node path as tv_tree_accept writes it: path[j] >= j).  A sequence
 * with kv_len[b] + N > Lmax is left unchanged.
 *
 *   k_tree, v_tree  [B, N, Hkv, D] bf16
 *   path [B, Dmax], accept_len [B]   as written by tv_tree_accept
 *   k_cache, v_cache [B, Lmax, Hkv, D] bf16, updated in place
 *   kv_len [B] int32, updated in place
 */
int tv_commit_path(const void* k_tree, const void* v_tree, const int32_t* path,
                   const int32_t* accept_len, void* k_cache, void* v_cache, int32_t* kv_len,
                   int B, int N, int Hkv, int D, int Lmax, int Dmax, hipStream_t stream);

/* tv_commit_path into a paged cache (layout as in
 * tv_tree_verify_attention_paged); the capacity is max_blocks * block_size. */
int tv_commit_path_paged(const void* k_tree, const void* v_tree, const int32_t* path,
                         const int32_t* accept_len, void* k_pool, void* v_pool,
                         const int32_t* block_table, int block_size, int max_blocks,
                         int num_blocks, int32_t* kv_len, int B, int N, int Hkv, int D, int Dmax,
                         hipStream_t stream);

/* Workspace bytes tv_tree_accept needs for these sizes (0 when invalid). */
size_t tv_tree_accept_workspace(int B, int N, int V);

/*
 * Greedy tree acceptance (Sec. 2.4; App. E).
 *
 *   logits     [B, N, V] bf16 or fp32  target logits at every tree node
 *   draft_tok  [B, N]    int32  drafted token of every node (node 0 ignored)
 *   parent     [B, N]    int32  as above
 *   accept_len [B]       int32  out: entries of the accepted path, root
 *                               included (>= 1), or -1 on a device error
 *   path       [B, Dmax] int32  out: node indices root first, -1 padded
 *   tgt_argmax [B, N]    int32  out (optional, may be NULL): first index of
 *                               the maximum logit of every node; the
 *                               correction token of sequence b is
 *                               tgt_argmax[b, path[b, accept_len[b]-1]]
 *
 * Ties in the argmax go to the lowest vocabulary index, values compared as
 * numbers (-0.0 == +0.0); logits must not be NaN.  Among equally deep
 * accepted nodes the lowest node index ends the path.
 * Requirements: 1 <= N <= TV_MAX_NODES, V >= 1, B >= 1, Dmax >= 1.
 */
int tv_tree_accept(const void* logits, int logits_dtype,
                   const int32_t* draft_tok, const int32_t* parent, int B,
                   int N, int V, int Dmax, int32_t* accept_len, int32_t* path,
                   int32_t* tgt_argmax, void* workspace,
                   size_t workspace_bytes, hipStream_t stream);

/*
 * tv_tree_accept without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, serving loops that must not
 * call hipMalloc, harnesses that forbid it.  Same arguments (minus the
 * workspace), results and device-side error behaviour as tv_tree_accept;
 * the same kernels run.
 *
 * The split keys go to a static device array of TV_ACCEPT_SCRATCH_BYTES
 * inside the library.  Every GPU the library runs on holds its own copy
 * from the library's load until the process ends; the call itself never
 * allocates or frees.  The copy used is that of the device `stream` belongs
 * to (the current device for the null stream); its address is looked up on
 * the first call on each device.  Nothing in it needs to start at zero: each
 * call writes every key before reading it.
 *
 * Sizes whose keys do not fit (tv_tree_accept_workspace(B, N, V) >
 * TV_ACCEPT_SCRATCH_BYTES: more than about 1M node rows B*N) return
 * TV_ERR_SCRATCH and launch nothing.  All calls on one GPU share its array:
 * calls that may overlap on that GPU (different streams without ordering
 * between them) race and give wrong results; order them, or use
 * tv_tree_accept with a workspace per stream.
 */
#define TV_ACCEPT_SCRATCH_BYTES (8u << 20)
int tv_tree_accept_noalloc(const void* logits, int logits_dtype,
                           const int32_t* draft_tok, const int32_t* parent, int B,
                           int N, int V, int Dmax, int32_t* accept_len, int32_t* path,
                           int32_t* tgt_argmax, hipStream_t stream);

/* ---- Budgeted tree drafting (the step before verification) ------------ */

/* Largest branching width W and draft depth the drafting calls accept. */
#define TV_MAX_WIDTH 16
#define TV_MAX_DRAFT_DEPTH 64

/* Workspace bytes tv_draft_topw needs for these sizes (0 when invalid). */
size_t tv_draft_topw_workspace(int B, int Nd, int V);

/*
 * Candidate children per draft depth (Sec. 2.4, parallel tree drafting: one
 * draft-head pass gives logits for every draft depth, of which the top-W
 * tokens and their log-probabilities are extracted; App. E uses k = W).
 *
 *   logits [B, Nd, V] bf16 or fp32  draft logits, row (b, d) for depth d+1
 *   tok    [B, Nd, W] int32  out: the W largest logits of each row, in
 *                            decreasing order, equal values by lower index
 *   logp   [B, Nd, W] fp32   out: their log-probabilities, logit minus the
 *                            row's log-sum-exp (computed in fp32)
 *
 * Requirements: 1 <= W <= min(V, TV_MAX_WIDTH), 1 <= Nd <= TV_MAX_DRAFT_DEPTH,
 * B >= 1; logits finite.
 */
int tv_draft_topw(const void* logits, int logits_dtype, int B, int Nd, int V, int W,
                  int32_t* tok, float* logp, void* workspace, size_t workspace_bytes,
                  hipStream_t stream);

/*
 * Best-first tree construction under a node budget (Alg. 1 with the
 * accumulated draft log-probability score of Sec. 2.4).
 *
 * Node 0 is the root (depth 0, score 0, token root_tok[b], or -1 when
 * root_tok is NULL).  Repeatedly the open node of highest score (equal
 * scores: lower node index) is taken; unless it is at depth Nd it gets up
 * to W children, child k of a depth-d node carrying tok[b, d, k] and score
 * fp32(score + logp[b, d, k]), numbered in creation order, until the tree
 * holds `budget` nodes or no open node is left.
 *
 *   tok, logp [B, Nd, W]   candidates as produced by tv_draft_topw
 *   root_tok  [B] int32    or NULL
 *   parent    [B, budget] int32  out: parent index, -1 for the root
 *   token     [B, budget] int32  out
 *   depth     [B, budget] int32  out
 *   score     [B, budget] fp32   out, or NULL
 *   n_nodes   [B] int32          out: nodes built (<= budget)
 * Slots at or beyond n_nodes[b] hold parent = token = depth = -1 and score
 * -inf.  The parent/token arrays of a sequence with n_nodes[b] = budget are
 * directly the parent and draft_tok inputs of the verification calls.
 * Requirements: 1 <= budget <= TV_MAX_NODES, 1 <= W <= TV_MAX_WIDTH,
 * 1 <= Nd <= TV_MAX_DRAFT_DEPTH, B >= 1; logp finite.  No workspace.
 */
int tv_build_tree(const int32_t* tok, const float* logp, const int32_t* root_tok, int B,
                  int Nd, int W, int budget, int32_t* parent, int32_t* token, int32_t* depth,
                  float* score, int32_t* n_nodes, hipStream_t stream);

/*
 * Non-greedy (temperature) tree acceptance (Sec. 2.4: the speculative
 * sampling rule applied along the tree's branches, with a correction token
 * drawn from the target when the drafts are rejected), in the form that
 * keeps verification lossless (Sec. 2.2) for trees whose children are
 * deterministic drafts (top-W per depth, as tv_build_tree makes them).
 *
 * With p_v = softmax(logits[b, v] / T) the target's next-token
 * distribution at node v, a walk starts at the root.  At the current node v
 * the children c of v are tested in increasing index order: c (token y)
 * passes when u_accept[b, c] * (1 - S) < e, where e = p_v(y) if y is in
 * [0, V) and no earlier child of v has token y, else e = 0, and S is the
 * sum of p_v over the distinct tokens of v's earlier children.  (Each child
 * is a point-mass proposal; the test is u < min(1, p'(y)) for the target
 * residual p' left by the rejected ones.)  The first child that passes
 * becomes the current node.  The walk ends at a node none of whose children
 * passes: path and accept_len describe the walk as in tv_tree_accept.
 * correction[b] is drawn at the last node v from p_v with the tokens of v's
 * children removed (from p_v when that leaves no mass): the token x
 * maximising w(x) / -ln U(b, x), ties to the lower index, where U(b, x)
 * takes word x % 4 of Philox4x32-10 (Salmon et al., SC 2011) with counter
 * (x / 4, b, 0, 0) and key (seed & 0xFFFFFFFF, seed >> 32), mapped to (0, 1)
 * as ((word >> 9) + 0.5) / 2^23.  With uniforms drawn independently on
 * [0, 1), the first emitted token (accepted draft or correction) follows p
 * at the root, and the walk ends at v with probability (product of p along
 * v's root path) x (1 - sum of p_v over v's distinct child tokens).
 *
 *   logits     [B, N, V]  bf16 or fp32 (logits_dtype)  target logits
 *   draft_tok, parent [B, N] int32, as in tv_tree_accept
 *   u_accept   [B, N] fp32 uniforms in [0, 1) (entry 0 of a row unused)
 *   accept_len [B], path [B, Dmax], correction [B] int32 outputs; an invalid
 *     tree or a path longer than Dmax gives -1, a -1 path and correction -1.
 *
 * Requirements: temperature > 0 and finite; 1 <= N <= TV_MAX_NODES,
 * 1 <= V <= 2^23 (TV_ERR_UNSUPPORTED above), Dmax >= 1, B*N <= 2^24; logits
 * finite.  Workspace: tv_tree_accept_sampled_workspace(B, N, V) bytes,
 * 16-byte aligned (needs no zero fill).  The decisions are taken in fp32:
 * a test within about 1e-6 (relative) of its threshold may go either way.
 */
size_t tv_tree_accept_sampled_workspace(int B, int N, int V);
int tv_tree_accept_sampled(const void* logits, int logits_dtype, const int32_t* draft_tok,
                           const int32_t* parent, const float* u_accept,
                           unsigned long long seed, float temperature, int B, int N, int V,
                           int Dmax, int32_t* accept_len, int32_t* path, int32_t* correction,
                           void* workspace, size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* TREEVERIFY_H */
