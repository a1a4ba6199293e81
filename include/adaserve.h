/*
 * adaserve.h -- C ABI of the MI355X (gfx950) batched tree-verification library.
 *
 * One verification pass of SLO-customised speculative decoding (section 4.3,
 * step 4): the target model scores every node of every request's draft token
 * tree in one pass, and the tokens to commit are read off the logits of those
 * nodes (section 5.1).  The library provides the steps of that pass that run
 * after the projections:
 *
 *   adaserve_tree_attn_verify  paged tree attention: each node attends to its
 *                              request's cached prefix plus its own
 *                              root-to-node path (section 2, draft token tree;
 *                              section 3, Theorem 1's root-to-v paths);
 *   adaserve_node_argmax       the target's greedy choice at every node;
 *   adaserve_tree_accept       the longest accepted root path per request and
 *                              the tokens it commits;
 *   adaserve_tree_verify_step  the three above as one call (two launches);
 *   adaserve_tree_accept_sampled  the same for sampled decoding (speculative
 *                              sampling over the tree);
 *   adaserve_commit_accepted_kv  the accepted path's keys and values written
 *                              into the request's paged cache;
 *   adaserve_select_trees      (before the pass) the two selection phases that
 *                              turn candidate trees into the draft trees;
 *   adaserve_beam_step         (before selection) one beam-search step of the
 *                              speculation phase that grows the candidate trees.
 *
 * Conventions for every entry point:
 *  - Pointers without a _host suffix are DEVICE pointers owned by the caller;
 *    _host pointers are host memory read synchronously during the call and
 *    not retained.  Nothing is allocated or freed, and nothing synchronises:
 *    work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *    the call returns.
 *  - Every scalar, pointer and host-mirror value is validated on the host
 *    before anything is enqueued; on a non-OK status nothing was enqueued and
 *    adaserve_last_error() describes the problem.
 *  - Device-only contents (parent arrays, block tables, draft tokens) are
 *    checked in the kernels: malformed trees give accept_len = -1 in
 *    adaserve_tree_accept and unspecified (but in-bounds) attention output.
 *  - The library is stateless apart from a per-device architecture check and
 *    the thread-local error string; calls on different streams may overlap.
 *  - Only gfx950 devices are supported (ADASERVE_ERR_UNSUPPORTED otherwise).
 *
 * Tree encoding (all entry points): request r owns the global node rows
 * [node_indptr[r], node_indptr[r+1]); local node 0 is the root (the last
 * committed token); parent[] holds LOCAL parent ids with parent[root] = -1 and
 * 0 <= parent[i] < i for every other node (a parent is drafted before its
 * children, Appendix B).  1 <= N_r <= 128 nodes per request.
 */
#ifndef ADASERVE_H
#define ADASERVE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every entry point. */
#define ADASERVE_OK                   0
#define ADASERVE_ERR_INVALID_ARGUMENT 1  /* bad pointer, size, layout or host-mirror value   */
#define ADASERVE_ERR_UNSUPPORTED      2  /* valid but not built: head_dim, page size, device  */
#define ADASERVE_ERR_WORKSPACE        3  /* workspace missing or smaller than required        */
#define ADASERVE_ERR_DEVICE           4  /* a HIP runtime call or kernel launch failed        */

/* Element types of the floating-point tensors. */
#define ADASERVE_F32  0
#define ADASERVE_BF16 1

/* Maximum tree nodes per request. */
#define ADASERVE_MAX_TREE_NODES 128

/*
 * Bytes of device workspace adaserve_tree_attn_verify needs for this batch
 * (split-KV partial results).  Depends only on the arguments given here, so a
 * caller can size the workspace once per batch shape.  Returns 0 when no
 * workspace is needed and SIZE_MAX when the arguments are invalid (the
 * reason is in adaserve_last_error()).
 */
size_t adaserve_tree_attn_workspace_bytes(int32_t num_requests, const int32_t *node_indptr_host,
                                          const int32_t *prefix_len_host, int32_t num_q_heads,
                                          int32_t num_kv_heads, int32_t head_dim,
                                          int32_t page_size, int32_t dtype);

/*
 * Paged tree attention (section 4.3 step 4; section 2 draft token tree).
 *
 * For node i of request r and q-head h, with kv-head g = h / (Hq / Hkv)
 * (contiguous head groups), the output is softmax-weighted attention of
 * q[i, h] over, in this order,
 *   - the request's cached prefix: positions t = 0 .. L_r - 1, held in page
 *     block_table[r * block_table_stride + t / page_size], slot t % page_size;
 *   - the tree nodes on i's root-to-node path (root .. i, i included), whose
 *     keys and values are k_tree / v_tree rows of those nodes;
 * with scores sm_scale * <q, k>.  No other tree node is visible to i.  The
 * kernel applies no positional encoding: q and k_tree arrive post-RoPE.
 *
 * Layouts (row-major, dense):
 *   q, out            [T, Hq, D]              dtype
 *   k_tree, v_tree    [T, Hkv, D]             dtype
 *   k_pages, v_pages  [num_pages, Hkv, page_size, D]   dtype
 *   block_table       [num_requests, block_table_stride] int32 physical page ids
 *   prefix_len        [num_requests] int32 (device), prefix_len_host its host copy
 *   node_indptr       [num_requests + 1] int32 (device), node_indptr_host its copy
 * Supported: dtype F32 or BF16; head_dim 64 or 128; page_size 16; any
 * Hq % Hkv == 0 with Hq / Hkv <= 16; L_r >= 0 (L_r = 0: attention over the
 * root path only); sm_scale finite, and > 0 for BF16
 * (ADASERVE_ERR_UNSUPPORTED otherwise; F32 takes any finite scale).
 * BF16 computes Q.K^T and P.V on bf16 matrix cores with
 * fp32 accumulation and rounds the output to bf16 (nearest even); when a
 * prefix is split into chunks, each chunk's own normalised output is kept in
 * bf16 and the chunks are merged with fp32 weights.  F32 computes in fp32
 * throughout.
 * Slots past L_r in the last page and pages not listed for r are never read
 * into the result (they may hold NaN).  Block-table entries outside
 * [0, num_pages) are treated as all-zero pages.  The device arrays must equal
 * their host mirrors.  workspace must hold at least
 * adaserve_tree_attn_workspace_bytes(...) bytes (256-byte aligned; contents
 * need no initialisation); calls that share a workspace must not overlap in
 * time.  When some prefix is split, a second kernel (the split-KV merge) is
 * enqueued after the attention kernel on the same stream.
 */
int32_t adaserve_tree_attn_verify(int32_t num_requests, const int32_t *node_indptr,
                                  const int32_t *node_indptr_host, const int32_t *parent,
                                  const void *q, const void *k_tree, const void *v_tree,
                                  const void *k_pages, const void *v_pages, int32_t num_pages,
                                  const int32_t *block_table, int32_t block_table_stride,
                                  const int32_t *prefix_len, const int32_t *prefix_len_host,
                                  int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                  int32_t page_size, float sm_scale, int32_t dtype, void *out,
                                  void *workspace, size_t workspace_bytes, void *stream);

/* Bytes of the static split-KV scratch of adaserve_tree_attn_verify_noalloc. */
#define ADASERVE_TREE_ATTN_SCRATCH_BYTES (32u << 20)

/*
 * adaserve_tree_attn_verify without a workspace argument, for callers that
 * cannot allocate device memory: code under HIP graph capture, serving loops
 * that must not allocate, harnesses that forbid hipMalloc.  It calls no
 * allocator of any kind.
 *
 * Arguments, layouts, results and errors are those of
 * adaserve_tree_attn_verify (same plan, same kernels, bit-identical output);
 * the split-KV partial results go to a static array of
 * ADASERVE_TREE_ATTN_SCRATCH_BYTES bytes that the library holds on every
 * device it runs on until the process ends.  A batch whose plan needs more
 * than that (adaserve_tree_attn_workspace_bytes(...) > the limit) is
 * rejected with ADASERVE_ERR_WORKSPACE before anything is enqueued.  Every
 * call on one device shares that device's array: calls that overlap in time
 * on one device (other streams, other threads) race and give undefined
 * results; calls on one stream are ordered and safe.  The array's contents
 * need no initialisation.
 */
int32_t adaserve_tree_attn_verify_noalloc(int32_t num_requests, const int32_t *node_indptr,
                                          const int32_t *node_indptr_host, const int32_t *parent,
                                          const void *q, const void *k_tree, const void *v_tree,
                                          const void *k_pages, const void *v_pages, int32_t num_pages,
                                          const int32_t *block_table, int32_t block_table_stride,
                                          const int32_t *prefix_len, const int32_t *prefix_len_host,
                                          int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                          int32_t page_size, float sm_scale, int32_t dtype, void *out,
                                          void *stream);

/*
 * Per-node vocabulary argmax of the verification logits (section 5.1: the
 * logits of every node come back from verification and the verified tokens
 * are identified from them; greedy reading: the target's choice is its
 * highest-scoring token).
 *
 * logits: [num_rows, row_stride] of dtype, row i = logits + i * row_stride
 * elements, columns 0 .. vocab - 1 compared (the rest of a row is never read).
 * argmax_out: [num_rows] int32, the LOWEST index holding the row's maximum
 * (values compare after exact widening to fp32; +0 == -0).  NaN inputs give
 * an unspecified index in [0, vocab).  Requires vocab >= 1 when num_rows > 0,
 * row_stride >= vocab.  num_rows = 0 is a no-op.
 */
int32_t adaserve_node_argmax(const void *logits, int64_t row_stride, int32_t num_rows,
                             int32_t vocab, int32_t dtype, int32_t *argmax_out, void *stream);

/*
 * Longest-accepted-path acceptance (greedy tree verification, section 4.3
 * step 4, read with section 2's tree and Algorithm 2's count of the root as
 * one accepted token).
 *
 * Node j > 0 matches when draft_tokens[j] == target_argmax[parent(j)]; j is
 * accepted when every non-root node on its root-to-node path matches; the
 * root is always accepted and its draft token is never compared.  With d* the
 * largest depth of an accepted node (root depth 0) and i* the smallest local
 * id among accepted nodes of that depth:
 *   accept_len[r]              = d* + 1
 *   accept_nodes[r][k]         = local id of the depth-k node on the root..i*
 *                                path, k = 0..d*
 *   accept_tokens[r][k]        = draft token of accept_nodes[r][k + 1], k < d*
 *   accept_tokens[r][d*]       = target_argmax[i*]  (the target's next token)
 *   slots k > d*               = -1
 * Outputs are [num_requests, max_accept] int32 rows (row stride max_accept).
 * A request whose tree is malformed (N_r outside 1..128, indptr outside
 * [0, total_nodes], parent[root] != -1, a parent not earlier than its child)
 * or deeper than max_accept - 1 gets accept_len = -1 and -1 in every slot.
 * draft_tokens, target_argmax: [total_nodes] int32 (device).
 */
int32_t adaserve_tree_accept(int32_t num_requests, int32_t total_nodes,
                             const int32_t *node_indptr, const int32_t *parent,
                             const int32_t *draft_tokens, const int32_t *target_argmax,
                             int32_t max_accept, int32_t *accept_len, int32_t *accept_tokens,
                             int32_t *accept_nodes, void *stream);

/*
 * The whole verification pass in one call (section 4.3 step 4: every tree
 * of the batch scored in one pass, then the tokens to commit read off the
 * node logits, section 5.1): tree attention as adaserve_tree_attn_verify,
 * the per-node argmax as adaserve_node_argmax over the logits' T rows, and
 * the acceptance as adaserve_tree_accept on that argmax.  Every output is
 * bit-identical to those three calls in that order on the same stream.
 *
 * The attention arguments, workspace (size:
 * adaserve_tree_attn_workspace_bytes) and limits are those of
 * adaserve_tree_attn_verify; logits [T, logits_row_stride] have the
 * attention's dtype (columns 0 .. vocab - 1 compared); draft_tokens [T],
 * target_argmax [T], accept_len [num_requests], accept_tokens and
 * accept_nodes [num_requests, max_accept] are as in adaserve_node_argmax
 * and adaserve_tree_accept (all device memory).  Errors: the union of those
 * calls' checks, all made before anything is enqueued.
 *
 * BF16 runs in two launches: the attention workgroups followed, in the same
 * grid, by one argmax workgroup per node (they take the CUs no attention
 * work unit holds and the attention's tail, so the logits stream beside the
 * attention instead of after it); then the split-KV merge (when a prefix is
 * split) together with one acceptance wave per request.  F32 enqueues the
 * three calls' kernels one after another.  Calls that share a workspace
 * must not overlap in time.
 */
int32_t adaserve_tree_verify_step(int32_t num_requests, const int32_t *node_indptr,
                                  const int32_t *node_indptr_host, const int32_t *parent,
                                  const void *q, const void *k_tree, const void *v_tree,
                                  const void *k_pages, const void *v_pages, int32_t num_pages,
                                  const int32_t *block_table, int32_t block_table_stride,
                                  const int32_t *prefix_len, const int32_t *prefix_len_host,
                                  int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                  int32_t page_size, float sm_scale, int32_t dtype,
                                  const void *logits, int64_t logits_row_stride, int32_t vocab,
                                  const int32_t *draft_tokens, int32_t max_accept, void *out,
                                  int32_t *target_argmax, int32_t *accept_len,
                                  int32_t *accept_tokens, int32_t *accept_nodes, void *workspace,
                                  size_t workspace_bytes, void *stream);

/*
 * Accepted-path KV commit: the keys and values of the accepted path enter
 * the request's paged cache, so the next iteration's prefix holds them
 * (section 5.1: once verified, a request's tokens return with it to the pool
 * of requests that the next iteration draws from; section 2: the root is the
 * last generated token, whose K/V, like every tree node's, was computed in
 * the verification pass).
 *
 * For request r with len = accept_len[r] >= 1 and L = prefix_len[r], row
 * k = 0 .. len-1 copies the tree row of local node accept_nodes[r][k]
 * (k_tree/v_tree row node_indptr[r] + node, every kv-head) to cache position
 * L + k: page block_table[r][(L + k) / page_size], slot (L + k) % page_size.
 * Rows are committed in order up to the first row that cannot be: node
 * outside [0, N_r), position past the block-table row, or a page id outside
 * [0, num_pages); nothing at or after that row is written.
 * new_prefix_len[r] = L + (rows committed).  A request with accept_len < 1
 * (e.g. -1 from adaserve_tree_accept), accept_len > max_accept or
 * accept_len > ADASERVE_MAX_TREE_NODES commits nothing and keeps L.  new_prefix_len may be the prefix_len array itself.
 * No other byte of k_pages / v_pages is written.
 *
 * Layouts as in adaserve_tree_attn_verify: k_tree, v_tree [total_nodes, Hkv,
 * D]; k_pages, v_pages [num_pages, Hkv, page_size, D]; accept_nodes
 * [num_requests, max_accept] int32 (device).  dtype F32 or BF16; head_dim * element
 * size a multiple of 16 bytes; page_size >= 1.  All arrays are device
 * memory; the copy is bit-exact.
 */
int32_t adaserve_commit_accepted_kv(int32_t num_requests, const int32_t *node_indptr,
                                    const int32_t *accept_len, const int32_t *accept_nodes,
                                    int32_t max_accept, const void *k_tree, const void *v_tree,
                                    void *k_pages, void *v_pages, int32_t num_pages,
                                    const int32_t *block_table, int32_t block_table_stride,
                                    const int32_t *prefix_len, int32_t num_kv_heads,
                                    int32_t head_dim, int32_t page_size, int32_t dtype,
                                    int32_t *new_prefix_len, void *stream);

/*
 * Draft-tree selection: the SLO-customised and throughput-optimised selection
 * phases of Algorithm 2 (section 4.3 steps 2 and 3), run on the candidate
 * token trees the speculation phase built; the result is the draft token
 * trees the verification pass scores.
 *
 * Request r owns candidates [cand_indptr[r], cand_indptr[r+1]) (root not
 * included); cand_parent holds LOCAL parents, -1 for a child of the root;
 * cand_prob is each candidate's path probability f(v).  Every well-formed
 * request starts with its root (one budget unit).  Requests are visited in
 * descending order of need (NaN: last; ties by index); each adds its best
 * remaining candidate while the float32 sum of its added path probabilities
 * (from 0, in the order added) is below need[r], its tree has fewer than
 * n_max nodes (root included) and budget remains (section 4.3 step 2; need[r]
 * is A_cap(r) minus the root's 1).  Then the best remaining candidates of
 * the whole batch are added while budget remains (step 3).  "Best" is the
 * highest path probability, ties to the smaller depth (so a parent always
 * precedes its child and every tree stays connected), then the smaller
 * request, then the smaller local index.  The budget loops run while
 * budget > 0 (the printed "B >= 0" would select one node past the budget).
 *
 * Outputs: tree_size[r] = nodes selected (root included); row r of
 * tree_parent / tree_cand ([num_requests, max_nodes] int32) lists the root
 * first (-1, -1), then the selected candidates by (depth, local index) with
 * their tree-local parent and their local candidate index; -1 past
 * tree_size.  These rows are a valid tree for adaserve_tree_attn_verify.
 * A request with more than 127 candidates, a parent that is not -1 or an
 * earlier candidate, or a path probability outside (0, 1] or above its
 * parent's (the root's is 1) takes no part: no budget, tree_size -1, rows of
 * -1.  If cand_indptr does not start at 0, decreases, or does not end at
 * num_candidates, every request gets -1.
 * Limits: num_requests <= 512, num_candidates <= 8192, max_nodes >= 128.
 * All arrays are device memory.
 */
int32_t adaserve_select_trees(int32_t num_requests, int32_t num_candidates,
                              const int32_t *cand_indptr, const int32_t *cand_parent,
                              const float *cand_prob, const float *need, int32_t budget,
                              int32_t n_max, int32_t max_nodes, int32_t *tree_size,
                              int32_t *tree_parent, int32_t *tree_cand, void *stream);

/*
 * One beam-search speculation step (section 4.3 step 1): every beam node of
 * a request expands into all vocabulary tokens, a child's path probability
 * being the beam's path probability times the draft model's softmax
 * probability of the token (section 4.2's product of draft probabilities
 * along the path), and each request keeps the beam_out children with the
 * highest path probability.  The first step has one beam per request (the
 * root, log path probability 0); later steps have beam_in = the previous
 * step's beam_out.
 *
 * Row b of request r is logits row r * beam_in + b: the draft model's logits
 * after beam node b, columns 0 .. vocab - 1 (row_stride elements apart; the
 * rest of a row is never read).  beam_logprob [num_requests * beam_in]
 * holds each beam's natural-log path probability; -inf marks an unused beam
 * slot, whose logits row is not read.  A child's score is
 *   beam_logprob[b] + x[b, t] - log(sum over t' of exp(x[b, t'])),
 * computed in fp32 (the log-sum-exp over the row accumulated in fp32).
 * Children are ranked by score (higher first), ties to the smaller beam, then
 * the smaller token (children of one beam whose fp32 scores coincide only
 * through rounding keep the order of their logits); the beam_out best
 * children with a finite score are written best first to row r of
 *   out_parent  [num_requests, beam_out] int32  beam index in [0, beam_in)
 *   out_token   [num_requests, beam_out] int32  token id in [0, vocab)
 *   out_logprob [num_requests, beam_out] fp32   the child's score
 * and slots past them hold -1, -1, -inf.  Logits are finite or -inf (a -inf
 * logit is a token of probability 0, never kept); NaN or +inf logits give
 * unspecified (in-range) outputs.
 *
 * dtype F32 or BF16 logits; logits 16-byte aligned and row_stride * element
 * size a multiple of 16 bytes; 1 <= beam_in, beam_out <= 64; vocab <= 2^20
 * (ADASERVE_ERR_UNSUPPORTED above).  workspace: at
 * least adaserve_beam_step_workspace_bytes(...) bytes of device memory,
 * 256-byte aligned, no initialisation needed; calls sharing a workspace must
 * not overlap in time.  Two kernels are enqueued on `stream` (a scan of
 * every live logits row, then a per-request merge).  num_requests = 0 is a
 * no-op.
 */
size_t adaserve_beam_step_workspace_bytes(int32_t num_requests, int32_t beam_in, int32_t vocab,
                                          int32_t beam_out, int32_t dtype);

int32_t adaserve_beam_step(int32_t num_requests, int32_t beam_in, const void *logits,
                           int64_t row_stride, int32_t vocab, int32_t dtype,
                           const float *beam_logprob, int32_t beam_out, int32_t *out_parent,
                           int32_t *out_token, float *out_logprob, void *workspace,
                           size_t workspace_bytes, void *stream);

/*
 * Tree verification for sampled decoding: multi-step speculative sampling
 * over each request's draft token tree (the tree-based verification of prior
 * work that section 4.3 step 4 delegates to; lossless -- the emitted tokens
 * follow the target distribution -- when each node's children were drawn
 * independently from the draft distribution at that node).  The greedy
 * counterpart is adaserve_tree_accept.
 *
 * Row u of target_logits / draft_logits ([total_nodes, row_stride], dtype)
 * holds the target / draft model's logits after node u's root path, already
 * divided by the sampling temperature; p_u / q_u are their softmax over
 * columns 0 .. vocab - 1.  Draft rows of leaves are not read (q at a leaf
 * enters no test and no residual).  From the
 * root, the children of the current node u are tried in index order: child
 * c with token t = draft_tokens[c] is accepted when
 *   u_accept[c] * q_u(t) < p_res(t)
 * (probability min(1, p_res(t) / q_u(t)) for u_accept uniform in [0, 1)),
 * where p_res starts as p_u at every node; a rejection replaces p_res by
 * max(0, p_res - q_u), renormalised.  The accepted child becomes the current
 * node and its token is emitted; when no child is accepted (or u is a leaf)
 * the bonus token -- the smallest v whose cumulative p_res, in token order,
 * exceeds u_bonus[u] -- is emitted and the walk ends.  A rejection that
 * leaves p_res without mass (possible only through rounding) ends the walk
 * with the bonus drawn from p_res before it.  Arithmetic is fp32.
 *
 * Outputs as adaserve_tree_accept: accept_len[r] = accepted drafts + 1,
 * accept_nodes[r] = the path from the root, accept_tokens[r] = the accepted
 * drafts' tokens then the bonus token, -1 past them; accept_len = -1 and rows
 * of -1 for a malformed tree (as adaserve_tree_accept), a draft token of a
 * non-root node outside [0, vocab), a tree deeper than max_accept - 1, or a
 * node with children whose draft row has no logit above -inf (NaN counts as
 * none: q is then no distribution).  node_indptr must
 * be increasing (requests of consecutive, disjoint node ranges): where it is
 * not, requests that share nodes may also get -1.
 * u_accept, u_bonus: [total_nodes] fp32 (device).  Logits 16-byte aligned,
 * row_stride * element size a multiple of 16 bytes.  workspace: at least
 * adaserve_tree_accept_sampled_workspace_bytes(total_nodes) bytes of device
 * memory (1 KB per node: every node's softmax statistics, in parts of 16
 * bytes, up to 64 per node), 16-byte aligned,
 * no initialisation needed; calls sharing a workspace must not overlap in
 * time.  Two kernels are enqueued on `stream`: the statistics of every node
 * (the whole chip), then the walks, one workgroup per request.
 */
size_t adaserve_tree_accept_sampled_workspace_bytes(int32_t total_nodes);

int32_t adaserve_tree_accept_sampled(int32_t num_requests, int32_t total_nodes,
                                     const int32_t *node_indptr, const int32_t *parent,
                                     const int32_t *draft_tokens, const void *target_logits,
                                     const void *draft_logits, int64_t row_stride, int32_t vocab,
                                     int32_t dtype, const float *u_accept, const float *u_bonus,
                                     int32_t max_accept, int32_t *accept_len,
                                     int32_t *accept_tokens, int32_t *accept_nodes,
                                     void *workspace, size_t workspace_bytes, void *stream);

/* Message describing the last non-OK status returned on this thread. */
const char *adaserve_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ADASERVE_H */
