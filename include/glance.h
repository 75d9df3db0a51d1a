/*
 * glance.h -- C ABI of the GLANCE decode-round hot path on MI355X (gfx950).
 *
 * One GLANCE round (arXiv 2609.00355, Algorithm 1, App. B) runs two forward
 * passes and a walk.  This library provides the data-parallel core of each:
 *
 *   glance_block_draft_attn  attention of the one-pass block draft (Sec. 3.2):
 *                            the block (pending root b + B-1 mask tokens) attends
 *                            to the whole cached multimodal context and,
 *                            bidirectionally, to itself;
 *   glance_tree_verify_attn  attention of the one-pass tree verification
 *                            (Def. 1, Sec. 3.3): root b and the candidate tree
 *                            are packed behind an ancestor mask, so node i sees
 *                            the context plus exactly its ancestors and itself;
 *   glance_greedy_accept     the target-greedy token of every verified row
 *                            (vocabulary argmax, lowest index on ties) and the
 *                            walk of Algorithm 1: the longest root-to-node path
 *                            whose every edge carries the parent row's argmax,
 *                            plus the bonus token that becomes the next root;
 *   glance_greedy_accept_entropy  the same, plus the entropy of each root row
 *                            (the predictor of Sec. 4's entropy law);
 *   glance_greedy_accept_noalloc  the same, with no workspace argument and no
 *                            allocation (a static per-GPU scratch buffer);
 *   glance_sample_accept     the same walk under sampling at temperature T:
 *                            each row's token is a Gumbel-max draw from
 *                            softmax(z / T) with counter-based noise;
 *   glance_commit_path       the commit of a round: the keys and values of the
 *                            root and the accepted nodes join the context
 *                            cache, whose length advances (Def. 1, Eq. 1);
 *   glance_build_tree        the candidate tree of Algorithm 1's second step:
 *                            the N strings of highest plug-in score
 *                            prod_j q_j(y_j) over the drafter's marginals
 *                            (Assumption 1, Sec. 3.2; Sec. 3.3), as parent
 *                            and token arrays ready for tree verification.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Data pointers marked "device" are HIP device pointers owned by the caller.
 *    The library never allocates, frees or copies to the host on these paths;
 *    all scratch memory is the caller's `workspace`, sized by the matching
 *    *_workspace_size() call.  Inputs are never written.
 *  - Work is enqueued on `stream` (0 = the null stream) and the call returns
 *    without synchronising.  Calls on different streams must use different
 *    workspaces; calls that share a workspace must be ordered on one stream.
 *  - The return status covers everything checkable on the host: null or
 *    misaligned (16-byte) pointers, unsupported shapes and a workspace that is
 *    too small.  These checks run before any HIP call.  A failed kernel launch
 *    returns GLANCE_ERR_HIP.  glance_last_error() gives the detail of the
 *    calling thread's last non-OK status.
 *  - Device integer inputs (ctx_lens, parents, tokens) are not checked on the
 *    hot path (that would need a device-to-host copy).  They are made safe to
 *    read: each ctx_len is clamped to [0, ctx_capacity], and a parent index
 *    that is not in [0, node) ends that node's ancestor chain.  Use
 *    glance_validate_tree() on host copies to reject malformed trees.
 *  - All arithmetic accumulates in fp32.  Q, K, V and O share one dtype.
 */
#ifndef GLANCE_H
#define GLANCE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GLANCE_OK = 0,
  GLANCE_ERR_INVALID_ARG = -1, /* null/misaligned pointer, bad size or shape */
  GLANCE_ERR_UNSUPPORTED = -2, /* well-formed but outside this build's limits */
  GLANCE_ERR_WORKSPACE = -3,   /* workspace null or smaller than required */
  GLANCE_ERR_HIP = -4          /* a HIP call failed; see glance_last_error() */
} glance_status;

typedef enum { GLANCE_F32 = 0, GLANCE_BF16 = 1 } glance_dtype;

/*
 * Shape of one attention call.
 *   batch         sequences in the call, >= 1
 *   n_new         new rows per sequence: the block size B (draft) or the tree
 *                 rows including the root (verify); 1..64 (one 64-bit ancestor
 *                 word per node; the paper's trees have 63 nodes + root, Sec. 3.3)
 *   n_q_heads     query heads Hq; n_q_heads % n_kv_heads == 0 and
 *                 n_q_heads / n_kv_heads <= 16.  Query head h reads KV head
 *                 h / (Hq/Hkv) (contiguous grouped-query attention).
 *   n_kv_heads    KV heads Hkv, >= 1
 *   head_dim      D, 64 or 128
 *   ctx_capacity  token stride of the context cache (>= every ctx_len), >= 0
 *   sm_scale      softmax scale; <= 0 selects 1/sqrt(head_dim)
 *   dtype         dtype of Q, K, V and O
 */
typedef struct {
  int32_t batch;
  int32_t n_new;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t ctx_capacity;
  float sm_scale;
  glance_dtype dtype;
} glance_attn_shape;

/*
 * Block-draft attention (Sec. 3.2).  For every sequence b, query head h and
 * block row i:
 *     keys = [K_ctx[b, g, 0:ctx_b] ; K_new[b, 0:n_new, g]],   g = h / (Hq/Hkv)
 *     out[b,i,h] = softmax(sm_scale * q[b,i,h] . keys^T) . values
 * with every key visible to every row (the block is bidirectional and sees
 * the whole context).  Row 0 is the pending root b, rows 1.. are mask tokens;
 * the kernel is position-agnostic (Q and K are post-rotary).
 *
 *   q         device [batch][n_new][Hq][D]              dtype
 *   k_ctx     device [batch][Hkv][ctx_capacity][D]      dtype (may be NULL iff ctx_capacity == 0)
 *   v_ctx     device [batch][Hkv][ctx_capacity][D]      dtype (idem)
 *   k_new     device [batch][n_new][Hkv][D]             dtype, keys of the block rows
 *   v_new     device [batch][n_new][Hkv][D]             dtype
 *   ctx_lens  device [batch] int32, context tokens per sequence (root excluded)
 *   out       device [batch][n_new][Hq][D]              dtype
 *   lse       device [batch][n_new][Hq] float32 natural-log sum-exp of the
 *             scaled scores, or NULL
 *   workspace device, >= glance_attn_workspace_size(s, 0) bytes, 256-byte aligned
 */
glance_status glance_block_draft_attn(const glance_attn_shape* s, const void* q, const void* k_ctx,
                                      const void* v_ctx, const void* k_new, const void* v_new,
                                      const int32_t* ctx_lens, void* out, float* lse,
                                      void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Tree-verify attention (Def. 1, Sec. 3.3; "pack b and T with an ancestor
 * mask", Algorithm 1).  Same as the draft except for the new keys: row i sees
 * new key j iff j == i or j is an ancestor of i in the tree given by
 *   parents   device [batch][n_new] int32; parents[b][0] = -1 (row 0 is the
 *             root b) and 0 <= parents[b][i] < i for i >= 1.
 * The row of a depth-d node then carries the target's conditioning on
 * x o b o y_{1:d}.  Positions (ctx_b + depth) are the caller's business:
 * Q and K arrive post-rotary.
 */
glance_status glance_tree_verify_attn(const glance_attn_shape* s, const void* q, const void* k_ctx,
                                      const void* v_ctx, const void* k_new, const void* v_new,
                                      const int32_t* ctx_lens, const int32_t* parents, void* out,
                                      float* lse, void* workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/*
 * Greedy acceptance (Algorithm 1's loop; Def. 1's accepted length A(T)).
 *   logits      device [batch][n_nodes][vocab], dtype logits_dtype (F32 or BF16);
 *               row v is the verified distribution of node v, row 0 the root's
 *   parents     device [batch][n_nodes] int32 (as for tree verify)
 *   tokens      device [batch][n_nodes] int32; tokens[b][0] = root b,
 *               tokens[b][c] = token on the edge into node c
 *   argmax_out  device [batch][n_nodes] int32: argmax of each row.  Ties go to
 *               the lowest index; +0 and -0 are equal; a NaN counts as larger
 *               than every number and the first NaN wins.
 *   accept_len  device [batch] int32: a, the number of accepted tree tokens
 *   accept_path device [batch][path_stride] int32: node ids from the root to
 *               the last accepted node (a + 1 entries), then -1.  Entries past
 *               path_stride are dropped (accept_len still counts them);
 *               path_stride >= 16 holds any tree of depth <= 15.
 *   next_root   device [batch] int32: the bonus token argmax_out[b][last node],
 *               which the round commits after the a accepted tokens and which
 *               becomes the next round's root.
 *   workspace   device, >= glance_accept_workspace_size(batch, n_nodes, vocab)
 *               bytes, 256-byte aligned
 * Walk: v = 0; t = argmax(row v); if some child c of v has tokens[c] == t
 * (lowest such c if siblings repeat a token), append c and continue from c,
 * else stop.  Each step moves to a larger node index, so the walk ends within
 * n_nodes steps even for malformed device data.
 *   1 <= n_nodes <= 64, 1 <= vocab <= 2^30, path_stride >= 1.
 */
glance_status glance_greedy_accept(int32_t batch, int32_t n_nodes, int32_t vocab,
                                   glance_dtype logits_dtype, const void* logits,
                                   const int32_t* parents, const int32_t* tokens,
                                   int32_t* argmax_out, int32_t* accept_len, int32_t* accept_path,
                                   int32_t path_stride, int32_t* next_root,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * glance_greedy_accept plus the root entropy (Sec. 4's entropy law predicts
 * the accepted length from the target's next-token entropy at the round
 * root):
 *   root_entropy device [batch] float32, not NULL: the entropy (nats) of the
 *               softmax of row 0 of each sequence.  Computed in the same
 *               launch (fp32 sums relative to each chunk's maximum; the root
 *               row's workgroups read their chunk a second time); -inf logits
 *               carry probability 0; undefined if row 0 holds a NaN or +inf.
 * All other arguments, outputs and the workspace as for glance_greedy_accept.
 */
glance_status glance_greedy_accept_entropy(int32_t batch, int32_t n_nodes, int32_t vocab,
                                           glance_dtype logits_dtype, const void* logits,
                                           const int32_t* parents, const int32_t* tokens,
                                           int32_t* argmax_out, int32_t* accept_len, int32_t* accept_path,
                                           int32_t path_stride, int32_t* next_root, float* root_entropy,
                                           void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * glance_greedy_accept for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same argmax and walk with the same outputs, but no
 * workspace argument.  The scratch (the chunk words of every row) lives in a
 * static 1 MiB device buffer that the library holds on every GPU it runs on
 * until the process ends; the call allocates nothing.  Shapes whose scratch
 * exceeds 1 MiB are rejected with GLANCE_ERR_UNSUPPORTED before any HIP call
 * (batch * n_nodes up to 32768 always fit).  All calls on one GPU share its
 * buffer: calls that overlap on one GPU (different streams without ordering,
 * or several host threads) race and must be serialised by the caller.
 * The first call on a device looks up that device's buffer address (one HIP
 * symbol query, no allocation).
 */
glance_status glance_greedy_accept_noalloc(int32_t batch, int32_t n_nodes, int32_t vocab,
                                           glance_dtype logits_dtype, const void* logits,
                                           const int32_t* parents, const int32_t* tokens,
                                           int32_t* argmax_out, int32_t* accept_len, int32_t* accept_path,
                                           int32_t path_stride, int32_t* next_root, hipStream_t stream);

/*
 * Sampling acceptance at temperature T > 0 (the Limitations section: under
 * sampling the walk draws a token from the verified row of its node and
 * descends while the draw is a child in the tree, so every committed token
 * is a draw from the target's own distribution; the Sampling paragraph of
 * the Implementation Details appendix runs this at T = 1).
 * Every row v of sequence b gets one draw from softmax(z / T) by the
 * Gumbel-max rule:  draw = argmax_w  z_w / T + g_w,  g_w = -ln(-ln u_w),
 * lowest index on ties, where
 *   u_w = ((x >> 9) + 0.5) * 2^-23  and  x = word (w mod 4) of
 *   Philox4x32-10(counter = (w / 4, v, b, round), key = (seed low 32 bits,
 *   seed high 32 bits))   (Salmon et al., SC'11),
 * and both logarithms use one fixed fp32 recipe (t = m 2^e with m in
 * [sqrt(1/2), sqrt(2)), then e ln 2 + 2 s (1 + s^2/3 + s^4/5 + s^6/7 + s^8/9),
 * s = (m - 1) / (m + 1); IEEE-rounded operations without fused multiply-add;
 * z / T is one IEEE division, bf16 logits widened exactly).  The draws are
 * therefore a pure function of (logits, T, seed, round, b, v), reproducible
 * bit for bit on any IEEE machine.  The walk is glance_greedy_accept's with
 * the draws in place of the argmax: from v = 0, descend to the lowest child
 * c of v whose token equals draw(v); next_root is the draw of the last node.
 * The draws of rows the walk does not visit are returned but unused.
 *
 *   temperature  finite, >= 2^-126 (a normal float); T = 0 is
 *                glance_greedy_accept
 *   seed, round  the generator's key and the round number (callers advance
 *                round every round so that draws never repeat)
 *   round_counter device uint32, or NULL: when given, the round number used
 *                is round + *round_counter (read before any draw), and the
 *                call adds 1 to *round_counter after its draws, in stream
 *                order.  A HIP graph that captures the call then draws fresh
 *                noise on every replay (a captured by-value round would
 *                repeat one round's noise).  Calls sharing a counter must be
 *                ordered on one stream.
 *   draws_out    device [batch][n_nodes] int32: each row's draw
 *   other arguments, shapes, output layouts and the workspace: as for
 *   glance_greedy_accept (glance_accept_workspace_size); no root entropy.
 * NaN logits count as larger than every number (the first NaN wins); -inf
 * is a token of probability 0.
 */
glance_status glance_sample_accept(int32_t batch, int32_t n_nodes, int32_t vocab,
                                   glance_dtype logits_dtype, const void* logits,
                                   const int32_t* parents, const int32_t* tokens, float temperature,
                                   uint64_t seed, uint32_t round, uint32_t* round_counter, int32_t* draws_out,
                                   int32_t* accept_len, int32_t* accept_path, int32_t path_stride,
                                   int32_t* next_root, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * Commit of a round's accepted path into a context cache (the walk of Def. 1
 * commits the pending root and the accepted tokens y_1..y_a; Eq. 1 counts
 * them with the bonus token, which becomes the next root and is not cached).
 * The verify pass computed every node's keys and values at position
 * ctx + depth, which for the nodes of the accepted path is exactly the slot
 * the token takes in the prefix, so for each sequence b, with a = accept_len[b]
 * and ctx = ctx_lens[b]:
 *     k_ctx[b, :, ctx + i, :] = k_new[b, accept_path[b][i], :, :]    (i = 0..a)
 *     (likewise v), then ctx_lens[b] = ctx + a + 1.
 * The cache then equals what autoregressive decoding would have built.
 *
 *   k_new, v_new   device [batch][n_nodes][Hkv][D], dtype: the verify pass's
 *                  post-rotary keys and values of the packed rows
 *   accept_len     device [batch] int32, accept_path device [batch][path_stride]
 *                  int32: glance_greedy_accept's outputs (node 0 first)
 *   k_ctx, v_ctx   device [batch][Hkv][ctx_capacity][D], dtype; written in place
 *   ctx_lens       device [batch] int32; read, then advanced in place
 * Device data is made safe: a row count of min(a + 1, path_stride, n_nodes)
 * (none if a < 0), the copy stops at the first path entry outside
 * [0, n_nodes), ctx is clamped to [0, ctx_capacity], slots at or past the
 * capacity are not written and the length stops at ctx_capacity.  The length
 * grows by the path rows copied, so path_stride must hold a + 1 entries
 * (>= 16 for trees of depth <= 15) for the whole path to be committed.
 *   1 <= n_nodes <= 64, 1 <= head_dim <= 1024, ctx_capacity >= 1,
 *   path_stride >= 1; pointers aligned to their element size.  No workspace.
 */
glance_status glance_commit_path(int32_t batch, int32_t n_nodes, int32_t n_kv_heads, int32_t head_dim,
                                 int32_t ctx_capacity, glance_dtype dtype, const void* k_new,
                                 const void* v_new, const int32_t* accept_len, const int32_t* accept_path,
                                 int32_t path_stride, void* k_ctx, void* v_ctx, int32_t* ctx_lens,
                                 hipStream_t stream);

/*
 * Draft tree builder (Algorithm 1, second step; Sec. 3.3 with the plug-in
 * score of Assumption 1, Sec. 3.2).  From the drafter's logits z_j at offsets
 * j = 1..horizon, q_j = softmax(z_j), keep the `budget` strings y_{1:l}
 * (1 <= l <= horizon) of highest score  s(y) = sum_{j<=l} log q_j(y_j)  and
 * pack them as a tree below the root b.
 *
 *   draft_logits  device, dtype logits_dtype (F32 or BF16); sequence b's
 *                 offset-j row is the `vocab` values at element offset
 *                 b * seq_stride + (j - 1) * vocab.  NaN and +inf are outside
 *                 the contract (results unspecified, memory-safe); -inf is a
 *                 token of probability 0, and a row of all -inf gives
 *                 log q = -inf throughout.
 *   seq_stride    elements between sequences, >= horizon * vocab (e.g. the
 *                 block head's [batch][B][vocab] rows with row 0, the root's,
 *                 skipped: pointer + vocab and seq_stride = B * vocab)
 *   roots         device [batch] int32, the pending root token b
 *   parents       device [batch][budget + 1] int32 out: -1 for node 0 (the
 *                 root), then 0 <= parents[i] < i
 *   tokens        device [batch][budget + 1] int32 out: roots[b], then the
 *                 token on the edge into each node
 *   scores        device [batch][budget + 1] float32 out, or NULL: 0 for the
 *                 root, then s(y) of each node's string
 *   workspace     device, >= glance_tree_workspace_size(...) bytes, 256-byte aligned
 *
 * Nodes 1..budget are the kept strings in ranking order: score descending,
 * then the shorter string, then the string whose tokens rank better offset by
 * offset (a token's rank at an offset is its place in logit-descending,
 * index-ascending order).  The kept set is prefix-closed and every node's
 * children carry the best-ranked tokens of their offset.  Scores are fp32:
 * log q = z - logsumexp(z), summed from the first offset on; strings whose
 * scores differ by less than the rounding of that sum may be ranked either
 * way.
 *   1 <= horizon <= 15, 1 <= budget <= 63 (so budget + 1 <= 64 rows fit
 *   glance_tree_verify_attn), 1 <= vocab <= 2^30, batch * horizon <= 65535,
 *   and at least `budget` strings of length <= horizon must exist.
 */
glance_status glance_build_tree(int32_t batch, int32_t horizon, int32_t vocab, int32_t budget,
                                glance_dtype logits_dtype, const void* draft_logits, int64_t seq_stride,
                                const int32_t* roots, int32_t* parents, int32_t* tokens, float* scores,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes glance_build_tree needs (0 if the sizes are invalid). Host only. */
size_t glance_tree_workspace_size(int32_t batch, int32_t horizon, int32_t vocab, int32_t budget);

/* Workspace bytes an attention call with shape *s needs (0 if *s is invalid):
 * is_verify = 0 for glance_block_draft_attn, 1 for glance_tree_verify_attn.
 * The two sizes are equal in this build, so one workspace serves both calls
 * of a shape.  The size depends on the shape only. Host only. */
size_t glance_attn_workspace_size(const glance_attn_shape* s, int is_verify);

/* Workspace bytes glance_greedy_accept, glance_greedy_accept_entropy and
 * glance_sample_accept need (0 if the sizes are invalid).  Host only. */
size_t glance_accept_workspace_size(int32_t batch, int32_t n_nodes, int32_t vocab);

/*
 * Host-side check of one candidate tree (Def. 1): parents[0] == -1,
 * 0 <= parents[i] < i, depth <= max_depth (max_depth < 0: no limit) and, when
 * tokens_host is not NULL, distinct tokens among siblings (the tree is a set
 * of strings).  Returns GLANCE_OK or GLANCE_ERR_INVALID_ARG with the reason in
 * glance_last_error().  Host pointers; no GPU needed.
 */
glance_status glance_validate_tree(int32_t n, const int32_t* parents_host, const int32_t* tokens_host,
                                   int32_t max_depth);

/* Static description of a status code. */
const char* glance_status_string(glance_status status);

/* Detail of the calling thread's last non-OK status ("" if none). */
const char* glance_last_error(void);

/*
 * Profiling hook.  When both events are non-NULL, the next attention, accept,
 * commit or tree-builder call on this thread records `start` on its stream
 * right before its main kernel (the attention kernel without its merge pass,
 * the vocabulary argmax kernel without the walk, the commit kernel, or all
 * passes of the tree builder) and `stop` right after it, then forgets the
 * pair.  Arguments are hipEvent_t handles created by the caller.  Pass NULLs
 * to clear.
 */
glance_status glance_set_kernel_events(void* start_event, void* stop_event);

/* Library version: major * 10000 + minor * 100 + patch. */
int32_t glance_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GLANCE_H */
