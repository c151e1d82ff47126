/*
 * treeverify: target-model tree verification on AMD Instinct MI355X (gfx950).
 *
 * One verification step of tree-based speculative decoding, as the paper
 * "Make Every Draft Count: Hidden State based Speculative Decoding" states
 * it: the target model verifies a draft token tree in one parallel pass
 * under a tree-shaped attention mask (§2.1; §8 cites SpecInfer's tree
 * masking), accepts one path of the tree and produces a bonus token (§5.3),
 * decoding greedily (§7.1: temperature 0), over a paged KV cache (§7.1).
 * The three calls below are that step's data-parallel part:
 *
 *   tree_verify_attention  every node's query heads attend to the sequence's
 *                          committed prefix and to the node's own root path;
 *   tree_argmax_accept     per-node vocabulary argmax, greedy longest accepted
 *                          path, bonus token;
 *   kv_compact_accepted    the accepted path's K/V rows are written into the
 *                          cache right after the committed prefix.
 *
 * Conventions shared by every call
 *   - Every pointer argument is a DEVICE pointer, owned by the caller. The
 *     library never allocates, frees or retains device memory.
 *   - bf16 tensors are passed as uint16_t bit patterns. Index tensors are
 *     int32. Every tensor is dense, row-major (C order), in the layout given.
 *   - Calls are asynchronous on `stream` (0 = the null stream) and never
 *     synchronize. The return value is a status: TV_OK (0) or a negative
 *     TV_ERR_* code. Argument checks are done on the host before anything is
 *     launched; on an error nothing is launched and no output is written.
 *     TV_ERR_HIP reports a failure of this call's own launches (each launch
 *     is checked by its own status, so an error an earlier unrelated HIP call
 *     left pending is neither reported nor cleared); asynchronous execution
 *     errors surface through the HIP runtime as usual.
 *   - The library keeps no state between calls apart from a per-device cache
 *     of the compute-unit count. Calls are safe from several host threads as
 *     long as their output buffers do not overlap.
 *
 * Tree format
 *   Node i of sequence b has parent[b][i] in [-1, i-1] (topological order: a
 *   parent precedes its children). parent == -1 marks a root: the anchor a
 *   draft tree hangs from (the last verified token, or the ground-truth token
 *   a re-sampled tree is rooted at, §5.3 / Alg. 2). Roots are always accepted;
 *   several roots form a forest. A node sees itself and its ancestors.
 *
 * Ragged batches (verification fusion, §6.2: the previous round's re-sampled
 *   trees are verified together with this round's trees, so sequences carry
 *   forests of different sizes). The calls that take `num_nodes` accept a
 *   device array [B] of node counts, or NULL for N nodes everywhere. Sequence
 *   b then has n_b = num_nodes[b] nodes (clamped to [0, N]); nodes
 *   n_b .. N-1 are padding: none of their inputs (q, tree K/V, parent, draft
 *   token, logits row) is read into any result, and work is not spent on them.
 *
 * Content contract (not checked in the fast path; tv_validate_inputs checks
 * it): parent[b][i] in [-1, i-1]; kv_len[b] >= 0; every page id the prefix
 * and the compacted rows touch lies in [0, num_pages); and
 * ceil((kv_len[b] + accepted rows) / P) <= max_pages. Kernels clamp or skip
 * out-of-range ids and never read or write outside the buffers described
 * here, but results for inputs that break the contract are unspecified.
 */
#ifndef TREEVERIFY_H
#define TREEVERIFY_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(TREEVERIFY_BUILD)
#define TV_API __attribute__((visibility("default")))
#else
#define TV_API
#endif

#define TV_ABI_VERSION 5

/* Size of the static device scratch of tree_argmax_accept_noalloc (per GPU). */
#define TV_NOALLOC_SCRATCH_BYTES (4u << 20)

enum tv_status {
    TV_OK = 0,
    TV_ERR_NULL = -1,        /* a required pointer is NULL                      */
    TV_ERR_SHAPE = -2,       /* a size or count is outside the supported range  */
    TV_ERR_ALIGN = -3,       /* a tensor pointer is not 16-byte aligned         */
    TV_ERR_WORKSPACE = -4,   /* workspace missing or smaller than required      */
    TV_ERR_HIP = -5,         /* a HIP runtime call or kernel launch failed      */
    TV_ERR_DEVICE = -6,      /* the current device is not gfx950                */
    TV_ERR_SCRATCH = -7      /* more scratch needed than the static buffer holds */
};

/* TV_ABI_VERSION of the built library. */
TV_API int tv_abi_version(void);

/* Static English text for a status code (never NULL). */
TV_API const char *tv_status_string(int status);

/* ------------------------------------------------------------------------
 * tree_verify_attention
 *
 * For sequence b, node i and query head h (KV head g = h / (Hq / Hkv)):
 *   visible keys  R(b, i) = prefix positions 0 .. kv_len[b]-1
 *                           U { tree node j : j == i or j is an ancestor of i }
 *   s_j  = scale * <q[b,i,h,:], k_j[g,:]>
 *   out[b,i,h,:] = sum_j softmax(s)_j * v_j[g,:]      (bf16, round to nearest even)
 *   lse[b,i,h]   = log sum_j exp(s_j)                  (fp32, natural log)
 * Prefix key t of sequence b lives at
 *   k_cache[page_table[b][t / P]][t % P][g][:]  (v_cache likewise).
 * Tree node j's own key/value is k_tree[b][j][g][:] / v_tree[b][j][g][:].
 * (§2.1 tree-shaped attention; §8 tree masking; §1 attention over the cached
 * prefix; §7.1 paged KV cache.) Keys and values are post-positional-encoding
 * inputs; positions are the caller's concern.
 *
 *   q           [B, N, Hq, D]              bf16
 *   k_tree      [B, N, Hkv, D]             bf16
 *   v_tree      [B, N, Hkv, D]             bf16
 *   k_cache     [num_pages, P, Hkv, D]     bf16
 *   v_cache     [num_pages, P, Hkv, D]     bf16 (slots past kv_len may hold
 *                                          anything, NaN included: they are
 *                                          never read into the result)
 *   page_table  [B, max_pages]             int32
 *   kv_len      [B]                        int32, committed prefix lengths
 *   parent      [B, N]                     int32
 *   num_nodes   [B]                        int32 node counts, or NULL (see
 *                                          "Ragged batches"); rows of padding
 *                                          nodes get out = 0 and lse = -inf
 *   out         [B, N, Hq, D]              bf16, every element written
 *   lse         [B, N, Hq]                 fp32, or NULL
 *   workspace   >= tv_attention_workspace_size(...) bytes of device memory,
 *               16-byte aligned; contents on entry do not matter; clobbered.
 *
 * Supported: D in {64, 128}; 1 <= N <= 256; Hq % Hkv == 0 and
 * (Hq / Hkv) * N <= 2048; Hkv * D < 2^23; 0 <= B <= 1024; P a power of two
 * in [1, 256]; max_pages >= 1; num_pages >= 1.
 * max_kv_len is a host-side upper bound of kv_len[] used only to size the
 * launch; results never depend on it (an understated bound costs speed only).
 * scale <= 0 selects 1/sqrt(D). q, k_tree, v_tree, k_cache, v_cache, out and
 * workspace must be 16-byte aligned.
 * ------------------------------------------------------------------------ */
TV_API size_t tv_attention_workspace_size(int B, int N, int Hq, int Hkv, int D);

TV_API int tree_verify_attention(const uint16_t *q, const uint16_t *k_tree,
                                 const uint16_t *v_tree, const uint16_t *k_cache,
                                 const uint16_t *v_cache, const int32_t *page_table,
                                 const int32_t *kv_len, const int32_t *parent,
                                 const int32_t *num_nodes, int B, int N, int Hq, int Hkv, int D,
                                 int P, int max_pages, int num_pages,
                                 int max_kv_len, float scale, uint16_t *out, float *lse,
                                 void *workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * tree_argmax_accept
 *
 * Greedy verification (§7.1 temperature 0; §5.3 accepted path and bonus
 * token; Alg. 2 names the bonus the ground-truth token):
 *   argmax_out[b,i]  = lowest v maximising logits[b,i,v] (IEEE compare, so
 *                      -0 == +0; a NaN counts as the maximum, the first NaN wins)
 *   accepted(i)      = parent[i] == -1, or accepted(parent[i]) and
 *                      draft_tokens[b,i] == argmax_out[b,parent[i]]
 *   sel              = accepted node of greatest depth (root depth 0),
 *                      lowest index on a tie
 *   accept_len[b]    = depth(sel) + 1          (path nodes, root included, >= 1
 *                                              unless the sequence has no nodes)
 *   accept_idx[b,:]  = root .. sel node ids, then -1 up to N
 *   bonus_token[b]   = argmax_out[b, sel]
 *
 *   logits        [B, N, V]  fp32 (V * 4 bytes per row; rows need no alignment)
 *   draft_tokens  [B, N]     int32
 *   parent        [B, N]     int32
 *   num_nodes     [B]        int32 node counts, or NULL (see "Ragged batches"):
 *                            only nodes i < n_b take part; argmax_out is -1 for
 *                            padding nodes; a sequence with n_b == 0 gets
 *                            accept_len 0, bonus_token -1 and accept_idx all -1
 *   argmax_out    [B, N]     int32
 *   accept_len    [B]        int32
 *   accept_idx    [B, N]     int32
 *   bonus_token   [B]        int32
 *   workspace     >= tv_argmax_workspace_size(B, N, V) bytes, 8-byte aligned.
 * Supported: 0 <= B <= 65535, 1 <= N <= 256, 1 <= V < 2^31.
 * ------------------------------------------------------------------------ */
TV_API size_t tv_argmax_workspace_size(int B, int N, int V);

TV_API int tree_argmax_accept(const float *logits, const int32_t *draft_tokens,
                              const int32_t *parent, const int32_t *num_nodes, int B, int N,
                              int V, int32_t *argmax_out,
                              int32_t *accept_len, int32_t *accept_idx, int32_t *bonus_token,
                              void *workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * tree_argmax_accept_noalloc
 *
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): exactly
 * tree_argmax_accept (same arguments apart from the workspace, same kernels,
 * same results), with its per-(node, vocabulary segment) keys kept in a static
 * device buffer of TV_NOALLOC_SCRATCH_BYTES (4 MiB) that the library holds on
 * every GPU it runs on until the process ends. The call allocates nothing:
 * the buffer's device address is looked up once per device on the first call
 * (hipGetSymbolAddress, no allocation). Every key the call reads is written
 * earlier in the same call, so nothing needs clearing between calls.
 *
 * Limit: tv_argmax_workspace_size(B, N, V) <= TV_NOALLOC_SCRATCH_BYTES
 * (B * N <= 524256 node rows, whatever V); larger batches return
 * TV_ERR_SCRATCH and launch nothing. All calls on one GPU share its buffer:
 * calls that can overlap in time on one GPU (several streams, several host
 * threads) race on it and must be serialised by the caller.
 * ------------------------------------------------------------------------ */
TV_API int tree_argmax_accept_noalloc(const float *logits, const int32_t *draft_tokens,
                                      const int32_t *parent, const int32_t *num_nodes, int B,
                                      int N, int V, int32_t *argmax_out, int32_t *accept_len,
                                      int32_t *accept_idx, int32_t *bonus_token,
                                      hipStream_t stream);

/* ------------------------------------------------------------------------
 * kv_compact_accepted
 *
 * Keep the accepted path's keys/values (§1: the KV cache holds committed
 * tokens; rejected branches are discarded): for j < accept_len[b],
 *   pos = kv_len[b] + j
 *   k_cache[page_table[b][pos / P]][pos % P][:][:] = k_tree[b][accept_idx[b,j]][:][:]
 *   v_cache likewise.
 * No other cache byte changes. kv_len is NOT modified: the caller advances
 * it by accept_len after this call. Source and destination never overlap.
 *
 *   k_tree, v_tree     [B, N, Hkv, D]          bf16
 *   k_cache, v_cache   [num_pages, P, Hkv, D]  bf16, written in place
 *   page_table [B, max_pages], kv_len [B], accept_idx [B, N], accept_len [B] int32
 * Supported: 0 <= B <= 65535, 1 <= N <= 256, Hkv * D a multiple of 8,
 * P a power of two in [1, 256]. Rows whose node id or page id is out of
 * range are skipped (contract violation).
 * ------------------------------------------------------------------------ */
TV_API int kv_compact_accepted(const uint16_t *k_tree, const uint16_t *v_tree, uint16_t *k_cache,
                               uint16_t *v_cache, const int32_t *page_table,
                               const int32_t *kv_len, const int32_t *accept_idx,
                               const int32_t *accept_len, int B, int N, int Hkv, int D, int P,
                               int max_pages, int num_pages, hipStream_t stream);

/* ------------------------------------------------------------------------
 * tv_validate_inputs (debug aid)
 *
 * Checks the content contract on the device and writes a bit set to
 * *status_word (device int32): bit 0 parent out of [-1, i-1]; bit 1 negative
 * kv_len; bit 2 a prefix or compaction page index beyond max_pages; bit 3 a
 * page id the prefix or the tree rows would use outside [0, num_pages); bit 4
 * a node count outside [0, N]. 0 means the inputs satisfy the contract for up
 * to n_b compacted rows per sequence.
 * num_nodes: device [B] node counts of a ragged batch, or NULL (N everywhere).
 * With it, parents of padding nodes are not checked, and a sequence without
 * nodes has no pages checked (no call reads its prefix).
 * ------------------------------------------------------------------------ */
TV_API int tv_validate_inputs(const int32_t *page_table, const int32_t *kv_len,
                              const int32_t *parent, const int32_t *num_nodes, int B, int N,
                              int P, int max_pages, int num_pages, int32_t *status_word,
                              hipStream_t stream);

/* ------------------------------------------------------------------------
 * tree_build  (draft-tree construction by token-info sampling, Alg. 1 of
 *              §5.2, followed by the verification-budget pruning of §5.2;
 *              the hot-token table of §6.1)
 *
 * For each sequence b: the root is root_token[b] (the last verified token,
 * probability and joint probability 1) and forms the first frontier. At step
 * i = 0 .. S-1, every frontier node (in frontier order) takes the k most
 * probable tokens of softmax(logits[b][i] + r) as its children, in rank order,
 * where r is the node token's row of the token-info table (§5.1: the collapsed
 * token-info embedding adds to the logits); a child's joint probability is its
 * parent's times its own. The next frontier is the k children of the step with
 * the largest joint probabilities, largest first. After the last step the
 * `budget` nodes of largest joint probability are kept, in creation order
 * (root first; a node's parent always precedes it and is always kept).
 *
 * Hot tokens (§6.1): token-info exists for the H hot tokens only.
 * hot_vocab[c] is the vocabulary id of hot token c (distinct ids) and
 * hot_index[v] = c for v = hot_vocab[c], -1 for every other v. token_info is
 * [H, H] bf16: entry (row, col) is added to the logit of hot token col when
 * the expanded node's token is hot token row. A node whose token is not hot,
 * and every non-hot candidate, get nothing added. With H = 0 the three hot
 * arrays may be NULL.
 *
 * Arithmetic: candidates are ranked by the fp32 sum logit + entry (ties to
 * the lower vocabulary id); probabilities and joint probabilities are fp64
 * (ties in joint probability go to the node created first: step, frontier
 * rank, child rank).
 *
 *   logits       [B, S, V]   fp32, finite (the draft model's logits per step)
 *   root_token   [B]         int32 in [0, V)
 *   token_info   [H, H]      bf16; hot_vocab [H], hot_index [V] int32
 *   parent       [B, budget] int32 out: parent slot, -1 for the root and padding
 *   token        [B, budget] int32 out: the node's token, -1 for padding
 *   joint        [B, budget] fp32 out: joint probability, 0 for padding
 *   num_nodes    [B]         int32 out: min(budget, 1 + k + (S-1) k^2); slots
 *                            from num_nodes[b] on are padding. (parent, token,
 *                            num_nodes) are the tree inputs of
 *                            tree_verify_attention / tree_argmax_accept.
 *   workspace    >= tv_tree_build_workspace_size(...) bytes of device memory,
 *                8-byte aligned; contents on entry do not matter; clobbered.
 *
 * Supported: 0 <= B <= 65535, 1 <= S <= 16, 1 <= k <= 16, k <= V,
 * 0 <= H <= V, 1 <= budget <= 256. Contract (not checked): consistent hot
 * maps, root tokens in range. Out-of-range hot ids are skipped; results for
 * inputs that break the contract are unspecified.
 * ------------------------------------------------------------------------ */
TV_API size_t tv_tree_build_workspace_size(int B, int S, int V, int H, int k);

/* ------------------------------------------------------------------------
 * tree_resample  (re-sampling after verification, Alg. 2 of §5.3)
 *
 * The draft logits of the rejected steps are reused with the verified token's
 * information: for each sequence b, bonus_token[b] (the verification's bonus
 * token, i.e. the ground truth at the first rejected position) roots a new
 * tree. The first rejected position is accept_len[b] (the accepted path of
 * tree_argmax_accept counts the root, so the token at depth accept_len[b] was
 * rejected); the remaining logits are rows accept_len[b] .. S-1 of
 * logits[b], N_remain = S - accept_len[b]. If N_remain > r the tree is built
 * from them exactly as tree_build builds a tree (same token-info table, k,
 * pruning to `budget`); otherwise it is the single node bonus_token[b].
 * A sequence with accept_len[b] <= 0 verified nothing and gets no tree
 * (num_nodes[b] = 0, all slots padding). The output feeds the next
 * verification, e.g. as the second root of a fused forest.
 *
 *   bonus_token, accept_len   [B] int32 (device), as tree_argmax_accept wrote them
 *   r                         re-sampling threshold, >= 0
 * Everything else, the limits and the workspace (tv_tree_build_workspace_size)
 * are those of tree_build.
 * ------------------------------------------------------------------------ */
TV_API int tree_resample(const float *logits, const int32_t *bonus_token,
                         const int32_t *accept_len, const uint16_t *token_info,
                         const int32_t *hot_vocab, const int32_t *hot_index, int B, int S, int V,
                         int H, int k, int r, int budget, int32_t *parent, int32_t *token,
                         float *joint, int32_t *num_nodes, void *workspace,
                         size_t workspace_bytes, hipStream_t stream);
TV_API int tree_build(const float *logits, const int32_t *root_token, const uint16_t *token_info,
                      const int32_t *hot_vocab, const int32_t *hot_index, int B, int S, int V,
                      int H, int k, int budget, int32_t *parent, int32_t *token, float *joint,
                      int32_t *num_nodes, void *workspace, size_t workspace_bytes,
                      hipStream_t stream);

/* ------------------------------------------------------------------------
 * tree_lm_head_argmax_accept  (LM head fused with greedy verification)
 *
 * The logits tree_argmax_accept consumes are the target model's LM head
 * applied to every node's final hidden state, all nodes in one matrix
 * product (the paper computes the draft's logits of many positions the same
 * way, §4.2). This call takes the hidden states and the head weight instead
 * and never stores logits:
 *   logit[r, v]  = sum_i hidden[r, i] * w_head[v, i]    (bf16 products, fp32
 *                                                       accumulation on the
 *                                                       matrix cores)
 *   argmax_out[b, i] = lowest v maximising logit[b * N + i, v] as computed
 *                      (same ordering as tree_argmax_accept: -0 == +0, NaN
 *                      counts as the maximum)
 * and then exactly the acceptance of tree_argmax_accept (accept_len,
 * accept_idx, bonus_token, num_nodes handling). Where two logits of a row
 * lie within the fp32 accumulation error of each other, which of them wins
 * depends on the accumulation order; the result is then one of them.
 *
 *   hidden       [B, N, d]   bf16, 16-byte aligned
 *   w_head       [V, d]      bf16, 16-byte aligned (row v = token v's weights)
 *   draft_tokens, parent [B, N], num_nodes [B] (or NULL), argmax_out [B, N],
 *   accept_len [B], accept_idx [B, N], bonus_token [B]: as tree_argmax_accept.
 *                Padding rows are multiplied with the rest (fixed tile shape)
 *                but take no part in any result.
 *   workspace    >= tv_lm_head_workspace_size(B, N, V, d) bytes of device
 *                memory, 8-byte aligned; contents on entry do not matter.
 * Supported: 0 <= B <= 65535, 1 <= N <= 256, 1 <= V <= 2^31 - 257, d a
 * multiple of 64 (>= 64; the weight streams in 64-deep units of whole
 * 128-byte lines), and at most 2^31 - 1 workgroups (V/256 x B N/256,
 * rounded up). Other shapes return TV_ERR_SHAPE.
 * ------------------------------------------------------------------------ */
TV_API size_t tv_lm_head_workspace_size(int B, int N, int V, int d);

TV_API int tree_lm_head_argmax_accept(const uint16_t *hidden, const uint16_t *w_head,
                                      const int32_t *draft_tokens, const int32_t *parent,
                                      const int32_t *num_nodes, int B, int N, int V, int d,
                                      int32_t *argmax_out, int32_t *accept_len,
                                      int32_t *accept_idx, int32_t *bonus_token,
                                      void *workspace, size_t workspace_bytes,
                                      hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* TREEVERIFY_H */
