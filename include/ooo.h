/*
 * ooo.h - C ABI of libooo, the MI355X (gfx950) tree-verification library.
 *
 * One verification step of greedy speculative decoding at batch one, as the
 * OoO-Spec paper describes it (Section 3, "Target authority" with Eq. 1 and
 * "The ToolSpec decoding loop"; Section 4.5, "Verify and commit"):
 *
 *   ooo_hint_merge     hint-bank continuations of the committed suffix, then
 *                      native candidates, as the lanes of one round
 *   ooo_pack_tree      merge priority-ordered draft continuations into a trie
 *   ooo_tree_attn      per layer: every trie node attends to the committed
 *                      prefix and to its own ancestors (one pass for the tree)
 *   ooo_lmhead_argmax  LM head over all nodes and the greedy token of each
 *                      (ooo_lmhead_pack lays the weight out for streaming)
 *   ooo_accept         longest root path whose tokens agree with the greedy
 *                      tokens, plus the target's own next (bonus) token
 *   ooo_kv_compact     move the accepted nodes' K/V rows into the committed
 *                      cache, directly after the prefix
 *
 * The target decoder layer around the path (the target scores the tree in
 * one forward pass, Section 4.5; Qwen3 targets, Section 5):
 *
 *   ooo_embed_rows     residual rows of the trie's tokens
 *   ooo_rmsnorm        RMSNorm of residual rows (fp32 in, bf16 out)
 *   ooo_linear         x W^T with a fused epilogue: the projections
 *                      (ooo_linear_pack lays a weight out for streaming)
 *   ooo_qk_norm_rope   per-head q/k norms, rotation at position P + depth,
 *                      q out, node k/v into the layer's cache rows
 *   ooo_swiglu         silu(gate) * up of the fused MLP projection
 *   ooo_linear_add_rmsnorm   a projection added into the residual rows,
 *                      fused with the RMSNorm that follows it
 *   ooo_linear_qk_norm_rope  the q/k/v projection fused with the q/k norms,
 *                      the rotation and the cache writes
 *
 * Conventions shared by every entry point
 *   - Return value: OOO_OK (0) or a negative ooo_status.  On error nothing has
 *     been enqueued and ooo_last_error() returns a message (thread-local,
 *     valid until the next call on the same thread).
 *   - Arguments are validated on the host before any device work is queued.
 *   - Device entry points are asynchronous on `stream` (a hipStream_t; NULL is
 *     the null stream) and return after enqueueing.  Buffers must stay valid
 *     until that work completes.  They never allocate device memory; scratch
 *     comes from the caller's `workspace`, sized by the *_workspace query.
 *   - The caller owns every buffer.  Outputs must not alias inputs unless an
 *     entry point says so.  No entry point keeps state between calls.
 *   - Calls sharing a workspace must not run concurrently.
 *   - dtype: OOO_F32 (float32 everywhere) or OOO_BF16 (bfloat16 storage,
 *     float32 accumulation and softmax).
 *   - Results are deterministic: identical inputs give bitwise-identical
 *     outputs (no floating-point atomics).
 */
#ifndef OOO_H
#define OOO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OOO_ABI_VERSION 1

typedef enum {
  OOO_OK = 0,
  OOO_ERR_INVALID = -1,     /* null pointer, bad size, inconsistent shape */
  OOO_ERR_UNSUPPORTED = -2, /* valid request this build has no kernel for */
  OOO_ERR_CAPACITY = -3,    /* an output or workspace is too small */
  OOO_ERR_HIP = -4          /* the HIP runtime reported a launch error */
} ooo_status;

typedef enum { OOO_F32 = 0, OOO_BF16 = 1 } ooo_dtype;

/* Message for the last non-OK status on this thread ("" if none). */
const char* ooo_last_error(void);

/* OOO_ABI_VERSION of the loaded library. */
int ooo_version(void);

/*
 * ooo_pack_tree - candidate trie (Section 3, ToolSpec loop: candidates are
 * combined into one tree; Section 4.4: Merge_B keeps a fixed candidate
 * budget and hint lanes come first; Section 4.5: hint and native
 * continuations are compiled into the same tree).
 *
 * HOST memory only, synchronous.
 *   root_token      the token the target committed last (node 0)
 *   cand_tokens     concatenated candidate continuations (after the root)
 *   cand_offsets    [n_cand + 1] CSR offsets into cand_tokens, in priority
 *                   order, non-decreasing, cand_offsets[0] == 0
 *   max_nodes       node budget (1..1024), including the root
 *   max_depth       depth cap (>= 0); the root has depth 0
 *   token, parent, depth   [max_nodes] int32 outputs; parent[0] == -1
 *   anc_mask        [max_nodes * mask_words] uint64 output; bit j of row i is
 *                   set iff node j is an ancestor of node i or i itself
 *   mask_words      words per mask row; must satisfy 64 * mask_words >= max_nodes
 *   n_nodes         number of nodes written
 *   n_truncated     candidate tokens dropped by the depth cap or the budget
 * Nodes appear in first-appearance order over the candidates, so
 * parent[i] < i and siblings carry distinct tokens.  A token equal to an
 * existing child is shared; once the budget is full no node is added and the
 * rest of each candidate from its first unplaceable token is dropped.
 * Host memory only; synchronous; keeps no state between calls and allocates
 * nothing.
 * Errors: OOO_ERR_INVALID for null pointers, n_cand < 0, max_nodes < 1,
 * max_depth < 0, non-monotone offsets, negative tokens, or too few mask words;
 * OOO_ERR_UNSUPPORTED for max_nodes > 1024 (the device kernels' limit).
 */
int ooo_pack_tree(int32_t root_token, const int32_t* cand_tokens, const int32_t* cand_offsets,
                  int32_t n_cand, int32_t max_nodes, int32_t max_depth, int32_t* token,
                  int32_t* parent, int32_t* depth, uint64_t* anc_mask, int32_t mask_words,
                  int32_t* n_nodes, int32_t* n_truncated);

/*
 * ooo_hint_merge - candidate lanes of one retrieval round (Section 4.4,
 * Suffix matching and Eq. 3): continuations that the request's hint bank
 * proposes for the next position come first, the native candidates fill the
 * remaining lanes.  The result feeds ooo_pack_tree, which applies the node
 * budget.
 *
 * HOST memory only, synchronous, deterministic.
 *   bank, bank_len   the hint bank: tokenized views separated by eos_token;
 *                    bank_len 0 (hints not ready, or none) gives the native
 *                    candidates alone
 *   committed, n_committed   committed tokens, oldest first; the last one is
 *                    the root of the next trie
 *   max_suffix       longest suffix tried (the paper uses 7), >= 1
 *   max_len          tokens per hint continuation, >= 1
 *   native_tokens, native_offsets, n_native   native candidates, CSR in
 *                    priority order (native_offsets[0] == 0, non-decreasing)
 *   n_lanes          lanes of the round, >= 0
 *   out_tokens       merged candidate tokens, capacity out_cap
 *   out_offsets      [n_lanes + 1] CSR offsets of the merged candidates
 *   n_out            merged candidates written (<= n_lanes)
 *   n_hint           how many of them come from the bank (they come first)
 *   suffix_len       length n of the suffix whose occurrences proposed them
 *                    (0 when the bank proposed nothing)
 * For n = min(max_suffix, n_committed) down to 1, every occurrence of the last
 * n committed tokens in the bank proposes the tokens after it, up to the next
 * eos_token (exclusive) and at most max_len of them; the first n with a
 * non-empty proposal is used, and its proposals are taken in bank order,
 * each distinct one once.
 * Errors: OOO_ERR_INVALID (null pointers, negative sizes, max_suffix or
 * max_len < 1, bad native offsets, negative tokens), OOO_ERR_CAPACITY (the
 * merged tokens exceed out_cap; *n_out is then 0).
 */
int ooo_hint_merge(const int32_t* bank, int64_t bank_len, int32_t eos_token, const int32_t* committed,
                   int32_t n_committed, int32_t max_suffix, int32_t max_len, const int32_t* native_tokens,
                   const int32_t* native_offsets, int32_t n_native, int32_t n_lanes, int32_t* out_tokens,
                   int64_t out_cap, int32_t* out_offsets, int32_t* n_out, int32_t* n_hint,
                   int32_t* suffix_len);

/*
 * ooo_tree_attn - one layer of tree-masked attention (Section 4.5: the target
 * scores the whole candidate tree in one forward pass; each node sees what
 * sequential greedy decoding of its own path would see).
 *
 * DEVICE pointers.
 *   q          [n_nodes][n_q_heads][head_dim] queries (post-RoPE)
 *   k_cache, v_cache   one layer, [n_kv_heads][cap][head_dim]: rows [0, P) are
 *              the committed prefix, row P + i holds node i's key/value
 *   cap        rows per KV head; P + n_nodes <= cap
 *   prefix_len P >= 0
 *   prefix_len_dev  NULL, or a device int32 holding the prefix length to use
 *              at run time (a decode loop that replays one captured step
 *              while P grows); prefix_len is then its upper bound, used for
 *              validation and planning, and a device value outside
 *              [0, prefix_len] is clamped into it
 *   anc_mask   [n_nodes][mask_words] from ooo_pack_tree (device copy)
 *   scale      score scale, normally 1/sqrt(head_dim)
 *   out        [n_nodes][n_q_heads][head_dim], same dtype; must not alias
 * Query head h reads KV head h / (n_q_heads / n_kv_heads).  For node i the
 * keys are prefix rows 0..P-1 and rows P + j for every j set in anc_mask[i];
 * softmax in float32.
 * Supported: head_dim 64 or 128; any n_q_heads / n_kv_heads;
 * n_nodes <= 64 * mask_words <= 1024.
 * workspace, ws_bytes  device scratch of ooo_tree_attn_workspace() bytes (0
 *            when the plan needs none; then workspace may be NULL): the bf16
 *            path splits the keys over workgroups, and a second kernel on the
 *            same stream merges the splits' partial results from it.
 * Errors: OOO_ERR_INVALID (null pointers, n_nodes < 1, prefix_len < 0,
 * P + n_nodes > cap, n_q_heads % n_kv_heads != 0, 64 * mask_words < n_nodes),
 * OOO_ERR_UNSUPPORTED, OOO_ERR_CAPACITY (ws_bytes below the query),
 * OOO_ERR_HIP.
 *
 * Relative to the plain signature of this step (Q, the layer's K/V cache, P,
 * N, the ancestor masks, head counts, scale, dtype, out, workspace, stream),
 * two arguments are additions: prefix_len_dev (one captured step replayed as
 * P grows) and the explicit head_dim.
 */
size_t ooo_tree_attn_workspace(int32_t n_nodes, int32_t n_q_heads, int32_t n_kv_heads,
                               int32_t head_dim, int32_t prefix_len, ooo_dtype dt);
int ooo_tree_attn(const void* q, const void* k_cache, const void* v_cache, int64_t cap,
                  int32_t prefix_len, const int32_t* prefix_len_dev, int32_t n_nodes,
                  const uint64_t* anc_mask,
                  int32_t mask_words, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                  float scale, ooo_dtype dt, void* out, void* workspace, size_t ws_bytes,
                  void* stream);

/*
 * ooo_tree_attn_noalloc - ooo_tree_attn without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops that must not call the allocator, harnesses that forbid it).
 *
 * Arguments as for ooo_tree_attn, without workspace and ws_bytes.  The split
 * partials go to a scratch array built into the library, 16 MiB per GPU
 * (ooo_tree_attn_noalloc_scratch_bytes()), held until the process ends; its
 * device address is looked up on the first call on each device.  The call
 * allocates nothing.  Every call on one GPU shares that GPU's scratch, so
 * calls that may overlap on one GPU (different streams without ordering)
 * race; calls ordered on one stream do not.  Nothing in the scratch needs to
 * start at zero.
 * Errors: those of ooo_tree_attn, and OOO_ERR_CAPACITY when the shape's
 * partials (ooo_tree_attn_workspace()) exceed the scratch.
 */
int ooo_tree_attn_noalloc(const void* q, const void* k_cache, const void* v_cache, int64_t cap,
                          int32_t prefix_len, const int32_t* prefix_len_dev, int32_t n_nodes,
                          const uint64_t* anc_mask, int32_t mask_words, int32_t n_q_heads, int32_t n_kv_heads,
                          int32_t head_dim, float scale, ooo_dtype dt, void* out, void* stream);
size_t ooo_tree_attn_noalloc_scratch_bytes(void);

/*
 * ooo_tree_attn_ex, ooo_tree_attn_workspace_ex - ooo_tree_attn with the
 * planner's choices overridden, for tests and tuning.
 *   force_splits  0: the planner's split count; > 0: that many key splits
 *                 (clamped to 1..32 and to the key tiles)
 *   variant       0: the default kernel; 1: one wave per 32-row group at
 *                 head_dim 128 (the head_dim 64 kernel's scheme)
 * Results stay within the same tolerance; each setting is deterministic.
 * The workspace query must be made with the same force_splits.
 */
size_t ooo_tree_attn_workspace_ex(int32_t n_nodes, int32_t n_q_heads, int32_t n_kv_heads,
                                  int32_t head_dim, int32_t prefix_len, ooo_dtype dt, int32_t force_splits);
int ooo_tree_attn_ex(const void* q, const void* k_cache, const void* v_cache, int64_t cap,
                     int32_t prefix_len, const int32_t* prefix_len_dev, int32_t n_nodes,
                     const uint64_t* anc_mask, int32_t mask_words, int32_t n_q_heads, int32_t n_kv_heads,
                     int32_t head_dim, float scale, ooo_dtype dt, void* out, void* workspace,
                     size_t ws_bytes, void* stream, int32_t force_splits, int32_t variant);

/*
 * ooo_lmhead_pack - one-time re-layout of the LM-head weight for streaming.
 *
 * The LM head reads all of W once per step and is bound by HBM bandwidth.
 * In nn.Linear layout each 128-row tile of W is read 128 bytes per row at a
 * time from rows hidden_dim*2 bytes apart; the packed layout stores each
 * (128-row tile, 64-column chunk) block as one contiguous 16 KiB run, with
 * rows past `vocab` zero-filled, so the kernel streams W strictly in order.
 * Model weights are static, so the packing runs once when the weight is
 * loaded, not per step.
 *
 * DEVICE pointers; OOO_BF16 only; asynchronous on `stream`.
 *   weight   [vocab][hidden_dim] (nn.Linear layout), read only
 *   packed   ooo_lmhead_packed_bytes(vocab, hidden_dim, dt) bytes; must not
 *            alias `weight`
 * Errors: OOO_ERR_INVALID (null pointers, non-positive sizes),
 * OOO_ERR_UNSUPPORTED (dtype other than OOO_BF16, hidden_dim % 64 != 0),
 * OOO_ERR_CAPACITY (packed_bytes too small), OOO_ERR_HIP.
 */
typedef enum { OOO_W_ROWS = 0, OOO_W_PACKED = 1 } ooo_weight_layout;
size_t ooo_lmhead_packed_bytes(int32_t vocab, int32_t hidden_dim, ooo_dtype dt);
int ooo_lmhead_pack(const void* weight, int32_t vocab, int32_t hidden_dim, ooo_dtype dt, void* packed,
                    size_t packed_bytes, void* stream);

/*
 * ooo_lmhead_argmax - LM head and greedy token of every node (Eq. 1: the
 * committed token is the target's most likely next token).
 *
 * DEVICE pointers.
 *   hidden     [n_nodes][hidden_dim] final hidden rows
 *   weight     OOO_W_ROWS: [vocab][hidden_dim] (nn.Linear layout);
 *              OOO_W_PACKED: the output of ooo_lmhead_pack (OOO_BF16 only)
 *   argmax_ids [n_nodes] int32: lowest vocabulary index among equal maxima
 *   max_logit  [n_nodes] float32: the logit at argmax_ids
 *   logits     NULL, or [n_nodes][vocab] float32 (validation dump)
 * Logits are float32 sums of exact products, added in the same order for
 * every vocabulary row, so identical weight rows give identical logits.
 * Supported: OOO_BF16 needs hidden_dim % 64 == 0 and n_nodes <= 256;
 * OOO_F32 needs hidden_dim % 4 == 0 and the OOO_W_ROWS layout.
 * Errors: OOO_ERR_INVALID (null pointers, non-positive sizes, unknown
 * layout), OOO_ERR_UNSUPPORTED, OOO_ERR_CAPACITY, OOO_ERR_HIP.
 */
size_t ooo_lmhead_workspace(int32_t n_nodes, int32_t hidden_dim, int32_t vocab, ooo_dtype dt);
int ooo_lmhead_argmax(const void* hidden, const void* weight, int32_t n_nodes,
                      int32_t hidden_dim, int32_t vocab, ooo_dtype dt, int32_t weight_layout,
                      int32_t* argmax_ids, float* max_logit, float* logits, void* workspace,
                      size_t ws_bytes, void* stream);

/*
 * ooo_accept - longest greedy-agreeing root path (Section 4.5, Verify and
 * commit: draft tokens are kept while they equal the target's greedy token
 * at their parent; at the first disagreement the rest is rejected and the
 * target's own token is used).
 *
 * DEVICE pointers.
 *   token, parent, depth, anc_mask   the packed trie (ooo_pack_tree layout)
 *   argmax_ids   [n_nodes] greedy token of every node
 *   max_depth    the deepest node depth the trie may hold (the max_depth it
 *                was packed with)
 *   path_cap     entries in `path`; at least max_depth + 1
 *   path         [path_cap] int32 out: path[d] = accepted node at depth d for
 *                d <= L, -1 beyond; path[0] == 0
 *   accept_len   [1] int32 out: L, the number of accepted draft nodes
 *   bonus_token  [1] int32 out: argmax_ids[path[L]]
 * The step commits token[path[1..L]] followed by the bonus token (L + 1
 * tokens).  Precondition (guaranteed by ooo_pack_tree): parent[i] < i and
 * siblings carry distinct tokens.  A trie whose accepted path runs deeper
 * than path_cap - 1 (deeper than the max_depth it was declared with) is
 * reported on the device, not shortened: accept_len = -1, bonus_token = -1
 * and path all -1, and ooo_kv_compact then moves no row.
 * Errors: OOO_ERR_INVALID (null pointers, n_nodes < 1, max_depth < 0,
 * path_cap < 1, 64 * mask_words < n_nodes, mask_words > 16),
 * OOO_ERR_CAPACITY (path_cap < max_depth + 1), OOO_ERR_HIP.
 * Relative to the plain signature of this step, path_cap is an addition (the
 * size of `path`, checked against max_depth).
 */
int ooo_accept(const int32_t* token, const int32_t* parent, const int32_t* depth,
               const uint64_t* anc_mask, int32_t mask_words, const int32_t* argmax_ids,
               int32_t n_nodes, int32_t max_depth, int32_t path_cap, int32_t* path,
               int32_t* accept_len, int32_t* bonus_token, void* stream);

/*
 * ooo_kv_compact - commit the accepted states (Section 4.5: only states on
 * the accepted path enter the committed KV cache).
 *
 * DEVICE pointers.
 *   k_cache, v_cache   [n_layers][n_kv_heads][cap][head_dim], updated in place
 *   prefix_len         P, the committed length before this step
 *   prefix_len_dev     NULL, or a device int32 holding the prefix length to
 *                      use at run time (a decode loop that replays one
 *                      captured step while P grows); prefix_len is then its
 *                      upper bound, used for validation and planning, and a
 *                      device value outside [0, prefix_len] is clamped into it
 *   n_nodes            trie size of the step; node rows are [P, P + n_nodes)
 *   path, accept_len   outputs of ooo_accept (read on the device, so no host
 *                      synchronisation is needed in between)
 *   path_cap           entries in `path`
 * For every layer, KV head, K and V: row P + path[d] moves to row P + d for
 * d = 0..L.  The committed length becomes P + L + 1; rows beyond it are free.
 * Rows [0, P] are never written.  Overlapping source and destination rows are
 * handled (every source is read before its row can be overwritten).
 * Precondition: path is strictly increasing (true for any root path of a
 * packed trie).  Entries with path[d] >= n_nodes or L >= path_cap are
 * ignored on the device rather than read out of bounds; accept_len = -1
 * (ooo_accept's report of a path deeper than path_cap - 1) moves no row.
 * Errors: OOO_ERR_INVALID (null pointers, sizes < 1, prefix_len < 0,
 * prefix_len + n_nodes > cap), OOO_ERR_UNSUPPORTED (head_dim * element size
 * not a multiple of 16 bytes), OOO_ERR_HIP.
 */
int ooo_kv_compact(void* k_cache, void* v_cache, int32_t n_layers, int32_t n_kv_heads,
                   int64_t cap, int32_t head_dim, ooo_dtype dt, int32_t prefix_len,
                   const int32_t* prefix_len_dev, int32_t n_nodes, const int32_t* path,
                   const int32_t* accept_len, int32_t path_cap, void* stream);

/*
 * ooo_embed_rows - residual rows of the trie's tokens (the input of the
 * target's first layer; Section 4.5: one forward pass over the tree).
 *
 * DEVICE pointers; asynchronous on `stream`.
 *   table    [vocab][hidden_dim] bf16 embedding table
 *   tokens   [n_nodes] int32 (the packed trie's tokens)
 *   h        [n_nodes][hidden_dim] float32 output
 * A token outside [0, vocab) gives a row of NaN.
 * Errors: OOO_ERR_INVALID (null pointers, sizes < 1), OOO_ERR_UNSUPPORTED
 * (hidden_dim % 8 != 0), OOO_ERR_HIP.
 */
int ooo_embed_rows(const void* table, const int32_t* tokens, int32_t n_nodes, int32_t hidden_dim,
                   int32_t vocab, float* h, void* stream);

/*
 * ooo_rmsnorm - out = h / sqrt(mean(h^2) + eps) * weight per row (the
 * target's pre-attention, pre-MLP and final norms; Section 5, Qwen3).
 *
 * DEVICE pointers; asynchronous on `stream`.
 *   h        [n_rows][dim] float32 residual rows
 *   weight   [dim] bf16
 *   out      [n_rows][dim] bf16; must not alias h
 * Errors: OOO_ERR_INVALID (null pointers, sizes < 1, eps < 0),
 * OOO_ERR_UNSUPPORTED (dim not a multiple of 4 or above 8192), OOO_ERR_HIP.
 */
int ooo_rmsnorm(const float* h, const void* weight, int32_t n_rows, int32_t dim, float eps, void* out,
                void* stream);

/*
 * ooo_linear - the target's projections (q/k/v, output, gate/up, down) over
 * the trie's rows: y = x W^T, bf16 operands, float32 accumulation, with the
 * epilogue fused (Section 4.5: one forward pass over the tree; Section 5:
 * Qwen3 targets).
 *
 * DEVICE pointers; asynchronous on `stream`.
 *   x        [n_rows][in_dim] bf16, n_rows <= 256, in_dim % 64 == 0
 *   weight   [out_dim][in_dim] bf16 (nn.Linear layout, OOO_W_ROWS), or its
 *            ooo_linear_pack layout (OOO_W_PACKED, the fast path)
 *   out      [n_rows][out_dim] float32 (OOO_EPI_STORE_F32: y; OOO_EPI_ADD_F32:
 *            out += y, e.g. the residual rows) or bf16 (OOO_EPI_STORE_BF16:
 *            y); OOO_EPI_SWIGLU_BF16: weight holds the gate rows then the up
 *            rows (out_dim = 2 I, I % 128 == 0) and out [n_rows][I] bf16 gets
 *            silu(gate) * up.  out must not alias x or weight.
 *   workspace, ws_bytes   ooo_linear_workspace(n_rows, in_dim, out_dim)
 *            bytes of partial sums (fp16 times a power of two per 32 output
 *            columns, so a float32 output carries a relative rounding error
 *            of about 2^-11 per partial sum; they are added in float32)
 * Deterministic: partial sums are added in a fixed order (no atomics).
 * Errors: OOO_ERR_INVALID (null pointers, sizes < 1, unknown layout or
 * epilogue), OOO_ERR_UNSUPPORTED (in_dim % 64, n_rows > 256, SwiGLU with
 * out_dim % 256), OOO_ERR_CAPACITY (workspace too small), OOO_ERR_HIP.
 */
typedef enum {
  OOO_EPI_STORE_F32 = 0,
  OOO_EPI_STORE_BF16 = 1,
  OOO_EPI_ADD_F32 = 2,
  OOO_EPI_SWIGLU_BF16 = 3
} ooo_epilogue;
size_t ooo_linear_workspace(int32_t n_rows, int32_t in_dim, int32_t out_dim);
size_t ooo_linear_packed_bytes(int32_t out_dim, int32_t in_dim);
/* One-time re-layout of a [out_dim][in_dim] bf16 weight into 16 KiB blocks
 * of 128 rows x 64 columns (the layout of ooo_lmhead_pack); same errors. */
int ooo_linear_pack(const void* weight, int32_t out_dim, int32_t in_dim, void* packed, size_t packed_bytes,
                    void* stream);
int ooo_linear(const void* x, const void* weight, int32_t n_rows, int32_t in_dim, int32_t out_dim,
               int32_t weight_layout, ooo_epilogue epilogue, void* out, void* workspace, size_t ws_bytes,
               void* stream);

/*
 * ooo_linear_add_rmsnorm - a projection whose output is added into the
 * residual rows, fused with the RMSNorm that follows it in the target's
 * layer (o_proj then the post-attention norm; down then the next layer's
 * input norm or the final norm; Section 4.5: one forward pass over the tree).
 *
 * DEVICE pointers; asynchronous on `stream`.
 *   x, weight, n_rows, in_dim, out_dim, weight_layout, workspace, ws_bytes
 *                as for ooo_linear (workspace sized by ooo_linear_workspace)
 *   residual     [n_rows][out_dim] float32, updated in place:
 *                residual += x weight^T
 *   norm_weight  [out_dim] bf16
 *   normed_out   [n_rows][out_dim] bf16:
 *                residual / sqrt(mean(residual^2) + eps) * norm_weight
 * The partial sums are added in the same order as ooo_linear's
 * OOO_EPI_ADD_F32, so `residual` matches that epilogue bitwise.
 * Errors: those of ooo_linear; OOO_ERR_INVALID (null residual, norm_weight
 * or normed_out, eps < 0); OOO_ERR_UNSUPPORTED (out_dim % 4 != 0 or
 * out_dim > 8192).
 */
int ooo_linear_add_rmsnorm(const void* x, const void* weight, int32_t n_rows, int32_t in_dim, int32_t out_dim,
                           int32_t weight_layout, float* residual, const void* norm_weight, float eps,
                           void* normed_out, void* workspace, size_t ws_bytes, void* stream);

/*
 * ooo_linear_qk_norm_rope - the fused q/k/v projection of the trie's rows
 * followed by what ooo_qk_norm_rope does with it (per-head norms of q and
 * k, rotation at position P + depth[i], q to q_out, k and v to cache row
 * P + i; Section 4.5), computed from the projection's float32 sums (no bf16
 * rounding in between).
 *
 * DEVICE pointers; asynchronous on `stream`.
 *   x, weight, n_rows, in_dim, weight_layout, workspace, ws_bytes   as for
 *                ooo_linear, with out_dim = (n_q_heads + 2 n_kv_heads)
 *                head_dim (q rows, then k rows, then v rows)
 *   the rest as for ooo_qk_norm_rope (n_rows trie nodes; prefix_len_dev
 *   NULL or the device prefix length that prefix_len bounds)
 * Errors: those of ooo_linear and ooo_qk_norm_rope; OOO_ERR_UNSUPPORTED when
 * (n_q_heads + 2 n_kv_heads) head_dim is not a multiple of 128.
 */
int ooo_linear_qk_norm_rope(const void* x, const void* weight, int32_t n_rows, int32_t in_dim,
                            int32_t weight_layout, const void* q_norm, const void* k_norm, float eps,
                            const int32_t* depth, int32_t prefix_len, const int32_t* prefix_len_dev,
                            double rope_theta, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                            void* q_out, void* k_cache, void* v_cache, int64_t cap, void* workspace,
                            size_t ws_bytes, void* stream);

/*
 * ooo_qk_norm_rope - queries of the trie nodes and their keys/values in the
 * cache (Section 4.5: one forward pass over the tree).  Node i takes the
 * rotary position P + depth[i], the position sequential decoding of its own
 * root path would give it; its key and value go to cache row P + i, where
 * ooo_tree_attn reads them.
 *
 * DEVICE pointers; asynchronous on `stream`.
 *   qkv       [n_nodes][(n_q_heads + 2 n_kv_heads) head_dim] bf16: the fused
 *             projection, q heads, then k heads, then v heads
 *   q_norm, k_norm   [head_dim] bf16 per-head RMSNorm weights of q and k
 *             (Qwen3), or NULL for no norm
 *   depth     [n_nodes] int32 (the packed trie's depths)
 *   prefix_len P; prefix_len_dev as for ooo_tree_attn (NULL, or the device
 *             prefix length that prefix_len bounds)
 *   q_out     [n_nodes][n_q_heads][head_dim] bf16
 *   k_cache, v_cache   one layer, [n_kv_heads][cap][head_dim] bf16; rows
 *             P .. P + n_nodes - 1 are written
 * Rotation: the pair (j, j + head_dim/2) turns by the angle
 * (P + depth[i]) * rope_theta^(-2j/head_dim), computed in double precision.
 * Norms in float32 with epsilon eps.
 * Errors: OOO_ERR_INVALID (null pointers, sizes < 1, P + n_nodes > cap,
 * rope_theta <= 0), OOO_ERR_UNSUPPORTED (head_dim other than 64 or 128),
 * OOO_ERR_HIP.
 */
int ooo_qk_norm_rope(const void* qkv, const void* q_norm, const void* k_norm, float eps,
                     const int32_t* depth, int32_t n_nodes, int32_t prefix_len,
                     const int32_t* prefix_len_dev, double rope_theta,
                     int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, void* q_out,
                     void* k_cache, void* v_cache, int64_t cap, void* stream);

/*
 * ooo_swiglu - out[n][j] = silu(g) * u with g = gate_up[n][j] and
 * u = gate_up[n][intermediate + j] (the target's MLP activation; the fused
 * projection holds the gate rows, then the up rows).
 *
 * DEVICE pointers; asynchronous on `stream`.
 *   gate_up  [n_rows][2 intermediate] float32
 *   out      [n_rows][intermediate] bf16
 * Errors: OOO_ERR_INVALID (null pointers, sizes < 1), OOO_ERR_HIP.
 */
int ooo_swiglu(const float* gate_up, int32_t n_rows, int32_t intermediate, void* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OOO_H */
