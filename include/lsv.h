/*
 * lsv.h -- C-ABI of the LibraSpec verification hot path on AMD MI355X (gfx950).
 *
 * LibraSpec (arXiv 2608.08721) decodes with a diffusion drafter and a target
 * model.  Each round (Sec. 3.1, Algorithm 1):
 *   1. lsv_select_length  -- choose how many drafted tokens to verify from the
 *      drafter's confidences (Sec. 3.2-3.4);
 *   2. lsv_verify_block   -- one target forward pass over the drafted block,
 *      giving the target distribution at every drafted position (Sec. 3.1);
 *   3. lsv_accept         -- compare draft and target, keep the accepted prefix
 *      and emit one corrected or bonus token (Sec. 3.1).
 * Around them: lsv_verify_tree / lsv_accept_tree / lsv_commit_tree (blocks whose drafts
 * form a tree), lsv_select_joint (one length allocation for a whole batch),
 * lsv_next_length_g4 (the G4-style baseline rule of the comparison experiments),
 * and lsv_pack_block / lsv_next_roots, which carry tokens from one round to the
 * next on the device.
 *
 * Conventions for every entry point
 *   - All buffers are caller-owned.  "d_" arguments are device pointers, all
 *     other pointers are host pointers.  The library never allocates device
 *     memory; scratch space comes from a caller-provided workspace.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = default stream),
 *     perform no host<->device copies and no synchronisation, and may be
 *     captured in a HIP graph.  Per-round shapes live in device arrays
 *     (row offsets, cached lengths); host integers are upper bounds.
 *   - Host-side argument checks run before any HIP call; a failed check returns
 *     LSV_ERR_INVALID_ARG (or LSV_ERR_UNSUPPORTED) and launches nothing.
 *     lsv_last_error() then describes the failure (thread-local).
 *   - Problems only the device can see (a token id out of range, a cache slab
 *     overflow, non-finite logits or confidences) are reported per sequence in
 *     a d_status array; that sequence's outputs are then unspecified but no
 *     memory outside the documented buffers is touched.
 *   - A workspace must not be shared by calls that may run concurrently.
 */
#ifndef LSV_H
#define LSV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ status */
enum {
  LSV_OK = 0,
  LSV_ERR_INVALID_ARG = -1,
  LSV_ERR_UNSUPPORTED = -2,
  LSV_ERR_HIP = -3,
  LSV_ERR_CAPACITY = -4,
  LSV_ERR_NONFINITE = -5
};

/* Static description of a status code. */
const char* lsv_status_string(int status);
/* Detail of the last failing call on this host thread ("" if none). */
const char* lsv_last_error(void);
/* ABI version: bumped whenever a signature or a documented layout changes. */
int lsv_abi_version(void);

/* ------------------------------------------------------------------ model */
enum { LSV_DTYPE_F32 = 0, LSV_DTYPE_BF16 = 1 };

/* Pre-norm decoder of the Llama family: RMSNorm, rotary position embedding
 * (rotate-half pairs (i, i + head_dim/2), angle = pos * rope_base^(-2i/head_dim)),
 * SwiGLU feed-forward, grouped-query attention where query head h reads kv head
 * h / (n_q_heads / n_kv_heads).  No biases; untied LM head.
 * dtype is the storage and matrix-operand type of weights, KV cache and
 * activations between kernels; residual stream, softmax and logits are fp32.
 * Supported: head_dim in {64, 128}; n_q_heads % n_kv_heads == 0;
 * d_model % 64 == 0, d_model <= 8192; every packed projection, the LM head
 * included, below 4 GiB (vocab < 262,144 at d_model 8192 in bf16: the kernels
 * address each with 32-bit byte offsets); rope applies to q and k. */
typedef struct lsv_model_config {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t d_ff;
  int32_t vocab;
  int32_t dtype;     /* LSV_DTYPE_F32 | LSV_DTYPE_BF16 */
  float rms_eps;     /* RMSNorm epsilon, e.g. 1e-5 */
  float reserved0;   /* must be 0 */
  double rope_base;  /* e.g. 10000.0 */
} lsv_model_config;

/* --------------------------------------------------------- packed weights */
/* The forward pass reads weights from one device buffer in a library-defined
 * layout ("packed"): each projection is cut into 16-row x (32 bf16 | 16 fp32)
 * fragments stored contiguously in the order the matrix cores consume them,
 * zero-padded to whole fragments.  Packing is a one-time re-layout (not part of
 * a verify step) from the usual row-major [out_features, in_features] matrices
 * (torch.nn.Linear.weight layout) in the model dtype.
 *
 * lsv_packed_model_bytes: size of the packed buffer for `cfg` (0 if cfg is
 * invalid).  lsv_pack_globals / lsv_pack_layer: write the embedding table
 * [vocab, d_model], the final norm gain [d_model] and the LM head
 * [vocab, d_model], respectively one layer's projections and norm gains, into
 * d_packed.  The projections are stored unchanged; each RMSNorm gain is stored
 * beside them in fp32, and the forward pass forms every projection's input as
 * a = R(h / sqrt(mean(h^2) + rms_eps) * g), rounded to the model dtype once, after
 * the gain (the normalised activation of the model's definition).  Source pointers
 * are device pointers in the model dtype; they may be freed once the stream has
 * passed the call.  Layers may be packed in any order. */
size_t lsv_packed_model_bytes(const lsv_model_config* cfg);
int lsv_pack_globals(const lsv_model_config* cfg, const void* d_embed, const void* d_final_norm,
                     const void* d_lm_head, void* d_packed, void* stream);
int lsv_pack_layer(const lsv_model_config* cfg, int32_t layer,
                   const void* d_wq,   /* [n_q_heads*head_dim, d_model]  */
                   const void* d_wk,   /* [n_kv_heads*head_dim, d_model] */
                   const void* d_wv,   /* [n_kv_heads*head_dim, d_model] */
                   const void* d_wo,   /* [d_model, n_q_heads*head_dim]  */
                   const void* d_wg,   /* [d_ff, d_model] */
                   const void* d_wu,   /* [d_ff, d_model] */
                   const void* d_wd,   /* [d_model, d_ff] */
                   const void* d_attn_norm, const void* d_ffn_norm, /* [d_model] */
                   void* d_packed, void* stream);

/* ---------------------------------------------------------------- KV cache */
/* One device buffer in the model dtype.  For layer l the K block precedes the V
 * block; each holds batch x capacity / 64 blocks of 64 positions, and a block holds
 * the n_kv_heads heads side by side (the same layout as a page of the paged cache
 * below, the blocks of sequence b being its pages in order):
 *   blk(l, kv, b, p, h) = ((((l * 2 + kv) * batch + b) * (capacity / 64) + p) * n_kv_heads + h)
 *                         * 64 * head_dim
 * with kv = 0 for K and 1 for V, p = pos / 64 and j = pos % 64.
 *   K (after the rotary embedding) is row-major [64][head_dim] per block and head:
 *     K(l, b, h, pos, i) at blk(l, 0, b, p, h) + j * head_dim + i
 *   V is transposed, [head_dim][64] per block and head, with positions permuted inside
 *   each aligned run of 32 so that the keys one matrix-core lane consumes are adjacent:
 *     V(l, b, h, pos, i) at blk(l, 1, b, p, h) + i * 64 + LSV_V_COLUMN(j)
 * Sequence b owns `capacity` positions; d_seq_len[b] of them are valid.  capacity must
 * be a positive multiple of LSV_KV_ALIGN (lsv_kv_cache_bytes returns 0 and
 * lsv_verify_block LSV_ERR_INVALID_ARG otherwise). */
enum { LSV_KV_ALIGN = 64, LSV_KV_PAGE = 64 };
#define LSV_V_COLUMN(pos) (((pos) & ~31) | (((pos) & 12) << 1) | (((pos) & 16) >> 2) | ((pos) & 3))
size_t lsv_kv_cache_bytes(const lsv_model_config* cfg, int32_t batch, int32_t capacity);

/* Paged KV cache, for serving many sequences of changing lengths from one pool (the
 * joint batched selection, lsv_select_joint, hands a batch lengths that vary per round and
 * sequence).  One device buffer in the model dtype: per layer a K pool then a V pool, each
 * of n_pages pages of LSV_KV_PAGE positions for every kv head:
 *   pool(l, kv) = (l * 2 + kv) * n_pages * n_kv_heads * LSV_KV_PAGE * head_dim
 *   K(l, page, h, j, i) at pool(l, 0) + ((page * n_kv_heads + h) * LSV_KV_PAGE + j) * head_dim + i
 *   V(l, page, h, j, i) at pool(l, 1) + ((page * n_kv_heads + h) * head_dim + i) * LSV_KV_PAGE
 *                                     + LSV_V_COLUMN(j)
 * i.e. a page is laid out like a block of the slab cache above.  Position pos of sequence b lives in page
 * d_page_table[b * max_pages + pos / 64] at j = pos % 64; a table entry outside
 * [0, n_pages) reads as zeros and is never written.  The caller owns the pool and the table
 * (any page order; pages need not be contiguous).  A layer's K pool must stay under 2 GiB
 * ((n_pages + 1) * n_kv_heads * 64 * head_dim * element size < 2^31).
 * lsv_kv_pool_bytes: size of the buffer (0 if cfg is invalid). */
size_t lsv_kv_pool_bytes(const lsv_model_config* cfg, int32_t n_pages);

/* ------------------------------------------------------------ verify step */
/* Workspace for lsv_verify_block with the given bounds.  The workspace must be
 * zero-filled once after allocation (e.g. with lsv_workspace_clear): the padding
 * columns of its activation buffers are never written and must read as zero.  It
 * carries no state from one call to the next, and a workspace sized for the largest
 * bounds serves calls with any smaller batch, max_rows or max_ctx. */
size_t lsv_verify_workspace_bytes(const lsv_model_config* cfg, int32_t batch, int32_t max_rows,
                                  int32_t max_ctx);
int lsv_workspace_clear(void* d_workspace, size_t workspace_bytes, void* stream);

/* One forward pass of the target over a block of rows per sequence
 * (Sec. 3.1: all drafted positions are scored in parallel in one pass).
 *
 * Rows: sequence b owns rows d_row_offsets[b] .. d_row_offsets[b+1]-1 of
 * d_tokens; in a verify step they are [root, x_1, ..., x_g] where root is the
 * pending token emitted by the previous round and x_v are drafts.  Row r of
 * sequence b sits at position d_seq_len[b] + (r - d_row_offsets[b]); its K/V
 * are written to those cache positions, and it attends to cache positions
 * 0 .. its own position (causal).  d_seq_len is NOT modified (lsv_accept
 * commits).  The same call with d_seq_len[b] = 0 and the prompt as the block
 * is a prefill; long prompts may be fed in chunks.
 *
 *   cfg, d_packed      model and its packed weights
 *   d_kv, capacity     KV cache (layout above) with `capacity` positions per sequence,
 *                      capacity % LSV_KV_ALIGN == 0 and a sequence's share of a layer's
 *                      K block under 2 GiB (n_kv_heads * capacity * head_dim * element
 *                      size < 2^31)
 *   batch              number of sequences (1..LSV_MAX_BATCH)
 *   d_seq_len          [batch] int32, cached positions before this block
 *   d_tokens           [rows] int32 token ids
 *   d_row_offsets      [batch+1] int32, non-decreasing, d_row_offsets[0] = 0; a sequence
 *                      may have no rows (it is left untouched; status LSV_OK)
 *   max_rows           host bound: d_row_offsets[batch] <= max_rows <= LSV_MAX_ROWS
 *   max_ctx            host bound: d_seq_len[b] + rows_b <= max_ctx <= capacity
 *   d_logits           [max_rows, vocab] fp32 out; rows >= d_row_offsets[batch] untouched
 *   d_status           [batch] int32 out (nullable): LSV_OK, LSV_ERR_INVALID_ARG (token id
 *                      out of range), LSV_ERR_CAPACITY (block exceeds max_ctx)
 *   d_workspace        lsv_verify_workspace_bytes(cfg, batch, max_rows, max_ctx) bytes */
enum { LSV_MAX_BATCH = 64, LSV_MAX_ROWS = 512 };
/* Performance note: bf16 blocks whose host bound max_rows lies in (64, LSV_WIDE_ROWS]
 * run the batched GEMM path (every row in one workgroup, activations shared through
 * LDS, matrix-core bound); other bounds process rows in chunks of 64. */
enum { LSV_WIDE_ROWS = 272 };
int lsv_verify_block(const lsv_model_config* cfg, const void* d_packed, void* d_kv, int32_t capacity,
                     int32_t batch, const int32_t* d_seq_len, const int32_t* d_tokens,
                     const int32_t* d_row_offsets, int32_t max_rows, int32_t max_ctx, float* d_logits,
                     int32_t* d_status, void* d_workspace, size_t workspace_bytes, void* stream);

/* Tree blocks (Sec. 4.3, Table 2: tree drafts such as DDTree, verified in one target pass;
 * Appendix B gives node budgets of 64 to 512).  The same call as lsv_verify_block, except
 * that each sequence's rows form a tree:
 *   d_parents     [rows] int32: the parent of row r as a row index within its sequence's
 *                 block (0-based); the first row of every sequence is the root (the pending
 *                 token) with parent -1, and every other row's parent precedes it.  A
 *                 sequence has at most LSV_MAX_ROWS rows.
 * Row r of sequence b (local index i) is stored at cache slot d_seq_len[b] + i, takes the
 * rotary position d_seq_len[b] + depth(i), and attends to the cached positions below
 * d_seq_len[b] and to the slots of its ancestors and itself.  Its logits are those of a
 * plain block over its root-to-node path.  A sequence whose parents do not form such a
 * tree gets LSV_ERR_INVALID_ARG in d_status.  Workspace: lsv_verify_workspace_bytes. */
int lsv_verify_tree(const lsv_model_config* cfg, const void* d_packed, void* d_kv, int32_t capacity, int32_t batch,
                    const int32_t* d_seq_len, const int32_t* d_tokens, const int32_t* d_row_offsets,
                    const int32_t* d_parents, int32_t max_rows, int32_t max_ctx, float* d_logits, int32_t* d_status,
                    void* d_workspace, size_t workspace_bytes, void* stream);

/* lsv_verify_block (d_parents NULL) or lsv_verify_tree (d_parents given) over a paged KV cache
 * (layout above): the same arguments, rules and results, with d_kv_pool / n_pages /
 * d_page_table / max_pages in place of d_kv / capacity.  Positions per sequence are bounded by
 * max_pages * LSV_KV_PAGE (max_ctx must not exceed it); a block position whose page entry is
 * outside the pool is not written (its keys read as zero). */
int lsv_verify_paged(const lsv_model_config* cfg, const void* d_packed, void* d_kv_pool, int32_t n_pages,
                     const int32_t* d_page_table, int32_t max_pages, int32_t batch, const int32_t* d_seq_len,
                     const int32_t* d_tokens, const int32_t* d_row_offsets, const int32_t* d_parents, int32_t max_rows,
                     int32_t max_ctx, float* d_logits, int32_t* d_status, void* d_workspace, size_t workspace_bytes,
                     void* stream);

/* -------------------------------------------------------------- acceptance */
/* Compare drafts with the target's scores (Sec. 3.1).  Per sequence b with
 * g_b = rows_b - 1 drafts, row v of the block scores draft x_{v+1}.
 *
 * LSV_ACC_GREEDY (temperature 0): argmax = smallest index of the row maximum;
 *   a_b = longest prefix with argmax(row v-1) == x_v; emitted tokens are
 *   x_1..x_{a_b} followed by argmax(row a_b).
 * LSV_ACC_SAMPLE (temperature T > 0), speculative rejection sampling:
 *   p_v = softmax(logits_v / T); draft v is accepted iff u_v * q_v(x_v) < p_{v-1}(x_v);
 *   at the first rejection the emitted token is drawn from max(0, p_a - q_{a+1})
 *   renormalised (from p_a if that is identically zero); if every draft passes
 *   the bonus token is drawn from p_g.  Draws use the exponential race
 *   argmin_x (-ln U_x) / w_x.  Uniforms come from Philox4x64-10 (Salmon et al.,
 *   SC'11) with U = ((w >> 12) + 0.5) * 2^-52 and
 *     ratio test of draft v:  key (seed, 1), counter (0, v | b << 32, round, 0), word 0
 *     draw from row r:        key (seed, 2), counter (x >> 2, r | b << 32, round, 0), word x & 3.
 *   Draft distributions: d_draft_probs row (d_row_offsets[b] - b + v - 1) is q_v of
 *   sequence b, [*, vocab] fp32.
 *
 *   d_logits           [rows, vocab] fp32 (as written by lsv_verify_block)
 *   max_rows           host bound on d_row_offsets[batch] (<= LSV_MAX_ROWS)
 *   max_rows_per_seq   host bound on rows_b (<= LSV_MAX_SEQ_ROWS: one wave decides a
 *                      sequence); width of d_out_tokens
 *   d_accept_len       [batch] out: a_b
 *   d_out_tokens       [batch, max_rows_per_seq] out: emitted tokens, then -1
 *   d_seq_len          [batch] in/out, nullable: if given, d_seq_len[b] += a_b + 1
 *                      (root and accepted drafts stay cached) for sequences with status OK
 *   d_status           [batch] in/out (nullable).  In: a sequence whose d_status[b] is not
 *                      LSV_OK (e.g. lsv_verify_block's LSV_ERR_CAPACITY for this block) is
 *                      skipped: accept_len 0, out_tokens all -1, no commit, status kept.
 *                      Pass the verify call's status array, or one set to LSV_OK.
 *                      Out: LSV_OK; LSV_ERR_NONFINITE (a non-finite logit in the sequence's
 *                      rows, or a non-finite draft probability read); LSV_ERR_INVALID_ARG if
 *                      the sequence has no rows or more than max_rows_per_seq (sampling: then
 *                      every sequence of the batch that arrived OK), or the rows run past
 *                      max_rows
 *   d_workspace        lsv_accept_workspace_bytes(batch, max_rows, vocab) bytes */
enum { LSV_ACC_GREEDY = 0, LSV_ACC_SAMPLE = 1 };
enum { LSV_MAX_SEQ_ROWS = 64 };
size_t lsv_accept_workspace_bytes(int32_t batch, int32_t max_rows, int32_t vocab);
int lsv_accept(int32_t mode, int32_t batch, int32_t vocab, const float* d_logits,
               const int32_t* d_row_offsets, int32_t max_rows, int32_t max_rows_per_seq,
               const int32_t* d_tokens, const float* d_draft_probs, float temperature, uint64_t seed,
               uint64_t round, int32_t* d_accept_len, int32_t* d_out_tokens, int32_t* d_seq_len,
               int32_t* d_status, void* d_workspace, size_t workspace_bytes, void* stream);

/* lsv_accept without a caller workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops or harnesses that forbid allocation).  Same
 * arguments, rules and outputs as lsv_accept.  Its scratch lives in a device array that the
 * library owns: LSV_ACCEPT_NOALLOC_BYTES per GPU, held until the process ends; nothing is
 * allocated per call.  A call whose lsv_accept_workspace_bytes(batch, max_rows, vocab)
 * exceeds that returns LSV_ERR_UNSUPPORTED and launches nothing (e.g. 512 rows fit up to a
 * vocabulary of about 190K entries).  Every call on one GPU uses the same array: calls that
 * may overlap on one GPU (other streams, other threads) race and must not be issued. */
enum { LSV_ACCEPT_NOALLOC_BYTES = 512 * 1024 };
int lsv_accept_noalloc(int32_t mode, int32_t batch, int32_t vocab, const float* d_logits,
                       const int32_t* d_row_offsets, int32_t max_rows, int32_t max_rows_per_seq,
                       const int32_t* d_tokens, const float* d_draft_probs, float temperature, uint64_t seed,
                       uint64_t round, int32_t* d_accept_len, int32_t* d_out_tokens, int32_t* d_seq_len,
                       int32_t* d_status, void* stream);

/* Greedy acceptance of tree blocks (after lsv_verify_tree): a node is accepted with its
 * parent when its token is the argmax of the parent's row (first index of the maximum); the
 * accepted path runs from the root to the deepest node whose ancestors below the root are all
 * accepted (the smallest node index among equally deep ones), i.e. the longest root-to-node
 * path that greedy acceptance of a chain would keep.  With a = its depth:
 *   d_accept_len  [batch] out: a
 *   d_out_tokens  [batch, width] out: the tokens of the path's nodes at depths 1..a, then the
 *                 argmax of the last node's row, then -1
 *   d_path        [batch, width] out: the node (row index within the block) at depth
 *                 0..a, then -1
 *   d_seq_len     [batch] in/out, nullable: += a + 1 for sequences with status OK
 *   d_status      [batch] in/out, nullable: as for lsv_accept (an incoming error skips the
 *                 sequence); out: LSV_OK, LSV_ERR_NONFINITE, or LSV_ERR_INVALID_ARG (invalid
 *                 parents, rows outside [1, LSV_MAX_ROWS] or past max_rows, a path of more
 *                 than width - 1 drafts)
 *   width         1..LSV_MAX_SEQ_ROWS;  d_workspace: lsv_accept_workspace_bytes(batch, max_rows, vocab)
 * lsv_commit_tree then moves each accepted path's K and V to consecutive positions: with
 * C = d_seq_len[b] - a - 1 (call it after lsv_accept_tree committed d_seq_len), the node at
 * depth k moves from slot C + d_path[b, k] to position C + k, k = 1..a, in every layer and kv
 * head, so that the cache holds what a plain block over the path would have written (the
 * rotary position of that node was already C + k).  Sequences whose status is not LSV_OK are
 * left alone.  One launch. */
int lsv_accept_tree(int32_t batch, int32_t vocab, const float* d_logits, const int32_t* d_row_offsets,
                    const int32_t* d_parents, const int32_t* d_tokens, int32_t max_rows, int32_t width,
                    int32_t* d_accept_len, int32_t* d_out_tokens, int32_t* d_path, int32_t* d_seq_len,
                    int32_t* d_status, void* d_workspace, size_t workspace_bytes, void* stream);
int lsv_commit_tree(const lsv_model_config* cfg, void* d_kv, int32_t capacity, int32_t batch, const int32_t* d_seq_len,
                    const int32_t* d_accept_len, const int32_t* d_path, int32_t width, const int32_t* d_status,
                    void* stream);
/* The same commit on a paged KV cache (layout above). */
int lsv_commit_tree_paged(const lsv_model_config* cfg, void* d_kv_pool, int32_t n_pages, const int32_t* d_page_table,
                          int32_t max_pages, int32_t batch, const int32_t* d_seq_len, const int32_t* d_accept_len,
                          const int32_t* d_path, int32_t width, const int32_t* d_status, void* stream);

/* -------------------------------------------------------- length selection */
/* Choose the speculative length gamma_b per sequence from drafter confidences
 * q_1..q_G (Assumption 3.7 uses them in place of the target's acceptance
 * probabilities).  All arithmetic is binary64, one rounding per operation, in
 * the order below (no fused multiply-add):
 *   P_j = P_{j-1} * q_j (P_0 = 1);  N(d) = [BONUS] + sum_{j<=d} P_j;  f(d) = N(d) / cost[d]
 *   (Eq. 2, the simplified speedup objective, up to a constant).
 * LSV_SEL_EXHAUSTIVE: smallest d in [1, d_max] maximising f.
 * LSV_SEL_MARGINAL:   from d = clamp(d_init, 1, d_max), repeat single beneficial
 *   adjustments (Def. 3.1): d += 1 while f(d+1) > f(d), else d -= 1 while
 *   f(d-1) >= f(d).  By Thm. 3.5/3.6 this reaches the EXHAUSTIVE answer when the
 *   cost table is convex.  aux = number of steps.
 * LSV_SEL_ALG1: Algorithm 1 with block size n = block_n and trade-off alpha.  With
 *   eps*(d) = min_{i<=d} floor(alpha * S_i + i), S_i = sum_{j=i}^{d} prod_{k=i}^{j} q_k
 *   (the position-wise bounds of Thm. 3.3 over the current length d), the length starts
 *   at min(n, d_max), climbs to min(eps*(d), d_max) while eps*(d) > d, and settles on
 *   eps*(d) at the first d where eps*(d) <= d (the single rollback); d_max also stops it.
 *   cost is not read.  aux = drafter blocks of n used: ceil(d_peak / n), d_peak the
 *   highest length reached (Algorithm 1's budget of drafted but unused tokens).
 *   With LSV_SEL_DRAFTED (blocks on demand) d_aux is in/out: in, the blocks of n drafted
 *   so far for the sequence (>= 1); only the first min(aux * n, G) confidences are read.
 *   When the length reaches past them (the budget goes negative) the rule stops with
 *   gamma = 0 and aux = ceil(d / n), the blocks it needs before it is run again; run
 *   again with those blocks it takes the same steps, so after at most ceil(d_max / n)
 *   calls it ends where the rule over all G confidences ends, with the same aux.
 *
 *   d_conf   [batch, G] fp32 confidences in [0, 1]
 *   d_cost   [G+1] fp64 verification cost of each length, cost[0] unused; cost[d] > 0
 *            for d <= d_max (MARGINAL / EXHAUSTIVE; may be NULL for ALG1)
 *   flags    LSV_SEL_BONUS: count the always-emitted token in N(d);
 *            LSV_SEL_DRAFTED: ALG1 with blocks on demand (above; needs d_aux)
 *   d_gamma  [batch] out (0: more blocks needed, LSV_SEL_DRAFTED only);
 *            d_aux [batch] out (nullable; in/out with LSV_SEL_DRAFTED)
 *   d_row_offsets [batch+1] out (nullable; needs batch <= LSV_MAX_BATCH): the row layout of
 *            the verify block that follows, row_offsets[0] = 0 and
 *            row_offsets[b+1] = row_offsets[b] + gamma_b + 1 (root plus gamma_b drafts), so
 *            select -> verify -> accept can run without a host round trip
 *   d_status [batch] out (nullable): LSV_OK, or LSV_ERR_INVALID_ARG when a confidence is
 *            outside [0, 1], a needed cost is not finite and positive, or (LSV_SEL_DRAFTED)
 *            the blocks drafted are fewer than one (then gamma = 0). */
enum { LSV_SEL_MARGINAL = 0, LSV_SEL_EXHAUSTIVE = 1, LSV_SEL_ALG1 = 2 };
enum { LSV_SEL_BONUS = 1, LSV_SEL_DRAFTED = 2 };
enum { LSV_MAX_G = 64 };
int lsv_select_length(int32_t mode, int32_t batch, int32_t G, const float* d_conf, const double* d_cost,
                      int32_t d_init, int32_t d_max, double alpha, int32_t block_n, uint32_t flags,
                      int32_t* d_gamma, int32_t* d_aux, int32_t* d_row_offsets, int32_t* d_status,
                      void* stream);

/* Joint batched selection: gamma_b in [1, d_max] for every sequence at once, maximising
 *   F(gamma) = sum_b N_b(gamma_b) / cost[R],  R = sum_b gamma_b,
 * the objective of Eq. 2 (expected accepted tokens per unit of verify time) over a batch
 * whose verify cost is shared.  The paper gives only the per-sequence rule; this batch
 * form is the library's extension.  N_b as for lsv_select_length (binary64, same order).
 * For each R the best allocation gives every sequence one draft and then the R - batch
 * largest increments P_{b,j}, j >= 2 (N_b has non-increasing increments), ties to the
 * smaller b, then the smaller j; F(R) sums N_b(gamma_b) over b in order; the smallest R
 * with the largest F wins.
 *
 *   d_conf        [batch, G] fp32 confidences in [0, 1]
 *   d_cost        [batch * d_max + 1] fp64: cost[R] = verify cost of a batch with R drafts in
 *                 total (root rows included in the cost); entries R < batch are not read;
 *                 entries R in [batch, batch * d_max] must be finite and > 0
 *   flags         LSV_SEL_BONUS as for lsv_select_length
 *   d_gamma       [batch] out;  d_total [1] out (nullable): R
 *   d_row_offsets [batch+1] out (nullable): row_offsets[b+1] = row_offsets[b] + gamma_b + 1
 *   d_status      [batch] out (nullable): LSV_OK, or LSV_ERR_INVALID_ARG for every sequence
 *                 when a confidence or a needed cost is invalid (then gamma = 0, R = 0 and
 *                 the row offsets give each sequence its root row only)
 * Host errors: batch outside [1, LSV_MAX_BATCH], G outside [1, LSV_MAX_G], d_max outside
 * [1, G], unknown flags, NULL d_conf / d_cost / d_gamma.  One workgroup on the caller's stream. */
int lsv_select_joint(int32_t batch, int32_t G, const float* d_conf, const double* d_cost, int32_t d_max,
                     uint32_t flags, int32_t* d_gamma, int32_t* d_total, int32_t* d_row_offsets, int32_t* d_status,
                     void* stream);

/* ------------------------------------------------------------ round plumbing */
/* Decoding runs in rounds (Sec. 3.1): each verifies the token emitted last (the root)
 * followed by the round's drafts, and emits the accepted drafts plus one token, which is
 * the next round's root.  These two calls carry tokens between the steps on the device,
 * so that select -> pack -> verify -> accept -> next roots needs no host round trip.
 *
 * lsv_pack_block: the verify block's token array from the row layout that
 *   lsv_select_length (or lsv_next_length_g4) wrote: for sequence b, row r0 = row_offsets[b]
 *   gets d_roots[b] and rows r0 + k, k = 1..rows_b - 1, get d_drafts[b * G + k - 1].
 *   d_row_offsets  [batch+1] in (device-written)
 *   max_rows       host bound: no row at or past it is written; d_tokens holds max_rows
 *   d_roots        [batch] in;  d_drafts [batch, G] in (may be NULL when G = 0)
 *   d_tokens       [max_rows] out
 *   d_status       [batch] out, nullable: LSV_OK, or LSV_ERR_INVALID_ARG when the
 *                  sequence's rows are empty, past max_rows or more than G + 1 (then none
 *                  of its rows is written)
 *   Host errors: batch outside [1, LSV_MAX_BATCH], G outside [0, LSV_MAX_SEQ_ROWS - 1],
 *   max_rows outside [1, LSV_MAX_ROWS], NULL pointers.
 * lsv_next_roots: d_roots[b] = d_out_tokens[b * width + d_accept_len[b]] (lsv_accept's
 *   outputs with max_rows_per_seq = width); a sequence whose status is not LSV_OK, or whose
 *   accept_len is outside [0, width), keeps its root.  d_status nullable.
 *   Host errors: batch < 1, width outside [1, LSV_MAX_SEQ_ROWS], NULL pointers. */
int lsv_pack_block(int32_t batch, int32_t G, const int32_t* d_row_offsets, int32_t max_rows, const int32_t* d_roots,
                   const int32_t* d_drafts, int32_t* d_tokens, int32_t* d_status, void* stream);
int lsv_next_roots(int32_t batch, const int32_t* d_accept_len, const int32_t* d_out_tokens, int32_t width,
                   const int32_t* d_status, int32_t* d_roots, void* stream);

/* Baseline length policy of the comparison experiments (Sec. 4.1; Appendix B,
 * baseline details: the dynamic-length rule adapted from Gemma 4's multi-token
 * prediction, "G4-style").  From the round just verified, where sequence b drafted
 * gamma_b tokens and accepted a_b of them (lsv_accept's d_accept_len):
 *   raw_b = gamma_b + 2  if a_b == gamma_b (no draft rejected),
 *           gamma_b - 1  otherwise;
 *   gamma_next_b = min(max(raw_b, d_min), d_max).
 * The rule states no bounds; the clamp to [d_min, d_max] is this library's reading.
 * A sequence whose round failed (d_status[b] != LSV_OK) has no outcome: raw_b = gamma_b.
 * A record outside 0 <= gamma_b < LSV_MAX_SEQ_ROWS, or (round OK) 0 <= a_b <= gamma_b,
 * restarts at d_min and is flagged in d_err.
 *
 *   d_gamma        [batch] int32 in: this round's gamma_b
 *   d_accept_len   [batch] int32 in: a_b
 *   d_status       [batch] int32 in, nullable: lsv_accept's status per sequence
 *   d_min, d_max   1 <= d_min <= d_max <= LSV_MAX_SEQ_ROWS - 1 (the next block must fit
 *                  lsv_accept's one-wave limit)
 *   d_gamma_next   [batch] out; may be the same buffer as d_gamma
 *   d_row_offsets  [batch+1] out, nullable (needs batch <= LSV_MAX_BATCH): the next verify
 *                  block's layout, row_offsets[b+1] = row_offsets[b] + gamma_next_b + 1
 *   d_err          [batch] out, nullable: LSV_OK or LSV_ERR_INVALID_ARG (see above)
 * Returns LSV_ERR_INVALID_ARG (nothing launched) for batch < 1, bounds outside the range
 * above, NULL d_gamma / d_accept_len / d_gamma_next, or row offsets with batch > LSV_MAX_BATCH.
 * One launch of one wave on the caller's stream. */
int lsv_next_length_g4(int32_t batch, const int32_t* d_gamma, const int32_t* d_accept_len, const int32_t* d_status,
                       int32_t d_min, int32_t d_max, int32_t* d_gamma_next, int32_t* d_row_offsets, int32_t* d_err,
                       void* stream);

/* ------------------------------------------------------------- measurement */
/* Kernel classes of lsv_verify_block, one launch per layer each (LM head once). */
enum {
  LSV_KERNEL_QKV = 0,
  LSV_KERNEL_O = 1,
  LSV_KERNEL_GATEUP = 2,
  LSV_KERNEL_DOWN = 3,
  LSV_KERNEL_LMHEAD = 4,
  LSV_KERNEL_ATTENTION = 5
};
/* While set (n_slots > 0), every lsv_verify_block records events[2i] just before
 * and events[2i+1] just after the i-th launch of kernel class `kernel` in that call
 * (i < n_slots), on the call's stream, with hipEventRecordWithFlags(record_flags):
 * pass hipEventRecordExternal (1) while capturing a graph so the records become
 * graph nodes, 0 otherwise.  `events` is a host array of 2 * n_slots hipEvent_t
 * created by the caller with timing enabled; the array is copied.  n_slots = 0
 * clears the hook.  Process-wide setting; set it while no other thread calls the
 * library. */
enum { LSV_MAX_TIMING_SLOTS = 256 };
int lsv_set_timing_events(int32_t kernel, void* const* events, int32_t n_slots, uint32_t record_flags);

#ifdef __cplusplus
}
#endif
#endif /* LSV_H */
