// Internal host/device declarations of liblsv (not part of the public ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "lsv.h"

namespace lsv {

// ---------------------------------------------------------------- selector
int launch_select(int mode, int batch, int G, const float* conf, const double* cost, int d_init, int d_max,
                  double alpha, int block_n, unsigned flags, int32_t* gamma, int32_t* aux, int32_t* row_offsets,
                  int32_t* status, hipStream_t stream);
int launch_select_joint(int batch, int G, const float* conf, const double* cost, int d_max, unsigned flags,
                        int32_t* gamma, int32_t* total, int32_t* row_offsets, int32_t* status, hipStream_t stream);
int launch_next_length_g4(int batch, const int32_t* gamma, const int32_t* accept_len, const int32_t* status,
                          int d_min, int d_max, int32_t* gamma_next, int32_t* row_offsets, int32_t* err,
                          hipStream_t stream);

// ---------------------------------------------------------------- rounds
int launch_pack_block(int batch, int G, const int32_t* row_offsets, int max_rows, const int32_t* roots,
                      const int32_t* drafts, int32_t* tokens, int32_t* status, hipStream_t stream);
int launch_next_roots(int batch, const int32_t* accept_len, const int32_t* out_tokens, int width,
                      const int32_t* status, int32_t* roots, hipStream_t stream);

// measurement hook (lsv_set_timing_events): called around each launch of a kernel class
void timing_before(int kernel, int index, hipStream_t st);
void timing_after(int kernel, int index, hipStream_t st);

// ---------------------------------------------------------------- accept
constexpr int kAcceptChunk = 4096;  // vocabulary entries per workgroup in the row scans
inline int accept_chunks(int vocab) { return (vocab + kAcceptChunk - 1) / kAcceptChunk; }
size_t accept_workspace_bytes(int batch, int max_rows, int vocab);
constexpr size_t kAcceptStaticBytes = LSV_ACCEPT_NOALLOC_BYTES;  // lsv_accept_noalloc's scratch per GPU
int accept_scratch(void** out);  // that scratch on the current device (looked up once per device)
int launch_accept(int mode, int batch, int vocab, const float* logits, const int32_t* row_offsets, int max_rows,
                  int max_rows_per_seq, const int32_t* tokens, const float* draft_probs, float temperature,
                  uint64_t seed, uint64_t round, int32_t* accept_len, int32_t* out_tokens, int32_t* seq_len,
                  int32_t* status, void* ws, hipStream_t stream);

// ---------------------------------------------------------------- forward
struct Shape {
  int L, d, nq, nkv, hd, F, V, dtype, es;  // es = element size of the storage type
  float eps;
  double rope_base;
};
Shape shape_of(const lsv_model_config* c);

// Packed matrix = fragments of 16 rows x KT columns (KT = 32 bf16 / 16 fp32), 1 KiB each.
struct PackedMat {
  size_t offset;  // byte offset in the packed model buffer
  int N, K;       // logical rows (out features) and columns (in features)
  int Nt, Kt;     // fragment counts (zero-padded)
};

// Fragment order of a packed matrix: the k range is cut into blocks of kFragBlock
// fragments; block b holds, for every fragment row in turn, that row's fragments of the
// block (the last block may be shorter).  A wave still streams contiguous KiB runs
// (kFragBlock fragments of one row), while the waves of a launch, which advance through
// k at the same pace, keep their concurrent reads within one block: a narrow window of
// DRAM pages instead of one page per fragment row.
constexpr int kFragBlock = 8;
__host__ __device__ inline size_t frag_index(int tn, int k, int Nt, int Kt) {
  const int b = k / kFragBlock, k0 = b * kFragBlock;
  const int bs = Kt - k0 < kFragBlock ? Kt - k0 : kFragBlock;  // size of block b
  return (size_t)k0 * Nt + (size_t)tn * bs + (k - k0);
}
// Activation operand layout (the B side of every projection): rows in tiles of 16, columns
// in k-steps of KT (32 bf16 or 16 fp32 columns, EPL = KT / 4 per lane).  The 16 x KT block
// of one (row tile, k-step) is one contiguous KiB in the lane order of the MFMA B operand:
// lane g * 16 + r holds row r, columns g * EPL .. g * EPL + EPL - 1.  A buffer of K columns
// has Kt = ceil(K / KT) k-steps per row tile (columns past K stay zero); a wave's activation
// load is then one contiguous KiB, as its weight loads are.
template <int KT>
__host__ __device__ inline size_t act_index(int m, int c, int Kt) {
  constexpr int EPL = KT / 4;
  return ((((size_t)(m >> 4) * Kt + c / KT) * 4 + (c % KT) / EPL) * 16 + (m & 15)) * EPL + c % EPL;
}
// Elements of an activation buffer of `rows` rows and K columns.
template <int KT>
__host__ __device__ inline size_t act_elems(int rows, int K) {
  return (size_t)((rows + 15) / 16) * 16 * (size_t)((K + KT - 1) / KT) * KT;
}

// RMSNorm gains are kept in fp32 beside the projections: the row-normalisation kernel
// applies them before the activation is rounded to the storage type.
struct ModelLayout {
  size_t embed;                     // raw row-major embedding [V, d]
  size_t final_norm;                // fp32 [d]
  PackedMat lm_head;
  size_t layer_base, layer_stride;  // per-layer block
  size_t attn_norm, ffn_norm;       // fp32 [d] each, offsets inside a layer block
  PackedMat qkv, o, gateup, down;   // offsets inside a layer block
  size_t total;
};
ModelLayout model_layout(const Shape& s);

enum PackKind { PACK_PLAIN = 0, PACK_QKV = 1, PACK_GATEUP = 2 };
int launch_pack(const Shape& s, PackKind kind, const PackedMat& pm, const void* src0, const void* src1,
                const void* src2, void* dst, hipStream_t stream);
// A norm gain [d] in the storage type -> fp32 at dst.
int launch_gain(const Shape& s, const void* src, void* dst, hipStream_t stream);

// Where a layer's cache entries live.  Slab mode (pages == NULL): `capacity` positions per
// sequence, in capacity / 64 consecutive blocks laid out like pages.  Paged mode: a pool of
// n_pages pages of LSV_KV_PAGE positions per layer; sequence b's positions p .. p + 63 (p a
// multiple of 64) are in page pages[b * max_pages + p / 64].
struct KvLayout {
  int capacity;
  const int32_t* pages;
  int max_pages, n_pages;
};

// Tree blocks: up to LSV_MAX_ROWS nodes per sequence; a node's ancestor set is a bit mask
// over its sequence's block rows.
constexpr int kTreeNodes = LSV_MAX_ROWS;
constexpr int kAncWords = kTreeNodes / 32;

size_t verify_workspace_bytes(const Shape& s, int batch, int max_rows, int max_ctx);
// parents: NULL for a chain block (row r's parent is r - 1), else the tree of each sequence's
// block (parent row index within the block, -1 for the root).
int launch_verify(const Shape& s, const ModelLayout& ml, const void* packed, void* kv, const KvLayout& kvl, int batch,
                  const int32_t* seq_len, const int32_t* tokens, const int32_t* row_offsets, const int32_t* parents,
                  int max_rows, int max_ctx, float* logits, int32_t* status, void* ws, size_t ws_bytes,
                  hipStream_t stream);
// Tree acceptance (accept.hip) and the commit of the accepted path's K/V (tree.hip).
int launch_accept_tree(int batch, int vocab, const float* logits, const int32_t* row_offsets, const int32_t* parents,
                       const int32_t* tokens, int max_rows, int width, int32_t* accept_len, int32_t* out_tokens,
                       int32_t* path, int32_t* seq_len, int32_t* status, void* ws, hipStream_t stream);
int launch_commit_tree(const Shape& s, void* kv, const KvLayout& kvl, int batch, const int32_t* seq_len,
                       const int32_t* accept_len, const int32_t* path, int width, const int32_t* status,
                       hipStream_t stream);

}  // namespace lsv
