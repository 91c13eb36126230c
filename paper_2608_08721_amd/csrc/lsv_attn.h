// Internal interface of the attention kernels (attention.hip).
#pragma once
#include "lsv_device.h"
#include "lsv_internal.h"

namespace lsv {

constexpr int kAttnChunk = 64;  // keys per LDS chunk in the bf16 split-context kernel

// Column of cached position p in a transposed V row: positions are permuted inside each
// aligned block of 32 so that the eight keys one lane feeds to a 16x16x32 MFMA (keys
// 4g..4g+3 and 16+4g..16+4g+3 of the block) are adjacent.
__host__ __device__ inline int v_column(int p) { return LSV_V_COLUMN(p); }

// Element offsets of K(b, h, pos, 0) and V(b, h, pos, 0) within the layer's K block / V block
// and the distance between V's head dimensions; false when the position has no valid page.
// Both modes store 64-position blocks with the kv heads of a block side by side ([nkv][64][hd]
// for K, [nkv][hd][64] for V^T): slab mode gives sequence b the blocks b * capacity / 64 ..
// in order (as if its page table were the identity), paged mode takes them from the page table.
// The attention's workgroups for the kv heads of one block then read neighbouring memory.
LSV_DEV bool kv_locate(const KvLayout& L, int nkv, int hd, int b, int h, int pos, size_t& k_off, size_t& v_off,
                       int& v_stride) {
  if (!L.pages) {
    const size_t blk = (((size_t)b * (L.capacity / kAttnChunk) + pos / kAttnChunk) * nkv + h) * kAttnChunk * hd;
    k_off = blk + (size_t)(pos % kAttnChunk) * hd;
    v_off = blk + v_column(pos % kAttnChunk);
    v_stride = kAttnChunk;
    return true;
  }
  const int blk = pos / kAttnChunk;
  if (pos < 0 || blk >= L.max_pages) return false;
  const int page = L.pages[(size_t)b * L.max_pages + blk];
  if (page < 0 || page >= L.n_pages) return false;
  const size_t base = ((size_t)page * nkv + h) * kAttnChunk * hd;
  k_off = base + (size_t)(pos % kAttnChunk) * hd;
  v_off = base + v_column(pos % kAttnChunk);
  v_stride = kAttnChunk;
  return true;
}

// Elements of one layer's K block (the V block follows it).
__host__ __device__ inline size_t kv_layer_block(const KvLayout& L, int batch, int nkv, int hd) {
  return L.pages ? (size_t)L.n_pages * nkv * kAttnChunk * hd : (size_t)batch * nkv * (size_t)L.capacity * hd;
}

struct AttnArgs {
  const void* q;  // [M][nq][hd] storage type
  const void* k;  // this layer's K block: [batch][capacity / 64][nkv][64][hd] (paged: [n_pages][nkv][64][hd])
  const void* v;  // this layer's V block: [batch][capacity / 64][nkv][hd][64], columns by
                  // v_column() (paged: [n_pages][nkv][hd][64])
  KvLayout kv;
  int capacity, ctx_limit, batch, nq, nkv, M_max;
  const int32_t* row_offsets;
  const int32_t* seq_len;
  float* o_part;   // [n_splits][M_max][nq][hd]  (bf16 path)
  float* ml_part;  // [n_splits][M_max][nq][2]: running max (log2 units), sum of exponentials
  void* out;       // nq*hd columns per row in the activation layout (act_index), storage type
  float scale_log2;
  int n_splits, chunks_per_split;
  // packed grid (a 1-D grid of n_splits * nkv * batch workgroups): workgroup i takes the i-th
  // (sequence, kv head, split) that holds keys instead of blockIdx = (split, kv head, sequence)
  int packed;
  // tree blocks: [M_max][kAncWords] ancestor-or-self masks; a block key (position >= the
  // cached length C) at slot C + j is visible to row m iff bit j of its mask is set.  NULL:
  // the causal block.
  const uint32_t* anc;
};

// Split of the context into n_splits ranges of chunks_per_split chunks (bf16 path); packed:
// the split kernel runs on a packed grid (AttnArgs::packed).
struct AttnPlan {
  int n_splits, chunks_per_split, packed;
};
AttnPlan plan_attention(int batch, int nkv, int max_ctx);

int launch_attention(int dtype, int hd, const AttnArgs& a, int max_rows, hipStream_t st);

}  // namespace lsv
