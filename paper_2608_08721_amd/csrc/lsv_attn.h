// Internal interface of the attention kernels (attention.hip).
#pragma once
#include "lsv_internal.h"

namespace lsv {

constexpr int kAttnChunk = 64;  // keys per LDS chunk in the bf16 split-context kernel

// Column of cached position p in a transposed V row: positions are permuted inside each
// aligned block of 32 so that the eight keys one lane feeds to a 16x16x32 MFMA (keys
// 4g..4g+3 and 16+4g..16+4g+3 of the block) are adjacent.
__host__ __device__ inline int v_column(int p) { return LSV_V_COLUMN(p); }

struct AttnArgs {
  const void* q;  // [M][nq][hd] storage type
  const void* k;  // this layer's K block: [batch][nkv][capacity][hd]
  const void* v;  // this layer's V block: [batch][nkv][hd][capacity], columns by v_column()
  int capacity, ctx_limit, batch, nq, nkv, M_max;
  const int32_t* row_offsets;
  const int32_t* seq_len;
  float* o_part;   // [n_splits][M_max][nq][hd]  (bf16 path)
  float* ml_part;  // [n_splits][M_max][nq][2]: running max (log2 units), sum of exponentials
  void* out;       // nq*hd columns per row in the activation layout (act_index), storage type
  float scale_log2;
  int n_splits, chunks_per_split;
  // tree blocks: [M_max][kAncWords] ancestor-or-self masks; a block key (position >= the
  // cached length C) at slot C + j is visible to row m iff bit j of its mask is set.  NULL:
  // the causal block.
  const uint32_t* anc;
};

// Split of the context into n_splits ranges of chunks_per_split chunks (bf16 path).
struct AttnPlan {
  int n_splits, chunks_per_split;
};
AttnPlan plan_attention(int batch, int nkv, int max_ctx);

int launch_attention(int dtype, int hd, const AttnArgs& a, int max_rows, hipStream_t st);

}  // namespace lsv
