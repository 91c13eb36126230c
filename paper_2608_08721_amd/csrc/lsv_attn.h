// Internal interface of the attention kernels (attention.hip).
#pragma once
#include "lsv_internal.h"

namespace lsv {

constexpr int kAttnChunk = 64;  // keys per workgroup in the bf16 split-context kernel

struct AttnArgs {
  const void* q;  // [M][nq][hd] storage type
  const void* k;  // this layer's K block: [batch][nkv][capacity][hd]
  const void* v;  // this layer's V block
  int capacity, ctx_limit, batch, nq, nkv, M_max;
  const int32_t* row_offsets;
  const int32_t* seq_len;
  float* o_part;   // [n_chunks][M_max][nq][hd]  (bf16 path)
  float* ml_part;  // [n_chunks][M_max][nq][2]
  void* out;       // [M][nq][hd] storage type
  float scale_log2;
};

int launch_attention(int dtype, int hd, const AttnArgs& a, int max_rows, int n_chunks, hipStream_t st);

}  // namespace lsv
