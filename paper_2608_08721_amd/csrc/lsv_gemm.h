// Internal interface of the skinny-M GEMM (gemm.hip).
#pragma once
#include "lsv_attn.h"
#include "lsv_device.h"
#include "lsv_internal.h"

namespace lsv {

template <typename T> struct FragTraits;
template <> struct FragTraits<bf16_t> {
  static constexpr int KT = 32, EPL = 8;  // k columns per fragment, elements per lane
};
template <> struct FragTraits<float> {
  static constexpr int KT = 16, EPL = 4;
};

enum { EPI_LOGITS = 0, EPI_QKV = 1, EPI_RESID = 2, EPI_SWIGLU = 3, EPI_PART = 4 };
enum GemmKind { GEMM_QKV = 0, GEMM_O = 1, GEMM_GATEUP = 2, GEMM_DOWN = 3, GEMM_LMHEAD = 4 };

struct GemmArgs {
  const uint4* W;  // packed fragments
  int N, K, Nt, Kt;
  int M_max, batch;
  const int32_t* row_offsets;  // [batch+1]; rows = row_offsets[batch]
  // B operand: activation rows in the storage type, fragment-major (act_index with Kt); for
  // QKV, gate/up and the LM head the normalised rows R(h / rms(h) * g)
  const void* x;
  // wide blocks: k-split partials [tiles][splits][M_max][128]
  float* part;
  size_t part_bytes;
  int splits;
  // EPI_LOGITS (and, for wide blocks, the normalised QKV projection before RoPE)
  float* out_f32;
  int ldo;
  // EPI_QKV
  void* q_out;  // [M][nq][hd]
  void* kv;     // KV cache base
  KvLayout kvl;  // slab or paged layout of the cache
  int capacity, layer, nq, nkv, hd;
  const int32_t* seq_len;
  const int32_t* depth;  // tree blocks: row m's rotary position is seq_len + depth[m] (else its slot)
  double log2_rope_base;
  // EPI_RESID
  float* h_out;  // [M][N] fp32 residual (row-major), updated in place
  // EPI_SWIGLU
  void* u_out;  // SwiGLU output, F columns (act_index)
  int F;
  int layer_index;  // host-side only: which layer a launch belongs to (measurement hook)
  // device row range a launch serves: it does nothing unless rows_lo < rows <= rows_hi,
  // rows = row_offsets[batch] (blocks under a batched bound launch both the 64-row kernel
  // and the batched one, and the device row count picks which of them works)
  int rows_lo, rows_hi;
};
constexpr int kRowsAny = 0x7fffffff;

// One launch: a workgroup per tile of output columns, the whole K per workgroup.
int launch_gemm(int dtype, GemmKind kind, int MT, const GemmArgs& a, hipStream_t st);

// Residual products (O, down) of bf16 models narrower than Llama-3-70B (fewer than 512 fragment
// rows of output, so two rows per stream would leave compute units idle): blocks of up to 64 rows
// (and every block of the 64-row kernel) stream two fragment rows over half of K each, one stream
// per fragment row, and leave the two halves' fp32 sums in a.part -- [tile][2][M_max][128], tile
// = 8 fragment rows, the layout of the batched partials -- for the row normalisation that follows,
// which adds them to h in half order.
constexpr int kGemmComputeUnits = 256;  // gfx950 (MI350X, MI355X)
__host__ __device__ inline bool residual_split_pairs(int kind, int Nt) {
  return (kind == GEMM_O || kind == GEMM_DOWN) && (Nt + 1) / 2 < kGemmComputeUnits;
}
__host__ __device__ inline size_t split_pair_floats(int Nt, int M_max) {
  return (size_t)((Nt + 7) / 8) * 2 * M_max * 128;
}

// Batched blocks (bf16, 64 < rows <= kWideRows): every row in one workgroup, activations via LDS.
constexpr int kWideRows = LSV_WIDE_ROWS;
constexpr int kWideFR = 8;               // fragment rows of a batched workgroup's column tile
constexpr int kWideCols = kWideFR * 16;  // its output columns: k-split partials are [tile][split][M_max][kWideCols]
struct WidePlan {
  int tiles, splits;
};
WidePlan plan_wide(int Nt, int Kt);
size_t wide_part_floats(const WidePlan& p, int M_max);
// Blocks under a batched bound: one launch whose workgroups take the 64-row body or the batched
// one from the device row count (plus the batched body's reduce, which returns for <= 64 rows).
// The residual products (GEMM_O, GEMM_DOWN) with more than one k-split leave their partials in
// a.part for more than 64 rows: the caller's next row normalisation adds them to h.
int launch_gemm_fused(GemmKind kind, const GemmArgs& a, const WidePlan& p, hipStream_t st);

}  // namespace lsv
