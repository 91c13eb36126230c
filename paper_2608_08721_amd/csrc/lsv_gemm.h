// Internal interface of the skinny-M GEMM (gemm.hip).
#pragma once
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

enum { PRO_RMS = 0, PRO_PLAIN = 1 };
enum { EPI_LOGITS = 0, EPI_QKV = 1, EPI_RESID = 2, EPI_SWIGLU = 3 };
enum GemmKind { GEMM_QKV = 0, GEMM_O = 1, GEMM_GATEUP = 2, GEMM_DOWN = 3, GEMM_LMHEAD = 4 };

struct GemmArgs {
  const uint4* W;  // packed fragments
  int N, K, Nt, Kt;
  int S, kf_max;
  int M_max, batch;
  const int32_t* row_offsets;  // [batch+1]; rows = row_offsets[batch]
  // prologue
  const float* h;      // PRO_RMS: fp32 [M][K]
  const float* stats;  // PRO_RMS: [P][M_max] partial sums of h^2 over 64-column groups
  int P;
  float eps;
  const void* gain;  // PRO_RMS: [K] storage type
  const void* x;     // PRO_PLAIN: [M][ldx] storage type
  int ldx;
  // split-K
  float* part;    // [S][M_max][Nt*16]
  int* counters;  // [groups], zero on entry and on exit
  // EPI_LOGITS
  float* out_f32;
  int ldo;
  // EPI_QKV
  void* q_out;  // [M][nq][hd]
  void* kv;     // KV cache base
  int capacity, layer, nq, nkv, hd;
  const int32_t* seq_len;
  double rope_base;
  // EPI_RESID
  float* h_out;      // [M][N] updated in place
  float* stats_out;  // [N/64][M_max]
  // EPI_SWIGLU
  void* u_out;  // [M][F]
  int F;
};

struct GemmPlan {
  int groups, S, kf_max;
  size_t lds_bytes;
};

GemmPlan plan_gemm(int Nt, int Kt, int KT, int es, int MT, int TPW, int want_wgs, int max_splits);
int gemm_tpw(GemmKind kind);
int launch_gemm(int dtype, GemmKind kind, int MT, const GemmArgs& a, const GemmPlan& p, hipStream_t st);

}  // namespace lsv
