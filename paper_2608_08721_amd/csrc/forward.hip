// Verify forward pass: packed-model layout, workspace layout, embedding kernel
// and the per-layer launch sequence (LibraSpec Sec. 3.1: one target pass over all
// drafted positions).
//
// Per layer, five launches (+1 attention merge for bf16):
//   QKV GEMM   : 1/rms row scaling, RoPE, K/V cache append
//   attention  : split-context running softmax (+ merge)
//   O GEMM     : residual add, storage-type copy of h, row sum-of-squares partials
//   gate/up    : 1/rms row scaling, SwiGLU
//   down GEMM  : residual add, storage-type copy of h, sum-of-squares partials
// then the LM head (1/rms row scaling) writes fp32 logits.
#include "lsv_attn.h"
#include "lsv_device.h"
#include "lsv_gemm.h"

namespace lsv {

static size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

Shape shape_of(const lsv_model_config* c) {
  Shape s;
  s.L = c->n_layers;
  s.d = c->d_model;
  s.nq = c->n_q_heads;
  s.nkv = c->n_kv_heads;
  s.hd = c->head_dim;
  s.F = c->d_ff;
  s.V = c->vocab;
  s.dtype = c->dtype;
  s.es = c->dtype == LSV_DTYPE_BF16 ? 2 : 4;
  s.eps = c->rms_eps;
  s.rope_base = c->rope_base;
  return s;
}

static PackedMat packed(size_t& off, int N, int K, int KT, int Nt_override = -1) {
  PackedMat p;
  p.offset = off;
  p.N = N;
  p.K = K;
  p.Nt = Nt_override >= 0 ? Nt_override : (N + 15) / 16;
  p.Kt = (K + KT - 1) / KT;
  off = al256(off + (size_t)p.Nt * p.Kt * 1024);
  return p;
}

ModelLayout model_layout(const Shape& s) {
  const int KT = s.dtype == LSV_DTYPE_BF16 ? 32 : 16;
  ModelLayout m;
  size_t off = 0;
  m.embed = off;
  off = al256(off + (size_t)s.V * s.d * s.es);
  m.lm_head = packed(off, s.V, s.d, KT);
  m.layer_base = off;
  size_t lo = 0;
  m.qkv = packed(lo, (s.nq + 2 * s.nkv) * s.hd, s.d, KT);
  m.o = packed(lo, s.d, s.nq * s.hd, KT);
  m.gateup = packed(lo, 2 * s.F, s.d, KT, 2 * ((s.F + 15) / 16));
  m.down = packed(lo, s.d, s.F, KT);
  m.layer_stride = lo;
  m.total = m.layer_base + (size_t)s.L * lo;
  return m;
}

// ------------------------------------------------------------------ workspace
struct VerifyWs {
  float* h;        // [M_max][d] fp32 residual stream (row-major)
  void* hx;        // storage-type copy of h, d columns (activation layout, act_index)
  float* stats;    // [M_max][d/16] per-16-column sums of squares of h
  void* q;         // [M_max][nq][hd]
  void* attn;      // attention output, nq*hd columns (activation layout)
  void* u;         // SwiGLU output, d_ff columns (activation layout; padding columns stay zero)
  float* o_part;   // attention split partials
  float* ml_part;
  float* part;     // wide blocks: k-split partials
  float* qkv_y;    // wide blocks with an unsplit QKV: [M_max][N_qkv] projection before RoPE
  size_t total;
};

struct VerifyPlan {
  int MT, batch;
  bool wide;  // bf16 blocks of 64 < rows <= kWideRows: all rows per workgroup, activations via LDS
  WidePlan w[5];
  size_t part_floats;
  AttnPlan attn;
};

static VerifyPlan plan_verify(const Shape& s, const ModelLayout& ml, int batch, int max_rows, int max_ctx) {
  VerifyPlan v;
  v.batch = batch;
  v.MT = max_rows > 64 ? 4 : (max_rows + 15) / 16;  // activation tiles per 64-row chunk
  v.wide = s.dtype == LSV_DTYPE_BF16 && max_rows > 64 && max_rows <= kWideRows;
  v.part_floats = 0;
  if (v.wide) {
    const PackedMat* mats[5] = {&ml.qkv, &ml.o, &ml.gateup, &ml.down, &ml.lm_head};
    for (int k = 0; k < 5; ++k) {
      v.w[k] = plan_wide(mats[k]->Nt, mats[k]->Kt);
      const size_t pf = wide_part_floats(v.w[k], max_rows);
      v.part_floats = pf > v.part_floats ? pf : v.part_floats;
    }
  }
  v.attn = plan_attention(batch, s.nkv, max_ctx);
  return v;
}

static VerifyWs carve_verify(const Shape& s, const ModelLayout& ml, const VerifyPlan& v, int max_rows, void* base) {
  VerifyWs w;
  char* p = (char*)base;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* r = p ? p + off : nullptr;
    off = al256(off + bytes);
    return (void*)r;
  };
  // activation buffers hold whole 16-row tiles and whole k-steps
  auto act_bytes = [&](int K) {
    return (size_t)s.es * (s.dtype == LSV_DTYPE_BF16 ? act_elems<32>(max_rows, K) : act_elems<16>(max_rows, K));
  };
  w.h = (float*)take(sizeof(float) * (size_t)max_rows * s.d);
  w.hx = take(act_bytes(s.d));
  w.stats = (float*)take(sizeof(float) * (size_t)(s.d / 16) * max_rows);
  w.q = take((size_t)s.es * max_rows * s.nq * s.hd);
  w.attn = take(act_bytes(s.nq * s.hd));
  w.u = take(act_bytes(s.F));
  if (s.dtype == LSV_DTYPE_BF16) {
    w.o_part = (float*)take(sizeof(float) * (size_t)v.attn.n_splits * max_rows * s.nq * s.hd);
    w.ml_part = (float*)take(sizeof(float) * (size_t)v.attn.n_splits * max_rows * s.nq * 2);
  } else {
    w.o_part = w.ml_part = nullptr;
  }
  w.part = (float*)take(sizeof(float) * v.part_floats);
  // the unsplit wide QKV projection goes through an fp32 copy before the rotary embedding
  w.qkv_y = v.wide && v.w[GEMM_QKV].splits == 1 ? (float*)take(sizeof(float) * (size_t)max_rows * ml.qkv.N) : nullptr;
  w.total = off;
  return w;
}

size_t verify_workspace_bytes(const Shape& s, int batch, int max_rows, int max_ctx) {
  (void)batch;
  ModelLayout ml = model_layout(s);
  VerifyPlan v = plan_verify(s, ml, batch, max_rows, max_ctx);
  return carve_verify(s, ml, v, max_rows, nullptr).total;
}

// ------------------------------------------------------------------ embedding
// h[m] = E[token_m] (fp32), its storage-type copy in the activation layout and
// per-16-column sums of squares for the first RMSNorm.  Workgroup 0 also validates every
// sequence: token ids in range and the block within max_ctx.  Invalid tokens embed as zeros.
template <typename T>
__global__ void __launch_bounds__(256) embed_kernel(const T* __restrict__ E, int V, int d, const int32_t* tokens,
                                                    const int32_t* row_offsets, const int32_t* seq_len, int batch,
                                                    int ctx_limit, int M_max, float* h, T* hx, float* stats,
                                                    int32_t* status) {
  const int m = blockIdx.x;
  if (m == 0 && status) {
    for (int b = threadIdx.x; b < batch; b += blockDim.x) {
      const int r0 = row_offsets[b], r1 = row_offsets[b + 1];
      int st = LSV_OK;
      if (r1 < r0 || seq_len[b] < 0 || seq_len[b] + (r1 - r0) > ctx_limit) st = LSV_ERR_CAPACITY;
      if (r0 < 0 || r1 > M_max) {
        status[b] = LSV_ERR_INVALID_ARG;
        continue;
      }
      for (int r = r0; r < r1; ++r)
        if (tokens[r] < 0 || tokens[r] >= V) st = LSV_ERR_INVALID_ARG;
      status[b] = st;
    }
  }
  if (m >= GL(row_offsets)[batch] || m >= M_max) return;
  const int tok_in = GL(tokens)[m];
  const bool ok = tok_in >= 0 && tok_in < V;
  const int tok = ok ? tok_in : 0;  // invalid ids read row 0 and are zeroed below
  // one 16-column group per thread: 16-byte loads and stores, the group's sum of squares
  constexpr int PER16 = 16 * sizeof(T) / 16;  // 16-byte pieces per 16 elements
  const GLOBAL u32x4_t* src = (const GLOBAL u32x4_t*)(GL(E) + (size_t)tok * d);
  for (int p = threadIdx.x; p < d / 16; p += blockDim.x) {
    u32x4_t raw[PER16];
#pragma unroll
    for (int i = 0; i < PER16; ++i) {
      const u32x4_t v = src[p * PER16 + i];
      raw[i] = ok ? v : u32x4_t{0u, 0u, 0u, 0u};
    }
    float x[16];
#pragma unroll
    for (int i = 0; i < PER16; ++i)
#pragma unroll
      for (int e = 0; e < 16 / PER16; ++e) {
        if (sizeof(T) == 2) {
          const uint32_t w = raw[i][e >> 1];
          x[i * 8 + e] = __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
        } else {
          x[i * 4 + e] = __uint_as_float(raw[i][e]);
        }
      }
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) ss += x[e] * x[e];
    GLOBAL f32x4_t* hp = (GLOBAL f32x4_t*)(GL(h) + (size_t)m * d + 16 * p);
#pragma unroll
    for (int i = 0; i < 4; ++i) hp[i] = f32x4_t{x[4 * i], x[4 * i + 1], x[4 * i + 2], x[4 * i + 3]};
    // a 16-byte piece is one lane's run of a fragment (EPL = 16 / sizeof(T) columns)
    constexpr int KT = 64 / sizeof(T), EPL = KT / 4;
    const int Kt = (d + KT - 1) / KT;
#pragma unroll
    for (int i = 0; i < PER16; ++i) *(GLOBAL u32x4_t*)(GL(hx) + act_index<KT>(m, 16 * p + i * EPL, Kt)) = raw[i];
    GL(stats)[(size_t)m * (d / 16) + p] = ss;
  }
}

int launch_verify(const Shape& s, const ModelLayout& ml, const void* packed, void* kv, int capacity, int batch,
                  const int32_t* seq_len, const int32_t* tokens, const int32_t* row_offsets, int max_rows,
                  int max_ctx, float* logits, int32_t* status, void* ws, size_t ws_bytes, hipStream_t st) {
  const VerifyPlan v = plan_verify(s, ml, batch, max_rows, max_ctx);
  const VerifyWs w = carve_verify(s, ml, v, max_rows, ws);
  if (w.total > ws_bytes) return LSV_ERR_INVALID_ARG;
  if (v.part_floats * sizeof(float) >= ((size_t)1 << 31)) return LSV_ERR_UNSUPPORTED;  // 32-bit buffer offsets
  const char* P = (const char*)packed;
  const bool bf16 = s.dtype == LSV_DTYPE_BF16;

  if (bf16)
    hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(max_rows), dim3(256), 0, st, (const bf16_t*)(P + ml.embed), s.V,
                       s.d, tokens, row_offsets, seq_len, batch, max_ctx, max_rows, w.h, (bf16_t*)w.hx, w.stats,
                       status);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(max_rows), dim3(256), 0, st, (const float*)(P + ml.embed), s.V, s.d,
                       tokens, row_offsets, seq_len, batch, max_ctx, max_rows, w.h, (float*)w.hx, w.stats, status);
  if (hipGetLastError() != hipSuccess) return LSV_ERR_HIP;

  GemmArgs base = {};
  base.M_max = max_rows;
  base.batch = batch;
  base.row_offsets = row_offsets;
  base.stats = w.stats;
  base.P = s.d / 16;
  base.eps = s.eps;
  base.seq_len = seq_len;
  base.kv = kv;
  base.capacity = capacity;
  base.nq = s.nq;
  base.nkv = s.nkv;
  base.hd = s.hd;
  base.log2_rope_base = log2(s.rope_base);
  base.F = s.F;

  auto gemm = [&](GemmKind kind, const PackedMat& pm, const char* layer_base, GemmArgs a) {
    a.W = (const uint4*)(layer_base + pm.offset);
    a.N = pm.N;
    a.K = pm.K;
    a.Nt = pm.Nt;
    a.Kt = pm.Kt;
    const int idx = kind == GEMM_LMHEAD ? 0 : a.layer_index;
    timing_before((int)kind, idx, st);
    int rc;
    if (v.wide) {
      a.part = w.part;
      a.part_bytes = sizeof(float) * v.part_floats;
      if (kind == GEMM_QKV) a.out_f32 = w.qkv_y;
      rc = launch_gemm_wide(kind, a, v.w[kind], st);
    } else {
      rc = launch_gemm(s.dtype, kind, v.MT, a, st);
    }
    timing_after((int)kind, idx, st);
    return rc;
  };

  const size_t kv_layer_elems = (size_t)2 * batch * s.nkv * (size_t)capacity * s.hd;
  int rc;
  for (int l = 0; l < s.L; ++l) {
    const char* LB = P + ml.layer_base + (size_t)l * ml.layer_stride;
    // QKV (normalised input) + RoPE + cache append
    GemmArgs a = base;
    a.layer_index = l;
    a.layer = l;
    a.x = w.hx;
    a.q_out = w.q;
    if ((rc = gemm(GEMM_QKV, ml.qkv, LB, a)) != LSV_OK) return rc;
    // attention
    AttnArgs at;
    at.q = w.q;
    at.k = (const char*)kv + (size_t)l * kv_layer_elems * s.es;
    at.v = (const char*)at.k + kv_layer_elems / 2 * s.es;
    at.capacity = capacity;
    at.ctx_limit = max_ctx;
    at.batch = batch;
    at.nq = s.nq;
    at.nkv = s.nkv;
    at.M_max = max_rows;
    at.row_offsets = row_offsets;
    at.seq_len = seq_len;
    at.o_part = w.o_part;
    at.ml_part = w.ml_part;
    at.out = w.attn;
    at.scale_log2 = (float)(1.4426950408889634 / sqrt((double)s.hd));
    at.n_splits = v.attn.n_splits;
    at.chunks_per_split = v.attn.chunks_per_split;
    timing_before(LSV_KERNEL_ATTENTION, l, st);
    if ((rc = launch_attention(s.dtype, s.hd, at, max_rows, st)) != LSV_OK) return rc;
    timing_after(LSV_KERNEL_ATTENTION, l, st);
    // O projection + residual
    a = base;
    a.layer_index = l;
    a.x = w.attn;
    a.h_out = w.h;
    a.hx_out = w.hx;
    a.stats_out = w.stats;
    if ((rc = gemm(GEMM_O, ml.o, LB, a)) != LSV_OK) return rc;
    // gate/up (normalised input) + SwiGLU
    a = base;
    a.layer_index = l;
    a.x = w.hx;
    a.u_out = w.u;
    if ((rc = gemm(GEMM_GATEUP, ml.gateup, LB, a)) != LSV_OK) return rc;
    // down + residual
    a = base;
    a.layer_index = l;
    a.x = w.u;
    a.h_out = w.h;
    a.hx_out = w.hx;
    a.stats_out = w.stats;
    if ((rc = gemm(GEMM_DOWN, ml.down, LB, a)) != LSV_OK) return rc;
  }
  GemmArgs a = base;
  a.x = w.hx;
  a.out_f32 = logits;
  a.ldo = s.V;
  return gemm(GEMM_LMHEAD, ml.lm_head, P, a);
}

}  // namespace lsv
