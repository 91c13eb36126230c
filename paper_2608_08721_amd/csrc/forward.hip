// Verify forward pass: packed-model layout, workspace layout, embedding kernel
// and the per-layer launch sequence (LibraSpec Sec. 3.1: one target pass over all
// drafted positions).
//
// Per layer, seven launches (+1 attention merge for bf16):
//   QKV GEMM   : RoPE, K/V cache append
//   attention  : split-context running softmax (+ merge)
//   O GEMM     : residual add
//   norm       : a = R(h / rms(h) * g_ffn)
//   gate/up    : SwiGLU
//   down GEMM  : residual add
//   norm       : a = R(h / rms(h) * g) with the next layer's attention gain (final gain last)
// then the LM head writes fp32 logits.  The embedding kernel writes layer 0's first a.
// R() rounds to the storage type once, after the gain: the normalised activation is what a
// projection multiplies, as in the model's definition.
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
  m.final_norm = off;
  off = al256(off + sizeof(float) * (size_t)s.d);
  m.lm_head = packed(off, s.V, s.d, KT);
  m.layer_base = off;
  size_t lo = 0;
  m.attn_norm = lo;
  lo = al256(lo + sizeof(float) * (size_t)s.d);
  m.ffn_norm = lo;
  lo = al256(lo + sizeof(float) * (size_t)s.d);
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
  void* a;         // normalised rows R(h / rms(h) * g), d columns (activation layout, act_index)
  void* q;         // [M_max][nq][hd]
  void* attn;      // attention output, nq*hd columns (activation layout)
  void* u;         // SwiGLU output, d_ff columns (activation layout; padding columns stay zero)
  float* o_part;   // attention split partials
  float* ml_part;
  float* part;     // wide blocks: k-split partials
  float* qkv_y;    // wide blocks with an unsplit QKV: [M_max][N_qkv] projection before RoPE
  int32_t* depth;  // tree blocks: [M_max] depth of each row in its sequence's tree
  uint32_t* anc;   // tree blocks: [M_max][kAncWords] ancestor-or-self masks over block rows
  int32_t* bad;    // tree blocks: [M_max] 1 where a row's parent chain is not a valid tree
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
  if (s.dtype == LSV_DTYPE_BF16 && residual_split_pairs(GEMM_O, ml.o.Nt))  // O and down: Nt = d / 16
    v.part_floats = split_pair_floats(ml.o.Nt, max_rows);
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
  w.a = take(act_bytes(s.d));
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
  w.depth = (int32_t*)take(sizeof(int32_t) * (size_t)max_rows);
  w.anc = (uint32_t*)take(sizeof(uint32_t) * (size_t)max_rows * kAncWords);
  w.bad = (int32_t*)take(sizeof(int32_t) * (size_t)max_rows);
  w.total = off;
  return w;
}

size_t verify_workspace_bytes(const Shape& s, int batch, int max_rows, int max_ctx) {
  (void)batch;
  ModelLayout ml = model_layout(s);
  VerifyPlan v = plan_verify(s, ml, batch, max_rows, max_ctx);
  return carve_verify(s, ml, v, max_rows, nullptr).total;
}

// ------------------------------------------------------------------ row normalisation
// a[m] = R(h[m] / sqrt(mean(h[m]^2) + eps) * g) of one row, by one 256-thread workgroup.
// Thread t holds the lane runs of EPL columns t, t + 256, ... of the row (EPL = 8 bf16 or 4 fp32
// columns: one 16-byte store of the operand each) in registers from a single read;
// its sum of squares runs over them in order, the wave adds its lanes in a fixed shuffle
// tree and wave 0 adds the four waves' sums in order.  Every element is then scaled,
// multiplied by its gain and rounded once.
// part (NULL: none): the k-split partial sums [tile][split][M_max][kWideCols] that the residual
// product before it left; the `splits` pieces of each of the thread's columns (up to four in
// flight at once, issued once h has arrived) are added in split order, ((0 + p_0) + p_1) + ...,
// and the sum joins the residual stream, h += sum, which is stored before the row is normalised
// from the same registers.
template <typename T>
LSV_DEV void normalise_row(float* __restrict__ hrow, int d, const float* __restrict__ gain, float eps, int m,
                           T* __restrict__ a, const float* __restrict__ part, int splits, int M_max) {
  constexpr int KT = 64 / sizeof(T), EPL = KT / 4;
  constexpr int RUNS = 8192 / (256 * EPL);  // d_model <= 8192
  constexpr int JB = 4;                     // splits whose pieces are in flight together
  __shared__ float wsum[4];
  const int t = threadIdx.x;
  // the row and the gains of the thread's columns are loaded together (the gains do not depend on
  // the row, and loading them after the reduction would add a memory round trip); columns past d
  // load the last piece (in bounds, no branch) and count as zeros
  f32x4_t x[RUNS][EPL / 4], gv[RUNS][EPL / 4];
#pragma unroll
  for (int r = 0; r < RUNS; ++r) {
    const int c = (t + 256 * r) * EPL;
#pragma unroll
    for (int e = 0; e < EPL / 4; ++e) {
      const int cc = min(c + 4 * e, d - 4);
      x[r][e] = *(const GLOBAL f32x4_t*)(GL(hrow) + cc);
      gv[r][e] = *(const GLOBAL f32x4_t*)(GL(gain) + cc);
    }
  }
#pragma unroll
  for (int r = 0; r < RUNS; ++r)
#pragma unroll
    for (int e = 0; e < EPL / 4; ++e)
      if ((t + 256 * r) * EPL >= d) x[r][e] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  if (part && splits > 1) {
    const size_t jstride = (size_t)M_max * kWideCols;
    f32x4_t acc[RUNS][EPL / 4];
#pragma unroll
    for (int r = 0; r < RUNS; ++r)
#pragma unroll
      for (int e = 0; e < EPL / 4; ++e) acc[r][e] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 < splits; j0 += JB) {
      f32x4_t v[JB][RUNS][EPL / 4];
#pragma unroll
      for (int r = 0; r < RUNS; ++r)
#pragma unroll
        for (int e = 0; e < EPL / 4; ++e) {
          const int c = min((t + 256 * r) * EPL + 4 * e, d - 4);  // columns past d read the last piece
          const GLOBAL float* p = GL(part) + ((size_t)(c / kWideCols) * splits * M_max + m) * kWideCols + c % kWideCols;
#pragma unroll
          for (int i = 0; i < JB; ++i) v[i][r][e] = *(const GLOBAL f32x4_t*)(p + (size_t)min(j0 + i, splits - 1) * jstride);
        }
#pragma unroll
      for (int i = 0; i < JB; ++i)
        if (j0 + i < splits)
#pragma unroll
          for (int r = 0; r < RUNS; ++r)
#pragma unroll
            for (int e = 0; e < EPL / 4; ++e) acc[r][e] += v[i][r][e];
    }
#pragma unroll
    for (int r = 0; r < RUNS; ++r) {
      const int c = (t + 256 * r) * EPL;
#pragma unroll
      for (int e = 0; e < EPL / 4; ++e)
        if (c < d) {
          x[r][e] = x[r][e] + acc[r][e];
          *(GLOBAL f32x4_t*)(GL(hrow) + c + 4 * e) = x[r][e];
        }
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int r = 0; r < RUNS; ++r)
#pragma unroll
    for (int e = 0; e < EPL / 4; ++e)
#pragma unroll
      for (int q = 0; q < 4; ++q) ss += x[r][e][q] * x[r][e][q];
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, kWave);
  if ((t & 63) == 0) wsum[t >> 6] = ss;
  __syncthreads();
  const float inv = 1.0f / sqrtf(((wsum[0] + wsum[1]) + (wsum[2] + wsum[3])) / (float)d + eps);
  const int Kt = (d + KT - 1) / KT;
#pragma unroll
  for (int r = 0; r < RUNS; ++r) {
    const int c = (t + 256 * r) * EPL;
    if (c >= d) break;
    float y[EPL];
#pragma unroll
    for (int e = 0; e < EPL; e += 4)
#pragma unroll
      for (int q = 0; q < 4; ++q) y[e + q] = x[r][e / 4][q] * inv * gv[r][e / 4][q];
    u32x4_t out;
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = (uint32_t)f2bf(y[2 * i]) | ((uint32_t)f2bf(y[2 * i + 1]) << 16);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) out[i] = __float_as_uint(y[i]);
    }
    *(GLOBAL u32x4_t*)(GL(a) + act_index<KT>(m, c, Kt)) = out;
  }
}

// The consumer operand of the next projection, one workgroup per block row.  part: the k-split
// partial sums [tile][split][M_max][kWideCols] that the residual product before it left -- the
// batched body for a block of more than 64 rows (splits_hi of them), the split pairs of the
// narrower models otherwise (splits_lo = 2); a count of 1 means none.  normalise_row adds them to
// the residual stream before it normalises the row.
template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_kernel(float* __restrict__ h, int d, const float* gain, float eps,
                                                      const int32_t* row_offsets, int batch, int M_max, T* a,
                                                      const float* __restrict__ part, int splits_lo, int splits_hi) {
  const int m = blockIdx.x;
  const int M = min(GL(row_offsets)[batch], M_max);
  if (m >= M) return;
  normalise_row<T>(h + (size_t)m * d, d, gain, eps, m, a, part, M > 64 ? splits_hi : splits_lo, M_max);
}

// ------------------------------------------------------------------ tree blocks
// Per block row m (one thread each): its depth in its sequence's tree and the bit mask of
// its ancestors and itself over the sequence's block rows, by walking its parent chain.
// A row whose chain leaves the tree shape (the first row's parent is not -1, or a parent
// does not precede its child) is flagged in bad[m]; its depth is 0 and its mask itself.
__global__ void __launch_bounds__(256) tree_prep_kernel(const int32_t* __restrict__ parents,
                                                        const int32_t* __restrict__ row_offsets, int batch, int M_max,
                                                        int32_t* __restrict__ depth, uint32_t* __restrict__ anc,
                                                        int32_t* __restrict__ bad) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  const int M = min(GL(row_offsets)[batch], M_max);
  if (m >= M) return;
  const int b = seq_of_row(row_offsets, batch, m);
  const int r0 = GL(row_offsets)[b], i = m - r0;
  uint32_t bits[kAncWords];
#pragma unroll
  for (int w = 0; w < kAncWords; ++w) bits[w] = 0u;
  if (r0 < 0 || i < 0 || i >= kTreeNodes) {  // row offsets the embedding kernel will refuse
    GL(depth)[m] = 0;
    GL(bad)[m] = 1;
#pragma unroll
    for (int w = 0; w < kAncWords; ++w) GL(anc)[(size_t)m * kAncWords + w] = 0u;
    return;
  }
  bool ok = GL(parents)[r0] == -1;
  int d = 0;
  for (int cur = i; ok && cur != 0;) {  // each step moves to a smaller index: at most i steps
    const int p = GL(parents)[r0 + cur];
    if (p < 0 || p >= cur) {
      ok = false;
      break;
    }
    bits[p >> 5] |= 1u << (p & 31);
    cur = p;
    ++d;
  }
  if (!ok) {
#pragma unroll
    for (int w = 0; w < kAncWords; ++w) bits[w] = 0u;
    d = 0;
  }
  bits[i >> 5] |= 1u << (i & 31);
  GL(depth)[m] = d;
  GL(bad)[m] = ok ? 0 : 1;
#pragma unroll
  for (int w = 0; w < kAncWords; ++w) GL(anc)[(size_t)m * kAncWords + w] = bits[w];
}

// ------------------------------------------------------------------ embedding
// h[m] = E[token_m] (fp32) and the first normalised operand a[m] = R(h / rms(h) * g) with
// layer 0's attention gain.  Workgroup 0 also validates every sequence: token ids in range
// and the block within max_ctx.  Invalid tokens embed as zeros.
template <typename T>
__global__ void __launch_bounds__(256) embed_kernel(const T* __restrict__ E, int V, int d, const int32_t* tokens,
                                                    const int32_t* row_offsets, const int32_t* seq_len, int batch,
                                                    int ctx_limit, int M_max, float* h, const float* gain, float eps,
                                                    T* a, const int32_t* tree_bad, int32_t* status) {
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
        if (tokens[r] < 0 || tokens[r] >= V || (tree_bad && tree_bad[r])) st = LSV_ERR_INVALID_ARG;
      status[b] = st;
    }
  }
  if (m >= GL(row_offsets)[batch] || m >= M_max) return;
  const int tok_in = GL(tokens)[m];
  const bool ok = tok_in >= 0 && tok_in < V;
  const int tok = ok ? tok_in : 0;  // invalid ids read row 0 and are zeroed below
  const GLOBAL T* src = GL(E) + (size_t)tok * d;
  float* hrow = h + (size_t)m * d;
  for (int c = threadIdx.x * 4; c < d; c += 256 * 4) {
    f32x4_t v;
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = ok ? to_f32<T>(src[c + r]) : 0.f;
    *(GLOBAL f32x4_t*)(GL(hrow) + c) = v;
  }
  __syncthreads();  // the workgroup's stores of the row are visible to its own loads below
  normalise_row<T>(hrow, d, gain, eps, m, a, nullptr, 1, M_max);
}

int launch_verify(const Shape& s, const ModelLayout& ml, const void* packed, void* kv, const KvLayout& kvl, int batch,
                  const int32_t* seq_len, const int32_t* tokens, const int32_t* row_offsets, const int32_t* parents,
                  int max_rows, int max_ctx, float* logits, int32_t* status, void* ws, size_t ws_bytes,
                  hipStream_t st) {
  const VerifyPlan v = plan_verify(s, ml, batch, max_rows, max_ctx);
  const VerifyWs w = carve_verify(s, ml, v, max_rows, ws);
  if (w.total > ws_bytes) return LSV_ERR_INVALID_ARG;
  if (v.part_floats * sizeof(float) >= ((size_t)1 << 31)) return LSV_ERR_UNSUPPORTED;  // 32-bit buffer offsets
  const char* P = (const char*)packed;
  const bool bf16 = s.dtype == LSV_DTYPE_BF16;

  auto layer_gain = [&](int l, size_t which) {
    return (const float*)(P + ml.layer_base + (size_t)l * ml.layer_stride + which);
  };
  if (parents)
    hipLaunchKernelGGL(tree_prep_kernel, dim3((max_rows + 255) / 256), dim3(256), 0, st, parents, row_offsets, batch,
                       max_rows, w.depth, w.anc, w.bad);
  const int32_t* tree_bad = parents ? w.bad : nullptr;
  if (bf16)
    hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(max_rows), dim3(256), 0, st, (const bf16_t*)(P + ml.embed), s.V,
                       s.d, tokens, row_offsets, seq_len, batch, max_ctx, max_rows, w.h, layer_gain(0, ml.attn_norm),
                       s.eps, (bf16_t*)w.a, tree_bad, status);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(max_rows), dim3(256), 0, st, (const float*)(P + ml.embed), s.V, s.d,
                       tokens, row_offsets, seq_len, batch, max_ctx, max_rows, w.h, layer_gain(0, ml.attn_norm), s.eps,
                       (float*)w.a, tree_bad, status);
  if (hipGetLastError() != hipSuccess) return LSV_ERR_HIP;
  // a = R(h / rms(h) * gain) for the next projection
  // a = R(h / rms(h) * gain) for the next projection, after the k-split partials of the
  // residual product before it (batched bounds) join h
  auto rmsnorm = [&](const float* gain, GemmKind after) {
    const int lo = bf16 && residual_split_pairs(after, ml.o.Nt) ? 2 : 1;  // O and down share Nt = d / 16
    const int hi = v.wide ? v.w[after].splits : lo;
    const float* part = lo > 1 || hi > 1 ? w.part : nullptr;
    if (bf16)
      hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(max_rows), dim3(256), 0, st, w.h, s.d, gain, s.eps, row_offsets,
                         batch, max_rows, (bf16_t*)w.a, part, lo, hi);
    else
      hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(max_rows), dim3(256), 0, st, w.h, s.d, gain, s.eps, row_offsets,
                         batch, max_rows, (float*)w.a, part, lo, hi);
    return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
  };

  GemmArgs base = {};
  base.rows_lo = -1;
  base.rows_hi = kRowsAny;
  base.M_max = max_rows;
  base.batch = batch;
  base.row_offsets = row_offsets;
  base.seq_len = seq_len;
  base.depth = parents ? w.depth : nullptr;
  base.kv = kv;
  base.kvl = kvl;
  base.capacity = kvl.capacity;
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
    a.part = w.part;  // the residual products' split pairs (narrower bf16 models) or batched split-K
    a.part_bytes = sizeof(float) * v.part_floats;
    if (v.wide) {
      // a batched bound: one launch whose workgroups run the 64-row body (the weights streamed
      // once) for blocks of up to 64 device rows and the batched body for larger ones
      if (kind == GEMM_QKV) a.out_f32 = w.qkv_y;
      rc = launch_gemm_fused(kind, a, v.w[kind], st);
    } else {
      rc = launch_gemm(s.dtype, kind, v.MT, a, st);
    }
    timing_after((int)kind, idx, st);
    return rc;
  };

  const size_t kv_block = kv_layer_block(kvl, batch, s.nkv, s.hd);  // elements of one layer's K (or V) block
  int rc;
  for (int l = 0; l < s.L; ++l) {
    const char* LB = P + ml.layer_base + (size_t)l * ml.layer_stride;
    // QKV (normalised input) + RoPE + cache append
    GemmArgs a = base;
    a.layer_index = l;
    a.layer = l;
    a.x = w.a;
    a.q_out = w.q;
    if ((rc = gemm(GEMM_QKV, ml.qkv, LB, a)) != LSV_OK) return rc;
    // attention
    AttnArgs at;
    at.q = w.q;
    at.k = (const char*)kv + 2 * (size_t)l * kv_block * s.es;
    at.v = (const char*)at.k + kv_block * s.es;
    at.kv = kvl;
    at.capacity = kvl.capacity;
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
    at.packed = v.attn.packed;
    at.anc = parents ? w.anc : nullptr;
    timing_before(LSV_KERNEL_ATTENTION, l, st);
    if ((rc = launch_attention(s.dtype, s.hd, at, max_rows, st)) != LSV_OK) return rc;
    timing_after(LSV_KERNEL_ATTENTION, l, st);
    // O projection + residual
    a = base;
    a.layer_index = l;
    a.x = w.attn;
    a.h_out = w.h;
    if ((rc = gemm(GEMM_O, ml.o, LB, a)) != LSV_OK) return rc;
    if ((rc = rmsnorm(layer_gain(l, ml.ffn_norm), GEMM_O)) != LSV_OK) return rc;
    // gate/up (normalised input) + SwiGLU
    a = base;
    a.layer_index = l;
    a.x = w.a;
    a.u_out = w.u;
    if ((rc = gemm(GEMM_GATEUP, ml.gateup, LB, a)) != LSV_OK) return rc;
    // down + residual
    a = base;
    a.layer_index = l;
    a.x = w.u;
    a.h_out = w.h;
    if ((rc = gemm(GEMM_DOWN, ml.down, LB, a)) != LSV_OK) return rc;
    // the next projection's operand: the next layer's attention norm, or the final norm
    if ((rc = rmsnorm(l + 1 < s.L ? layer_gain(l + 1, ml.attn_norm) : (const float*)(P + ml.final_norm), GEMM_DOWN)) !=
        LSV_OK)
      return rc;
  }
  GemmArgs a = base;
  a.x = w.a;
  a.out_f32 = logits;
  a.ldo = s.V;
  return gemm(GEMM_LMHEAD, ml.lm_head, P, a);
}

}  // namespace lsv
