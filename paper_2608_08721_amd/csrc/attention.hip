// Causal grouped-query attention of the block rows over the KV cache.
//
// bf16 path (matrix cores), two kernels:
//  * split kernel: one workgroup of four waves per (context split, kv head, sequence).  A
//    split is a run of 64-key chunks.  Each chunk's K rows and transposed V rows go HBM ->
//    registers -> LDS with 16-byte accesses; the first chunk's loads are issued before any
//    device metadata is read, and each next chunk's loads are in flight while the current
//    one is consumed.  A wave owns up to kQpw tiles of 16 query vectors (block rows x query
//    heads of this kv head) and keeps a running softmax over the split:
//    S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_16x16x32_bf16.  The probabilities stay in
//    registers: the D layout of S^T is the B operand layout of P^T, and the V rows are
//    stored with their keys permuted (v_column) so that one 16-byte read is a fragment.
//    Output per split and query vector: running max (log2 units), sum, unnormalised O.
//  * merge kernel: per (row, query head) combines the splits in split order.
// fp32 path: a plain kernel, one wave per (row, query head).
#include <math.h>

#include "lsv_attn.h"
#include "lsv_device.h"

namespace lsv {

constexpr int kCh = kAttnChunk;  // keys per chunk
constexpr int kQpw = 1;          // query tiles per wave and pass
constexpr int kAttnWgs = 256;     // split-kernel workgroups aimed for
constexpr int kMaxChunksPerSplit = 16;  // a split walks its chunks in sequence

AttnPlan plan_attention(int batch, int nkv, int max_ctx) {
  const int n_chunks = (max_ctx + kCh - 1) / kCh;
  const int units = batch * nkv;
  // about one workgroup per compute unit, but no split longer than kMaxChunksPerSplit chunks
  int want = (kAttnWgs + units - 1) / units;
  const int by_length = (n_chunks + kMaxChunksPerSplit - 1) / kMaxChunksPerSplit;
  if (want < by_length) want = by_length;
  if (want > n_chunks) want = n_chunks;
  if (want < 1) want = 1;
  AttnPlan p;
  p.chunks_per_split = (n_chunks + want - 1) / want;
  p.n_splits = (n_chunks + p.chunks_per_split - 1) / p.chunks_per_split;
  return p;
}

template <int HD>
__global__ void __launch_bounds__(256) attn_split_bf16_kernel(AttnArgs a) {
  constexpr int P8 = HD / 8;             // 16-byte pieces per K row
  constexpr int NP = kCh * HD / 8 / 256;  // pieces of K (and of V^T) per thread and chunk
  constexpr int KPITCH = HD + 8, VPITCH = kCh + 8;  // padded LDS rows: conflict-free fragment reads
  __shared__ __align__(16) bf16_t Ks[kCh * KPITCH];
  __shared__ __align__(16) bf16_t Vt[HD * VPITCH];

  const int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, g4 = lane >> 4, l16 = lane & 15;
  const size_t slab = ((size_t)b * a.nkv + kvh) * (size_t)a.capacity * HD;
  const GLOBAL bf16_t* kb = GL((const bf16_t*)a.k) + slab;
  const GLOBAL bf16_t* vb = GL((const bf16_t*)a.v) + slab;
  // The grid covers the chunks of ctx_limit <= capacity and capacity is a multiple of the
  // chunk, so every chunk a workgroup may load lies inside its slab.
  const int c0 = s * a.chunks_per_split;

  u32x4_t kr[NP], vr[NP];
  auto load_chunk = [&](int c) {
    const int k0 = c * kCh;
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const int i = tid + 256 * j;
      kr[j] = *(const GLOBAL u32x4_t*)(kb + (size_t)(k0 + i / P8) * HD + (i % P8) * 8);
      vr[j] = *(const GLOBAL u32x4_t*)(vb + (size_t)(i >> 3) * a.capacity + k0 + (i & 7) * 8);
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const int i = tid + 256 * j;
      *(u32x4_t*)&Ks[(i / P8) * KPITCH + (i % P8) * 8] = kr[j];
      *(u32x4_t*)&Vt[(i >> 3) * VPITCH + (i & 7) * 8] = vr[j];
    }
  };
  load_chunk(c0);

  const int r0 = GL(a.row_offsets)[b], rows = GL(a.row_offsets)[b + 1] - r0, C = GL(a.seq_len)[b];
  if (r0 < 0 || rows <= 0 || r0 + rows > a.M_max) return;  // rows beyond the host bound are never touched
  const int group = a.nq / a.nkv, nqv = rows * group, n_qt = (nqv + 15) / 16;
  const int L = min(C + rows, a.ctx_limit);  // cached + block keys that exist
  const int nch = L > 0 ? (L + kCh - 1) / kCh : 0;
  const int c1 = min(c0 + a.chunks_per_split, nch);
  const size_t prow = (size_t)s * a.M_max + r0;  // this split's partial row of the sequence's first row
  if (c0 >= c1) {  // no key of this split exists for the sequence: mark its query vectors empty
    for (int i = tid; i < nqv; i += 256) {
      const size_t base = (prow + i / group) * a.nq + kvh * group + i % group;
      *(GLOBAL f32x2_t*)(a.ml_part + base * 2) = f32x2_t{-INFINITY, 0.f};
    }
    return;
  }

  for (int qbase = 0; qbase < n_qt; qbase += 4 * kQpw) {
    u32x4_t qf[kQpw][HD / 32];
    f32x4_t o[kQpw][HD / 16];
    float mrun[kQpw], lrun[kQpw];
    int qpos[kQpw];
    bool qval[kQpw];
#pragma unroll
    for (int j = 0; j < kQpw; ++j) {
      const int qv = (qbase + wave + 4 * j) * 16 + l16;
      qval[j] = qv < nqv;
      const int rr = qval[j] ? qv / group : 0, head = kvh * group + (qval[j] ? qv % group : 0);
      const GLOBAL bf16_t* qp = GL((const bf16_t*)a.q) + ((size_t)(r0 + rr) * a.nq + head) * HD + 8 * g4;
#pragma unroll
      for (int ds = 0; ds < HD / 32; ++ds) {  // rr = 0 for invalid columns: the load stays in bounds
        const u32x4_t t = *(const GLOBAL u32x4_t*)(qp + 32 * ds);
        qf[j][ds] = qval[j] ? t : u32x4_t{0u, 0u, 0u, 0u};
      }
      qpos[j] = C + rr;
      mrun[j] = -INFINITY;
      lrun[j] = 0.f;
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) o[j][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    if (qbase > 0) load_chunk(c0);  // a later pass over the same split

    for (int c = c0; c < c1; ++c) {
      __syncthreads();  // the previous chunk's LDS reads are done
      store_chunk();
      __syncthreads();
      if (c + 1 < c1) load_chunk(c + 1);
      const int k0 = c * kCh;
#pragma unroll
      for (int j = 0; j < kQpw; ++j) {
        if (qbase + wave + 4 * j >= n_qt) continue;  // wave-uniform
        f32x4_t sc[4];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          sc[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ds = 0; ds < HD / 32; ++ds) {
            const u32x4_t kf = *(const u32x4_t*)&Ks[(16 * kt + l16) * KPITCH + 32 * ds + 8 * g4];
            sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kf),
                                                             __builtin_bit_cast(bf16x8_t, qf[j][ds]), sc[kt], 0, 0, 0);
          }
        }
        // scale (log2 units), causal mask, running max over the split
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int kp = k0 + 16 * kt + 4 * g4 + r;
            const bool ok = qval[j] && kp < L && kp <= qpos[j];
            const float v = ok ? sc[kt][r] * a.scale_log2 : -INFINITY;
            sc[kt][r] = v;
            mx = fmaxf(mx, v);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
        mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
        const float mnew = fmaxf(mrun[j], mx);
        const float alpha = mrun[j] == -INFINITY ? 0.f : exp2f(mrun[j] - mnew);
        float sum = 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = mnew == -INFINITY ? 0.f : exp2f(sc[kt][r] - mnew);
            sc[kt][r] = p;
            sum += p;
          }
        sum += __shfl_xor(sum, 16, kWave);
        sum += __shfl_xor(sum, 32, kWave);
        mrun[j] = mnew;
        lrun[j] = lrun[j] * alpha + sum;
#pragma unroll
        for (int dt = 0; dt < HD / 16; ++dt) o[j][dt] *= alpha;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          bf16x8_t pb;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            pb[r] = (__bf16)sc[2 * ks][r];
            pb[4 + r] = (__bf16)sc[2 * ks + 1][r];
          }
#pragma unroll
          for (int dt = 0; dt < HD / 16; ++dt) {
            const u32x4_t vf = *(const u32x4_t*)&Vt[(16 * dt + l16) * VPITCH + 32 * ks + 8 * g4];
            o[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, vf), pb, o[j][dt], 0, 0, 0);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kQpw; ++j) {
      if (!qval[j]) continue;
      const int qv = (qbase + wave + 4 * j) * 16 + l16;
      const size_t base = (prow + qv / group) * a.nq + kvh * group + qv % group;
      GLOBAL float* op = GL(a.o_part) + base * HD;
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) *(GLOBAL f32x4_t*)(op + 16 * dt + 4 * g4) = o[j][dt];
      if (g4 == 0) *(GLOBAL f32x2_t*)(a.ml_part + base * 2) = f32x2_t{mrun[j], lrun[j]};
    }
  }
}

// Merge the split partials of one (row, query head): out = sum_s w_s o_s / sum_s w_s l_s,
// w_s = 2^(m_s - max_s m_s), splits in ascending order, 16 splits' loads in flight at a time.
// A wave covers 256 / HD heads of one row, four head dimensions per lane.
template <int HD>
__global__ void __launch_bounds__(64) attn_merge_bf16_kernel(AttnArgs a) {
  constexpr int LPH = HD / 4, HPW = 64 / LPH, NB = 16;
  const int m = blockIdx.x, head = blockIdx.y * HPW + threadIdx.x / LPH, d = (threadIdx.x % LPH) * 4;
  const int M = GL(a.row_offsets)[a.batch];
  if (head >= a.nq) return;
  const size_t stride = (size_t)a.M_max * a.nq, rh = (size_t)m * a.nq + head;
  const GLOBAL f32x2_t* ml = (const GLOBAL f32x2_t*)a.ml_part;
  const GLOBAL float* op = GL(a.o_part);
  float mx_all = -INFINITY, den = 0.f;
  f32x4_t num = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < a.n_splits; s0 += NB) {
    f32x2_t mv[NB];
    f32x4_t ov[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const size_t s = (size_t)min(s0 + i, a.n_splits - 1);
      mv[i] = ml[s * stride + rh];
      ov[i] = *(const GLOBAL f32x4_t*)(op + (s * stride + rh) * HD + d);
    }
    float mx = mx_all;
#pragma unroll
    for (int i = 0; i < NB; ++i)
      if (s0 + i < a.n_splits) mx = fmaxf(mx, mv[i][0]);
    const float al = mx_all == -INFINITY ? 0.f : exp2f(mx_all - mx);
    den *= al;
    num *= al;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      // empty splits (max -inf) contribute nothing; their O was never written
      if (s0 + i < a.n_splits && mv[i][0] != -INFINITY) {
        const float w = exp2f(mv[i][0] - mx);
        den += w * mv[i][1];
        num += w * ov[i];
      }
    }
    mx_all = mx;
  }
  if (m >= M) return;
  const f32x4_t r = num / den;
  const u32x2_t packed = {(uint32_t)f2bf(r[0]) | ((uint32_t)f2bf(r[1]) << 16),
                          (uint32_t)f2bf(r[2]) | ((uint32_t)f2bf(r[3]) << 16)};
  *(GLOBAL u32x2_t*)(GL((bf16_t*)a.out) + rh * HD + d) = packed;
}

// fp32 path: one wave per (row, query head); scores in LDS.
__global__ void __launch_bounds__(64) attn_f32_kernel(AttnArgs a, int hd) {
  extern __shared__ float sc[];  // [ctx_limit]
  const int m = blockIdx.x, head = blockIdx.y, t = threadIdx.x;
  if (m >= a.row_offsets[a.batch]) return;
  const int b = seq_of_row(a.row_offsets, a.batch, m);
  const int r0 = a.row_offsets[b], rows = a.row_offsets[b + 1] - r0;
  const int pos = a.seq_len[b] + (m - r0);
  const int L = min(min(pos + 1, a.seq_len[b] + rows), a.ctx_limit);
  const int kvh = head / (a.nq / a.nkv);
  const size_t slab = ((size_t)b * a.nkv + kvh) * (size_t)a.capacity * hd;
  const float* K = (const float*)a.k + slab;
  const float* Vt = (const float*)a.v + slab;
  const float* q = (const float*)a.q + ((size_t)m * a.nq + head) * hd;
  const float scale = rsqrtf((float)hd);
  float mx = -INFINITY;
  for (int j = t; j < L; j += 64) {
    float s = 0.f;
    for (int i = 0; i < hd; ++i) s += q[i] * K[(size_t)j * hd + i];
    s *= scale;
    sc[j] = s;
    mx = fmaxf(mx, s);
  }
  mx = wave_max(mx);
  float sum = 0.f;
  for (int j = t; j < L; j += 64) {
    const float p = expf(sc[j] - mx);
    sc[j] = p;
    sum += p;
  }
  sum = wave_sum(sum);
  __syncthreads();
  for (int i = t; i < hd; i += 64) {
    const float* vrow = Vt + (size_t)i * a.capacity;
    float o = 0.f;
    for (int j = 0; j < L; ++j) o += sc[j] * vrow[v_column(j)];
    ((float*)a.out)[((size_t)m * a.nq + head) * hd + i] = o / sum;
  }
}

int launch_attention(int dtype, int hd, const AttnArgs& a, int max_rows, hipStream_t st) {
  if (dtype == LSV_DTYPE_BF16) {
    const dim3 grid(a.n_splits, a.nkv, a.batch);
    const int hpw = 256 / hd;
    const dim3 mgrid(max_rows, (a.nq + hpw - 1) / hpw);
    if (hd == 128) {
      hipLaunchKernelGGL(attn_split_bf16_kernel<128>, grid, dim3(256), 0, st, a);
      hipLaunchKernelGGL(attn_merge_bf16_kernel<128>, mgrid, dim3(64), 0, st, a);
    } else if (hd == 64) {
      hipLaunchKernelGGL(attn_split_bf16_kernel<64>, grid, dim3(256), 0, st, a);
      hipLaunchKernelGGL(attn_merge_bf16_kernel<64>, mgrid, dim3(64), 0, st, a);
    } else {
      return LSV_ERR_UNSUPPORTED;
    }
  } else {
    hipLaunchKernelGGL(attn_f32_kernel, dim3(max_rows, a.nq), dim3(64), sizeof(float) * (size_t)a.ctx_limit, st, a,
                       hd);
  }
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

}  // namespace lsv
