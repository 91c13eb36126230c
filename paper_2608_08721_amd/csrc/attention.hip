// Causal grouped-query attention of the block rows over the KV cache.
//
// bf16 path (matrix cores): one workgroup per (64-key chunk, kv head, sequence)
// stages the chunk's K rows and transposed V rows in LDS with coalesced loads,
// then each wave takes 16 query vectors (block rows x query heads of this kv head)
// at a time: S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_16x16x32_bf16, with the
// softmax of each query column reduced across the four lane groups.  The
// probabilities never leave registers: the D layout of S^T is already the B
// operand layout of the P^T product.  Per-chunk (max, sum, unnormalised O) go to
// the workspace and a second kernel merges the chunks in chunk order.
// fp32 path: a plain kernel, one wave per (row, query head).
#include <math.h>

#include "lsv_attn.h"
#include "lsv_device.h"

namespace lsv {

constexpr int kCh = kAttnChunk;  // keys per chunk

template <int HD>
__global__ void __launch_bounds__(256) attn_chunk_bf16_kernel(AttnArgs a) {
  const int c = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, g4 = lane >> 4, l16 = lane & 15;
  const int r0 = GL(a.row_offsets)[b], rows = GL(a.row_offsets)[b + 1] - r0, C = GL(a.seq_len)[b];
  if (r0 < 0 || r0 + rows > a.M_max) return;  // rows beyond the host bound are never read
  const int group = a.nq / a.nkv;
  const int L = min(C + rows, a.ctx_limit);  // cached + block keys that exist
  const int k0 = c * kCh;
  if (k0 >= L || rows <= 0) return;

  __shared__ __align__(16) bf16_t Ks[kCh][HD + 8];
  __shared__ __align__(16) bf16_t Vt[HD][kCh + 8];
  const size_t slab = ((size_t)b * a.nkv + kvh) * (size_t)a.capacity * HD;
  const auto* kbase = GL((const bf16_t*)a.k) + slab;
  const auto* vbase = GL((const bf16_t*)a.v) + slab;
  constexpr int C8 = HD / 8;  // 16-byte chunks per row
  for (int i = threadIdx.x; i < kCh * C8; i += blockDim.x) {
    const int key = i / C8, d8 = i % C8;
    u32x4_t x = {0u, 0u, 0u, 0u};
    if (k0 + key < L) x = *(const GLOBAL u32x4_t*)(kbase + (size_t)(k0 + key) * HD + d8 * 8);
    *(u32x4_t*)&Ks[key][d8 * 8] = x;
  }
  for (int i = threadIdx.x; i < kCh * C8; i += blockDim.x) {
    const int key = i % kCh, d8 = i / kCh;
    u32x4_t x = {0u, 0u, 0u, 0u};
    if (k0 + key < L) x = *(const GLOBAL u32x4_t*)(vbase + (size_t)(k0 + key) * HD + d8 * 8);
    const bf16_t* e = (const bf16_t*)&x;
#pragma unroll
    for (int j = 0; j < 8; ++j) Vt[d8 * 8 + j][key] = e[j];
  }
  __syncthreads();

  const int nqv = rows * group, qtiles = (nqv + 15) / 16;
  for (int qt = wave; qt < qtiles; qt += 4) {
    const int qv = qt * 16 + l16;
    const bool qvalid = qv < nqv;
    const int rr = qvalid ? qv / group : 0, head = kvh * group + (qvalid ? qv % group : 0);
    const auto* qp = GL((const bf16_t*)a.q) + ((size_t)(r0 + rr) * a.nq + head) * HD + 8 * g4;
    u32x4_t qf[HD / 32];
#pragma unroll
    for (int ds = 0; ds < HD / 32; ++ds) {  // rr = 0 for invalid columns: the load stays in bounds
      const u32x4_t t = *(const GLOBAL u32x4_t*)(qp + 32 * ds);
      qf[ds] = qvalid ? t : u32x4_t{0u, 0u, 0u, 0u};
    }

    f32x4_t s[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      s[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < HD / 32; ++ds) {
        const u32x4_t kf = *(const u32x4_t*)&Ks[16 * kt + l16][32 * ds + 8 * g4];
        s[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kf),
                                                        __builtin_bit_cast(bf16x8_t, qf[ds]), s[kt], 0, 0, 0);
      }
    }
    // scale (log2 units), causal mask, column max / sum over the chunk's 64 keys
    const int qpos = C + rr;
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kp = k0 + 16 * kt + 4 * g4 + r;
        const bool ok = qvalid && kp < L && kp <= qpos;
        const float v = ok ? s[kt][r] * a.scale_log2 : -INFINITY;
        s[kt][r] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    float sum = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = mx == -INFINITY ? 0.f : exp2f(s[kt][r] - mx);
        s[kt][r] = p;
        sum += p;
      }
    sum += __shfl_xor(sum, 16, kWave);
    sum += __shfl_xor(sum, 32, kWave);

    f32x4_t o[HD / 16];
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8_t pb;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pb[r] = (__bf16)s[2 * ks][r];
        pb[4 + r] = (__bf16)s[2 * ks + 1][r];
      }
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) {
        const u32x2_t lo = *(const u32x2_t*)&Vt[16 * dt + l16][32 * ks + 4 * g4];
        const u32x2_t hi = *(const u32x2_t*)&Vt[16 * dt + l16][32 * ks + 16 + 4 * g4];
        const u32x4_t vf = {lo[0], lo[1], hi[0], hi[1]};
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, vf), pb, o[dt], 0, 0, 0);
      }
    }
    if (qvalid) {
      const size_t base = ((size_t)c * a.M_max + (r0 + rr)) * a.nq + head;
      auto* op = GL(a.o_part) + base * HD;
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) *(GLOBAL f32x4_t*)(op + 16 * dt + 4 * g4) = o[dt];
      if (g4 == 0) *(GLOBAL f32x2_t*)(a.ml_part + base * 2) = f32x2_t{mx, sum};
    }
  }
}

// Merge the chunk partials of one (row, query head): out = sum_c w_c o_c / sum_c w_c l_c,
// w_c = 2^(m_c - max_c m_c), chunks in ascending order.
template <typename T>
__global__ void attn_merge_kernel(AttnArgs a, int hd) {
  const int m = blockIdx.x, head = blockIdx.y, d = threadIdx.x;
  if (m >= GL(a.row_offsets)[a.batch] || m >= a.M_max) return;
  const int b = seq_of_row(a.row_offsets, a.batch, m);
  const int rows = GL(a.row_offsets)[b + 1] - GL(a.row_offsets)[b];
  const int L = min(GL(a.seq_len)[b] + rows, a.ctx_limit);
  const int n_used = (L + kCh - 1) / kCh;
  const auto* ml = (const GLOBAL f32x2_t*)a.ml_part;
  const auto* op = GL(a.o_part);
  const size_t stride = (size_t)a.M_max * a.nq;  // between chunks, in (row, head) units
  const size_t rh = (size_t)m * a.nq + head;
  float M = -INFINITY;
#pragma unroll 8
  for (int c = 0; c < n_used; ++c) M = fmaxf(M, ml[c * stride + rh][0]);
  float num = 0.f, den = 0.f;
#pragma unroll 8
  for (int c = 0; c < n_used; ++c) {
    const f32x2_t v = ml[c * stride + rh];
    const float w = v[0] == -INFINITY ? 0.f : exp2f(v[0] - M);
    den += w * v[1];
    num += w * op[(c * stride + rh) * hd + d];
  }
  GL((T*)a.out)[rh * hd + d] = from_f32<T>(num / den);
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
  const float* V = (const float*)a.v + slab;
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
    float o = 0.f;
    for (int j = 0; j < L; ++j) o += sc[j] * V[(size_t)j * hd + i];
    ((float*)a.out)[((size_t)m * a.nq + head) * hd + i] = o / sum;
  }
}

int launch_attention(int dtype, int hd, const AttnArgs& a, int max_rows, int n_chunks, hipStream_t st) {
  if (dtype == LSV_DTYPE_BF16) {
    dim3 grid(n_chunks, a.nkv, a.batch);
    if (hd == 128)
      hipLaunchKernelGGL(attn_chunk_bf16_kernel<128>, grid, dim3(256), 0, st, a);
    else if (hd == 64)
      hipLaunchKernelGGL(attn_chunk_bf16_kernel<64>, grid, dim3(256), 0, st, a);
    else
      return LSV_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(attn_merge_kernel<bf16_t>, dim3(max_rows, a.nq), dim3(hd), 0, st, a, hd);
  } else {
    hipLaunchKernelGGL(attn_f32_kernel, dim3(max_rows, a.nq), dim3(64), sizeof(float) * (size_t)a.ctx_limit, st, a,
                       hd);
  }
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

}  // namespace lsv
