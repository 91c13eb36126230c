// Weight packing and the skinny-M matrix-core GEMM of the verify forward pass.
//
// Y[M, N] = X[M, K] * W[N, K]^T with M = the block's rows (a few to 64) and N, K
// in the thousands: the product streams W from HBM once, so the kernel is built
// around that stream.  W is pre-packed into 1 KiB fragments (16 rows x 32 bf16,
// or 16 rows x 16 fp32) laid out in the order a wave consumes them; each lane
// loads 16 contiguous bytes, so one wave-wide load is one contiguous KiB.  The
// fragment is the A operand of v_mfma_f32_16x16x32_bf16 (fp32: four
// v_mfma_f32_16x16x4_f32), with weight rows as the MFMA rows; the activation rows
// are the MFMA columns, staged once per workgroup in LDS with the RMSNorm
// prologue applied.  The k order inside a fragment is any permutation shared by
// A and B, so the packed layout is free to be the one that streams best.
//
// Work split: blockIdx.x = a group of 4 waves x TPW fragment rows (64*TPW
// output columns), blockIdx.y = a split of K.  With several splits every
// workgroup writes fp32 partials and the last one to arrive (device-scope
// counter) sums them in split order -- deterministic -- and runs the epilogue.
#include <math.h>

#include "lsv_device.h"
#include "lsv_gemm.h"

namespace lsv {

// ------------------------------------------------------------------ packing
template <typename T>
__global__ void __launch_bounds__(256) pack_kernel(int kind, int N, int K, int Nt, int Kt, const T* __restrict__ s0,
                                                   const T* __restrict__ s1, const T* __restrict__ s2, int nq_rows,
                                                   int nkv_rows, int hd, T* __restrict__ dst) {
  constexpr int EPL = FragTraits<T>::EPL, KT = FragTraits<T>::KT;
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t frag = gid >> 6;
  const int lane = (int)(gid & 63);
  if (frag >= (size_t)Nt * Kt) return;
  const int tn = (int)(frag / Kt), tk = (int)(frag % Kt);
  const int pr = 16 * tn + (lane & 15);
  const int col0 = tk * KT + (lane >> 4) * EPL;
  const T* src = nullptr;
  int row = -1;
  if (kind == PACK_PLAIN) {
    src = s0;
    row = pr < N ? pr : -1;
  } else if (kind == PACK_QKV) {
    // q and k rows are reordered inside each head so that packed rows (2i, 2i+1)
    // hold dims (i, i + hd/2), the two halves of a rotary pair
    int base = 0;
    if (pr < nq_rows) {
      src = s0;
    } else if (pr < nq_rows + nkv_rows) {
      src = s1;
      base = nq_rows;
    } else if (pr < nq_rows + 2 * nkv_rows) {
      src = s2;
      base = nq_rows + nkv_rows;
    }
    if (src) {
      int local = pr - base;
      if (src != s2) {
        int head = local / hd, p = local % hd;
        local = head * hd + ((p & 1) ? (p >> 1) + hd / 2 : (p >> 1));
      }
      row = local;
    }
  } else {  // PACK_GATEUP: fragment rows alternate 16 gate rows, 16 up rows
    src = (tn & 1) ? s1 : s0;
    int r = 16 * (tn >> 1) + (lane & 15);
    row = r < N ? r : -1;
  }
  T* out = dst + frag * 64 * EPL + (size_t)lane * EPL;
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    int c = col0 + e;
    out[e] = (row >= 0 && c < K) ? src[(size_t)row * K + c] : from_f32<T>(0.f);
  }
}

int launch_pack(const Shape& s, PackKind kind, const PackedMat& pm, const void* src0, const void* src1,
                const void* src2, void* dst, hipStream_t stream) {
  const size_t threads = (size_t)pm.Nt * pm.Kt * 64;
  dim3 grid((unsigned)((threads + 255) / 256));
  char* d = (char*)dst + pm.offset;
  const int nq_rows = s.nq * s.hd, nkv_rows = s.nkv * s.hd;
  const int n_logical = kind == PACK_GATEUP ? s.F : pm.N;
  if (s.dtype == LSV_DTYPE_BF16)
    hipLaunchKernelGGL(pack_kernel<bf16_t>, grid, dim3(256), 0, stream, (int)kind, n_logical, pm.K, pm.Nt, pm.Kt,
                       (const bf16_t*)src0, (const bf16_t*)src1, (const bf16_t*)src2, nq_rows, nkv_rows, s.hd,
                       (bf16_t*)d);
  else
    hipLaunchKernelGGL(pack_kernel<float>, grid, dim3(256), 0, stream, (int)kind, n_logical, pm.K, pm.Nt, pm.Kt,
                       (const float*)src0, (const float*)src1, (const float*)src2, nq_rows, nkv_rows, s.hd,
                       (float*)d);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

// ------------------------------------------------------------------ MFMA on fragments
LSV_DEV void mfma_frag(const uint4& a, const uint4& b, f32x4_t& acc, bf16_t) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                acc, 0, 0, 0);
}
LSV_DEV void mfma_frag(const uint4& a, const uint4& b, f32x4_t& acc, float) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// 4 consecutive storage elements <-> floats
LSV_DEV void load4(const float* p, float v[4]) {
  float4 x = *(const float4*)p;
  v[0] = x.x, v[1] = x.y, v[2] = x.z, v[3] = x.w;
}
LSV_DEV void load4(const bf16_t* p, float v[4]) {
  uint2 x = *(const uint2*)p;
  v[0] = __uint_as_float(x.x << 16), v[1] = __uint_as_float(x.x & 0xffff0000u);
  v[2] = __uint_as_float(x.y << 16), v[3] = __uint_as_float(x.y & 0xffff0000u);
}
LSV_DEV void store4(float* p, const float v[4]) { *(float4*)p = make_float4(v[0], v[1], v[2], v[3]); }
LSV_DEV void store4(bf16_t* p, const float v[4]) {
  uint2 x;
  x.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
  x.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
  *(uint2*)p = x;
}

// ------------------------------------------------------------------ the GEMM
template <typename T, int MT, int TPW, int PRO, int EPI>
__global__ void __launch_bounds__(256) gemm_kernel(GemmArgs a) {
  constexpr int KT = FragTraits<T>::KT, EPL = FragTraits<T>::EPL;
  constexpr int WAVES = 4;
  constexpr int U = TPW == 1 ? 8 : 4;  // fragments per wave per pipeline stage (per tile)
  constexpr int ROWS = MT * 16;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int group = blockIdx.x, split = blockIdx.y;
  const int M = min(a.row_offsets[a.batch], a.M_max);  // never trust device rows beyond the host bound
  const int kf0 = (int)((long long)split * a.Kt / a.S), kf1 = (int)((long long)(split + 1) * a.Kt / a.S);
  const int nkf = kf1 - kf0;
  const int ldsx = a.kf_max * KT + 16 / (int)sizeof(T);

  extern __shared__ __align__(16) char smem[];
  T* X = (T*)smem;                                                  // [ROWS][ldsx]
  float* inv_rms = (float*)(smem + (size_t)ROWS * ldsx * sizeof(T));  // [ROWS]
  float* red = inv_rms + ROWS;                                      // [WAVES*TPW][ROWS]
  int* flag = (int*)(red + WAVES * TPW * ROWS);

  const int tn0 = (group * WAVES + wave) * TPW;
  bool tvalid[TPW];
  const uint4* wp[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    tvalid[t] = tn0 + t < a.Nt;
    wp[t] = a.W + ((size_t)(tvalid[t] ? tn0 + t : 0) * a.Kt + kf0) * 64 + lane;
  }
  const uint4 zero4 = make_uint4(0, 0, 0, 0);
  uint4 cur[U][TPW], nxt[U][TPW];
  auto load_stage = [&](uint4 (&buf)[U][TPW], int kb) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < TPW; ++t)
        buf[u][t] = (kb + u < nkf && tvalid[t]) ? wp[t][(size_t)(kb + u) * 64] : zero4;
  };
  load_stage(cur, 0);  // weight stream starts before the activation prologue

  // ---- prologue: activations for this K split -> LDS (RMSNorm applied), zero-padded
  if (PRO == PRO_RMS) {
    for (int m = threadIdx.x; m < ROWS; m += blockDim.x) {
      float ss = 0.f;
      if (m < M)
        for (int p = 0; p < a.P; ++p) ss += a.stats[(size_t)p * a.M_max + m];
      inv_rms[m] = m < M ? 1.0f / sqrtf(ss / (float)a.K + a.eps) : 0.f;
    }
    __syncthreads();
  }
  {
    const int kcols = nkf * KT;  // multiple of 4
    const int units = ROWS * (kcols >> 2);
    for (int i = threadIdx.x; i < units; i += blockDim.x) {
      const int m = i / (kcols >> 2), c4 = (i % (kcols >> 2)) * 4;
      const int k = kf0 * KT + c4;
      float v[4] = {0.f, 0.f, 0.f, 0.f};
      if (m < M && k < a.K) {
        if (PRO == PRO_RMS) {
          float g[4];
          load4(a.h + (size_t)m * a.K + k, v);
          load4((const T*)a.gain + k, g);
          const float r = inv_rms[m];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = v[e] * r * g[e];
        } else {
          load4((const T*)a.x + (size_t)m * a.ldx + k, v);
        }
      }
      store4(X + (size_t)m * ldsx + c4, v);
    }
  }
  __syncthreads();

  // ---- main loop: stream weight fragments, B operand from LDS
  f32x4_t acc[TPW][MT];
#pragma unroll
  for (int t = 0; t < TPW; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const T* xrow = X + (size_t)(lane & 15) * ldsx + (lane >> 4) * EPL;
  for (int kb = 0; kb < nkf; kb += U) {
    if (kb + U < nkf) load_stage(nxt, kb + U);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kb + u < nkf) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const uint4 bf = *(const uint4*)(xrow + (size_t)mt * 16 * ldsx + (kb + u) * KT);
#pragma unroll
          for (int t = 0; t < TPW; ++t) mfma_frag(cur[u][t], bf, acc[t][mt], T{});
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < TPW; ++t) cur[u][t] = nxt[u][t];
  }

  // ---- split-K: partials, last workgroup reduces in split order
  const int Np = a.Nt * 16;
  if (a.S > 1) {
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + (lane & 15), n = (tn0 + t) * 16 + 4 * (lane >> 4);
        if (m < M && tvalid[t]) *(f32x4_t*)(a.part + ((size_t)split * a.M_max + m) * Np + n) = acc[t][mt];
      }
    if (!arrive_last(&a.counters[group], a.S, flag)) return;
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + (lane & 15), n = (tn0 + t) * 16 + 4 * (lane >> 4);
        f32x4_t s = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if (m < M && tvalid[t])
          for (int sp = 0; sp < a.S; ++sp) s += *(const f32x4_t*)(a.part + ((size_t)sp * a.M_max + m) * Np + n);
        acc[t][mt] = s;
      }
    reset_counter(&a.counters[group]);
  }

  // ---- epilogues; lane holds rows n0..n0+3 (weights) x column m (activation row)
  if (EPI == EPI_LOGITS) {
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + (lane & 15), n0 = (tn0 + t) * 16 + 4 * (lane >> 4);
        if (m >= M || !tvalid[t]) continue;
        float* o = a.out_f32 + (size_t)m * a.ldo;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (n0 + r < a.N) o[n0 + r] = acc[t][mt][r];
      }
  } else if (EPI == EPI_QKV) {
    const int qrows = a.nq * a.hd, krows = a.nkv * a.hd;
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + (lane & 15), n0 = (tn0 + t) * 16 + 4 * (lane >> 4);
        if (m >= M || !tvalid[t] || n0 >= qrows + 2 * krows) continue;
        const int b = seq_of_row(a.row_offsets, a.batch, m);
        const int pos = a.seq_len[b] + (m - a.row_offsets[b]);
        const f32x4_t v = acc[t][mt];
        if (n0 < qrows + krows) {
          const bool isq = n0 < qrows;
          const int local = isq ? n0 : n0 - qrows;
          const int head = local / a.hd, i0 = (local % a.hd) >> 1;  // pairs (i0, i0+hd/2), (i0+1, i0+1+hd/2)
          float out[4];
#pragma unroll
          for (int pr = 0; pr < 2; ++pr) {
            const int i = i0 + pr;
            const double inv_freq = pow(a.rope_base, -2.0 * (double)i / (double)a.hd);
            const double ang = (double)pos * inv_freq;
            const float c = (float)cos(ang), s = (float)sin(ang);
            const float x1 = v[2 * pr], x2 = v[2 * pr + 1];
            out[2 * pr] = x1 * c - x2 * s;
            out[2 * pr + 1] = x2 * c + x1 * s;
          }
          T* dst;
          if (isq) {
            dst = (T*)a.q_out + ((size_t)m * a.nq + head) * a.hd;
          } else {
            if (pos < 0 || pos >= a.capacity) continue;
            dst = (T*)a.kv + ((((size_t)a.layer * 2 + 0) * a.batch + b) * a.nkv + head) * (size_t)a.capacity * a.hd +
                  (size_t)pos * a.hd;
          }
          dst[i0] = from_f32<T>(out[0]);
          dst[i0 + a.hd / 2] = from_f32<T>(out[1]);
          dst[i0 + 1] = from_f32<T>(out[2]);
          dst[i0 + 1 + a.hd / 2] = from_f32<T>(out[3]);
        } else {
          if (pos < 0 || pos >= a.capacity) continue;
          const int local = n0 - qrows - krows;
          const int head = local / a.hd, d0 = local % a.hd;
          T* dst = (T*)a.kv + ((((size_t)a.layer * 2 + 1) * a.batch + b) * a.nkv + head) * (size_t)a.capacity * a.hd +
                   (size_t)pos * a.hd + d0;
          float out[4] = {v[0], v[1], v[2], v[3]};
          store4(dst, out);
        }
      }
  } else if (EPI == EPI_RESID) {
    // h += y; then per-row sums of squares of the new h over each 64-column group
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + (lane & 15), n0 = (tn0 + t) * 16 + 4 * (lane >> 4);
        float ss = 0.f;
        if (m < M && tvalid[t]) {
          float* hp = a.h_out + (size_t)m * a.N + n0;
          float4 h4 = *(float4*)hp;
          h4.x += acc[t][mt][0];
          h4.y += acc[t][mt][1];
          h4.z += acc[t][mt][2];
          h4.w += acc[t][mt][3];
          *(float4*)hp = h4;
          ss = ((h4.x * h4.x + h4.y * h4.y) + h4.z * h4.z) + h4.w * h4.w;
        }
        ss += __shfl_xor(ss, 16, kWave);
        ss += __shfl_xor(ss, 32, kWave);
        if (lane < 16) red[(wave * TPW + t) * ROWS + mt * 16 + lane] = ss;
      }
    __syncthreads();
    // 64-column groups: tiles 4p..4p+3 of this workgroup, summed in order
    constexpr int PARTS = WAVES * TPW / 4;
    for (int i = threadIdx.x; i < PARTS * ROWS; i += blockDim.x) {
      const int p = i / ROWS, m = i % ROWS;
      if (m >= M) continue;
      const int gp = group * PARTS + p;
      if (gp * 64 >= a.N) continue;
      const float s = ((red[(4 * p + 0) * ROWS + m] + red[(4 * p + 1) * ROWS + m]) + red[(4 * p + 2) * ROWS + m]) +
                      red[(4 * p + 3) * ROWS + m];
      a.stats_out[(size_t)gp * a.M_max + m] = s;
    }
  } else if (EPI == EPI_SWIGLU) {
    static_assert(EPI != EPI_SWIGLU || TPW == 2, "SwiGLU pairs a gate and an up fragment row");
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = mt * 16 + (lane & 15), f0 = (tn0 >> 1) * 16 + 4 * (lane >> 4);
      if (m >= M || !tvalid[0]) continue;
      float out[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float g = acc[0][mt][r], u = acc[TPW - 1][mt][r];
        out[r] = g / (1.0f + expf(-g)) * u;
      }
      T* dst = (T*)a.u_out + (size_t)m * a.F + f0;
      if (f0 + 3 < a.F) {
        store4(dst, out);
      } else {
        for (int r = 0; r < 4; ++r)
          if (f0 + r < a.F) dst[r] = from_f32<T>(out[r]);
      }
    }
  }
}

// ------------------------------------------------------------------ planning and launch
GemmPlan plan_gemm(int Nt, int Kt, int KT, int es, int MT, int TPW, int want_wgs, int max_splits) {
  GemmPlan p;
  p.groups = (Nt + 4 * TPW - 1) / (4 * TPW);
  const int rows = MT * 16;
  // LDS budget for the activation tile: 60 KiB (the whole workgroup stays under 64 KiB)
  const int lds_cap_frags = (int)((61440 / (rows * es) - 16 / es) / KT);
  int S = (want_wgs + p.groups - 1) / p.groups;
  S = S < 1 ? 1 : S;
  const int min_s_lds = (Kt + lds_cap_frags - 1) / lds_cap_frags;
  S = S < min_s_lds ? min_s_lds : S;
  S = S > Kt ? Kt : S;
  S = S > max_splits ? max_splits : S;
  if ((Kt + S - 1) / S > lds_cap_frags) S = min_s_lds;  // LDS wins over the split cap
  p.S = S;
  p.kf_max = (Kt + S - 1) / S;
  const int ldsx = p.kf_max * KT + 16 / es;
  p.lds_bytes = (size_t)rows * ldsx * es + sizeof(float) * (size_t)rows * (1 + 4 * TPW) + 16;
  return p;
}

template <typename T, int MT, int TPW, int PRO, int EPI>
static void launch_one(const GemmArgs& a, const GemmPlan& p, hipStream_t st) {
  hipLaunchKernelGGL((gemm_kernel<T, MT, TPW, PRO, EPI>), dim3(p.groups, p.S), dim3(256), p.lds_bytes, st, a);
}

template <typename T, int TPW, int PRO, int EPI>
static int launch_mt(int MT, const GemmArgs& a, const GemmPlan& p, hipStream_t st) {
  switch (MT) {
    case 1: launch_one<T, 1, TPW, PRO, EPI>(a, p, st); break;
    case 2: launch_one<T, 2, TPW, PRO, EPI>(a, p, st); break;
    case 3: launch_one<T, 3, TPW, PRO, EPI>(a, p, st); break;
    case 4: launch_one<T, 4, TPW, PRO, EPI>(a, p, st); break;
    default: return LSV_ERR_UNSUPPORTED;
  }
  return LSV_OK;
}

template <typename T>
static int launch_typed(GemmKind kind, int MT, const GemmArgs& a, const GemmPlan& p, hipStream_t st) {
  switch (kind) {
    case GEMM_QKV: return launch_mt<T, 1, PRO_RMS, EPI_QKV>(MT, a, p, st);
    case GEMM_O: return launch_mt<T, 1, PRO_PLAIN, EPI_RESID>(MT, a, p, st);
    case GEMM_GATEUP: return launch_mt<T, 2, PRO_RMS, EPI_SWIGLU>(MT, a, p, st);
    case GEMM_DOWN: return launch_mt<T, 1, PRO_PLAIN, EPI_RESID>(MT, a, p, st);
    case GEMM_LMHEAD: return launch_mt<T, 1, PRO_RMS, EPI_LOGITS>(MT, a, p, st);
  }
  return LSV_ERR_UNSUPPORTED;
}

int launch_gemm(int dtype, GemmKind kind, int MT, const GemmArgs& a, const GemmPlan& p, hipStream_t st) {
  int rc = dtype == LSV_DTYPE_BF16 ? launch_typed<bf16_t>(kind, MT, a, p, st) : launch_typed<float>(kind, MT, a, p, st);
  if (rc != LSV_OK) return rc;
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

int gemm_tpw(GemmKind kind) { return kind == GEMM_GATEUP ? 2 : 1; }

}  // namespace lsv
