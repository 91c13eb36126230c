// Weight packing and the skinny-M matrix-core GEMM of the verify forward pass.
//
// Y[M, N] = X[M, K] * W[N, K]^T with M = the block's rows (a few to 64) and N, K
// in the thousands: the product streams W from HBM once, so the kernel is built
// around that stream.  W is pre-packed into 1 KiB fragments (16 rows x 32 bf16,
// or 16 rows x 16 fp32) laid out in the order a wave consumes them; each lane
// loads 16 contiguous bytes, so one wave-wide load is one contiguous KiB.  The
// fragment is the A operand of v_mfma_f32_16x16x32_bf16 (fp32: four
// v_mfma_f32_16x16x4_f32), weight rows being the MFMA rows.  The B operand --
// activation rows as MFMA columns -- is read the same way straight from the
// (L2-resident) activation buffer.  The k order inside a fragment is any
// permutation shared by A and B.
//
// RMSNorm: rmsnorm(h) g W^T = inv_rms[m] * (h (W o g)^T).  The gain g is folded
// into W when packing, the producer of h writes a storage-type copy of h and
// per-16-column sums of squares, and the consumer scales row m by inv_rms[m] in
// its epilogue.
//
// Work split: a workgroup owns one tile of TPW fragment rows (16*TPW output columns)
// over the whole K.  Its KS waves take balanced contiguous k-slices, each running its
// own software pipeline of NS stages x U k-steps; the slices meet in LDS and wave 0
// adds them in slice order (deterministic) and runs the epilogue.  No data crosses
// workgroups, so there are no partial buffers, counters or fences.  The residual a
// tile adds to is loaded ahead of the weight stream; inputs that need dependent loads
// (1/rms, cache positions) are read in the epilogue.
#include <math.h>

#include "lsv_device.h"
#include "lsv_attn.h"
#include "lsv_gemm.h"

namespace lsv {

// ------------------------------------------------------------------ packing
// dst fragment element (row pr, col c) = src[row][c] * gain[c] (rounded to the storage type).
template <typename T>
__global__ void __launch_bounds__(256) pack_kernel(int kind, int N, int K, int Nt, int Kt, const T* __restrict__ s0,
                                                   const T* __restrict__ s1, const T* __restrict__ s2,
                                                   const T* __restrict__ gain, int nq_rows, int nkv_rows, int hd,
                                                   T* __restrict__ dst) {
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
    const int c = col0 + e;
    float v = 0.f;
    if (row >= 0 && c < K) {
      v = to_f32<T>(src[(size_t)row * K + c]);
      if (gain) v *= to_f32<T>(gain[c]);
    }
    out[e] = from_f32<T>(v);
  }
}

int launch_pack(const Shape& s, PackKind kind, const PackedMat& pm, const void* src0, const void* src1,
                const void* src2, const void* gain, void* dst, hipStream_t stream) {
  const size_t threads = (size_t)pm.Nt * pm.Kt * 64;
  dim3 grid((unsigned)((threads + 255) / 256));
  char* d = (char*)dst + pm.offset;
  const int nq_rows = s.nq * s.hd, nkv_rows = s.nkv * s.hd;
  const int n_logical = kind == PACK_GATEUP ? s.F : pm.N;
  if (s.dtype == LSV_DTYPE_BF16)
    hipLaunchKernelGGL(pack_kernel<bf16_t>, grid, dim3(256), 0, stream, (int)kind, n_logical, pm.K, pm.Nt, pm.Kt,
                       (const bf16_t*)src0, (const bf16_t*)src1, (const bf16_t*)src2, (const bf16_t*)gain, nq_rows,
                       nkv_rows, s.hd, (bf16_t*)d);
  else
    hipLaunchKernelGGL(pack_kernel<float>, grid, dim3(256), 0, stream, (int)kind, n_logical, pm.K, pm.Nt, pm.Kt,
                       (const float*)src0, (const float*)src1, (const float*)src2, (const float*)gain, nq_rows,
                       nkv_rows, s.hd, (float*)d);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

// ------------------------------------------------------------------ MFMA on fragments
LSV_DEV void mfma_frag(const u32x4_t& a, const u32x4_t& b, f32x4_t& acc, bf16_t) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                acc, 0, 0, 0);
}
LSV_DEV void mfma_frag(const u32x4_t& a, const u32x4_t& b, f32x4_t& acc, float) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[e]), __uint_as_float(b[e]), acc, 0, 0, 0);
}

LSV_DEV u32x2_t pack_bf16x4(const f32x4_t v) {
  return u32x2_t{(uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16), (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16)};
}
// 4 consecutive outputs to global memory in the storage type
LSV_DEV void store4(float* p, const f32x4_t v) { *(GLOBAL f32x4_t*)p = v; }
LSV_DEV void store4(bf16_t* p, const f32x4_t v) { *(GLOBAL u32x2_t*)p = pack_bf16x4(v); }

constexpr int kMaxStatParts = 512;  // d_model / 16 for d_model <= 8192

// 1 / rms of activation row m from the producer's per-16-column sums of squares
// (stats[m][0..P)).  The four lanes sharing (lane & 15) take every fourth float4 of
// the row and combine their sums with a fixed shuffle tree: deterministic and the
// same in every lane.
LSV_DEV float inv_rms_of_row(const GemmArgs& a, int m, int g4) {
  const GLOBAL f32x4_t* st = (const GLOBAL f32x4_t*)(a.stats + (size_t)min(m, a.M_max - 1) * a.P);
  const int P4 = a.P >> 2;  // float4s per row (P is a multiple of 4)
  f32x4_t v[kMaxStatParts / 16];
#pragma unroll
  for (int j = 0; j < kMaxStatParts / 16; ++j) {
    const int i = g4 + 4 * j;
    v[j] = i < P4 ? st[i] : f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxStatParts / 16; ++j) ss += ((v[j][0] + v[j][1]) + v[j][2]) + v[j][3];
  ss += __shfl_xor(ss, 16, kWave);
  ss += __shfl_xor(ss, 32, kWave);
  return 1.0f / sqrtf(ss / (float)a.K + a.eps);
}

// ------------------------------------------------------------------ the GEMM
template <typename T, int MT, int TPW, int KS, int U, int NS, int EPI, int MT_MAX>
LSV_DEV void gemm_body(const GemmArgs& a, const int M, const int tile, const int m0,
                       f32x4_t (*red)[TPW][MT_MAX][kWave]) {
  constexpr int KT = FragTraits<T>::KT, EPL = FragTraits<T>::EPL;
  constexpr bool RMS = EPI != EPI_RESID;  // consumer of a normalised activation
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, l16 = lane & 15, g4 = lane >> 4;
  // this workgroup: fragment rows tn0 .. tn0+TPW-1 over the whole K, activation rows
  // m0 .. min(M, m0 + 16 MT) - 1; wave = k-slice
  const int tn0 = tile * TPW;
  const int k0 = (int)((long long)wave * a.Kt / KS), k1 = (int)((long long)(wave + 1) * a.Kt / KS);
  const int nk = k1 - k0;  // >= 0, and k0 < Kt for every wave
  bool tvalid[TPW];
  const GLOBAL u32x4_t* wp[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    tvalid[t] = tn0 + t < a.Nt;
    wp[t] = (const GLOBAL u32x4_t*)a.W + ((size_t)(tvalid[t] ? tn0 + t : 0) * a.Kt + k0) * 64 + lane;
  }

  // ---- the residual this tile adds to (EPI_RESID, wave 0 runs the epilogue): its loads are
  // issued ahead of the weight stream and retire with it
  f32x4_t hpre[TPW][MT];
  if (EPI == EPI_RESID && wave == 0) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = min(m0 + mt * 16 + l16, a.M_max - 1);
#pragma unroll
      for (int t = 0; t < TPW; ++t) {
        const int n0 = (tvalid[t] ? tn0 + t : 0) * 16 + 4 * g4;
        hpre[t][mt] = *(const GLOBAL f32x4_t*)(a.h_out + (size_t)m * a.N + n0);
      }
    }
  }

  // B operand: activation rows (clamped into the buffer; columns of rows >= M are never
  // stored, so their contents do not matter)
  const GLOBAL T* xp[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = min(m0 + mt * 16 + l16, a.M_max - 1);
    xp[mt] = (const GLOBAL T*)a.x + (size_t)m * a.ldx + (size_t)k0 * KT + g4 * EPL;
  }

  f32x4_t acc[TPW][MT];
#pragma unroll
  for (int t = 0; t < TPW; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  {
    // NS pipeline stages of U k-steps.  Every load hits an in-bounds fragment (index
    // clamped): a conditional load would become a select between addresses and a generic
    // access.  Steps past the range re-read the last one and are never used.
    u32x4_t wa[NS][U][TPW], xb[NS][U][MT];
    auto load_stage = [&](int st, int kb) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kf = max(min(kb + u, nk - 1), 0);  // a slice may be empty when Kt < KS
#pragma unroll
        for (int t = 0; t < TPW; ++t) wa[st][u][t] = wp[t][(size_t)kf * 64];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) xb[st][u][mt] = *(const GLOBAL u32x4_t*)(xp[mt] + (size_t)kf * KT);
      }
    };
    auto compute_stage = [&](int st, int kb, bool tail) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (!tail || kb + u < nk)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int t = 0; t < TPW; ++t) mfma_frag(wa[st][u][t], xb[st][u][mt], acc[t][mt], T{});
    };
    // Scheduling barriers keep the loads issued -- and so retired, vmcnt counting in
    // order -- stage by stage, and the loop body has no branches: while one stage is
    // multiplied the later ones are in flight.
    const int nfull = nk - nk % (NS * U);
#pragma unroll
    for (int st = 0; st < NS; ++st) {
      load_stage(st, st * U);
      __builtin_amdgcn_sched_barrier(0);
    }
    for (int kb = 0; kb < nfull; kb += NS * U) {
#pragma unroll
      for (int st = 0; st < NS; ++st) {
        compute_stage(st, kb + st * U, false);
        __builtin_amdgcn_sched_barrier(0);
        load_stage(st, kb + (NS + st) * U);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int st = 0; st < NS; ++st) compute_stage(st, nfull + st * U, true);
  }

  // ---- k-slices: waves 1.. hand their sums to wave 0 through LDS; summed in slice order
  if (KS > 1) {
    if (wave > 0) {
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) red[wave - 1][t][mt][lane] = acc[t][mt];
    }
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int w = 1; w < KS; ++w)
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[t][mt] += red[w - 1][t][mt][lane];
  }

  // ---- epilogues (wave 0); lane holds output columns n0..n0+3 (weight rows) of activation row m.
  // Row inputs that need dependent loads (1/rms, cache positions) are read here, off the
  // weight stream's critical path.
  float inv[MT];
  if (RMS) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) inv[mt] = inv_rms_of_row(a, m0 + mt * 16 + l16, g4);
  }
  int qkv_b[MT], qkv_pos[MT];
  if (EPI == EPI_QKV) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = min(m0 + mt * 16 + l16, a.M_max - 1);
      const int b = seq_of_row(a.row_offsets, a.batch, m);
      qkv_b[mt] = b;
      qkv_pos[mt] = GL(a.seq_len)[b] + (m - GL(a.row_offsets)[b]);
    }
  }
  if (EPI == EPI_LOGITS) {
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = m0 + mt * 16 + l16, n0 = (tn0 + t) * 16 + 4 * g4;
        if (m >= M || !tvalid[t]) continue;
        const f32x4_t v = acc[t][mt] * inv[mt];
        GLOBAL float* o = GL(a.out_f32) + (size_t)m * a.ldo;
        if (n0 + 3 < a.N && (a.ldo & 3) == 0) {
          *(GLOBAL f32x4_t*)(o + n0) = v;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (n0 + r < a.N) o[n0 + r] = v[r];
        }
      }
  } else if (EPI == EPI_QKV) {
      const int qrows = a.nq * a.hd, krows = a.nkv * a.hd;
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = m0 + mt * 16 + l16, n0 = (tn0 + t) * 16 + 4 * g4;
          if (m >= M || !tvalid[t] || n0 >= qrows + 2 * krows) continue;
          const int b = qkv_b[mt], pos = qkv_pos[mt];
          const f32x4_t v = acc[t][mt] * inv[mt];
          if (n0 < qrows + krows) {
            const bool isq = n0 < qrows;
            const int local = isq ? n0 : n0 - qrows;
            const int head = local / a.hd, i0 = (local % a.hd) >> 1;  // pairs (i0, i0+hd/2), (i0+1, i0+1+hd/2)
            float out[4];
#pragma unroll
            for (int pr = 0; pr < 2; ++pr) {
              // angle = pos * base^(-2i/hd) in fp64, reduced to [-pi, pi] in fp64, then fp32 sin/cos
              const int i = i0 + pr;
              const double inv_freq = exp2(-(double)(2 * i) / (double)a.hd * a.log2_rope_base);
              const double ang = (double)pos * inv_freq;
              const double red2pi = ang - 6.283185307179586 * rint(ang * 0.15915494309189535);
              float sn, cs;
              sincosf((float)red2pi, &sn, &cs);
              const float x1 = v[2 * pr], x2 = v[2 * pr + 1];
              out[2 * pr] = x1 * cs - x2 * sn;
              out[2 * pr + 1] = x2 * cs + x1 * sn;
            }
            T* dst;
            if (isq) {
              dst = (T*)a.q_out + ((size_t)m * a.nq + head) * a.hd;
            } else {
              if (pos < 0 || pos >= a.capacity) continue;
              dst = (T*)a.kv + ((((size_t)a.layer * 2 + 0) * a.batch + b) * a.nkv + head) * (size_t)a.capacity * a.hd +
                    (size_t)pos * a.hd;
            }
            GLOBAL T* gd = GL(dst);
            gd[i0] = from_f32<T>(out[0]);
            gd[i0 + a.hd / 2] = from_f32<T>(out[1]);
            gd[i0 + 1] = from_f32<T>(out[2]);
            gd[i0 + 1 + a.hd / 2] = from_f32<T>(out[3]);
          } else {
            if (pos < 0 || pos >= a.capacity) continue;
            // V rows are stored transposed: [head_dim][capacity], column v_column(pos)
            const int local = n0 - qrows - krows;
            const int head = local / a.hd, d0 = local % a.hd;
            GLOBAL T* dst = GL((T*)a.kv) +
                            ((((size_t)a.layer * 2 + 1) * a.batch + b) * a.nkv + head) * (size_t)a.capacity * a.hd +
                            (size_t)d0 * a.capacity + v_column(pos);
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[(size_t)r * a.capacity] = from_f32<T>(v[r]);
          }
        }
    } else if (EPI == EPI_RESID) {
      // h += y; the storage-type copy of h for the next consumer; per-row sum of squares of
      // the new h over this fragment row's 16 columns (stats[m][n / 16])
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = m0 + mt * 16 + l16, n0 = (tn0 + t) * 16 + 4 * g4;
          float ss = 0.f;
          if (m < M && tvalid[t]) {
            const f32x4_t h4 = hpre[t][mt] + acc[t][mt];
            *(GLOBAL f32x4_t*)(a.h_out + (size_t)m * a.N + n0) = h4;
            if (a.hx_out) store4((T*)a.hx_out + (size_t)m * a.N + n0, h4);
            ss = ((h4[0] * h4[0] + h4[1] * h4[1]) + h4[2] * h4[2]) + h4[3] * h4[3];
          }
          ss += __shfl_xor(ss, 16, kWave);
          ss += __shfl_xor(ss, 32, kWave);
          if (g4 == 0 && m < M && tvalid[t]) GL(a.stats_out)[(size_t)m * (a.N / 16) + tn0 + t] = ss;
        }
    } else if (EPI == EPI_SWIGLU) {
      static_assert(EPI != EPI_SWIGLU || TPW == 2, "SwiGLU pairs a gate and an up fragment row");
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = m0 + mt * 16 + l16, f0 = (tn0 >> 1) * 16 + 4 * g4;
        if (m >= M || !tvalid[0]) continue;
        f32x4_t out;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float gt = acc[0][mt][r] * inv[mt], up = acc[TPW - 1][mt][r] * inv[mt];
          out[r] = gt / (1.0f + expf(-gt)) * up;
        }
        T* dst = (T*)a.u_out + (size_t)m * a.ldu + f0;
        if (f0 + 3 < a.F) {
          store4(dst, out);
        } else {
          for (int r = 0; r < 4; ++r)
            if (f0 + r < a.F) GL(dst)[r] = from_f32<T>(out[r]);
        }
      }
    }
}

// Launch configuration of each product: fragment rows per wave (TPW), k-slices = waves
// per workgroup (KS), k-steps per pipeline stage (U) and stages in flight (NS).  Chosen by
// measurement on the Llama-3-8B shapes: enough bytes in flight per compute unit, a wave
// count that spreads evenly over the 256 compute units, and few waves per tile for the
// long products.
template <int KIND> struct GemmCfg;
template <> struct GemmCfg<GEMM_QKV> { static constexpr int TPW = 1, KS = 2, U = 8, NS = 2, EPI = EPI_QKV; };
template <> struct GemmCfg<GEMM_O> { static constexpr int TPW = 1, KS = 4, U = 8, NS = 2, EPI = EPI_RESID; };
template <> struct GemmCfg<GEMM_GATEUP> { static constexpr int TPW = 2, KS = 1, U = 4, NS = 3, EPI = EPI_SWIGLU; };
template <> struct GemmCfg<GEMM_DOWN> { static constexpr int TPW = 1, KS = 4, U = 8, NS = 2, EPI = EPI_RESID; };
template <> struct GemmCfg<GEMM_LMHEAD> { static constexpr int TPW = 2, KS = 1, U = 4, NS = 3, EPI = EPI_LOGITS; };

// Wide activation tiles (prefill bounds) use a shallower pipeline to stay in registers.
template <int KIND, int MT_MAX> struct GemmShape {
  using C = GemmCfg<KIND>;
  static constexpr int TPW = C::TPW, KS = C::KS, EPI = C::EPI;
  static constexpr int U = MT_MAX <= 2 ? C::U : 4, NS = MT_MAX <= 2 ? C::NS : 2;
};

// Rows come in chunks of 64 (4 activation tiles); a chunk's workgroups read the same
// weights, so the grid puts the chunks of one column tile on the same XCD (workgroup
// ids congruent mod 8 share one) where the repeated reads hit its L2.  The host bound
// on rows fixes MT_MAX; the kernel runs the body for the activation tiles that the
// device row count of its chunk actually needs, so a generous bound costs nothing.
template <typename T, int KIND, int MT_MAX>
__global__ void __launch_bounds__(64 * GemmCfg<KIND>::KS) gemm_kernel(GemmArgs a) {
  using S = GemmShape<KIND, MT_MAX>;
  __shared__ f32x4_t red[S::KS > 1 ? S::KS - 1 : 1][S::TPW][MT_MAX][kWave];  // k-slice sums
  const int tiles = (a.Nt + S::TPW - 1) / S::TPW, nch = (a.M_max + 63) / 64;
  const int round = blockIdx.x >> 3, chunk = round % nch, tile = (round / nch) * 8 + (blockIdx.x & 7);
  if (tile >= tiles) return;
  const int M = min(GL(a.row_offsets)[a.batch], a.M_max);  // never trust device rows beyond the host bound
  const int m0 = chunk * 64;
  if (m0 >= M) return;
  const int Mc = min(M - m0, 64);
  const int M_end = m0 + Mc;
  const int mt = Mc <= 16 ? 1 : (Mc <= 32 ? 2 : (Mc <= 48 ? 3 : 4));
  if (mt <= 1 || MT_MAX == 1)
    gemm_body<T, 1, S::TPW, S::KS, S::U, S::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, red);
  else if (mt == 2 || MT_MAX == 2)
    gemm_body<T, (MT_MAX >= 2 ? 2 : 1), S::TPW, S::KS, S::U, S::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, red);
  else if (mt == 3 || MT_MAX == 3)
    gemm_body<T, (MT_MAX >= 3 ? 3 : 1), S::TPW, S::KS, S::U, S::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, red);
  else
    gemm_body<T, MT_MAX, S::TPW, S::KS, S::U, S::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, red);
}

// ------------------------------------------------------------------ planning and launch
template <typename T, int KIND, int MT_MAX>
static void launch_one(const GemmArgs& a, hipStream_t st) {
  constexpr int TPW = GemmCfg<KIND>::TPW, KS = GemmCfg<KIND>::KS;
  const int tiles = (a.Nt + TPW - 1) / TPW, nch = (a.M_max + 63) / 64;
  const unsigned grid = (unsigned)((tiles + 7) / 8 * 8 * nch);
  hipLaunchKernelGGL((gemm_kernel<T, KIND, MT_MAX>), dim3(grid), dim3(64 * KS), 0, st, a);
}

template <typename T, int KIND>
static int launch_mt(int MT, const GemmArgs& a, hipStream_t st) {
  switch (MT) {
    case 1: launch_one<T, KIND, 1>(a, st); break;
    case 2: launch_one<T, KIND, 2>(a, st); break;
    case 3: launch_one<T, KIND, 3>(a, st); break;
    case 4: launch_one<T, KIND, 4>(a, st); break;
    default: return LSV_ERR_UNSUPPORTED;
  }
  return LSV_OK;
}

template <typename T>
static int launch_typed(GemmKind kind, int MT, const GemmArgs& a, hipStream_t st) {
  switch (kind) {
    case GEMM_QKV: return launch_mt<T, GEMM_QKV>(MT, a, st);
    case GEMM_O: return launch_mt<T, GEMM_O>(MT, a, st);
    case GEMM_GATEUP: return launch_mt<T, GEMM_GATEUP>(MT, a, st);
    case GEMM_DOWN: return launch_mt<T, GEMM_DOWN>(MT, a, st);
    case GEMM_LMHEAD: return launch_mt<T, GEMM_LMHEAD>(MT, a, st);
  }
  return LSV_ERR_UNSUPPORTED;
}

int launch_gemm(int dtype, GemmKind kind, int MT, const GemmArgs& a, hipStream_t st) {
  int rc = dtype == LSV_DTYPE_BF16 ? launch_typed<bf16_t>(kind, MT, a, st) : launch_typed<float>(kind, MT, a, st);
  if (rc != LSV_OK) return rc;
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

}  // namespace lsv
