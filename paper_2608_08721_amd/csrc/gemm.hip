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
// (L2-resident) activation buffer: no LDS staging, no barrier in front of the
// stream, every wave runs its own two-stage software pipeline.  The k order
// inside a fragment is any permutation shared by A and B.
//
// RMSNorm: rmsnorm(h) g W^T = inv_rms[m] * (h (W o g)^T).  The gain g is folded
// into W when packing, the producer of h writes a bf16 copy of h and per-64-
// column sums of squares, and the consumer scales row m by inv_rms[m] in its
// epilogue.
//
// Work split (stream-K): a workgroup of 4 waves processes "steps" = one k-fragment
// of a tile group (4 waves x TPW fragment rows = 64*TPW output columns).  The
// groups x Kt steps are cut into gridDim.x equal contiguous ranges, so every
// workgroup streams the same number of bytes and the launch has no tail round.
// A group covered by one workgroup runs its epilogue directly; otherwise each
// contributor publishes an fp32 partial with 16-byte device-scope stores and bumps
// a device-scope counter, and the last to arrive reads the partials back (device
// scope) in k order -- deterministic -- and runs the epilogue.  Device-scope
// accesses go through the coherent path, so no cache write-back is needed between
// a contributor and the reducer.
#include <math.h>

#include "lsv_device.h"
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

// 1 / rms of activation row m from the producer's per-64-column sums of squares.
// The four lanes sharing (lane & 15) split the partials (p = g, g+4, ...) and
// combine them with a fixed shuffle tree: deterministic and the same in every lane.
// All loads are issued before the first use (P <= kMaxStatParts), then summed in order.
constexpr int kMaxStatParts = 128;  // d_model <= 8192
LSV_DEV float inv_rms_of_row(const GemmArgs& a, int m, int g4) {
  const GLOBAL float* st = GL(a.stats) + (m < a.M_max ? m : 0);
  float v[kMaxStatParts / 4];
#pragma unroll
  for (int j = 0; j < kMaxStatParts / 4; ++j) {
    const int p = g4 + 4 * j;
    v[j] = p < a.P ? st[(size_t)min(p, a.P - 1) * a.M_max] : 0.f;
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxStatParts / 4; ++j) ss += v[j];
  ss += __shfl_xor(ss, 16, kWave);
  ss += __shfl_xor(ss, 32, kWave);
  return 1.0f / sqrtf(ss / (float)a.K + a.eps);
}

// ------------------------------------------------------------------ the GEMM
// Raw buffer resource over the partials (word 3 = the gfx9-family raw-buffer format).
LSV_DEV __amdgpu_buffer_rsrc_t part_rsrc(float* base, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, (int)(bytes > 0x7fffffffu ? 0x7fffffffu : bytes), 0x00020000);
}
constexpr int kDeviceScope = 16;  // buffer cache policy: sc1 (coherent at device scope)

// Which workgroup's step range contains step i (ranges start at floor(w T / W)).
LSV_DEV int owner_of(long long i, long long T, int W) { return (int)(((i + 1) * W - 1) / T); }

template <typename T, int MT, int TPW, int EPI, int ROWS_SH>
LSV_DEV void gemm_body(const GemmArgs& a, const int M, float (*red)[ROWS_SH], int& flag) {
  constexpr int KT = FragTraits<T>::KT, EPL = FragTraits<T>::EPL;
  constexpr int WAVES = 4, U = 4;  // U k-steps per pipeline stage
  constexpr bool RMS = EPI != EPI_RESID;  // consumer of a normalised activation
  constexpr int ROWS = MT * 16, GCOLS = 64 * TPW;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, l16 = lane & 15, g4 = lane >> 4;
  const int W = gridDim.x, w = blockIdx.x;
  const long long Tsteps = (long long)a.groups * a.Kt;
  const long long s_begin = (long long)w * Tsteps / W, s_end = (long long)(w + 1) * Tsteps / W;


  // B operand: activation rows (clamped into the buffer; columns of rows >= M are never
  // stored, so their contents do not matter)
  const GLOBAL T* xp[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = min(mt * 16 + l16, a.M_max - 1);
    xp[mt] = (const GLOBAL T*)a.x + (size_t)m * a.ldx + g4 * EPL;
  }
  float inv[MT];  // computed at the first epilogue, off the weight stream's critical path
  bool inv_ready = false;
  const __amdgpu_buffer_rsrc_t prs = part_rsrc(a.part, a.part_bytes);

  for (long long g = s_begin / a.Kt; g * a.Kt < s_end; ++g) {
    const int k0 = (int)(max(s_begin, g * a.Kt) - g * a.Kt), k1 = (int)(min(s_end, (g + 1) * a.Kt) - g * a.Kt);
    const int nk = k1 - k0;
    const int tn0 = ((int)g * WAVES + wave) * TPW;
    bool tvalid[TPW];
    const GLOBAL u32x4_t* wp[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      tvalid[t] = tn0 + t < a.Nt;
      wp[t] = (const GLOBAL u32x4_t*)a.W + ((size_t)(tvalid[t] ? tn0 + t : 0) * a.Kt + k0) * 64 + lane;
    }
    // Every load hits an in-bounds fragment (index clamped): a conditional load would become
    // a select between addresses and a generic access.  Steps past the range are never used.
    u32x4_t wa[2][U][TPW], xb[2][U][MT];
    auto load_stage = [&](int st, int kb) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kf = min(kb + u, nk - 1);
#pragma unroll
        for (int t = 0; t < TPW; ++t) wa[st][u][t] = wp[t][(size_t)kf * 64];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) xb[st][u][mt] = *(const GLOBAL u32x4_t*)(xp[mt] + (size_t)(k0 + kf) * KT);
      }
    };
    f32x4_t acc[TPW][MT];
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    auto compute_stage = [&](int st) {  // all U steps, no per-step conditions
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int t = 0; t < TPW; ++t) mfma_frag(wa[st][u][t], xb[st][u][mt], acc[t][mt], T{});
    };
    auto compute_tail = [&](int st, int kb) {  // the last (< 2U) steps
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (kb + u < nk)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int t = 0; t < TPW; ++t) mfma_frag(wa[st][u][t], xb[st][u][mt], acc[t][mt], T{});
    };
    // Scheduling barriers keep the loads issued -- and so retired, vmcnt counting in
    // order -- stage by stage, and the loop body has no branches: while one stage is
    // multiplied the other is in flight.  Loads past the range re-read the last step.
    const int nfull = nk - nk % (2 * U);
    load_stage(0, 0);
    __builtin_amdgcn_sched_barrier(0);
    load_stage(1, U);
    __builtin_amdgcn_sched_barrier(0);
    for (int kb = 0; kb < nfull; kb += 2 * U) {
      compute_stage(0);
      __builtin_amdgcn_sched_barrier(0);
      load_stage(0, kb + 2 * U);
      __builtin_amdgcn_sched_barrier(0);
      compute_stage(1);
      __builtin_amdgcn_sched_barrier(0);
      load_stage(1, kb + 3 * U);
      __builtin_amdgcn_sched_barrier(0);
    }
    compute_tail(0, nfull);
    compute_tail(1, nfull + U);

    // ---- groups shared with other workgroups: device-scope partials, last arrival reduces
    const int first = owner_of(g * a.Kt, Tsteps, W), last = owner_of(g * a.Kt + a.Kt - 1, Tsteps, W);
    const int contributors = last - first + 1;
    if (contributors > 1) {
      const size_t slot = (size_t)g * a.cmax + (w - first);
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = mt * 16 + l16, col = (wave * TPW + t) * 16 + 4 * g4;
          if (m < M) {
            const int off = (int)(((slot * a.M_max + m) * GCOLS + col) * sizeof(float));
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, acc[t][mt]), prs, off, 0, kDeviceScope);
          }
        }
      __builtin_amdgcn_s_waitcnt(0);  // this thread's partials have reached the coherent level
      __syncthreads();
      if (threadIdx.x == 0)
        flag = __hip_atomic_fetch_add(&a.counters[g], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == contributors - 1;
      __syncthreads();
      const bool is_last = flag != 0;
      __syncthreads();  // flag is rewritten by the next group
      if (!is_last) continue;
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = mt * 16 + l16, col = (wave * TPW + t) * 16 + 4 * g4;
          f32x4_t sum = f32x4_t{0.f, 0.f, 0.f, 0.f};
          if (m < M) {
            for (int j = 0; j < contributors; ++j) {
              const size_t sl = (size_t)g * a.cmax + j;
              const int off = (int)(((sl * a.M_max + m) * GCOLS + col) * sizeof(float));
              sum += __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(prs, off, 0, kDeviceScope));
            }
          }
          acc[t][mt] = sum;
        }
      if (threadIdx.x == 0) __hip_atomic_store(&a.counters[g], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }

    // ---- epilogues; lane holds output columns n0..n0+3 (weight rows) of activation row m
    if (RMS && !inv_ready) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) inv[mt] = inv_rms_of_row(a, mt * 16 + l16, g4);
      inv_ready = true;
    }
    if (EPI == EPI_LOGITS) {
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = mt * 16 + l16, n0 = (tn0 + t) * 16 + 4 * g4;
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
          const int m = mt * 16 + l16, n0 = (tn0 + t) * 16 + 4 * g4;
          if (m >= M || !tvalid[t] || n0 >= qrows + 2 * krows) continue;
          const int b = seq_of_row(a.row_offsets, a.batch, m);
          const int pos = GL(a.seq_len)[b] + (m - GL(a.row_offsets)[b]);
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
            const int local = n0 - qrows - krows;
            const int head = local / a.hd, d0 = local % a.hd;
            T* dst = (T*)a.kv + ((((size_t)a.layer * 2 + 1) * a.batch + b) * a.nkv + head) * (size_t)a.capacity * a.hd +
                     (size_t)pos * a.hd + d0;
            store4(dst, v);
          }
        }
    } else if (EPI == EPI_RESID) {
      // h += y; the storage-type copy of h for the next consumer; per-row sums of squares of
      // the new h over each 64-column group
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = mt * 16 + l16, n0 = (tn0 + t) * 16 + 4 * g4;
          float ss = 0.f;
          if (m < M && tvalid[t]) {
            GLOBAL f32x4_t* hp = (GLOBAL f32x4_t*)(a.h_out + (size_t)m * a.N + n0);
            const f32x4_t h4 = *hp + acc[t][mt];
            *hp = h4;
            if (a.hx_out) store4((T*)a.hx_out + (size_t)m * a.N + n0, h4);
            ss = ((h4[0] * h4[0] + h4[1] * h4[1]) + h4[2] * h4[2]) + h4[3] * h4[3];
          }
          ss += __shfl_xor(ss, 16, kWave);
          ss += __shfl_xor(ss, 32, kWave);
          if (lane < 16) red[wave * TPW + t][mt * 16 + lane] = ss;
        }
      __syncthreads();
      // 64-column groups: tiles 4p..4p+3 of this tile group, summed in order
      constexpr int PARTS = WAVES * TPW / 4;
      for (int i = threadIdx.x; i < PARTS * ROWS; i += blockDim.x) {
        const int p = i / ROWS, m = i % ROWS;
        if (m >= M) continue;
        const int gp = (int)g * PARTS + p;
        if (gp * 64 >= a.N) continue;
        const float sm = ((red[4 * p + 0][m] + red[4 * p + 1][m]) + red[4 * p + 2][m]) + red[4 * p + 3][m];
        GL(a.stats_out)[(size_t)gp * a.M_max + m] = sm;
      }
      __syncthreads();  // red is rewritten by the next group
    } else if (EPI == EPI_SWIGLU) {
      static_assert(EPI != EPI_SWIGLU || TPW == 2, "SwiGLU pairs a gate and an up fragment row");
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + l16, f0 = (tn0 >> 1) * 16 + 4 * g4;
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
}


// The host bound on rows fixes MT_MAX; the kernel runs the body for the activation
// tiles that the device row count actually needs, so a generous bound costs nothing.
template <typename T, int MT_MAX, int TPW, int EPI>
__global__ void __launch_bounds__(256) gemm_kernel(GemmArgs a) {
  __shared__ float red[4 * TPW][MT_MAX * 16];  // residual epilogue: per-16-column sums of squares
  __shared__ int flag;
  const int M = min(GL(a.row_offsets)[a.batch], a.M_max);  // never trust device rows beyond the host bound
  const int mt = M <= 16 ? 1 : (M <= 32 ? 2 : (M <= 48 ? 3 : 4));
  if (mt <= 1 || MT_MAX == 1) gemm_body<T, 1, TPW, EPI, MT_MAX * 16>(a, M, red, flag);
  else if (mt == 2 || MT_MAX == 2) gemm_body<T, (MT_MAX >= 2 ? 2 : 1), TPW, EPI, MT_MAX * 16>(a, M, red, flag);
  else if (mt == 3 || MT_MAX == 3) gemm_body<T, (MT_MAX >= 3 ? 3 : 1), TPW, EPI, MT_MAX * 16>(a, M, red, flag);
  else gemm_body<T, MT_MAX, TPW, EPI, MT_MAX * 16>(a, M, red, flag);
}

// ------------------------------------------------------------------ planning and launch
GemmPlan plan_gemm(int Nt, int Kt, int TPW, int want_wgs, int min_steps_per_wg) {
  GemmPlan p;
  p.groups = (Nt + 4 * TPW - 1) / (4 * TPW);
  const long long T = (long long)p.groups * Kt;
  long long W = want_wgs;
  if (W > T / min_steps_per_wg) W = T / min_steps_per_wg;
  if (W < 1) W = 1;
  p.wgs = (int)W;
  // largest number of workgroups sharing one tile group
  p.cmax = 1;
  for (int g = 0; g < p.groups; ++g) {
    const long long i0 = (long long)g * Kt, i1 = i0 + Kt - 1;
    const int c = (int)(((i1 + 1) * W - 1) / T - ((i0 + 1) * W - 1) / T) + 1;
    p.cmax = c > p.cmax ? c : p.cmax;
  }
  return p;
}

template <typename T, int MT, int TPW, int EPI>
static void launch_one(const GemmArgs& a, const GemmPlan& p, hipStream_t st) {
  hipLaunchKernelGGL((gemm_kernel<T, MT, TPW, EPI>), dim3(p.wgs), dim3(256), 0, st, a);
}

template <typename T, int TPW, int EPI>
static int launch_mt(int MT, const GemmArgs& a, const GemmPlan& p, hipStream_t st) {
  switch (MT) {
    case 1: launch_one<T, 1, TPW, EPI>(a, p, st); break;
    case 2: launch_one<T, 2, TPW, EPI>(a, p, st); break;
    case 3: launch_one<T, 3, TPW, EPI>(a, p, st); break;
    case 4: launch_one<T, 4, TPW, EPI>(a, p, st); break;
    default: return LSV_ERR_UNSUPPORTED;
  }
  return LSV_OK;
}

template <typename T>
static int launch_typed(GemmKind kind, int MT, const GemmArgs& a, const GemmPlan& p, hipStream_t st) {
  switch (kind) {
    case GEMM_QKV: return launch_mt<T, 1, EPI_QKV>(MT, a, p, st);
    case GEMM_O: return launch_mt<T, 1, EPI_RESID>(MT, a, p, st);
    case GEMM_GATEUP: return launch_mt<T, 2, EPI_SWIGLU>(MT, a, p, st);
    case GEMM_DOWN: return launch_mt<T, 1, EPI_RESID>(MT, a, p, st);
    case GEMM_LMHEAD: return launch_mt<T, 1, EPI_LOGITS>(MT, a, p, st);
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
