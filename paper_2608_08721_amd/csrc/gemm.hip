// Weight packing and the skinny-M matrix-core GEMM of the verify forward pass.
//
// Y[M, N] = X[M, K] * W[N, K]^T with M = the block's rows (a few to 64) and N, K
// in the thousands: the product streams W from HBM once, so the kernel is built
// around that stream.  W is pre-packed into 1 KiB fragments (16 rows x 32 bf16,
// or 16 rows x 16 fp32); each lane loads 16 contiguous bytes, so one wave-wide load
// is one contiguous KiB.  Fragments are ordered in k blocks (frag_index): runs of 8
// fragments of one row, all rows of a block before the next block.  The
// fragment is the A operand of v_mfma_f32_16x16x32_bf16 (fp32: four
// v_mfma_f32_16x16x4_f32), weight rows being the MFMA rows.  The B operand --
// activation rows as MFMA columns -- is read the same way straight from the
// (L2-resident) activation buffer.  The k order inside a fragment is any
// permutation shared by A and B.
//
// RMSNorm: the consumers of a normalised activation (QKV, gate/up, LM head) read the
// operand a = R(h / rms(h) * g) that the row-normalisation kernel (forward.hip) writes in
// the storage type, and multiply it by the plain weights; the producers of the residual
// (O, down) only update h.
//
// Work split: a workgroup owns one tile of TPW fragment rows (16*TPW output columns)
// over the whole K.  Its KS waves take balanced contiguous k-slices, each running its
// own software pipeline of NS stages x U k-steps; the slices meet in LDS and wave 0
// adds them in slice order (deterministic) and runs the epilogue.  No data crosses
// workgroups, so there are no partial buffers, counters or fences.  The residual a
// tile adds to is loaded ahead of the weight stream; inputs that need dependent loads
// (cache positions) are read in the epilogue.
#include <math.h>

#include <type_traits>

#include "lsv_device.h"
#include "lsv_attn.h"
#include "lsv_gemm.h"

namespace lsv {

// ------------------------------------------------------------------ packing
// dst fragment element (row pr, col c) = src[row][c].
template <typename T>
__global__ void __launch_bounds__(256) pack_kernel(int kind, int N, int K, int Nt, int Kt, const T* __restrict__ s0,
                                                   const T* __restrict__ s1, const T* __restrict__ s2, int nq_rows,
                                                   int nkv_rows, int hd, T* __restrict__ dst) {
  constexpr int EPL = FragTraits<T>::EPL, KT = FragTraits<T>::KT;
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t frag = gid >> 6;
  const int lane = (int)(gid & 63);
  if (frag >= (size_t)Nt * Kt) return;
  // inverse of frag_index: block of the k range, then row, then k inside the block
  const int b = (int)(frag / ((size_t)Nt * kFragBlock));
  const int k0 = b * kFragBlock, bs = Kt - k0 < kFragBlock ? Kt - k0 : kFragBlock;
  const size_t rem = frag - (size_t)k0 * Nt;
  const int tn = (int)(rem / bs), tk = k0 + (int)(rem % bs);
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
    out[e] = (row >= 0 && c < K) ? src[(size_t)row * K + c] : from_f32<T>(0.f);
  }
}

// RMSNorm gain [n] in the storage type -> fp32 (exact) in the packed buffer.
template <typename T>
__global__ void __launch_bounds__(256) gain_kernel(int n, const T* __restrict__ src, float* __restrict__ dst) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = to_f32<T>(src[i]);
}

int launch_gain(const Shape& s, const void* src, void* dst, hipStream_t stream) {
  const dim3 grid((unsigned)((s.d + 255) / 256));
  if (s.dtype == LSV_DTYPE_BF16)
    hipLaunchKernelGGL(gain_kernel<bf16_t>, grid, dim3(256), 0, stream, s.d, (const bf16_t*)src, (float*)dst);
  else
    hipLaunchKernelGGL(gain_kernel<float>, grid, dim3(256), 0, stream, s.d, (const float*)src, (float*)dst);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
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

// ------------------------------------------------------------------ QKV epilogue
// base^(-2i/hd) of the two rotary pairs held by output columns n0 .. n0+3 (packed rows
// (2i, 2i+1) of a q or k head are dims (i, i + hd/2)); they depend on the column only.
LSV_DEV void qkv_inv_freq(const GemmArgs& a, int n0, double (&f)[2]) {
  const int qrows = a.nq * a.hd;
  const int local = n0 < qrows ? n0 : n0 - qrows;
  const int i0 = (local % a.hd) >> 1;
#pragma unroll
  for (int pr = 0; pr < 2; ++pr) f[pr] = exp2(-(double)(2 * (i0 + pr)) / (double)a.hd * a.log2_rope_base);
}

// Output columns n0 .. n0+3 of row m of the normalised QKV projection (v), for a row of
// sequence b at cache position pos: rotary embedding of q and k, then the Q store or the
// cache append (V transposed).
template <typename T>
// pos: the cache slot; rpos: the rotary position (the slot, or for a tree node seq_len + its depth).
LSV_DEV void qkv_store4(const GemmArgs& a, int m, int n0, const f32x4_t v, int b, int pos, int rpos,
                        const double (&inv_freq)[2]) {
  const int qrows = a.nq * a.hd, krows = a.nkv * a.hd;
  if (n0 >= qrows + 2 * krows) return;
  if (n0 < qrows + krows) {
    const bool isq = n0 < qrows;
    const int local = isq ? n0 : n0 - qrows;
    const int head = local / a.hd, i0 = (local % a.hd) >> 1;  // pairs (i0, i0+hd/2), (i0+1, i0+1+hd/2)
    float out[4];
#pragma unroll
    for (int pr = 0; pr < 2; ++pr) {
      // angle = pos * base^(-2i/hd) in fp64, reduced to [-pi, pi] in fp64, then fp32 sin/cos
      const double ang = (double)rpos * inv_freq[pr];
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
      size_t ko, vo;
      int vs;
      if (pos < 0 || (!a.kvl.pages && pos >= a.capacity) || !kv_locate(a.kvl, a.nkv, a.hd, b, head, pos, ko, vo, vs))
        return;
      dst = (T*)a.kv + 2 * (size_t)a.layer * kv_layer_block(a.kvl, a.batch, a.nkv, a.hd) + ko;
    }
    GLOBAL T* gd = GL(dst);
    if constexpr (sizeof(T) == 2) {
      // dims (i0, i0+1) and (i0+hd/2, i0+1+hd/2) are adjacent pairs (i0 and hd/2 are even):
      // two 4-byte stores instead of four 2-byte ones
      *(GLOBAL uint32_t*)(gd + i0) = (uint32_t)f2bf(out[0]) | ((uint32_t)f2bf(out[2]) << 16);
      *(GLOBAL uint32_t*)(gd + i0 + a.hd / 2) = (uint32_t)f2bf(out[1]) | ((uint32_t)f2bf(out[3]) << 16);
    } else {
      gd[i0] = from_f32<T>(out[0]);
      gd[i0 + a.hd / 2] = from_f32<T>(out[1]);
      gd[i0 + 1] = from_f32<T>(out[2]);
      gd[i0 + 1 + a.hd / 2] = from_f32<T>(out[3]);
    }
  } else {
    // V rows are stored transposed: [head_dim][64] per 64-position block and kv head, column
    // v_column(pos % 64)
    const int local = n0 - qrows - krows;
    const int head = local / a.hd, d0 = local % a.hd;
    size_t ko, vo;
    int vs;
    if (pos < 0 || (!a.kvl.pages && pos >= a.capacity) || !kv_locate(a.kvl, a.nkv, a.hd, b, head, pos, ko, vo, vs))
      return;
    const size_t blk = kv_layer_block(a.kvl, a.batch, a.nkv, a.hd);
    GLOBAL T* dst = GL((T*)a.kv) + (2 * (size_t)a.layer + 1) * blk + vo + (size_t)d0 * vs;
#pragma unroll
    for (int r = 0; r < 4; ++r) dst[(size_t)r * vs] = from_f32<T>(v[r]);
  }
}

// ------------------------------------------------------------------ the GEMM
// Epilogue of one wave: lane holds output columns n0..n0+3 (weight rows) of activation
// row m for each of its TPW fragment rows and MT activation tiles.  Row inputs that need
// dependent loads (cache positions) are read here, off the weight stream's critical path.
// HPRE: the residual was loaded ahead into hpre (else it is read here).
template <typename T, int MT, int TPW, int EPI, bool HPRE>
LSV_DEV void gemm_epilogue(const GemmArgs& a, const int M, const int m0, const int tn0, const bool (&tvalid)[TPW],
                           f32x4_t (&acc)[TPW][MT], const f32x4_t (&hpre)[TPW][MT]) {
  constexpr int KT = FragTraits<T>::KT;
  const int lane = threadIdx.x & 63, l16 = lane & 15, g4 = lane >> 4;
  int qkv_b[MT], qkv_pos[MT], qkv_rpos[MT];
  if (EPI == EPI_QKV) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = min(m0 + mt * 16 + l16, a.M_max - 1);
      const int b = seq_of_row(a.row_offsets, a.batch, m);
      qkv_b[mt] = b;
      qkv_pos[mt] = GL(a.seq_len)[b] + (m - GL(a.row_offsets)[b]);
      qkv_rpos[mt] = a.depth ? GL(a.seq_len)[b] + GL(a.depth)[m] : qkv_pos[mt];
    }
  }
  if (EPI == EPI_LOGITS) {
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = m0 + mt * 16 + l16, n0 = (tn0 + t) * 16 + 4 * g4;
        if (m >= M || !tvalid[t]) continue;
        const f32x4_t v = acc[t][mt];
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
      double inv_freq[TPW][2];
#pragma unroll
      for (int t = 0; t < TPW; ++t) qkv_inv_freq(a, (tn0 + t) * 16 + 4 * g4, inv_freq[t]);
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = m0 + mt * 16 + l16, n0 = (tn0 + t) * 16 + 4 * g4;
          if (m >= M || !tvalid[t]) continue;
          qkv_store4<T>(a, m, n0, acc[t][mt], qkv_b[mt], qkv_pos[mt], qkv_rpos[mt], inv_freq[t]);
        }
    } else if (EPI == EPI_RESID) {
      // h += y (fp32 residual, row-major); the next norm reads it
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int m = m0 + mt * 16 + l16, n0 = (tn0 + t) * 16 + 4 * g4;
          if (m < M && tvalid[t]) {
            const f32x4_t hv = HPRE ? hpre[t][mt] : *(const GLOBAL f32x4_t*)(a.h_out + (size_t)m * a.N + n0);
            *(GLOBAL f32x4_t*)(a.h_out + (size_t)m * a.N + n0) = hv + acc[t][mt];
          }
        }
    } else if (EPI == EPI_SWIGLU) {
      // fragment rows come in (gate, up) pairs: even rows gate, odd rows up
      static_assert(EPI != EPI_SWIGLU || TPW % 2 == 0, "SwiGLU pairs a gate and an up fragment row");
#pragma unroll
      for (int t = 0; t < TPW; t += 2)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = m0 + mt * 16 + l16, f0 = ((tn0 + t) >> 1) * 16 + 4 * g4;
        if (m >= M || !tvalid[t]) continue;
        f32x4_t out;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float gt = acc[t][mt][r], up = acc[t + 1][mt][r];
          out[r] = gt / (1.0f + expf(-gt)) * up;
        }
        T* dst = (T*)a.u_out + act_index<KT>(m, f0, (a.F + KT - 1) / KT);  // f0 .. f0+3 are adjacent
        if (f0 + 3 < a.F) {
          store4(dst, out);
        } else {
          for (int r = 0; r < 4; ++r)
            if (f0 + r < a.F) GL(dst)[r] = from_f32<T>(out[r]);
        }
      }
    }
}

template <typename T, int MT, int TPW, int KS, int U, int NS, int EPI, int MT_MAX>
LSV_DEV void gemm_body(const GemmArgs& a, const int M, const int tile, const int m0,
                       f32x4_t (*red)[TPW][MT_MAX][kWave], const int kslice) {
  constexpr int EPL = FragTraits<T>::EPL;
  const int wave = kslice, lane = threadIdx.x & 63, l16 = lane & 15, g4 = lane >> 4;
  // this workgroup: fragment rows tn0 .. tn0+TPW-1 over the whole K, activation rows
  // m0 .. min(M, m0 + 16 MT) - 1; wave = k-slice
  const int tn0 = tile * TPW;
  const int k0 = (int)((long long)wave * a.Kt / KS), k1 = (int)((long long)(wave + 1) * a.Kt / KS);
  const int nk = k1 - k0;  // >= 0, and k0 < Kt for every wave
  bool tvalid[TPW];
  int tr[TPW];  // fragment row of each of the wave's tiles (row 0 stands in past the end)
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    tvalid[t] = tn0 + t < a.Nt;
    tr[t] = tvalid[t] ? tn0 + t : 0;
  }
  // the packed weights: fragment f is the KiB at byte f * 1024, this lane's 16 bytes at + lane * 16
  const __amdgpu_buffer_rsrc_t wrs = stream_rsrc(a.W, (size_t)a.Nt * a.Kt * 1024);

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

  // B operand: this lane's piece of each activation tile's fragments (rows >= M hold stale
  // but finite values; their output columns are never stored)
  const GLOBAL T* xp[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
    xp[mt] = (const GLOBAL T*)a.x + (((size_t)((m0 >> 4) + mt) * a.Kt + k0) * kWave + lane) * EPL;

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
        for (int t = 0; t < TPW; ++t) wa[st][u][t] = load_stream(wrs, (uint32_t)((frag_index(tr[t], k0 + kf, a.Nt, a.Kt) * 64 + lane) * 16));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) xb[st][u][mt] = *(const GLOBAL u32x4_t*)(xp[mt] + (size_t)kf * kWave * EPL);
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

  // ---- a k range of a split pair (EPI_PART, residual_split_pairs): this range's sums, k slice
  // `kslice` of 2, to the partials [tile][2][M_max][128] (tile = 8 fragment rows); rows past M
  // are not written
  if constexpr (EPI == EPI_PART) {
    static_assert(KS == 2 && MT_MAX >= MT, "two k ranges per fragment-row pair");
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = m0 + mt * 16 + l16, fr = tn0 + t;
        if (m < M && tvalid[t])
          *(GLOBAL f32x4_t*)(a.part + (((size_t)(fr >> 3) * 2 + kslice) * a.M_max + m) * kWideCols + (fr & 7) * 16 +
                             4 * g4) = acc[t][mt];
      }
    return;
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

  gemm_epilogue<T, MT, TPW, EPI, true>(a, M, m0, tn0, tvalid, acc, hpre);
}

// Launch configuration of each product: fragment rows per wave (TPW), k-slices = waves
// per workgroup (KS), k-steps per pipeline stage (U) and stages in flight (NS).  Chosen by
// measurement on the Llama-3-8B shapes: few long weight streams, each with many bytes in
// flight, beat many short ones (more concurrent streams read more scattered DRAM rows), so
// every product runs one wave per workgroup over the whole K.  A stream sustained about
// 11-14 GB/s however deep its pipeline (default-policy loads), so a product with few fragment rows needs one per
// wave: the QKV projection of Llama-3-70B (640 fragment rows) takes 38 us at two per wave
// and 34 us at one (a lane's four outputs hold whole rotary pairs either way).
template <int KIND> struct GemmCfg;
template <> struct GemmCfg<GEMM_QKV> { static constexpr int TPW = 1, KS = 1, U = 4, NS = 3, EPI = EPI_QKV; };
template <> struct GemmCfg<GEMM_O> { static constexpr int TPW = 1, KS = 1, U = 8, NS = 3, EPI = EPI_RESID; };
template <> struct GemmCfg<GEMM_GATEUP> { static constexpr int TPW = 4, KS = 1, U = 4, NS = 3, EPI = EPI_SWIGLU; };
template <> struct GemmCfg<GEMM_DOWN> { static constexpr int TPW = 1, KS = 1, U = 8, NS = 3, EPI = EPI_RESID; };
template <> struct GemmCfg<GEMM_LMHEAD> { static constexpr int TPW = 4, KS = 1, U = 4, NS = 3, EPI = EPI_LOGITS; };
// gate/up of the wider models (3072 or more fragment rows: Qwen2.5-32B, Llama-3-70B shapes):
// eight fragment rows per wave halve the workgroups and the activation loads per weight byte
// (measured 5.45 -> 5.72 TB/s at d 5120, 5.62 -> 5.94 TB/s at d 8192; at d 4096 it lost);
// blocks of up to 32 rows only
constexpr int kGateUpWide = 5;  // internal kind id of that configuration
constexpr int kGateUpWideRows = 3072;
template <> struct GemmCfg<kGateUpWide> { static constexpr int TPW = 8, KS = 1, U = 2, NS = 3, EPI = EPI_SWIGLU; };

// Bodies of three or four activation tiles (prefill bounds) use a shallower pipeline to stay in
// registers.
template <int KIND, int MT_MAX> struct GemmShape {
  using C = GemmCfg<KIND>;
  static constexpr int TPW = C::TPW, KS = C::KS, EPI = C::EPI;
  static constexpr int U = MT_MAX <= 2 ? C::U : 4, NS = MT_MAX <= 2 ? C::NS : 2;
};

// Two or more activation tiles: a product that streams one or two fragment rows per wave takes
// twice as many when that still leaves a stream per compute unit.  Each activation tile adds one
// load per k-step to every wave, and per-wave issue, not DRAM, bounds these streams, so this halves
// the activation loads per weight byte (lab, Llama-3-70B, 20 / 52 rows: down 102 -> 79 / 146 ->
// 116 us, O 31 -> 26 / 44 -> 36 us); with fewer streams than compute units it loses (Llama-3-8B
// at 17 rows: +0.5 ms per step), and four rows per wave lost everywhere.
constexpr int kComputeUnits = 256;
template <int KIND> struct MultiTile {
  static constexpr int TPW = GemmCfg<KIND>::TPW <= 2 ? 2 * GemmCfg<KIND>::TPW : GemmCfg<KIND>::TPW;
  LSV_DEV static bool use(int mt, int Nt) { return mt >= 2 && TPW != GemmCfg<KIND>::TPW && (Nt + TPW - 1) / TPW >= kComputeUnits; }
};

// One activation tile on the residual products (O, down): a one-row stream spends half of its
// load instructions on the block's activation fragments, so two fragment rows per wave -- while a
// stream per compute unit remains -- move more weight bytes per instruction (lab, Llama-3-70B at
// 16 rows: down 80.1 -> 68.3 us, O 24.3 -> 22.4 us; the QKV projection lost, 33 -> 37 us, and
// the same for two tiles lost).  Two k-steps per stage and six stages keep 24 KB in flight per
// stream, as one row at U 8 did; 32 KB lost.  A wave's products and sums are those of one row per
// wave, so the outputs are bit-identical either way.
template <int KIND> struct PairRows {
  static constexpr int TPW = 2, U = 2, NS = 6;
  LSV_DEV static bool use(int mt, int Nt) {
    return (KIND == GEMM_O || KIND == GEMM_DOWN) && mt == 1 && (Nt + TPW - 1) / TPW >= kComputeUnits;
  }
};

// The narrower residual products (residual_split_pairs): stream `s` of the launch takes fragment
// rows 2 (s / 2), +1 over k half s % 2 -- one stream per fragment row as before, with the
// activation loads of two rows per weight load -- and writes its half's sums (EPI_PART).  The
// pipeline is PairRows' for one or two activation tiles and shallower for three or four.
template <int MT, int MT_MAX>
LSV_DEV void split_pair_body(const GemmArgs& a, const int M, const int stream, const int m0) {
  if constexpr (MT <= 2)
    gemm_body<bf16_t, MT, 2, 2, 2, 6, EPI_PART, MT_MAX>(a, M, stream >> 1, m0, nullptr, stream & 1);
  else
    gemm_body<bf16_t, MT, 2, 2, 2, 3, EPI_PART, MT_MAX>(a, M, stream >> 1, m0, nullptr, stream & 1);
}

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
  const int rows = GL(a.row_offsets)[a.batch];
  if (rows <= a.rows_lo || rows > a.rows_hi) return;  // another launch serves this row count
  const int M = min(rows, a.M_max);  // never trust device rows beyond the host bound
  const int m0 = chunk * 64;
  if (m0 >= M) return;
  const int Mc = min(M - m0, 64);
  const int M_end = m0 + Mc;
  const int mt = Mc <= 16 ? 1 : (Mc <= 32 ? 2 : (Mc <= 48 ? 3 : 4));
  // one or two tiles keep the product's full pipeline under any bound (lab: down at 9 rows under a
  // 64-row bound, 41 -> 25 us); three or four take the shallower one
  using C = GemmCfg<KIND>;
  const int ks = threadIdx.x >> 6;
  if constexpr (std::is_same<T, bf16_t>::value && S::KS == 1 && (KIND == GEMM_O || KIND == GEMM_DOWN)) {
    if (residual_split_pairs(KIND, a.Nt)) {  // one stream per fragment row: tile < tiles = Nt
      if (mt <= 1 || MT_MAX == 1)
        split_pair_body<1, MT_MAX>(a, M_end, tile, m0);
      else if (mt == 2 || MT_MAX == 2)
        split_pair_body<(MT_MAX >= 2 ? 2 : 1), MT_MAX>(a, M_end, tile, m0);
      else if (mt == 3 || MT_MAX == 3)
        split_pair_body<(MT_MAX >= 3 ? 3 : 1), MT_MAX>(a, M_end, tile, m0);
      else
        split_pair_body<MT_MAX, MT_MAX>(a, M_end, tile, m0);
      return;
    }
    using P = PairRows<KIND>;
    if (P::use(mt, a.Nt)) {
      if (tile >= (a.Nt + P::TPW - 1) / P::TPW) return;
      gemm_body<T, 1, P::TPW, 1, P::U, P::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, nullptr, 0);
      return;
    }
  }
  if constexpr (std::is_same<T, bf16_t>::value && S::KS == 1 && MT_MAX >= 2) {
    using X = MultiTile<KIND>;
    if (X::use(mt, a.Nt)) {
      if (tile >= (a.Nt + X::TPW - 1) / X::TPW) return;
      if (mt == 2 || MT_MAX == 2)
        gemm_body<T, 2, X::TPW, 1, C::U, C::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, nullptr, 0);
      else if (mt == 3 || MT_MAX == 3)
        gemm_body<T, (MT_MAX >= 3 ? 3 : 2), X::TPW, 1, S::U, S::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, nullptr, 0);
      else
        gemm_body<T, MT_MAX, X::TPW, 1, S::U, S::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, nullptr, 0);
      return;
    }
  }
  if (mt <= 1 || MT_MAX == 1)
    gemm_body<T, 1, S::TPW, S::KS, C::U, C::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, red, ks);
  else if (mt == 2 || MT_MAX == 2)
    gemm_body<T, (MT_MAX >= 2 ? 2 : 1), S::TPW, S::KS, C::U, C::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, red, ks);
  else if (mt == 3 || MT_MAX == 3)
    gemm_body<T, (MT_MAX >= 3 ? 3 : 1), S::TPW, S::KS, S::U, S::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, red, ks);
  else
    gemm_body<T, MT_MAX, S::TPW, S::KS, S::U, S::NS, S::EPI, MT_MAX>(a, M_end, tile, m0, red, ks);
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
    case GEMM_GATEUP:
      if constexpr (std::is_same<T, bf16_t>::value) {
        if (a.Nt >= kGateUpWideRows && MT <= 2) {  // deeper row chunks would not fit its registers
          if (MT == 1)
            launch_one<T, kGateUpWide, 1>(a, st);
          else
            launch_one<T, kGateUpWide, 2>(a, st);
          return LSV_OK;
        }
      }
      return launch_mt<T, GEMM_GATEUP>(MT, a, st);
    case GEMM_DOWN: return launch_mt<T, GEMM_DOWN>(MT, a, st);
    case GEMM_LMHEAD: return launch_mt<T, GEMM_LMHEAD>(MT, a, st);
  }
  return LSV_ERR_UNSUPPORTED;
}

// ------------------------------------------------------------------ wide blocks
// Batched verification (64 < rows <= kWideRows): the matrix cores become the bound.
// Workgroup = 4 waves x 8 fragment rows (128 output columns) x one of `splits` k ranges;
// the waves share the 8 weight fragments of each k-step through LDS and split the rows:
// wave w keeps activation tiles w*MTW .. w*MTW+MTW-1 (MTW <= 5) in registers.  With more
// than one k range per tile, each workgroup writes fp32 partials and
// gemm_wide_reduce_kernel adds them in split order (deterministic) and runs the epilogue,
// one workgroup per (tile, 16 rows); the QKV reduce applies the rotary embedding and the Q
// store / cache append.  An unsplit QKV runs the plain epilogue into an fp32 buffer
// and qkv_rope_kernel does the rest.  The residual products (O, down) launch no reduce: the
// row normalisation that follows each of them adds their partials to the residual stream.
constexpr int kWideRingW = 10;  // k-steps of weight pieces in flight (register ring)
constexpr int kWideRingX = 2;   // k-steps of activation fragments in flight (from L2)

// The body for MTW activation tiles per wave.  The workgroup's 8 weight fragments of a
// k-step go HBM -> registers -> LDS (double buffered) and every wave reads all 8; each wave
// keeps its own MTW activation tiles (rows wave*16*MTW ..) in registers, straight from L2.
// A k-step is 8 LDS reads and 8 x MTW MFMAs per wave, each read feeding MTW of them.  Tiles
// past the device row count are computed on clamped rows and never stored.
// Ws: two buffers of 8 fragments.  The QKV projection never runs its fused epilogue here
// (split K: the reduce does; one split: the projection, then qkv_rope_kernel).
template <int EPI, int MTW>
LSV_DEV void gemm_wide_body(const GemmArgs& a, const int M, u32x4_t* Ws) {
  static_assert(EPI != EPI_QKV, "the batched QKV epilogue runs in the reduce or the RoPE kernel");
  using T = bf16_t;
  constexpr int FR = kWideFR;
  constexpr int RX = kWideRingX, RW = kWideRingW;
  constexpr int PPT = FR * kWave / 256;  // 16-byte weight pieces per thread and k-step
  static_assert(PPT * 256 == FR * kWave, "weight pieces divide over the threads");
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, l16 = lane & 15, g4 = lane >> 4;
  const int S = a.splits, tile = blockIdx.x / S, j = blockIdx.x % S;
  const int k0 = (int)((long long)j * a.Kt / S), k1 = (int)((long long)(j + 1) * a.Kt / S), nk = k1 - k0;
  const int tn0 = tile * FR, mt0 = wave * MTW;
  const int tiles_alloc = (a.M_max + 15) / 16;  // activation tiles in the buffer
  bool tvalid[FR];
#pragma unroll
  for (int f = 0; f < FR; ++f) tvalid[f] = tn0 + f < a.Nt;
  const GLOBAL u32x4_t* wg = (const GLOBAL u32x4_t*)a.W;
  const GLOBAL u32x4_t* xg = (const GLOBAL u32x4_t*)a.x + lane;
  int xt[MTW];  // activation tile of each of the wave's slots (clamped into the buffer)
#pragma unroll
  for (int mt = 0; mt < MTW; ++mt) xt[mt] = min(mt0 + mt, tiles_alloc - 1);

  // Register rings: weight pieces of the next RW k-steps (piece p = (fragment p / 64, lane
  // p % 64)), and this wave's activation fragments of the next RX.
  u32x4_t wst[RW][PPT], xr[RX][MTW];
  auto issue_w = [&](int sw, int k) {
    const int kk = max(min(k, nk - 1), 0);
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int p = tid + 256 * i, f = p / kWave, ln = p % kWave;
      const int fr = tn0 + f < a.Nt ? tn0 + f : 0;
      wst[sw][i] = load_stream(&wg[frag_index(fr, k0 + kk, a.Nt, a.Kt) * kWave + ln]);
    }
  };
  auto issue_x = [&](int sx, int k) {
    const int kk = max(min(k, nk - 1), 0);
#pragma unroll
    for (int mt = 0; mt < MTW; ++mt) xr[sx][mt] = xg[((size_t)xt[mt] * a.Kt + k0 + kk) * kWave];
  };
  auto store = [&](int sw, int buf) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) Ws[buf * FR * kWave + tid + 256 * i] = wst[sw][i];
  };
  f32x4_t acc[FR][MTW];
#pragma unroll
  for (int f = 0; f < FR; ++f)
#pragma unroll
    for (int mt = 0; mt < MTW; ++mt) acc[f][mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  u32x4_t xcur[MTW];
  auto compute = [&](int buf) {
#pragma unroll
    for (int f = 0; f < FR; ++f) {
      const u32x4_t w = Ws[(buf * FR + f) * kWave + lane];
#pragma unroll
      for (int mt = 0; mt < MTW; ++mt) mfma_frag(w, xcur[mt], acc[f][mt], T{});
    }
  };
  // k-step c: its weights sit in LDS buffer c & 1 (stored during step c - 1); the weights of
  // step c + 1 move from their register stage to the other buffer and that stage takes step
  // c + 1 + RW; the activation stage of step c takes step c + RX.  One barrier per step.
  // u = c mod UNR (a compile-time constant where step is called), so ring stages are static.
  constexpr int UNR = RX % RW == 0 ? RX : (RW % RX == 0 ? RW : RX * RW);
  auto step = [&](int c, int u) {
    const int sx = u % RX, sw = (u + 1) % RW;
#pragma unroll
    for (int mt = 0; mt < MTW; ++mt) xcur[mt] = xr[sx][mt];
    if (c + 1 < nk) store(sw, (c + 1) & 1);
    issue_w(sw, c + 1 + RW);
    issue_x(sx, c + RX);
    compute(c & 1);
    __syncthreads();
  };
#pragma unroll
  for (int sx = 0; sx < RX; ++sx) issue_x(sx, sx);
#pragma unroll
  for (int sw = 0; sw < RW; ++sw) issue_w(sw, sw);
  store(0, 0);
  issue_w(0, RW);
  __syncthreads();
  int c = 0;
  for (; c + UNR <= nk; c += UNR) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) step(c + u, u);
  }
#pragma unroll
  for (int u = 0; u < UNR; ++u)
    if (c + u < nk) step(c + u, u);

  if (S > 1) {  // partial sums of this k range: [tile][split][M_max][kWideCols]
#pragma unroll
    for (int f = 0; f < FR; ++f)
#pragma unroll
      for (int mt = 0; mt < MTW; ++mt) {
        const int m = (mt0 + mt) * 16 + l16, col = f * 16 + 4 * g4;
        if (m < M)
          *(GLOBAL f32x4_t*)(a.part + (((size_t)tile * S + j) * a.M_max + m) * kWideCols + col) = acc[f][mt];
      }
    return;
  }
  const f32x4_t none[FR][MTW] = {};
  gemm_epilogue<T, MTW, FR, EPI, false>(a, M, mt0 * 16, tn0, tvalid, acc, none);
}

// One launch for blocks under a batched row bound (64 < bound <= kWideRows).  Up to 64 device
// rows, each of a workgroup's four waves runs the 64-row body on a column tile of its own --
// tile (wave x grid + workgroup), so that the busy waves spread over the compute units -- and
// streams its weights once, as gemm_kernel does (gate/up of the wider models with up to 32 rows
// takes its eight-fragment-row configuration); more rows run the batched body on the
// workgroup's (tile, k-split).  One launch instead of one of each kind, one of which would
// find no work.
template <int KIND, int WIDE_EPI>
__global__ void __launch_bounds__(256) gemm_fused_kernel(GemmArgs a) {
  __shared__ u32x4_t Ws[2 * kWideFR * kWave];
  const int M = min(GL(a.row_offsets)[a.batch], a.M_max);  // never trust device rows beyond the host bound
  if (M <= 64) {
    if (M <= 0) return;
    const int vt = (int)(threadIdx.x >> 6) * (int)gridDim.x + (int)blockIdx.x;  // this wave's column tile
    const int mt = M <= 16 ? 1 : (M <= 32 ? 2 : (M <= 48 ? 3 : 4));
    if constexpr (KIND == GEMM_GATEUP) {
      if (a.Nt >= kGateUpWideRows && mt <= 2) {
        using W = GemmCfg<kGateUpWide>;
        if (vt >= (a.Nt + W::TPW - 1) / W::TPW) return;
        if (mt == 1)
          gemm_body<bf16_t, 1, W::TPW, 1, W::U, W::NS, W::EPI, 2>(a, M, vt, 0, nullptr, 0);
        else
          gemm_body<bf16_t, 2, W::TPW, 1, W::U, W::NS, W::EPI, 2>(a, M, vt, 0, nullptr, 0);
        return;
      }
    }
    using C = GemmCfg<KIND>;
    using S = GemmShape<KIND, 4>;
    static_assert(C::KS == 1, "one wave per column tile");
    if constexpr (KIND == GEMM_O || KIND == GEMM_DOWN) {
      if (residual_split_pairs(KIND, a.Nt)) {  // one stream per fragment row
        if (vt >= a.Nt) return;
        if (mt == 1)
          split_pair_body<1, 4>(a, M, vt, 0);
        else if (mt == 2)
          split_pair_body<2, 4>(a, M, vt, 0);
        else if (mt == 3)
          split_pair_body<3, 4>(a, M, vt, 0);
        else
          split_pair_body<4, 4>(a, M, vt, 0);
        return;
      }
      using P = PairRows<KIND>;
      if (P::use(mt, a.Nt)) {  // one activation tile on a wide residual product
        if (vt >= (a.Nt + P::TPW - 1) / P::TPW) return;
        gemm_body<bf16_t, 1, P::TPW, 1, P::U, P::NS, S::EPI, 4>(a, M, vt, 0, nullptr, 0);
        return;
      }
    }
    using X = MultiTile<KIND>;
    if (X::use(mt, a.Nt)) {  // two or more activation tiles on a wide product
      if (vt >= (a.Nt + X::TPW - 1) / X::TPW) return;
      if (mt == 2)
        gemm_body<bf16_t, 2, X::TPW, 1, C::U, C::NS, S::EPI, 4>(a, M, vt, 0, nullptr, 0);
      else if (mt == 3)
        gemm_body<bf16_t, 3, X::TPW, 1, S::U, S::NS, S::EPI, 4>(a, M, vt, 0, nullptr, 0);
      else
        gemm_body<bf16_t, 4, X::TPW, 1, S::U, S::NS, S::EPI, 4>(a, M, vt, 0, nullptr, 0);
      return;
    }
    if (vt >= (a.Nt + S::TPW - 1) / S::TPW) return;
    if (mt == 1)
      gemm_body<bf16_t, 1, S::TPW, 1, C::U, C::NS, S::EPI, 4>(a, M, vt, 0, nullptr, 0);
    else if (mt == 2)
      gemm_body<bf16_t, 2, S::TPW, 1, C::U, C::NS, S::EPI, 4>(a, M, vt, 0, nullptr, 0);
    else if (mt == 3)
      gemm_body<bf16_t, 3, S::TPW, 1, S::U, S::NS, S::EPI, 4>(a, M, vt, 0, nullptr, 0);
    else
      gemm_body<bf16_t, 4, S::TPW, 1, S::U, S::NS, S::EPI, 4>(a, M, vt, 0, nullptr, 0);
    return;
  }
  if ((int)blockIdx.x >= (a.Nt + kWideFR - 1) / kWideFR * a.splits) return;
  const int mtw = ((M + 15) / 16 + 3) / 4;  // activation tiles per wave
  if (mtw <= 1)
    gemm_wide_body<WIDE_EPI, 1>(a, M, Ws);
  else if (mtw == 2)
    gemm_wide_body<WIDE_EPI, 2>(a, M, Ws);
  else if (mtw == 3)
    gemm_wide_body<WIDE_EPI, 3>(a, M, Ws);
  else if (mtw == 4)
    gemm_wide_body<WIDE_EPI, 4>(a, M, Ws);
  else
    gemm_wide_body<WIDE_EPI, 5>(a, M, Ws);
}

// Split-K sums of the batched GEMM: one workgroup per (tile, 16 rows) adds the k ranges in
// split order and runs the product's epilogue (wave w: fragment rows of the tile's wave w).
template <int EPI>
__global__ void __launch_bounds__(256) gemm_wide_reduce_kernel(GemmArgs a) {
  constexpr int TPW = kWideFR / 4;  // wave w sums fragment rows w*TPW ..
  const int tile = blockIdx.x, m0 = blockIdx.y * 16, S = a.splits;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, l16 = lane & 15, g4 = lane >> 4;
  const int rows = GL(a.row_offsets)[a.batch];
  if (rows <= a.rows_lo || rows > a.rows_hi) return;
  const int M = min(rows, a.M_max);
  if (m0 >= M) return;
  const int tn0 = (tile * 4 + wave) * TPW, m = m0 + l16;
  bool tvalid[TPW];
  f32x4_t acc[TPW][1];
  const f32x4_t none[TPW][1] = {};
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    tvalid[t] = tn0 + t < a.Nt;
    acc[t][0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  if (m < M) {
    // the partials of up to RB splits are in flight at once; they are added in split order
    constexpr int RB = 8;
    const GLOBAL f32x4_t* p = (const GLOBAL f32x4_t*)(a.part + ((size_t)tile * S * a.M_max + m) * kWideCols) +
                              wave * TPW * 4 + g4;
    const size_t split_step = (size_t)a.M_max * kWideCols / 4;
    for (int j0 = 0; j0 < S; j0 += RB) {
      f32x4_t v[RB][TPW];
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int t = 0; t < TPW; ++t) v[i][t] = p[(size_t)min(j0 + i, S - 1) * split_step + 4 * t];
#pragma unroll
      for (int i = 0; i < RB; ++i)
        if (j0 + i < S)
#pragma unroll
          for (int t = 0; t < TPW; ++t) acc[t][0] += v[i][t];
    }
  }
  gemm_epilogue<bf16_t, 1, TPW, EPI, false>(a, M, m0, tn0, tvalid, acc, none);
}

// Rotary embedding and Q store / cache append of a normalised QKV projection y [M][N] (fp32),
// four columns per thread.
__global__ void __launch_bounds__(256) qkv_rope_kernel(GemmArgs a, const float* y) {
  const int rows = GL(a.row_offsets)[a.batch];
  if (rows <= a.rows_lo || rows > a.rows_hi) return;
  const int M = min(rows, a.M_max);
  const int groups = a.N / 4;
  const size_t n = (size_t)M * groups;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    const int m = (int)(i / groups), n0 = (int)(i % groups) * 4;
    const f32x4_t v = *(const GLOBAL f32x4_t*)(y + (size_t)m * a.N + n0);
    const int b = seq_of_row(a.row_offsets, a.batch, m);
    const int pos = GL(a.seq_len)[b] + (m - GL(a.row_offsets)[b]);
    const int rpos = a.depth ? GL(a.seq_len)[b] + GL(a.depth)[m] : pos;
    double f[2];
    qkv_inv_freq(a, n0, f);
    qkv_store4<bf16_t>(a, m, n0, v, b, pos, rpos, f);
  }
}

WidePlan plan_wide(int Nt, int Kt) {
  WidePlan p;
  p.tiles = (Nt + kWideFR - 1) / kWideFR;
  // one resident workgroup per compute unit (the accumulators fill the AGPRs); at least
  // eight k-steps per workgroup
  p.splits = 256 / p.tiles;
  const int most = Kt / 8;
  if (p.splits > most) p.splits = most;
  if (p.splits < 1) p.splits = 1;
  return p;
}

size_t wide_part_floats(const WidePlan& p, int M_max) {
  return p.splits > 1 ? (size_t)p.tiles * p.splits * M_max * kWideCols : 0;
}

// The fused launch of a product (and, for the batched body, its split-K reduce or the separate
// rotary-embedding pass; those return at once for blocks of up to 64 rows).
template <int KIND, int WIDE_EPI>
static void launch_fused_one(const GemmArgs& a, const WidePlan& p, hipStream_t st) {
  using S = GemmShape<KIND, 4>;
  const int skinny_wgs = ((a.Nt + S::TPW - 1) / S::TPW + 3) / 4;
  const int grid = p.tiles * p.splits > skinny_wgs ? p.tiles * p.splits : skinny_wgs;
  hipLaunchKernelGGL((gemm_fused_kernel<KIND, WIDE_EPI>), dim3((unsigned)grid), dim3(256), 0, st, a);
}

int launch_gemm_fused(GemmKind kind, const GemmArgs& a0, const WidePlan& p, hipStream_t st) {
  GemmArgs a = a0;
  a.splits = p.splits;
  GemmArgs big = a;  // the passes after the batched body: only for more than 64 rows
  big.rows_lo = 64;
  const dim3 rgrid((unsigned)p.tiles, (unsigned)((a.M_max + 15) / 16));
  switch (kind) {
    case GEMM_QKV:
      if (p.splits > 1) {
        launch_fused_one<GEMM_QKV, EPI_LOGITS>(a, p, st);
        hipLaunchKernelGGL(gemm_wide_reduce_kernel<EPI_QKV>, rgrid, dim3(256), 0, st, big);
      } else {
        if (!a.out_f32) return LSV_ERR_INVALID_ARG;
        a.ldo = a.N;  // the batched body writes the projection to out_f32; the 64-row body does not read it
        big.ldo = a.N;
        launch_fused_one<GEMM_QKV, EPI_LOGITS>(a, p, st);
        const size_t n = (size_t)a.M_max * (a.N / 4);
        hipLaunchKernelGGL(qkv_rope_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, big, big.out_f32);
      }
      break;
    case GEMM_O:  // k-split partials are added by the next row normalisation
      launch_fused_one<GEMM_O, EPI_RESID>(a, p, st);
      break;
    case GEMM_GATEUP:
      launch_fused_one<GEMM_GATEUP, EPI_SWIGLU>(a, p, st);
      if (p.splits > 1) hipLaunchKernelGGL(gemm_wide_reduce_kernel<EPI_SWIGLU>, rgrid, dim3(256), 0, st, big);
      break;
    case GEMM_DOWN:  // k-split partials are added by the next row normalisation
      launch_fused_one<GEMM_DOWN, EPI_RESID>(a, p, st);
      break;
    case GEMM_LMHEAD:
      launch_fused_one<GEMM_LMHEAD, EPI_LOGITS>(a, p, st);
      if (p.splits > 1) hipLaunchKernelGGL(gemm_wide_reduce_kernel<EPI_LOGITS>, rgrid, dim3(256), 0, st, big);
      break;
  }
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

int launch_gemm(int dtype, GemmKind kind, int MT, const GemmArgs& a, hipStream_t st) {
  int rc = dtype == LSV_DTYPE_BF16 ? launch_typed<bf16_t>(kind, MT, a, st) : launch_typed<float>(kind, MT, a, st);
  if (rc != LSV_OK) return rc;
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

}  // namespace lsv
