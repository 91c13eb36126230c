// Causal grouped-query attention of the block rows over the KV cache.
//
// bf16 path (matrix cores), two kernels:
//  * split kernel: one workgroup of four or eight waves per (context split, kv head,
//    sequence).  A split is a run of 64-key chunks.  Each chunk's K rows and transposed V
//    rows (a contiguous [64][hd] and [hd][64] block per chunk, next to the other kv heads'
//    blocks) go HBM -> registers -> LDS with 16-byte accesses; the first chunk's loads are issued before any device metadata is read, and
//    each next chunk's loads are in flight while the current one is consumed.  A wave owns one tile of 16 query vectors (block
//    rows x query heads of this kv head) per pass over the split -- eight waves cover up to
//    32 rows of a 4-query-head group in one pass -- and keeps a running softmax:
//    S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_16x16x32_bf16.  The probabilities stay in
//    registers: the D layout of S^T is the B operand layout of P^T, and the V rows are
//    stored with their keys permuted (v_column) so that one 16-byte read is a fragment.
//    Output per split and query vector: running max (log2 units), sum, unnormalised O.
//  * merge kernel: per (row, query head) combines the splits in split order.
// fp32 path: a plain kernel, one wave per (row, query head).
#include <math.h>

#include <type_traits>

#include "lsv_attn.h"
#include "lsv_device.h"

namespace lsv {

constexpr int kCh = kAttnChunk;  // keys per chunk
// Split plan: about kAttnWgs split workgroups, and no split longer than kMaxChunksPerSplit
// chunks (a split walks its chunks in sequence).  Fewer splits mean fewer partials to merge
// -- one batch of merge loads for up to 16 -- against longer chunk walks; 128 measured best
// for one sequence of 2K context (11 splits of 3 chunks).  The length cap keeps the
// workgroups of a batch with long contexts from running too long -- but never beyond one
// workgroup per compute unit: a grid larger than the chip runs its last workgroups in a
// second round, which costs more than longer splits (Llama-3-70B, four sequences of 8K
// context: 9 splits, 288 workgroups, 49 us; 8 splits, 256 workgroups, 34 us).
constexpr int kAttnWgs = 128;
constexpr int kMaxChunksPerSplit = 16;
constexpr int kComputeUnits = 256;  // gfx950 (MI350X, MI355X)

//
// Long contexts over many (sequence, kv head) pairs -- when one round's splits would walk more
// than twice the length cap -- take a whole number of rounds' worth of splits instead, on a
// packed grid: the splits that hold keys come first, so in a batch of ragged contexts the
// empty splits of the short sequences no longer hold compute units while a long sequence walks
// its splits (Llama-3-8B, batch 8, contexts of 1.7K-8.2K: 4 splits of 33 chunks become 12 of
// 11).  With every context at the bound, three rounds of a third of the length cost what one
// round costs.  Split boundaries still follow from the host bound alone, so a row's result does
// not depend on its block, its batch or the other sequences' lengths.
AttnPlan plan_attention(int batch, int nkv, int max_ctx) {
  const int n_chunks = (max_ctx + kCh - 1) / kCh;
  const int units = batch * nkv;
  int want = (kAttnWgs + units - 1) / units;
  const int by_length = (n_chunks + kMaxChunksPerSplit - 1) / kMaxChunksPerSplit;
  if (want < by_length) want = by_length;
  const int fit = kComputeUnits / units;  // splits per (sequence, kv head) in one round
  AttnPlan p;
  p.packed = fit >= 1 && by_length > 2 * fit;
  if (p.packed)
    want = (by_length + fit - 1) / fit * fit;
  else if (want > fit)
    want = fit;
  if (want > n_chunks) want = n_chunks;
  if (want < 1) want = 1;
  p.chunks_per_split = (n_chunks + want - 1) / want;
  p.n_splits = (n_chunks + p.chunks_per_split - 1) / p.chunks_per_split;
  return p;
}

// Splits of sequence b that hold keys: ceil(chunks / chunks_per_split), none for a sequence
// without rows (or rows past the host bound).  At most n_splits, since L <= ctx_limit.
LSV_DEV int active_splits(const AttnArgs& a, int r0, int rows, int C) {
  if (r0 < 0 || rows <= 0 || r0 + rows > a.M_max) return 0;
  const int L = min(C + rows, a.ctx_limit);
  const int nch = L > 0 ? (L + kCh - 1) / kCh : 0;
  return (nch + a.chunks_per_split - 1) / a.chunks_per_split;
}

// Packed grid: workgroup i takes the i-th split that holds keys -- every sequence's full splits
// first (ordered by sequence, split, kv head), then every sequence's last split (by sequence, kv
// head) -- so the longest splits start first.  One lane per sequence (batch <= 64); every wave
// computes the same answer, moved to scalar registers.  False: no split is left for i.
LSV_DEV bool packed_unit(const AttnArgs& a, int i, int& s, int& kvh, int& b) {
  const int lane = threadIdx.x & 63;
  int act = 0;
  if (lane < a.batch) {
    const int r0 = GL(a.row_offsets)[lane], r1 = GL(a.row_offsets)[lane + 1];
    act = active_splits(a, r0, r1 - r0, GL(a.seq_len)[lane]);
  }
  const int full = act > 0 ? (act - 1) * a.nkv : 0, last = act > 0 ? a.nkv : 0;
  int pf = full, pl = last;  // inclusive prefix sums over the lanes
  for (int o = 1; o < kWave; o <<= 1) {
    const int tf = __shfl_up(pf, o, kWave), tl = __shfl_up(pl, o, kWave);
    if (lane >= o) {
      pf += tf;
      pl += tl;
    }
  }
  const int F = __builtin_amdgcn_readfirstlane(__shfl(pf, kWave - 1, kWave));
  const int P = __builtin_amdgcn_readfirstlane(__shfl(pl, kWave - 1, kWave));
  const bool in_full = i < F;
  const int j = in_full ? i : i - F;
  if (!in_full && j >= P) return false;
  const unsigned long long over = __ballot(in_full ? pf > j : pl > j);  // lanes past unit j
  const int bb = __builtin_amdgcn_readfirstlane(__ffsll((long long)over) - 1);
  const int local = j - __builtin_amdgcn_readfirstlane(__shfl(in_full ? pf - full : pl - last, bb, kWave));
  b = bb;
  if (in_full) {
    s = local / a.nkv;
    kvh = local % a.nkv;
  } else {
    s = __builtin_amdgcn_readfirstlane(__shfl(act, bb, kWave)) - 1;
    kvh = local;
  }
  return true;
}

template <int HD, int NW>
__global__ void __launch_bounds__(64 * NW) attn_split_bf16_kernel(AttnArgs a) {
  constexpr int NG = NW / 4;               // wave groups: each loads one chunk per step
  constexpr int P8 = HD / 8;               // 16-byte pieces per K row
  constexpr int NP = kCh * HD / 8 / 256;   // pieces of K (and of V^T) per thread of a group and chunk
  // LDS rows padded by 32 bytes: on gfx950 a 16-byte pad still left 2.5 bank-conflict cycles per
  // LDS instruction (SQ_LDS_BANK_CONFLICT); 32 bytes leaves none
  constexpr int KPITCH = HD + 16, VPITCH = kCh + 16;
  static_assert(NG >= 1 && NG * 4 == NW && NP >= 1 && NP * 256 * 8 == kCh * HD, "four-wave groups");
  __shared__ __align__(16) bf16_t Ks[NG][kCh * KPITCH];  // one chunk buffer per group
  __shared__ __align__(16) bf16_t Vt[NG][HD * VPITCH];

  int s = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  if (a.packed && !packed_unit(a, blockIdx.x, s, kvh, b)) return;
  // the wave index in a scalar register: the group, its chunk offsets and the page-table reads
  // are then wave-uniform, and the buffer loads take their chunk offsets in scalar registers
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int g4 = lane >> 4, l16 = lane & 15;
  const int grp = wave >> 2, gtid = tid & 255;
  // A chunk is one 64-position block of the cache.  Slab mode: the grid covers the chunks of
  // ctx_limit <= capacity and capacity is a multiple of the chunk, so every chunk below
  // capacity / kCh is one of the sequence's blocks.  Paged mode: a chunk is a page; chunks
  // below max_pages have a page-table entry.
  const bool paged = a.kv.pages != nullptr;
  const int c0 = s * a.chunks_per_split, cap_chunks = paged ? a.kv.max_pages : a.capacity / kCh;

  // a step covers chunks c .. c+NG-1, group g loading chunk c+g into buffer g; the next
  // step's chunks are in flight in registers while the current ones are used. The loads go
  // through buffer descriptors -- over this sequence's blocks, or over the layer's page pool
  // -- with one 32-bit lane offset per operand and the chunk and piece offsets in scalar
  // registers; reads past the descriptor return zero (a page number outside the pool points
  // there).
  const GLOBAL bf16_t* kb = GL((const bf16_t*)a.k);
  const GLOBAL bf16_t* vb = GL((const bf16_t*)a.v);
  // V^T comes in blocks of one chunk, [hd][64], in both modes: the rows of a chunk's V^T are kCh
  // elements apart
  constexpr int vstride = kCh;
  int span_bytes;
  if (paged) {
    span_bytes = a.kv.n_pages * a.nkv * kCh * HD * (int)sizeof(bf16_t);  // < 2^31, checked on the host
  } else {
    const size_t seq = (size_t)b * a.nkv * a.capacity * HD;  // this sequence's blocks
    kb += seq;
    vb += seq;
    span_bytes = a.nkv * a.capacity * HD * (int)sizeof(bf16_t);  // < 2^31, checked on the host
  }
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc((void*)kb, 0, span_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc((void*)vb, 0, span_bytes, 0x00020000);
  const int koff = ((gtid / P8) * HD + (gtid % P8) * 8) * (int)sizeof(bf16_t);
  const int voff = ((gtid >> 3) * vstride + (gtid & 7) * 8) * (int)sizeof(bf16_t);
  // element offset of chunk c's K rows and of its V^T block (the same offset: a block starts a
  // [64][hd] K block and a [hd][64] V^T block for each kv head)
  auto chunk_base = [&](int c, int& kbase, int& vbase) {
    if (!paged) {
      kbase = vbase = (c * a.nkv + kvh) * kCh * HD;
      return;
    }
    int page = GL(a.kv.pages)[(size_t)b * a.kv.max_pages + c];
    if (page < 0 || page >= a.kv.n_pages) page = a.kv.n_pages;  // past the pool: reads zero
    kbase = vbase = (page * a.nkv + kvh) * kCh * HD;
  };
  u32x4_t kr[NP], vr[NP];
  auto load_chunk = [&](int c) {
    int kbase, vbase;
    chunk_base(c, kbase, vbase);
#pragma unroll
    for (int j = 0; j < NP; ++j) {  // piece gtid + 256 j: K row + j 256 / P8, V^T row + 32 j
      kr[j] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                              krs, koff, (kbase + j * (256 / P8) * HD) * (int)sizeof(bf16_t), kBufferStream));
      vr[j] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                                              vrs, voff, (vbase + j * 32 * vstride) * (int)sizeof(bf16_t), kBufferStream));
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const int i = gtid + 256 * j;
      *(u32x4_t*)&Ks[grp][(i / P8) * KPITCH + (i % P8) * 8] = kr[j];
      *(u32x4_t*)&Vt[grp][(i >> 3) * VPITCH + (i & 7) * 8] = vr[j];
    }
  };
  if (grp < a.chunks_per_split && c0 + grp < cap_chunks) load_chunk(c0 + grp);

  const int r0 = GL(a.row_offsets)[b], rows = GL(a.row_offsets)[b + 1] - r0, C = GL(a.seq_len)[b];
  if (r0 < 0 || rows <= 0 || r0 + rows > a.M_max) return;  // rows beyond the host bound are never touched
  const int group = a.nq / a.nkv, nqv = rows * group, n_qt = (nqv + 15) / 16;
  const int L = min(C + rows, a.ctx_limit);  // cached + block keys that exist
  const int nch = L > 0 ? (L + kCh - 1) / kCh : 0;
  const int c1 = min(c0 + a.chunks_per_split, nch);
  const size_t prow = (size_t)s * a.M_max + r0;  // this split's partial row of the sequence's first row
  if (c0 >= c1) return;  // no key of this split exists for the sequence: the merge does not read it
  // A pass over the split covers up to NW query tiles, one per wave, each wave running its
  // tile over all chunks in order.  Every tile takes the same chunk order and the same
  // arithmetic whatever the block's tile count, so a row's result does not depend on how
  // many rows share its block (decoding then emits the same tokens for every length).
  for (int qbase = 0; qbase < n_qt; qbase += NW) {
    const int qt = qbase + wave;
    const bool active = qt < n_qt;  // wave-uniform
    u32x4_t qf[HD / 32];
    f32x4_t o[HD / 16];
    float mrun = -INFINITY, lrun = 0.f;
    const int qv = qt * 16 + l16;
    const bool qval = active && qv < nqv;
    const int rr = qval ? qv / group : 0;
    const int qpos = C + rr;
    {
      const int head = kvh * group + (qval ? qv % group : 0);
      const GLOBAL bf16_t* qp = GL((const bf16_t*)a.q) + ((size_t)(r0 + rr) * a.nq + head) * HD + 8 * g4;
#pragma unroll
      for (int ds = 0; ds < HD / 32; ++ds) {  // rr = 0 for invalid columns: the load stays in bounds
        const u32x4_t t = *(const GLOBAL u32x4_t*)(qp + 32 * ds);
        qf[ds] = qval ? t : u32x4_t{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    if (qbase > 0 && c0 + grp < c1) load_chunk(c0 + grp);  // a later pass over the same split

    // scores and running-softmax update of this wave's tile for the chunk in buffer g.
    // A chunk below the cached length C is visible to every row of the block: no mask, and
    // its scores are finite (exp2 needs no guard); only chunks that reach the block's own
    // keys apply the causal and length mask.  Both take the same hardware exp2, so a key
    // contributes the same bits whether or not its chunk was masked.
    auto consume = [&](int g, int c, auto masked) {
      constexpr bool MASK = decltype(masked)::value;
      const int k0 = c * kCh;
      f32x4_t sc[4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        sc[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < HD / 32; ++ds) {
          const u32x4_t kf = *(const u32x4_t*)&Ks[g][(16 * kt + l16) * KPITCH + 32 * ds + 8 * g4];
          sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kf),
                                                           __builtin_bit_cast(bf16x8_t, qf[ds]), sc[kt], 0, 0, 0);
        }
      }
      // scale (log2 units), causal mask, running max over the split
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float v = sc[kt][r] * a.scale_log2;
          if (MASK) {
            const int kp = k0 + 16 * kt + 4 * g4 + r;
            bool vis;
            if (a.anc) {  // tree block: cached keys, then the slots of the row's ancestors and itself
              const int j = kp - C;
              vis = kp < C || (kp < L && j < kTreeNodes &&
                               ((GL(a.anc)[(size_t)(r0 + rr) * kAncWords + (j >> 5)] >> (j & 31)) & 1u));
            } else {
              vis = kp < L && kp <= qpos;
            }
            v = qval && vis ? v : -INFINITY;
          }
          sc[kt][r] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      const float mnew = fmaxf(mrun, mx);
      float alpha, sum = 0.f;
      if (MASK) {
        alpha = mrun == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mrun - mnew);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = mnew == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sc[kt][r] - mnew);
            sc[kt][r] = p;
            sum += p;
          }
      } else {  // mnew is finite; exp2(-inf) = 0 covers a first chunk (mrun = -inf)
        alpha = __builtin_amdgcn_exp2f(mrun - mnew);
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = __builtin_amdgcn_exp2f(sc[kt][r] - mnew);
            sc[kt][r] = p;
            sum += p;
          }
      }
      sum += __shfl_xor(sum, 16, kWave);
      sum += __shfl_xor(sum, 32, kWave);
      mrun = mnew;
      lrun = lrun * alpha + sum;
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) o[dt] *= alpha;
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
          const u32x4_t vf = *(const u32x4_t*)&Vt[g][(16 * dt + l16) * VPITCH + 32 * ks + 8 * g4];
          o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, vf), pb, o[dt], 0, 0, 0);
        }
      }
    };

    for (int c = c0; c < c1; c += NG) {
      __syncthreads();  // the previous step's LDS reads are done
      if (c + grp < c1) store_chunk();
      __syncthreads();
      if (c + NG + grp < c1) load_chunk(c + NG + grp);
      if (!active) continue;  // wave-uniform: a wave without a query tile in this pass
      using Masked = std::true_type;
      using Full = std::false_type;
#pragma unroll
      for (int g = 0; g < NG; ++g)
        if (c + g < c1) {
          if ((c + g + 1) * kCh <= C) consume(g, c + g, Full{});
          else consume(g, c + g, Masked{});
        }
    }

    if (active && qval) {
      const size_t base = (prow + qv / group) * a.nq + kvh * group + qv % group;
      GLOBAL float* op = GL(a.o_part) + base * HD;
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) *(GLOBAL f32x4_t*)(op + 16 * dt + 4 * g4) = o[dt];
      if (g4 == 0) *(GLOBAL f32x2_t*)(a.ml_part + base * 2) = f32x2_t{mrun, lrun};
    }
    __syncthreads();  // the next pass refills the chunk buffers
  }
}

// Merge the split partials of one (row, query head): out = sum_s w_s o_s / sum_s w_s l_s,
// w_s = 2^(m_s - max_s m_s), splits in ascending order, 16 splits' loads in flight at a time.
// Only the splits that hold keys of the row's sequence were written and are read.
// A wave covers 256 / HD heads of one row, four head dimensions per lane.
template <int HD>
__global__ void __launch_bounds__(64) attn_merge_bf16_kernel(AttnArgs a) {
  constexpr int LPH = HD / 4, HPW = 64 / LPH, NB = 16;
  const int m = blockIdx.x, head = blockIdx.y * HPW + threadIdx.x / LPH, d = (threadIdx.x % LPH) * 4;
  // lane t: sequence t (batch <= 64); the row's sequence is the number of sequences ending at
  // or before it
  int mr0 = 0, mr1 = 0, mC = 0;
  if ((int)threadIdx.x < a.batch) {
    mr0 = GL(a.row_offsets)[threadIdx.x];
    mr1 = GL(a.row_offsets)[threadIdx.x + 1];
    mC = GL(a.seq_len)[threadIdx.x];
  }
  const int M = __shfl(mr1, a.batch - 1, kWave);
  const int b = __popcll(__ballot((int)threadIdx.x < a.batch && mr1 <= m));
  const int r0 = __shfl(mr0, b, kWave), r1 = __shfl(mr1, b, kWave), C = __shfl(mC, b, kWave);
  if (m >= M || head >= a.nq) return;  // after the lane exchanges, which need every lane
  const int ns = active_splits(a, r0, r1 - r0, C);
  const size_t stride = (size_t)a.M_max * a.nq, rh = (size_t)m * a.nq + head;
  const GLOBAL f32x2_t* ml = (const GLOBAL f32x2_t*)a.ml_part;
  const GLOBAL float* op = GL(a.o_part);
  float mx_all = -INFINITY, den = 0.f;
  f32x4_t num = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < ns; s0 += NB) {
    f32x2_t mv[NB];
    f32x4_t ov[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const size_t s = (size_t)min(s0 + i, ns - 1);
      mv[i] = ml[s * stride + rh];
      ov[i] = *(const GLOBAL f32x4_t*)(op + (s * stride + rh) * HD + d);
    }
    float mx = mx_all;
#pragma unroll
    for (int i = 0; i < NB; ++i)
      if (s0 + i < ns) mx = fmaxf(mx, mv[i][0]);
    const float al = mx_all == -INFINITY ? 0.f : exp2f(mx_all - mx);
    den *= al;
    num *= al;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      // a split none of whose keys the row sees (max -inf) contributes nothing
      if (s0 + i < ns && mv[i][0] != -INFINITY) {
        const float w = exp2f(mv[i][0] - mx);
        den += w * mv[i][1];
        num += w * ov[i];
      }
    }
    mx_all = mx;
  }
  const f32x4_t r = num / den;
  const u32x2_t packed = {(uint32_t)f2bf(r[0]) | ((uint32_t)f2bf(r[1]) << 16),
                          (uint32_t)f2bf(r[2]) | ((uint32_t)f2bf(r[3]) << 16)};
  // the O projection's activation operand: column head * HD + d of row m (d .. d+3 adjacent)
  *(GLOBAL u32x2_t*)(GL((bf16_t*)a.out) + act_index<32>(m, head * HD + d, a.nq * HD / 32)) = packed;
}

// fp32 path: one wave per (row, query head); scores in LDS.
__global__ void __launch_bounds__(64) attn_f32_kernel(AttnArgs a, int hd) {
  extern __shared__ float sc[];  // [ctx_limit]
  const int m = blockIdx.x, head = blockIdx.y, t = threadIdx.x;
  if (m >= a.row_offsets[a.batch]) return;
  const int b = seq_of_row(a.row_offsets, a.batch, m);
  const int r0 = a.row_offsets[b], rows = a.row_offsets[b + 1] - r0;
  const int C = a.seq_len[b], pos = C + (m - r0);
  // causal: keys 0..pos; tree block: keys below C + rows, block keys masked to the row's ancestors
  const int L = a.anc ? min(C + rows, a.ctx_limit) : min(min(pos + 1, C + rows), a.ctx_limit);
  auto visible = [&](int j) {
    if (!a.anc || j < C) return true;
    const int i = j - C;
    return i < kTreeNodes && ((a.anc[(size_t)m * kAncWords + (i >> 5)] >> (i & 31)) & 1u) != 0;
  };
  const int kvh = head / (a.nq / a.nkv);
  const float* K = (const float*)a.k;
  const float* Vt = (const float*)a.v;
  const float* q = (const float*)a.q + ((size_t)m * a.nq + head) * hd;
  const float scale = rsqrtf((float)hd);
  float mx = -INFINITY;
  for (int j = t; j < L; j += 64) {
    float s = -INFINITY;
    size_t ko, vo;
    int vs;
    if (visible(j) && kv_locate(a.kv, a.nkv, hd, b, kvh, j, ko, vo, vs)) {
      s = 0.f;
      for (int i = 0; i < hd; ++i) s += q[i] * K[ko + i];
      s *= scale;
    }
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
    for (int j = 0; j < L; ++j) {
      size_t ko, vo;
      int vs;
      if (sc[j] != 0.f && kv_locate(a.kv, a.nkv, hd, b, kvh, j, ko, vo, vs)) o += sc[j] * Vt[vo + (size_t)i * vs];
    }
    ((float*)a.out)[act_index<16>(m, head * hd + i, a.nq * hd / 16)] = o / sum;
  }
}

int launch_attention(int dtype, int hd, const AttnArgs& a, int max_rows, hipStream_t st) {
  if (dtype == LSV_DTYPE_BF16) {
    const dim3 grid = a.packed ? dim3(a.n_splits * a.nkv * a.batch) : dim3(a.n_splits, a.nkv, a.batch);
    const int hpw = 256 / hd;
    const dim3 mgrid(max_rows, (a.nq + hpw - 1) / hpw);
    // query tiles per sequence (rows of a single sequence, else the mean over the batch): up
    // to four take four waves, more take eight so that one pass covers them
    const int rows_seq = (max_rows + a.batch - 1) / a.batch;
    const bool wide = (size_t)rows_seq * (a.nq / a.nkv) > 64;
    if (hd == 128) {
      if (wide)
        hipLaunchKernelGGL((attn_split_bf16_kernel<128, 8>), grid, dim3(512), 0, st, a);
      else
        hipLaunchKernelGGL((attn_split_bf16_kernel<128, 4>), grid, dim3(256), 0, st, a);
      hipLaunchKernelGGL(attn_merge_bf16_kernel<128>, mgrid, dim3(64), 0, st, a);
    } else if (hd == 64) {
      if (wide)
        hipLaunchKernelGGL((attn_split_bf16_kernel<64, 8>), grid, dim3(512), 0, st, a);
      else
        hipLaunchKernelGGL((attn_split_bf16_kernel<64, 4>), grid, dim3(256), 0, st, a);
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
