// Speculative-length selection (LibraSpec Sec. 3.2-3.4, Algorithm 1) on the GPU.
//
// One wave per sequence.  Everything is binary64 with one rounding per operation in
// a fixed order (fp-contract off), so the result is bit-identical to a sequential
// IEEE evaluation of the same formulas.
#include "lsv_device.h"
#include "lsv_internal.h"

#pragma clang fp contract(off)

namespace lsv {

// One wave per sequence; lane j stands for draft position j + 1 (G <= 64).  Every value is
// formed by the same binary64 operations in the same order as a sequential evaluation:
// the running products and sums are carried left to right (each lane keeps its prefix),
// and only independent quantities (one objective value or one S_i per lane) are computed
// side by side.

// Wave-uniform broadcast of lane j's value.
LSV_DEV double bcast(double v, int j) { return __shfl(v, j, kWave); }
LSV_DEV float bcastf(float v, int j) { return __shfl(v, j, kWave); }

// Lane d-1 gets f(d) = N(d) / cost[d] with P_j = P_{j-1} q_j, N(d) = bonus + sum_{j<=d} P_j
// (Eq. 2 objective), for d <= d_max.
LSV_DEV double objective_lane(float q, const double* cost, int d_max, bool bonus, int lane) {
  double p = 1.0, n = bonus ? 1.0 : 0.0, mine = 0.0;
  for (int j = 1; j <= d_max; ++j) {
    p = p * (double)bcastf(q, j - 1);
    n = n + p;
    if (lane == j - 1) mine = n;
  }
  return lane < d_max ? mine / cost[lane + 1] : -INFINITY;
}

// eps* = min_{i<=d} floor(alpha S_i + i), S_i = sum_{j=i}^{d} prod_{k=i}^{j} q_k (Algorithm 1);
// lane i-1 accumulates S_i over j = i..d.
LSV_DEV int eps_star_wave(float q, int d, double alpha, int lane) {
  const int i = lane + 1;
  double s = 0.0, p = 1.0;
  for (int j = 1; j <= d; ++j) {
    const double qj = (double)bcastf(q, j - 1);
    if (j >= i) {
      p = p * qj;
      s = s + p;
    }
  }
  int e = 0x7fffffff;
  if (i <= d) {
    const double t = alpha * s + (double)i;
    e = t >= 1.0e9 ? 1000000000 : (int)floor(t);  // any value > d_max acts alike
  }
  for (int o = 32; o > 0; o >>= 1) e = min(e, __shfl_xor(e, o, kWave));
  return e;
}

// Selection for sequence b by one wave; returns gamma (0 on invalid input) in every lane.
LSV_DEV int select_wave(int mode, int G, const float* __restrict__ conf, const double* __restrict__ cost, int d_init,
                        int d_max, double alpha, int block_n, unsigned flags, int b, int32_t* __restrict__ aux,
                        int32_t* __restrict__ status) {
  const int lane = threadIdx.x & 63;
  // blocks on demand (ALG1): only the first aux[b] * n confidences have been drafted, and
  // only those are read
  const bool on_demand = mode == LSV_SEL_ALG1 && (flags & LSV_SEL_DRAFTED);
  const int drafted = on_demand ? aux[b] : 0;
  const long long dn = (long long)drafted * block_n;
  const int avail = !on_demand ? G : (drafted < 1 ? 0 : (dn < G ? (int)dn : G));
  const float q = lane < avail ? conf[(size_t)b * G + lane] : 0.0f;
  bool bad = (lane < avail && !(q >= 0.0f && q <= 1.0f)) || (on_demand && drafted < 1);  // true for NaN
  if (mode != LSV_SEL_ALG1 && lane < d_max) {
    const double c = cost[lane + 1];
    bad = bad || !(c > 0.0 && c <= 1.7976931348623157e308);
  }
  const bool ok = !__any(bad);
  int d = 0, a = 0;
  if (ok) {
    if (mode == LSV_SEL_ALG1) {
      // Algorithm 1: from the block size the length climbs along d -> min(eps*(d), d_max)
      // while that raises it, and settles on eps*(d) (itself, or one step back) at the first d
      // where it does not.  Blocks: enough drafter blocks of n to cover the highest length.
      // A length past the drafted confidences (the budget went negative) stops the rule with
      // gamma 0 and the blocks it needs.
      d = block_n < d_max ? block_n : d_max;
      int settled = 0;  // eps* >= 1 always, so 0 means "still climbing"
      while (settled == 0 && d < d_max && d <= avail) {
        const int e = eps_star_wave(q, d, alpha, lane);
        if (e > d) d = e < d_max ? e : d_max;
        else settled = e;
      }
      a = (d + block_n - 1) / block_n;  // d >= 1 here, so at least one block
      if (settled) d = settled;
      else if (d > avail) d = 0;  // more blocks first
    } else {
      const double f = objective_lane(q, cost, d_max, (flags & LSV_SEL_BONUS) != 0, lane);
      if (mode == LSV_SEL_EXHAUSTIVE) {
        // smallest d whose f(d) is maximal (a strict '>' scan keeps the first maximum)
        double mx = f;
        for (int o = 32; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, kWave));
        const unsigned long long hit = __ballot(lane < d_max && f == mx);
        d = __ffsll((long long)hit);
      } else {
        d = d_init < 1 ? 1 : (d_init > d_max ? d_max : d_init);
        for (;;) {
          const double fd = bcast(f, d - 1);
          const double up = bcast(f, d < d_max ? d : d - 1), dn = bcast(f, d > 1 ? d - 2 : d - 1);
          if (d < d_max && up > fd) ++d;
          else if (d > 1 && dn >= fd) --d;
          else break;
          ++a;
        }
      }
    }
  }
  if (lane == 0) {
    if (aux) aux[b] = a;
    if (status) status[b] = ok ? LSV_OK : LSV_ERR_INVALID_ARG;
  }
  return d;
}

constexpr int kSelectWaves = 16;  // sequences selected side by side

// Wave w of workgroup g takes sequences (g * 16 + w) + k * 16 * gridDim.x.  With row offsets
// requested the grid is one workgroup (batch <= LSV_MAX_BATCH): gamma of every sequence is
// then scanned into the verify row offsets (rows = gamma + 1) by the first wave.
__global__ void __launch_bounds__(64 * kSelectWaves) select_length_kernel(
    int mode, int batch, int G, const float* __restrict__ conf, const double* __restrict__ cost, int d_init,
    int d_max, double alpha, int block_n, unsigned flags, int32_t* __restrict__ gamma, int32_t* __restrict__ aux,
    int32_t* __restrict__ row_offsets, int32_t* __restrict__ status) {
  __shared__ int s_gamma[LSV_MAX_BATCH];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int b = blockIdx.x * kSelectWaves + wave; b < batch; b += kSelectWaves * gridDim.x) {
    const int d = select_wave(mode, G, conf, cost, d_init, d_max, alpha, block_n, flags, b, aux, status);
    if (lane == 0) {
      gamma[b] = d;
      if (b < LSV_MAX_BATCH) s_gamma[b] = d;
    }
  }
  if (!row_offsets) return;
  __syncthreads();
  if (wave == 0) {  // inclusive scan of gamma + 1 (batch <= 64 = one wave)
    int v = lane < batch ? s_gamma[lane] + 1 : 0;
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(v, o, kWave);
      if (lane >= o) v += t;
    }
    if (lane < batch) row_offsets[lane + 1] = v;
    if (lane == 0) row_offsets[0] = 0;
  }
}

int launch_select(int mode, int batch, int G, const float* conf, const double* cost, int d_init, int d_max,
                  double alpha, int block_n, unsigned flags, int32_t* gamma, int32_t* aux, int32_t* row_offsets,
                  int32_t* status, hipStream_t stream) {
  // one workgroup when row offsets are written (the host checks batch <= LSV_MAX_BATCH then)
  const unsigned grid = row_offsets ? 1u : (unsigned)((batch + kSelectWaves - 1) / kSelectWaves);
  hipLaunchKernelGGL(select_length_kernel, dim3(grid), dim3(64 * kSelectWaves), 0, stream, mode, batch, G, conf,
                     cost, d_init, d_max, alpha, block_n, flags, gamma, aux, row_offsets, status);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

// Joint batched selection: gamma_b in [1, d_max] maximising sum_b N_b(gamma_b) / cost[R],
// R = sum_b gamma_b (Eq. 2's objective over a batch that shares one verify cost).  For each
// R the best allocation is every sequence's first draft plus the R - B largest increments
// P_{b,j} (j >= 2; N_b has non-increasing increments), ties to the smaller b, then j.  One
// workgroup: the increments' ranks in that order come from binary searches in each
// sequence's (non-increasing) list, the allocation for every R from binary searches in the
// ranks, and the objective for every R in the same binary64 order as a sequential
// evaluation (N_b left to right, summed over b in order).
constexpr int kJointThreads = 1024;

__global__ void __launch_bounds__(kJointThreads) select_joint_kernel(int batch, int G, const float* __restrict__ conf,
                                                                      const double* __restrict__ cost, int d_max,
                                                                      unsigned flags, int32_t* __restrict__ gamma,
                                                                      int32_t* __restrict__ total,
                                                                      int32_t* __restrict__ row_offsets,
                                                                      int32_t* __restrict__ status) {
  __shared__ double sP[LSV_MAX_BATCH][LSV_MAX_G];  // P_{b,j} at [b][j-1]
  __shared__ double sN[LSV_MAX_BATCH][LSV_MAX_G];  // N_b(j) at [b][j-1]
  __shared__ int sRank[LSV_MAX_BATCH][LSV_MAX_G];  // rank of increment (b, j >= 2) at [b][j-1]
  __shared__ double sBestF[kJointThreads / 64];
  __shared__ int sBestR[kJointThreads / 64], sBad;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const bool bonus = flags & LSV_SEL_BONUS;
  if (tid == 0) sBad = 0;
  __syncthreads();
  // 1. prefix products and expected accepted counts, one wave per sequence
  for (int b = wave; b < batch; b += kJointThreads / 64) {
    const float q = lane < G ? conf[(size_t)b * G + lane] : 0.0f;
    if (__any(lane < G && !(q >= 0.0f && q <= 1.0f))) sBad = 1;  // NaN fails both tests
    double p = 1.0, n = bonus ? 1.0 : 0.0;
    for (int j = 1; j <= d_max; ++j) {
      p = p * (double)bcastf(q, j - 1);
      n = n + p;
      if (lane == j - 1) {
        sP[b][lane] = p;
        sN[b][lane] = n;
      }
    }
  }
  const int Rmin = batch, Rmax = batch * d_max;
  for (int R = Rmin + tid; R <= Rmax; R += kJointThreads)
    if (!(cost[R] > 0.0 && cost[R] <= 1.7976931348623157e308)) sBad = 1;
  __syncthreads();
  if (sBad) {
    for (int b = tid; b < batch; b += kJointThreads) {
      gamma[b] = 0;
      if (status) status[b] = LSV_ERR_INVALID_ARG;
    }
    if (tid == 0 && total) *total = 0;
    if (row_offsets)
      for (int i = tid; i <= batch; i += kJointThreads) row_offsets[i] = i;  // root rows only
    return;
  }
  // 2. rank of every increment (b, j), 2 <= j <= d_max, in (value desc, b asc, j asc) order
  const int per = d_max - 1;  // increments per sequence
  for (int e = tid; e < batch * per; e += kJointThreads) {
    const int b = e / per, j = 2 + e % per;
    const double v = sP[b][j - 1];
    int rank = j - 2;  // the sequence's own earlier increments
    for (int o = 0; o < batch; ++o) {
      if (o == b) continue;
      // count of j' in [2, d_max] with P > v (o > b) or P >= v (o < b): a prefix of o's list
      int lo = 2, hi = d_max + 1;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        const double w = sP[o][mid - 1];
        if (o < b ? w >= v : w > v) lo = mid + 1;
        else hi = mid;
      }
      rank += lo - 2;
    }
    sRank[b][j - 1] = rank;
  }
  __syncthreads();
  // 3. objective for every total R; the best (largest f, then smallest R) per thread, then per wave
  double bestF = -1.0;
  int bestR = 0x7fffffff;
  for (int R = Rmin + tid; R <= Rmax; R += kJointThreads) {
    const int take = R - Rmin;  // increments beyond the first drafts
    double s = 0.0;
    for (int b = 0; b < batch; ++b) {
      int lo = 2, hi = d_max + 1;  // gamma_b = 1 + #{j >= 2 : rank < take} (ranks rise with j)
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (sRank[b][mid - 1] < take) lo = mid + 1;
        else hi = mid;
      }
      s = s + sN[b][lo - 2];  // N_b(gamma_b), gamma_b = lo - 1
    }
    const double f = s / cost[R];
    if (f > bestF) {  // R rises within a thread: ties keep the smaller R
      bestF = f;
      bestR = R;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const double f2 = __shfl_xor(bestF, o, kWave);
    const int r2 = __shfl_xor(bestR, o, kWave);
    if (f2 > bestF || (f2 == bestF && r2 < bestR)) {
      bestF = f2;
      bestR = r2;
    }
  }
  if (lane == 0) {
    sBestF[wave] = bestF;
    sBestR[wave] = bestR;
  }
  __syncthreads();
  if (wave != 0) return;
  bestF = lane < kJointThreads / 64 ? sBestF[lane] : -1.0;
  bestR = lane < kJointThreads / 64 ? sBestR[lane] : 0x7fffffff;
  for (int o = 32; o > 0; o >>= 1) {
    const double f2 = __shfl_xor(bestF, o, kWave);
    const int r2 = __shfl_xor(bestR, o, kWave);
    if (f2 > bestF || (f2 == bestF && r2 < bestR)) {
      bestF = f2;
      bestR = r2;
    }
  }
  // 4. the allocation at the best R, its status and the verify row offsets (batch <= 64)
  int g = 0;
  if (lane < batch) {
    const int take = bestR - Rmin;
    int lo = 2, hi = d_max + 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (sRank[lane][mid - 1] < take) lo = mid + 1;
      else hi = mid;
    }
    g = lo - 1;
    gamma[lane] = g;
    if (status) status[lane] = LSV_OK;
  }
  if (lane == 0 && total) *total = bestR;
  if (row_offsets) {
    int v = lane < batch ? g + 1 : 0;
    for (int o = 1; o < kWave; o <<= 1) {
      const int t = __shfl_up(v, o, kWave);
      if (lane >= o) v += t;
    }
    if (lane < batch) row_offsets[lane + 1] = v;
    if (lane == 0) row_offsets[0] = 0;
  }
}

int launch_select_joint(int batch, int G, const float* conf, const double* cost, int d_max, unsigned flags,
                        int32_t* gamma, int32_t* total, int32_t* row_offsets, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(select_joint_kernel, dim3(1), dim3(kJointThreads), 0, stream, batch, G, conf, cost, d_max, flags,
                     gamma, total, row_offsets, status);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

// Baseline length policy of the comparison experiments (Sec. 4.1; Appendix B, baseline
// details): the length rises by two after a round without a rejection and falls by one after a
// round with one, kept in [d_min, d_max].  Lane b of the single wave takes sequence b + 64 k;
// with row offsets requested (batch <= 64) the new lengths are scanned into them.  gamma_next
// may alias gamma: each element is read before the same lane writes it.
__global__ void __launch_bounds__(64) next_length_g4_kernel(int batch, const int32_t* gamma,
                                                             const int32_t* __restrict__ accept_len,
                                                             const int32_t* __restrict__ acc_status, int d_min,
                                                             int d_max, int32_t* gamma_next,
                                                             int32_t* __restrict__ row_offsets,
                                                             int32_t* __restrict__ err) {
  const int lane = threadIdx.x;
  int mine = 0;  // this lane's new length when b = lane (the scan's input)
  for (int b = lane; b < batch; b += kWave) {
    const int g = gamma[b], a = accept_len[b];
    const bool ok = acc_status == nullptr || acc_status[b] == LSV_OK;
    const bool valid = g >= 0 && g < LSV_MAX_SEQ_ROWS && (!ok || (a >= 0 && a <= g));
    const int raw = !valid ? d_min    // unusable round record: restart at the floor
                    : !ok ? g         // the round failed: no outcome to react to
                    : a == g ? g + 2  // every draft accepted
                             : g - 1; // a draft rejected
    const int next = min(max(raw, d_min), d_max);
    gamma_next[b] = next;
    if (err) err[b] = valid ? LSV_OK : LSV_ERR_INVALID_ARG;
    if (b == lane) mine = next;
  }
  if (!row_offsets) return;
  int v = lane < batch ? mine + 1 : 0;  // rows = root + gamma drafts
  for (int o = 1; o < kWave; o <<= 1) {
    const int t = __shfl_up(v, o, kWave);
    if (lane >= o) v += t;
  }
  if (lane < batch) row_offsets[lane + 1] = v;
  if (lane == 0) row_offsets[0] = 0;
}

int launch_next_length_g4(int batch, const int32_t* gamma, const int32_t* accept_len, const int32_t* status,
                          int d_min, int d_max, int32_t* gamma_next, int32_t* row_offsets, int32_t* err,
                          hipStream_t stream) {
  hipLaunchKernelGGL(next_length_g4_kernel, dim3(1), dim3(kWave), 0, stream, batch, gamma, accept_len, status, d_min,
                     d_max, gamma_next, row_offsets, err);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

}  // namespace lsv
