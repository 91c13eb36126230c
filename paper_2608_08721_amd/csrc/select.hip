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
  const float q = lane < G ? conf[(size_t)b * G + lane] : 0.0f;
  bool bad = lane < G && !(q >= 0.0f && q <= 1.0f);  // true for NaN
  if (mode != LSV_SEL_ALG1 && lane < d_max) {
    const double c = cost[lane + 1];
    bad = bad || !(c > 0.0 && c <= 1.7976931348623157e308);
  }
  const bool ok = !__any(bad);
  int d = 0, a = 0;
  if (ok) {
    if (mode == LSV_SEL_ALG1) {
      d = block_n < d_max ? block_n : d_max;
      long long B = 0;
      int blocks = 1;
      while (d < d_max) {
        int e = eps_star_wave(q, d, alpha, lane);
        if (e <= d) {  // single rollback, then stop
          d = e;
          break;
        }
        if (e > d_max) e = d_max;
        B -= (long long)(e - d);
        d = e;
        if (B < 0) {
          long long k = (-B + block_n - 1) / block_n;
          blocks += (int)k;
          B += k * block_n;
        }
      }
      a = blocks;
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
