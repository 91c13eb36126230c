// Speculative-length selection (LibraSpec Sec. 3.2-3.4, Algorithm 1) on the GPU.
//
// One lane per sequence.  Everything is binary64 with one rounding per
// operation in a fixed order (fp-contract off), so the result is bit-identical
// to any sequential IEEE evaluation of the same formulas.
#include "lsv_device.h"
#include "lsv_internal.h"

#pragma clang fp contract(off)

namespace lsv {

// P_j = P_{j-1} q_j; N(d) = bonus + sum_{j<=d} P_j; f(d) = N(d) / cost[d]  (Eq. 2 objective).
__device__ static void objective(const float* q, const double* cost, int G, bool bonus, double* f) {
  double p = 1.0, n = bonus ? 1.0 : 0.0;
  for (int j = 1; j <= G; ++j) {
    p = p * (double)q[j - 1];
    n = n + p;
    f[j] = n / cost[j];
  }
}

// S_i = sum_{j=i}^{d} prod_{k=i}^{j} q_k; eps* = min_i floor(alpha S_i + i)  (Algorithm 1).
__device__ static int eps_star(const float* q, int d, double alpha) {
  int best = 0x7fffffff;
  for (int i = 1; i <= d; ++i) {
    double s = 0.0, p = 1.0;
    for (int j = i; j <= d; ++j) {
      p = p * (double)q[j - 1];
      s = s + p;
    }
    double t = alpha * s + (double)i;
    int e = t >= 1.0e9 ? 1000000000 : (int)floor(t);  // any value > d_max acts alike
    best = e < best ? e : best;
  }
  return best;
}

__device__ static int select_one(int mode, int G, const float* __restrict__ conf, const double* __restrict__ cost,
                                 int d_init, int d_max, double alpha, int block_n, unsigned flags, int b,
                                 int32_t* __restrict__ aux, int32_t* __restrict__ status) {
  float q[LSV_MAX_G];
  bool ok = true;
  for (int j = 0; j < G; ++j) {
    q[j] = conf[(size_t)b * G + j];
    ok = ok && (q[j] >= 0.0f && q[j] <= 1.0f);  // false for NaN
  }
  if (mode != LSV_SEL_ALG1) {
    for (int d = 1; d <= d_max; ++d) {
      double c = cost[d];
      ok = ok && (c > 0.0 && c <= 1.7976931348623157e308);
    }
  }
  int d = 0, a = 0;
  if (ok) {
    if (mode == LSV_SEL_ALG1) {
      d = block_n < d_max ? block_n : d_max;
      long long B = 0;
      int blocks = 1;
      while (d < d_max) {
        int e = eps_star(q, d, alpha);
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
      double f[LSV_MAX_G + 1];
      objective(q, cost, d_max, (flags & LSV_SEL_BONUS) != 0, f);
      if (mode == LSV_SEL_EXHAUSTIVE) {
        d = 1;
        for (int j = 2; j <= d_max; ++j)
          if (f[j] > f[d]) d = j;
      } else {
        d = d_init < 1 ? 1 : (d_init > d_max ? d_max : d_init);
        for (;;) {
          if (d < d_max && f[d + 1] > f[d]) ++d;
          else if (d > 1 && f[d - 1] >= f[d]) --d;
          else break;
          ++a;
        }
      }
    }
  }
  if (aux) aux[b] = a;
  if (status) status[b] = ok ? LSV_OK : LSV_ERR_INVALID_ARG;
  return d;
}

__global__ void __launch_bounds__(64) select_length_kernel(int mode, int batch, int G, const float* __restrict__ conf,
                                                           const double* __restrict__ cost, int d_init, int d_max,
                                                           double alpha, int block_n, unsigned flags,
                                                           int32_t* __restrict__ gamma, int32_t* __restrict__ aux,
                                                           int32_t* __restrict__ row_offsets,
                                                           int32_t* __restrict__ status) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  int d = 0;
  if (b < batch) d = select_one(mode, G, conf, cost, d_init, d_max, alpha, block_n, flags, b, aux, status);
  if (b < batch) gamma[b] = d;
  if (row_offsets) {  // single wave (batch <= 64): inclusive scan of gamma + 1
    int v = b < batch ? d + 1 : 0;
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(v, o, 64);
      if ((threadIdx.x & 63) >= o) v += t;
    }
    if (b < batch) row_offsets[b + 1] = v;
    if (b == 0) row_offsets[0] = 0;
  }
}

int launch_select(int mode, int batch, int G, const float* conf, const double* cost, int d_init, int d_max,
                  double alpha, int block_n, unsigned flags, int32_t* gamma, int32_t* aux, int32_t* row_offsets,
                  int32_t* status, hipStream_t stream) {
  dim3 grid((batch + 63) / 64);
  hipLaunchKernelGGL(select_length_kernel, grid, dim3(64), 0, stream, mode, batch, G, conf, cost, d_init, d_max,
                     alpha, block_n, flags, gamma, aux, row_offsets, status);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

}  // namespace lsv
