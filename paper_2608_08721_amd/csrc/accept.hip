// Acceptance of a verified block (LibraSpec Sec. 3.1) on the GPU.
//
// Greedy: a row scan (vocabulary split over workgroups, partial (max, first
// argmax) per chunk), then one wave per sequence merges the partials in chunk
// order and finds the accepted prefix with a ballot.
// Sampling: a row scan for the softmax normalisers (max, sum of exponentials per
// chunk), one wave per sequence for the ratio tests, then a vocabulary-parallel
// exponential race for the correction / bonus token whose last workgroup commits.
#include <math.h>

#include <mutex>

#include "lsv_device.h"
#include "lsv_internal.h"

namespace lsv {

// ------------------------------------------------------------------ Philox4x64-10
// Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC'11).
struct U64x4 {
  uint64_t w[4];
};
LSV_DEV U64x4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0, uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    uint64_t hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
    uint64_t hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
    uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += W0;
    k1 += W1;
  }
  U64x4 o;
  o.w[0] = c0;
  o.w[1] = c1;
  o.w[2] = c2;
  o.w[3] = c3;
  return o;
}
LSV_DEV double unit52(uint64_t w) { return ((double)(w >> 12) + 0.5) * (1.0 / 4503599627370496.0); }
constexpr uint64_t kStreamAccept = 1, kStreamSample = 2;

// ------------------------------------------------------------------ workspace
struct RowPartial {  // greedy: (val, idx); sampling: (max z, sum exp(z - max))
  float a;
  float b;
  int idx;
  int bad;
};
struct SeqDecision {
  int status, a, row, residual;
  int draft_row;  // q row for the residual draw
  float m, z;     // softmax max and normaliser of the sampled row
  int pad;
};
struct RacePartial {
  double key_res, key_p;
  int idx_res, idx_p, bad, pad;
};

struct AcceptWs {
  RowPartial* rows;  // [max_rows][chunks]
  SeqDecision* seq;  // [batch]
  RacePartial* race; // [batch][chunks]
  int* counters;     // [batch]
};
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
static AcceptWs carve(void* ws, int batch, int max_rows, int vocab) {
  int nc = accept_chunks(vocab);
  char* p = (char*)ws;
  AcceptWs w;
  w.rows = (RowPartial*)p;
  p += align256(sizeof(RowPartial) * (size_t)max_rows * nc);
  w.seq = (SeqDecision*)p;
  p += align256(sizeof(SeqDecision) * (size_t)batch);
  w.race = (RacePartial*)p;
  p += align256(sizeof(RacePartial) * (size_t)batch * nc);
  w.counters = (int*)p;
  return w;
}
size_t accept_workspace_bytes(int batch, int max_rows, int vocab) {
  int nc = accept_chunks(vocab);
  return align256(sizeof(RowPartial) * (size_t)max_rows * nc) + align256(sizeof(SeqDecision) * (size_t)batch) +
         align256(sizeof(RacePartial) * (size_t)batch * nc) + align256(sizeof(int) * (size_t)batch);
}

// ------------------------------------------------------------------ row scans
// greedy: first index of the maximum over the chunk; sampling: (max z, sum exp(z - max)), z = l / T.
template <bool kSample>
__global__ void __launch_bounds__(256) row_scan_kernel(const float* __restrict__ logits, const int32_t* row_offsets,
                                                       int batch, int vocab, float temperature, RowPartial* out) {
  const int r = blockIdx.y, c = blockIdx.x, nc = gridDim.x;
  if (r >= row_offsets[batch]) return;
  const auto* row = GL(logits) + (size_t)r * vocab;
  const int x0 = c * kAcceptChunk, x1 = min(vocab, x0 + kAcceptChunk);
  float best = -INFINITY;
  int bidx = 0x7fffffff, bad = 0;
  // all of the thread's loads are issued before the first is used (one memory round trip);
  // the elements are then taken in increasing x, as a strided loop would
  constexpr int PER = kAcceptChunk / 256;
  static_assert(PER * 256 == kAcceptChunk, "whole strides per chunk");
  float vals[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int x = x0 + (int)threadIdx.x + 256 * i;
    vals[i] = x < x1 ? row[x] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int x = x0 + (int)threadIdx.x + 256 * i;
    if (x >= x1) break;
    float v = vals[i];
    if (!isfinite(v)) bad = 1;
    if (kSample) v = v / temperature;
    if (v > best || (v == best && x < bidx)) {
      best = v;
      bidx = x;
    }
  }
  float sum = 0.f;
  __shared__ float s_best[256];
  __shared__ int s_idx[256], s_bad[256];
  __shared__ float s_sum[256];
  s_best[threadIdx.x] = best;
  s_idx[threadIdx.x] = bidx;
  s_bad[threadIdx.x] = bad;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) {
      float ob = s_best[threadIdx.x + o];
      int oi = s_idx[threadIdx.x + o];
      if (ob > s_best[threadIdx.x] || (ob == s_best[threadIdx.x] && oi < s_idx[threadIdx.x])) {
        s_best[threadIdx.x] = ob;
        s_idx[threadIdx.x] = oi;
      }
      s_bad[threadIdx.x] |= s_bad[threadIdx.x + o];
    }
    __syncthreads();
  }
  const float cmax = s_best[0];
  if (kSample) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {  // the same elements, from registers, in the same order
      if (x0 + (int)threadIdx.x + 256 * i >= x1) break;
      sum += expf(vals[i] / temperature - cmax);
    }
    s_sum[threadIdx.x] = sum;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
      if (threadIdx.x < o) s_sum[threadIdx.x] += s_sum[threadIdx.x + o];
      __syncthreads();
    }
  }
  if (threadIdx.x == 0) {
    RowPartial p;
    p.a = cmax;
    p.b = kSample ? s_sum[0] : 0.f;
    p.idx = s_idx[0];
    p.bad = s_bad[0];
    out[(size_t)r * nc + c] = p;
  }
}

// ------------------------------------------------------------------ greedy
__global__ void __launch_bounds__(64) accept_greedy_kernel(const RowPartial* __restrict__ parts, int nc,
                                                           const int32_t* row_offsets, int max_rows,
                                                           const int32_t* tokens, int width, int32_t* accept_len,
                                                           int32_t* out_tokens, int32_t* seq_len, int32_t* status) {
  const int b = blockIdx.x, lane = threadIdx.x;
  // a sequence that arrives with an error (e.g. the verify step's capacity check) is skipped:
  // no tokens, accept_len 0, no commit, its status kept
  if (status && status[b] != LSV_OK) {
    if (lane < width) out_tokens[(size_t)b * width + lane] = -1;
    if (lane == 0) accept_len[b] = 0;
    return;
  }
  const int r0 = row_offsets[b], r1 = row_offsets[b + 1];
  const bool in_bounds = r0 >= 0 && r1 >= r0 && r1 <= max_rows;
  const int rows = in_bounds ? r1 - r0 : 0, g = rows - 1;
  int am = 0, bad = 0;
  const int next_tok = lane < g ? tokens[r0 + lane + 1] : 0;  // issued ahead of the partials' loads
  if (lane < rows) {
    float best = -INFINITY;
    int bi = 0x7fffffff;
    // chunks in ascending index order (strict '>' keeps the first maximum), eight partials'
    // loads in flight at a time
    constexpr int NB = 8;
    const RowPartial* rp = parts + (size_t)(r0 + lane) * nc;
    for (int c0 = 0; c0 < nc; c0 += NB) {
      RowPartial pb[NB];
#pragma unroll
      for (int i = 0; i < NB; ++i) pb[i] = rp[min(c0 + i, nc - 1)];
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        if (c0 + i >= nc) break;
        bad |= pb[i].bad;
        if (pb[i].a > best || bi == 0x7fffffff) {
          best = pb[i].a;
          bi = pb[i].idx;
        }
      }
    }
    am = bi;
  }
  const bool any_bad = __any(bad);
  const bool mismatch = lane < g && am != next_tok;
  const unsigned long long mm = __ballot(mismatch);
  const int a = mm ? __ffsll((long long)mm) - 1 : g;
  const int am_a = __shfl(am, a < 0 ? 0 : a, kWave);
  const int st = (rows < 1 || rows > width) ? LSV_ERR_INVALID_ARG : any_bad ? LSV_ERR_NONFINITE : LSV_OK;  // rows <= 64 = wave
  if (st != LSV_OK) {
    if (lane < width) out_tokens[(size_t)b * width + lane] = -1;
    if (lane == 0) {
      accept_len[b] = 0;
      if (status) status[b] = st;
    }
    return;
  }
  if (lane < width) {
    int t = -1;
    if (lane < a) t = tokens[r0 + lane + 1];
    else if (lane == a) t = am_a;
    out_tokens[(size_t)b * width + lane] = t;
  }
  if (lane == 0) {
    accept_len[b] = a;
    if (seq_len) seq_len[b] += a + 1;
    if (status) status[b] = LSV_OK;
  }
}

// ------------------------------------------------------------------ greedy, tree blocks
// One workgroup per sequence whose block is a tree (kTreeNodes nodes at most): every node's
// argmax from the row partials; a node is reachable when its token is its parent's argmax and
// its parent is reachable (the root always is); the accepted path ends at the deepest reachable
// node (the smallest index among equally deep ones).  Depth and reachability settle level by
// level: each round resolves the nodes whose parent was resolved before it.
__global__ void __launch_bounds__(256) accept_tree_kernel(const RowPartial* __restrict__ parts, int nc,
                                                          const int32_t* row_offsets, int max_rows,
                                                          const int32_t* parents, const int32_t* tokens, int width,
                                                          int32_t* accept_len, int32_t* out_tokens, int32_t* path,
                                                          int32_t* seq_len, int32_t* status) {
  __shared__ int s_par[kTreeNodes], s_tok[kTreeNodes], s_top[kTreeNodes], s_dep[kTreeNodes];
  __shared__ int s_reach[kTreeNodes];
  __shared__ int s_key[256];
  const int b = blockIdx.x, t = threadIdx.x;
  auto finish = [&](int st) {  // nothing accepted: -1 tokens and path, status st
    for (int j = t; j < width; j += 256) {
      out_tokens[(size_t)b * width + j] = -1;
      path[(size_t)b * width + j] = -1;
    }
    if (t == 0) {
      accept_len[b] = 0;
      if (status) status[b] = st;
    }
  };
  if (status && status[b] != LSV_OK) {  // a failed verify step: skipped, status kept
    finish(status[b]);
    return;
  }
  const int r0 = row_offsets[b], r1 = row_offsets[b + 1], n = r1 - r0;
  if (r0 < 0 || n < 1 || n > kTreeNodes || r1 > max_rows) {
    finish(LSV_ERR_INVALID_ARG);
    return;
  }
  int bad_tree = 0, bad_val = 0;
  for (int i = t; i < n; i += 256) {
    const int p = parents[r0 + i];
    s_par[i] = p;
    s_tok[i] = tokens[r0 + i];
    bad_tree |= i == 0 ? p != -1 : (p < 0 || p >= i);
    // argmax of row i: chunk partials in ascending order, strict '>' keeps the first maximum
    float best = -INFINITY;
    int bi = 0x7fffffff;
    const RowPartial* rp = parts + (size_t)(r0 + i) * nc;
    for (int c = 0; c < nc; ++c) {
      const RowPartial q = rp[c];
      bad_val |= q.bad;
      if (q.a > best || bi == 0x7fffffff) {
        best = q.a;
        bi = q.idx;
      }
    }
    s_top[i] = bi;
    s_dep[i] = i == 0 ? 0 : -1;
    s_reach[i] = i == 0;
  }
  const int any_tree = __syncthreads_or(bad_tree), any_val = __syncthreads_or(bad_val);
  if (any_tree || any_val) {
    finish(any_tree ? LSV_ERR_INVALID_ARG : LSV_ERR_NONFINITE);
    return;
  }
  // levels: a round reads the parents' state, then writes the nodes it resolves
  for (int round = 0; round < n; ++round) {
    int upd = 0;
    int nd[kTreeNodes / 256], nr[kTreeNodes / 256];
#pragma unroll
    for (int k = 0; k < kTreeNodes / 256; ++k) {
      const int i = t + 256 * k;
      nd[k] = -1;
      nr[k] = 0;
      if (i < n && i > 0 && s_dep[i] < 0) {
        const int p = s_par[i];
        if (s_dep[p] >= 0) {
          nd[k] = s_dep[p] + 1;
          nr[k] = s_reach[p] && s_tok[i] == s_top[p];
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kTreeNodes / 256; ++k)
      if (nd[k] >= 0) {
        s_dep[t + 256 * k] = nd[k];
        s_reach[t + 256 * k] = nr[k];
        upd = 1;
      }
    if (!__syncthreads_or(upd)) break;
  }
  // deepest reachable node, smallest index on ties: key = depth * 1024 + (1023 - index)
  int key = -1;
  for (int i = t; i < n; i += 256)
    if (s_reach[i]) key = max(key, s_dep[i] * 1024 + (1023 - i));
  s_key[t] = key;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) s_key[t] = max(s_key[t], s_key[t + o]);
    __syncthreads();
  }
  const int last = 1023 - (s_key[0] & 1023), a = s_key[0] >> 10;
  if (a + 1 > width) {
    finish(LSV_ERR_INVALID_ARG);
    return;
  }
  if (t == 0) {  // walk up from the last node: path[k] = the node at depth k
    int u = last, child = -1;
    for (int k = a; k >= 0; --k) {
      path[(size_t)b * width + k] = u;
      out_tokens[(size_t)b * width + k] = k == a ? s_top[last] : s_tok[child];
      child = u;
      u = s_par[u];
    }
    accept_len[b] = a;
    if (seq_len) seq_len[b] += a + 1;
    if (status) status[b] = LSV_OK;
  }
  for (int j = a + 1 + t; j < width; j += 256) {
    out_tokens[(size_t)b * width + j] = -1;
    path[(size_t)b * width + j] = -1;
  }
}

int launch_accept_tree(int batch, int vocab, const float* logits, const int32_t* row_offsets, const int32_t* parents,
                       const int32_t* tokens, int max_rows, int width, int32_t* accept_len, int32_t* out_tokens,
                       int32_t* path, int32_t* seq_len, int32_t* status, void* ws, hipStream_t stream) {
  const int nc = accept_chunks(vocab);
  AcceptWs w = carve(ws, batch, max_rows, vocab);
  hipLaunchKernelGGL(row_scan_kernel<false>, dim3(nc, max_rows), dim3(256), 0, stream, logits, row_offsets, batch,
                     vocab, 1.0f, w.rows);
  hipLaunchKernelGGL(accept_tree_kernel, dim3(batch), dim3(256), 0, stream, w.rows, nc, row_offsets, max_rows, parents,
                     tokens, width, accept_len, out_tokens, path, seq_len, status);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

// ------------------------------------------------------------------ sampling
__global__ void __launch_bounds__(64) accept_sample_decide_kernel(const RowPartial* __restrict__ parts, int nc,
                                                                  const float* __restrict__ logits, int vocab,
                                                                  const float* __restrict__ q, float temperature,
                                                                  const int32_t* row_offsets, int batch, int max_rows,
                                                                  int width, const int32_t* tokens, uint64_t seed,
                                                                  uint64_t round, const int32_t* status,
                                                                  SeqDecision* dec, int* counters) {
  const int b = blockIdx.x, lane = threadIdx.x;
  // a sequence that arrives with an error keeps it: the race kernel then emits nothing for it
  const int in_status = status ? status[b] : LSV_OK;
  if (in_status != LSV_OK) {
    if (lane == 0) {
      SeqDecision d = {};
      d.status = in_status;
      dec[b] = d;
      counters[b] = 0;
    }
    return;
  }
  // draft rows are indexed row_offsets[b] - b + v - 1, which needs every sequence to own 1..width rows
  bool shape_bad = false;
  for (int bb = lane; bb < batch; bb += kWave) {
    const int n = row_offsets[bb + 1] - row_offsets[bb];
    shape_bad |= n < 1 || n > width;
  }
  shape_bad = __any(shape_bad) || row_offsets[0] != 0 || row_offsets[batch] > max_rows;
  if (shape_bad) {
    if (lane == 0) {
      SeqDecision d = {};
      d.status = LSV_ERR_INVALID_ARG;
      dec[b] = d;
      counters[b] = 0;
    }
    return;
  }
  const int r0 = row_offsets[b], rows = row_offsets[b + 1] - r0, g = rows - 1;
  if (lane == 0) counters[b] = 0;  // the race kernel's arrival counter starts from zero
  float m = -INFINITY, z = 0.f;
  int bad = 0;
  if (lane < rows) {
    for (int c = 0; c < nc; ++c) m = fmaxf(m, parts[(size_t)(r0 + lane) * nc + c].a);
    for (int c = 0; c < nc; ++c) {  // fixed chunk order
      RowPartial p = parts[(size_t)(r0 + lane) * nc + c];
      bad |= p.bad;
      z += p.b * expf(p.a - m);
    }
  }
  // ratio test of draft v = lane + 1 against row lane
  bool reject = false;
  int qbad = 0;
  if (lane < g) {
    const int x = tokens[r0 + lane + 1];
    const float qx = q[(size_t)(r0 - b + lane) * vocab + x];
    qbad = !isfinite(qx);
    const float px = expf(logits[(size_t)(r0 + lane) * vocab + x] / temperature - m) / z;
    const U64x4 w = philox4x64_10(0, (uint64_t)(uint32_t)(lane + 1) | ((uint64_t)b << 32), round, 0, seed,
                                  kStreamAccept);
    const double u = unit52(w.w[0]);
    reject = !(u * (double)qx < (double)px);  // a non-finite q(x) always rejects
  }
  const bool rows_bad = __any(bad);
  const unsigned long long rj = __ballot(reject);
  const int a = rj ? __ffsll((long long)rj) - 1 : g;
  // the rule reads q(x_v) for drafts 1..a+1 only; earlier ones passed, so only draft a+1 can be bad
  const bool q_bad = a < g && __shfl(qbad, a, kWave);
  const float m_a = __shfl(m, a, kWave), z_a = __shfl(z, a, kWave);
  if (lane == 0) {
    SeqDecision d;
    d.status = (rows_bad || q_bad) ? LSV_ERR_NONFINITE : LSV_OK;
    d.a = a;
    d.row = r0 + a;
    d.residual = a < g;
    d.draft_row = r0 - b + a;
    d.m = m_a;
    d.z = z_a;
    d.pad = 0;
    dec[b] = d;
  }
}

__global__ void __launch_bounds__(256) accept_sample_race_kernel(
    const float* __restrict__ logits, int vocab, const float* __restrict__ q, float temperature,
    const int32_t* row_offsets, const int32_t* tokens, uint64_t seed, uint64_t round, const SeqDecision* dec,
    RacePartial* race, int* counters, int width, int32_t* accept_len, int32_t* out_tokens, int32_t* seq_len,
    int32_t* status) {
  const int c = blockIdx.x, b = blockIdx.y, nc = gridDim.x;
  const SeqDecision d = dec[b];
  const int x0 = c * kAcceptChunk, x1 = min(vocab, x0 + kAcceptChunk);
  double kr = INFINITY, kp = INFINITY;
  int ir = 0x7fffffff, ip = 0x7fffffff, bad = 0;
  if (d.status == LSV_OK) {
    const auto* row = GL(logits) + (size_t)d.row * vocab;
    const auto* qrow = d.residual ? GL(q) + (size_t)d.draft_row * vocab : nullptr;
    const uint64_t c1 = (uint64_t)(uint32_t)(d.a) | ((uint64_t)b << 32);
    // each thread owns groups of 4 consecutive tokens (one Philox call each)
    for (int x4 = (x0 >> 2) + threadIdx.x; x4 < ((x1 + 3) >> 2); x4 += blockDim.x) {
      const U64x4 w = philox4x64_10((uint64_t)x4, c1, round, 0, seed, kStreamSample);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int x = 4 * x4 + e;
        if (x < x0 || x >= x1) continue;
        const float p = expf(row[x] / temperature - d.m) / d.z;
        const double E = -log(unit52(w.w[e]));
        if (p > 0.f) {
          const double k = E / (double)p;
          if (k < kp) {
            kp = k;
            ip = x;
          }
        }
        if (qrow) {
          const float qx = qrow[x];
          if (!isfinite(qx)) bad = 1;
          const float wr = fmaxf(p - qx, 0.f);
          if (wr > 0.f) {
            const double k = E / (double)wr;
            if (k < kr) {
              kr = k;
              ir = x;
            }
          }
        }
      }
    }
  }
  // block argmin (ties -> smallest index)
  __shared__ double s_kr[256], s_kp[256];
  __shared__ int s_ir[256], s_ip[256], s_bad[256];
  __shared__ int s_last;
  const int t = threadIdx.x;
  s_kr[t] = kr;
  s_kp[t] = kp;
  s_ir[t] = ir;
  s_ip[t] = ip;
  s_bad[t] = bad;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) {
      if (s_kr[t + o] < s_kr[t] || (s_kr[t + o] == s_kr[t] && s_ir[t + o] < s_ir[t])) {
        s_kr[t] = s_kr[t + o];
        s_ir[t] = s_ir[t + o];
      }
      if (s_kp[t + o] < s_kp[t] || (s_kp[t + o] == s_kp[t] && s_ip[t + o] < s_ip[t])) {
        s_kp[t] = s_kp[t + o];
        s_ip[t] = s_ip[t + o];
      }
      s_bad[t] |= s_bad[t + o];
    }
    __syncthreads();
  }
  if (t == 0) {
    RacePartial p;
    p.key_res = s_kr[0];
    p.key_p = s_kp[0];
    p.idx_res = s_ir[0];
    p.idx_p = s_ip[0];
    p.bad = s_bad[0];
    p.pad = 0;
    race[(size_t)b * nc + c] = p;
  }
  if (!arrive_last(&counters[b], nc, &s_last)) return;
  // last workgroup of sequence b: merge in chunk order and commit
  if (t == 0) {
    double kr2 = INFINITY, kp2 = INFINITY;
    int ir2 = -1, ip2 = -1, bad2 = 0;
    for (int cc = 0; cc < nc; ++cc) {
      RacePartial p = race[(size_t)b * nc + cc];
      bad2 |= p.bad;
      if (p.key_res < kr2) {
        kr2 = p.key_res;
        ir2 = p.idx_res;
      }
      if (p.key_p < kp2) {
        kp2 = p.key_p;
        ip2 = p.idx_p;
      }
    }
    int st = d.status;
    if (st == LSV_OK && bad2) st = LSV_ERR_NONFINITE;
    const int y = (d.residual && ir2 >= 0) ? ir2 : ip2;
    s_ir[0] = st;
    s_ip[0] = y;
    reset_counter(&counters[b]);
  }
  __syncthreads();
  const int st = s_ir[0], y = s_ip[0];
  const int r0 = row_offsets[b];
  for (int j = t; j < width; j += blockDim.x) {
    int tok = -1;
    if (st == LSV_OK) {
      if (j < d.a) tok = tokens[r0 + 1 + j];
      else if (j == d.a) tok = y;
    }
    out_tokens[(size_t)b * width + j] = tok;
  }
  if (t == 0) {
    accept_len[b] = st == LSV_OK ? d.a : 0;
    if (status) status[b] = st;
    if (seq_len && st == LSV_OK) seq_len[b] += d.a + 1;
  }
}

// ------------------------------------------------------------------ library-owned scratch
// lsv_accept_noalloc: the same kernels on a device array the library owns (one copy per GPU,
// held until the process ends).  Host code must use the address hipGetSymbolAddress returns
// on the current device, never the array's name.
static __device__ __align__(256) unsigned char scratch[kAcceptStaticBytes];
constexpr int kMaxDevices = 64;
static void* g_scratch[kMaxDevices];
static std::mutex g_scratch_mu;

int accept_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return LSV_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return LSV_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return LSV_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return LSV_OK;
}

int launch_accept(int mode, int batch, int vocab, const float* logits, const int32_t* row_offsets, int max_rows,
                  int max_rows_per_seq, const int32_t* tokens, const float* draft_probs, float temperature,
                  uint64_t seed, uint64_t round, int32_t* accept_len, int32_t* out_tokens, int32_t* seq_len,
                  int32_t* status, void* ws, hipStream_t stream) {
  const int nc = accept_chunks(vocab);
  AcceptWs w = carve(ws, batch, max_rows, vocab);
  dim3 scan_grid(nc, max_rows);
  if (mode == LSV_ACC_GREEDY) {
    hipLaunchKernelGGL(row_scan_kernel<false>, scan_grid, dim3(256), 0, stream, logits, row_offsets, batch, vocab,
                       1.0f, w.rows);
    hipLaunchKernelGGL(accept_greedy_kernel, dim3(batch), dim3(64), 0, stream, w.rows, nc, row_offsets, max_rows,
                       tokens, max_rows_per_seq, accept_len, out_tokens, seq_len, status);
  } else {
    hipLaunchKernelGGL(row_scan_kernel<true>, scan_grid, dim3(256), 0, stream, logits, row_offsets, batch, vocab,
                       temperature, w.rows);
    hipLaunchKernelGGL(accept_sample_decide_kernel, dim3(batch), dim3(64), 0, stream, w.rows, nc, logits, vocab,
                       draft_probs, temperature, row_offsets, batch, max_rows, max_rows_per_seq, tokens, seed, round,
                       status, w.seq, w.counters);
    hipLaunchKernelGGL(accept_sample_race_kernel, dim3(nc, batch), dim3(256), 0, stream, logits, vocab, draft_probs,
                       temperature, row_offsets, tokens, seed, round, w.seq, w.race, w.counters, max_rows_per_seq,
                       accept_len, out_tokens, seq_len, status);
  }
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

}  // namespace lsv
