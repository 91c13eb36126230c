// Token plumbing between decoding rounds (Sec. 3.1: each round verifies the last emitted
// token followed by the drafted tokens, and its output token is the next round's first row),
// so that select -> verify -> accept -> next round runs without a host round trip.
#include "lsv_device.h"
#include "lsv_internal.h"

namespace lsv {

// Verify block rows of sequence b: row r0_b is the root, rows r0_b + k (k = 1..gamma_b) are
// drafts[b][k-1]; gamma_b = rows_b - 1 comes from the row offsets.  One workgroup per
// sequence; rows past max_rows are never written (the host bound).
__global__ void __launch_bounds__(64) pack_block_kernel(int G, const int32_t* __restrict__ row_offsets, int max_rows,
                                                        const int32_t* __restrict__ roots,
                                                        const int32_t* __restrict__ drafts,
                                                        int32_t* __restrict__ tokens, int32_t* __restrict__ status) {
  const int b = blockIdx.x;
  const int r0 = row_offsets[b], r1 = row_offsets[b + 1];
  const bool ok = r0 >= 0 && r1 > r0 && r1 <= max_rows && r1 - r0 - 1 <= G;
  if (status && threadIdx.x == 0) status[b] = ok ? LSV_OK : LSV_ERR_INVALID_ARG;
  if (!ok) return;
  for (int r = r0 + (int)threadIdx.x; r < r1; r += 64)
    tokens[r] = r == r0 ? roots[b] : drafts[(size_t)b * G + (r - r0 - 1)];
}

// The next round's root of each sequence: the token emitted after its accepted drafts,
// out_tokens[b][accept_len[b]].  A sequence whose round failed keeps its root.
__global__ void __launch_bounds__(64) next_roots_kernel(int batch, const int32_t* __restrict__ accept_len,
                                                        const int32_t* __restrict__ out_tokens, int width,
                                                        const int32_t* __restrict__ acc_status,
                                                        int32_t* __restrict__ roots) {
  const int b = blockIdx.x * 64 + threadIdx.x;
  if (b >= batch) return;
  const int a = accept_len[b];
  const bool ok = (acc_status == nullptr || acc_status[b] == LSV_OK) && a >= 0 && a < width;
  if (ok) roots[b] = out_tokens[(size_t)b * width + a];
}

int launch_pack_block(int batch, int G, const int32_t* row_offsets, int max_rows, const int32_t* roots,
                      const int32_t* drafts, int32_t* tokens, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(pack_block_kernel, dim3(batch), dim3(64), 0, stream, G, row_offsets, max_rows, roots, drafts,
                     tokens, status);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

int launch_next_roots(int batch, const int32_t* accept_len, const int32_t* out_tokens, int width,
                      const int32_t* status, int32_t* roots, hipStream_t stream) {
  hipLaunchKernelGGL(next_roots_kernel, dim3((batch + 63) / 64), dim3(64), 0, stream, batch, accept_len, out_tokens,
                     width, status, roots);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

}  // namespace lsv
