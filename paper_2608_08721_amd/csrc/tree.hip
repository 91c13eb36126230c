// Commit of an accepted tree path (Sec. 4.3: tree drafts verified in one pass).  The verify
// step stored node r of a sequence's tree at cache slot C + r with its rotary position
// C + depth(r); after acceptance the path's node at depth k belongs at position C + k.  Its
// K row and V column are copied there (k = 1..a; the root already sits at C).
//
// Order: path[k] >= k (a node at depth k has k ancestors of smaller index), so a copy's
// source C + path[k] is never the destination C + j of an earlier step j < k, while its
// destination C + k may be the source of an earlier step (path[j] = k for some j < k).  One
// thread owns one head dimension of one (layer, sequence, kv head) for every k, in
// increasing k, so each of its reads precedes every write that could clobber it.
#include "lsv_device.h"
#include "lsv_attn.h"

namespace lsv {

template <typename T>
__global__ void __launch_bounds__(128) commit_tree_kernel(T* kv, KvLayout kvl, int batch, int nkv, int hd,
                                                          const int32_t* __restrict__ seq_len,
                                                          const int32_t* __restrict__ accept_len,
                                                          const int32_t* __restrict__ path, int width,
                                                          const int32_t* __restrict__ status) {
  const int h = blockIdx.x, b = blockIdx.y, l = blockIdx.z, i = threadIdx.x;
  if (i >= hd) return;
  if (status && status[b] != LSV_OK) return;
  const int a = accept_len[b];
  const int C = seq_len[b] - a - 1;  // the committed length minus the root and the a accepted drafts
  if (a < 1 || a >= width || C < 0) return;
  const size_t blk = kv_layer_block(kvl, batch, nkv, hd);
  T* K = kv + 2 * (size_t)l * blk;
  T* V = K + blk;
  for (int k = 1; k <= a; ++k) {
    const int src = C + path[(size_t)b * width + k], dst = C + k;
    if (src <= dst) continue;  // src == dst needs no copy; src < dst is not a path the acceptance wrote
    size_t ks, vs_, kd, vd;
    int ss, sd;
    if (!kvl.pages && src >= kvl.capacity) continue;
    if (!kv_locate(kvl, nkv, hd, b, h, src, ks, vs_, ss) || !kv_locate(kvl, nkv, hd, b, h, dst, kd, vd, sd)) continue;
    K[kd + i] = K[ks + i];
    V[vd + (size_t)i * sd] = V[vs_ + (size_t)i * ss];
  }
}

int launch_commit_tree(const Shape& s, void* kv, const KvLayout& kvl, int batch, const int32_t* seq_len,
                       const int32_t* accept_len, const int32_t* path, int width, const int32_t* status,
                       hipStream_t stream) {
  const dim3 grid((unsigned)s.nkv, (unsigned)batch, (unsigned)s.L);
  if (s.dtype == LSV_DTYPE_BF16)
    hipLaunchKernelGGL(commit_tree_kernel<bf16_t>, grid, dim3(128), 0, stream, (bf16_t*)kv, kvl, batch, s.nkv, s.hd,
                       seq_len, accept_len, path, width, status);
  else
    hipLaunchKernelGGL(commit_tree_kernel<float>, grid, dim3(128), 0, stream, (float*)kv, kvl, batch, s.nkv, s.hd,
                       seq_len, accept_len, path, width, status);
  return hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP;
}

}  // namespace lsv
