// C-ABI of liblsv (declared in include/lsv.h): host-side validation, then launches.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "lsv_device.h"
#include "lsv_gemm.h"
#include "lsv_internal.h"

namespace {

thread_local char g_err[512] = "";

struct TimingHook {
  int kernel = 0, n = 0;
  unsigned flags = 0;
  hipEvent_t ev[2 * LSV_MAX_TIMING_SLOTS];
} g_timing;

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}
int ok() {
  g_err[0] = 0;
  return LSV_OK;
}
int hip_rc(int rc, const char* what) {
  if (rc == LSV_ERR_HIP && strncmp(g_err, "timing event", 12) == 0) return rc;
  if (rc == LSV_ERR_HIP) return fail(LSV_ERR_HIP, "%s: %s", what, hipGetErrorString(hipGetLastError()));
  if (rc == LSV_ERR_UNSUPPORTED) return fail(rc, "%s: unsupported shape", what);
  if (rc != LSV_OK) return fail(rc, "%s failed", what);
  return ok();
}

int check_config(const lsv_model_config* c) {
  if (!c) return fail(LSV_ERR_INVALID_ARG, "cfg is NULL");
  if (c->n_layers < 1 || c->d_model < 64 || c->d_model % 64 || c->n_q_heads < 1 || c->n_kv_heads < 1 ||
      c->n_q_heads % c->n_kv_heads || c->d_ff < 4 || c->d_ff % 4 || c->vocab < 1)
    return fail(LSV_ERR_INVALID_ARG, "bad model dimensions (d_model %% 64, n_q %% n_kv, d_ff %% 4 required)");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(LSV_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c->d_model > 8192) return fail(LSV_ERR_UNSUPPORTED, "d_model must be <= 8192");
  if (c->dtype != LSV_DTYPE_F32 && c->dtype != LSV_DTYPE_BF16) return fail(LSV_ERR_INVALID_ARG, "bad dtype");
  if (!(c->rms_eps > 0.f) || !(c->rope_base > 0.0) || !isfinite(c->rope_base) || c->reserved0 != 0.f)
    return fail(LSV_ERR_INVALID_ARG, "bad rms_eps / rope_base / reserved0");
  // the weight streams address a packed matrix with 32-bit byte offsets
  const lsv::ModelLayout ml = lsv::model_layout(lsv::shape_of(c));
  for (const lsv::PackedMat* p : {&ml.lm_head, &ml.qkv, &ml.o, &ml.gateup, &ml.down})
    if ((size_t)p->Nt * p->Kt * 1024 >= ((size_t)1 << 32))
      return fail(LSV_ERR_UNSUPPORTED, "a packed projection of %zu bytes reaches 4 GiB", (size_t)p->Nt * p->Kt * 1024);
  return LSV_OK;
}

}  // namespace

extern "C" {

const char* lsv_status_string(int s) {
  switch (s) {
    case LSV_OK: return "ok";
    case LSV_ERR_INVALID_ARG: return "invalid argument";
    case LSV_ERR_UNSUPPORTED: return "unsupported configuration";
    case LSV_ERR_HIP: return "HIP runtime error";
    case LSV_ERR_CAPACITY: return "KV-cache capacity exceeded";
    case LSV_ERR_NONFINITE: return "non-finite value";
  }
  return "unknown status";
}

const char* lsv_last_error(void) { return g_err; }
int lsv_abi_version(void) { return 3; }

size_t lsv_packed_model_bytes(const lsv_model_config* cfg) {
  if (check_config(cfg) != LSV_OK) return 0;
  return lsv::model_layout(lsv::shape_of(cfg)).total;
}

int lsv_pack_globals(const lsv_model_config* cfg, const void* d_embed, const void* d_final_norm, const void* d_lm_head,
                     void* d_packed, void* stream) {
  int rc = check_config(cfg);
  if (rc) return rc;
  if (!d_embed || !d_final_norm || !d_lm_head || !d_packed) return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  const lsv::Shape s = lsv::shape_of(cfg);
  const lsv::ModelLayout ml = lsv::model_layout(s);
  hipStream_t st = (hipStream_t)stream;
  char* P = (char*)d_packed;
  if (hipMemcpyAsync(P + ml.embed, d_embed, (size_t)s.V * s.d * s.es, hipMemcpyDeviceToDevice, st) != hipSuccess)
    return fail(LSV_ERR_HIP, "copy: %s", hipGetErrorString(hipGetLastError()));
  if ((rc = lsv::launch_pack(s, lsv::PACK_PLAIN, ml.lm_head, d_lm_head, nullptr, nullptr, P, st)) ||
      (rc = lsv::launch_gain(s, d_final_norm, P + ml.final_norm, st)))
    return hip_rc(rc, "pack globals");
  return ok();
}

int lsv_pack_layer(const lsv_model_config* cfg, int32_t layer, const void* d_wq, const void* d_wk, const void* d_wv,
                   const void* d_wo, const void* d_wg, const void* d_wu, const void* d_wd, const void* d_attn_norm,
                   const void* d_ffn_norm, void* d_packed, void* stream) {
  int rc = check_config(cfg);
  if (rc) return rc;
  if (layer < 0 || layer >= cfg->n_layers) return fail(LSV_ERR_INVALID_ARG, "layer %d out of range", layer);
  if (!d_wq || !d_wk || !d_wv || !d_wo || !d_wg || !d_wu || !d_wd || !d_attn_norm || !d_ffn_norm || !d_packed)
    return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  const lsv::Shape s = lsv::shape_of(cfg);
  const lsv::ModelLayout ml = lsv::model_layout(s);
  hipStream_t st = (hipStream_t)stream;
  char* LB = (char*)d_packed + ml.layer_base + (size_t)layer * ml.layer_stride;
  if ((rc = lsv::launch_pack(s, lsv::PACK_QKV, ml.qkv, d_wq, d_wk, d_wv, LB, st)) ||
      (rc = lsv::launch_pack(s, lsv::PACK_PLAIN, ml.o, d_wo, nullptr, nullptr, LB, st)) ||
      (rc = lsv::launch_pack(s, lsv::PACK_GATEUP, ml.gateup, d_wg, d_wu, nullptr, LB, st)) ||
      (rc = lsv::launch_pack(s, lsv::PACK_PLAIN, ml.down, d_wd, nullptr, nullptr, LB, st)) ||
      (rc = lsv::launch_gain(s, d_attn_norm, LB + ml.attn_norm, st)) ||
      (rc = lsv::launch_gain(s, d_ffn_norm, LB + ml.ffn_norm, st)))
    return hip_rc(rc, "pack layer");
  return ok();
}

size_t lsv_kv_cache_bytes(const lsv_model_config* cfg, int32_t batch, int32_t capacity) {
  if (check_config(cfg) != LSV_OK || batch < 1 || capacity < 1 || capacity % LSV_KV_ALIGN) return 0;
  const lsv::Shape s = lsv::shape_of(cfg);
  return (size_t)s.L * 2 * batch * s.nkv * (size_t)capacity * s.hd * s.es;
}

size_t lsv_verify_workspace_bytes(const lsv_model_config* cfg, int32_t batch, int32_t max_rows, int32_t max_ctx) {
  if (check_config(cfg) != LSV_OK || batch < 1 || max_rows < 1 || max_rows > LSV_MAX_ROWS || max_ctx < 1) return 0;
  return lsv::verify_workspace_bytes(lsv::shape_of(cfg), batch, max_rows, max_ctx);
}

__global__ void lsv_clear_kernel(uint4* p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0, 0, 0, 0);
}

int lsv_workspace_clear(void* d_workspace, size_t bytes, void* stream) {
  if (!d_workspace || bytes % 16 || ((uintptr_t)d_workspace & 15))
    return fail(LSV_ERR_INVALID_ARG, "workspace must be non-NULL, 16-byte aligned and a multiple of 16 bytes");
  const size_t n16 = bytes / 16;
  unsigned blocks = (unsigned)((n16 + 255) / 256);
  blocks = blocks > 4096 ? 4096 : (blocks == 0 ? 1 : blocks);
  hipLaunchKernelGGL(lsv_clear_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, (uint4*)d_workspace, n16);
  return hip_rc(hipGetLastError() == hipSuccess ? LSV_OK : LSV_ERR_HIP, "workspace clear");
}

namespace {
// Host checks of a cache description: a slab cache (pages NULL: capacity positions per sequence) or a
// page pool (n_pages pages of LSV_KV_PAGE positions, a page table of max_pages entries per sequence).
int check_kv(const lsv::Shape& s, const lsv::KvLayout& kvl) {
  if (!kvl.pages) {
    if (kvl.capacity < 1 || kvl.capacity % LSV_KV_ALIGN)
      return fail(LSV_ERR_INVALID_ARG, "capacity %d is not a positive multiple of %d", kvl.capacity, (int)LSV_KV_ALIGN);
    // offsets inside a sequence's blocks are 32-bit in the kernels
    if ((size_t)s.nkv * kvl.capacity * s.hd * s.es >= ((size_t)1 << 31))
      return fail(LSV_ERR_INVALID_ARG, "capacity %d: a sequence's KV block of %d x %d x %d elements reaches 2 GiB",
                  kvl.capacity, s.nkv, kvl.capacity, s.hd);
    return LSV_OK;
  }
  if (kvl.n_pages < 1 || kvl.max_pages < 1 || kvl.max_pages > (1 << 20))
    return fail(LSV_ERR_INVALID_ARG, "need n_pages >= 1 and 1 <= max_pages <= 2^20");
  // the attention reads a layer's pool through 32-bit offsets, one page past the end included
  if (((size_t)kvl.n_pages + 1) * s.nkv * LSV_KV_PAGE * s.hd * s.es >= ((size_t)1 << 31))
    return fail(LSV_ERR_INVALID_ARG, "a layer's K pool of %d pages reaches 2 GiB", kvl.n_pages);
  return LSV_OK;
}

int verify(const lsv_model_config* cfg, const void* d_packed, void* d_kv, const lsv::KvLayout& kvl, int32_t batch,
           const int32_t* d_seq_len, const int32_t* d_tokens, const int32_t* d_row_offsets, const int32_t* d_parents,
           int32_t max_rows, int32_t max_ctx, float* d_logits, int32_t* d_status, void* d_workspace,
           size_t workspace_bytes, void* stream) {
  int rc = check_config(cfg);
  if (rc) return rc;
  if (!d_packed || !d_kv || !d_seq_len || !d_tokens || !d_row_offsets || !d_logits || !d_workspace)
    return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  if (batch < 1 || batch > LSV_MAX_BATCH) return fail(LSV_ERR_INVALID_ARG, "batch %d not in [1, %d]", batch, LSV_MAX_BATCH);
  if (max_rows < 1 || max_rows > LSV_MAX_ROWS)
    return fail(LSV_ERR_INVALID_ARG, "max_rows %d not in [1, %d]", max_rows, LSV_MAX_ROWS);
  const int capacity = kvl.pages ? kvl.max_pages * LSV_KV_PAGE : kvl.capacity;  // positions per sequence
  if (capacity < 1 || max_ctx < 1 || max_ctx > capacity)
    return fail(LSV_ERR_INVALID_ARG, "need 1 <= max_ctx (%d) <= capacity (%d)", max_ctx, capacity);
  const lsv::Shape s = lsv::shape_of(cfg);
  if ((rc = check_kv(s, kvl)) != LSV_OK) return rc;
  if (s.dtype == LSV_DTYPE_F32 && max_ctx > 16384)
    return fail(LSV_ERR_UNSUPPORTED, "fp32 models support max_ctx <= 16384");
  const size_t need = lsv::verify_workspace_bytes(s, batch, max_rows, max_ctx);
  if (workspace_bytes < need)
    return fail(LSV_ERR_INVALID_ARG, "workspace %zu bytes < %zu required", workspace_bytes, need);
  const lsv::ModelLayout ml = lsv::model_layout(s);
  rc = lsv::launch_verify(s, ml, d_packed, d_kv, kvl, batch, d_seq_len, d_tokens, d_row_offsets, d_parents,
                          max_rows, max_ctx, d_logits, d_status, d_workspace, workspace_bytes, (hipStream_t)stream);
  return hip_rc(rc, "verify");
}

lsv::KvLayout slab_kv(int capacity) { return lsv::KvLayout{capacity, nullptr, 0, 0}; }
lsv::KvLayout paged_kv(const int32_t* pages, int max_pages, int n_pages) {
  return lsv::KvLayout{max_pages * LSV_KV_PAGE, pages, max_pages, n_pages};
}
}  // namespace

int lsv_verify_block(const lsv_model_config* cfg, const void* d_packed, void* d_kv, int32_t capacity, int32_t batch,
                     const int32_t* d_seq_len, const int32_t* d_tokens, const int32_t* d_row_offsets, int32_t max_rows,
                     int32_t max_ctx, float* d_logits, int32_t* d_status, void* d_workspace, size_t workspace_bytes,
                     void* stream) {
  return verify(cfg, d_packed, d_kv, slab_kv(capacity), batch, d_seq_len, d_tokens, d_row_offsets, nullptr, max_rows,
                max_ctx, d_logits, d_status, d_workspace, workspace_bytes, stream);
}

size_t lsv_kv_pool_bytes(const lsv_model_config* cfg, int32_t n_pages) {
  if (check_config(cfg) != LSV_OK || n_pages < 1) return 0;
  const lsv::Shape s = lsv::shape_of(cfg);
  return (size_t)s.L * 2 * (size_t)n_pages * s.nkv * LSV_KV_PAGE * s.hd * s.es;
}

int lsv_verify_paged(const lsv_model_config* cfg, const void* d_packed, void* d_kv_pool, int32_t n_pages,
                     const int32_t* d_page_table, int32_t max_pages, int32_t batch, const int32_t* d_seq_len,
                     const int32_t* d_tokens, const int32_t* d_row_offsets, const int32_t* d_parents, int32_t max_rows,
                     int32_t max_ctx, float* d_logits, int32_t* d_status, void* d_workspace, size_t workspace_bytes,
                     void* stream) {
  if (!d_page_table) return fail(LSV_ERR_INVALID_ARG, "NULL page table");
  return verify(cfg, d_packed, d_kv_pool, paged_kv(d_page_table, max_pages, n_pages), batch, d_seq_len, d_tokens,
                d_row_offsets, d_parents, max_rows, max_ctx, d_logits, d_status, d_workspace, workspace_bytes, stream);
}

int lsv_verify_tree(const lsv_model_config* cfg, const void* d_packed, void* d_kv, int32_t capacity, int32_t batch,
                    const int32_t* d_seq_len, const int32_t* d_tokens, const int32_t* d_row_offsets,
                    const int32_t* d_parents, int32_t max_rows, int32_t max_ctx, float* d_logits, int32_t* d_status,
                    void* d_workspace, size_t workspace_bytes, void* stream) {
  if (!d_parents) return fail(LSV_ERR_INVALID_ARG, "NULL parents");
  return verify(cfg, d_packed, d_kv, slab_kv(capacity), batch, d_seq_len, d_tokens, d_row_offsets, d_parents, max_rows,
                max_ctx, d_logits, d_status, d_workspace, workspace_bytes, stream);
}

int lsv_accept_tree(int32_t batch, int32_t vocab, const float* d_logits, const int32_t* d_row_offsets,
                    const int32_t* d_parents, const int32_t* d_tokens, int32_t max_rows, int32_t width,
                    int32_t* d_accept_len, int32_t* d_out_tokens, int32_t* d_path, int32_t* d_seq_len,
                    int32_t* d_status, void* d_workspace, size_t workspace_bytes, void* stream) {
  if (batch < 1 || batch > LSV_MAX_BATCH || vocab < 1) return fail(LSV_ERR_INVALID_ARG, "bad batch or vocab");
  if (max_rows < 1 || max_rows > LSV_MAX_ROWS || width < 1 || width > LSV_MAX_SEQ_ROWS)
    return fail(LSV_ERR_INVALID_ARG, "bad max_rows %d (<= %d) / width %d (<= %d)", max_rows, (int)LSV_MAX_ROWS, width,
                (int)LSV_MAX_SEQ_ROWS);
  if (!d_logits || !d_row_offsets || !d_parents || !d_tokens || !d_accept_len || !d_out_tokens || !d_path ||
      !d_workspace)
    return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  if (workspace_bytes < lsv::accept_workspace_bytes(batch, max_rows, vocab))
    return fail(LSV_ERR_INVALID_ARG, "accept workspace too small");
  return hip_rc(lsv::launch_accept_tree(batch, vocab, d_logits, d_row_offsets, d_parents, d_tokens, max_rows, width,
                                        d_accept_len, d_out_tokens, d_path, d_seq_len, d_status, d_workspace,
                                        (hipStream_t)stream),
                "accept_tree");
}

namespace {
int commit_tree(const lsv_model_config* cfg, void* d_kv, const lsv::KvLayout& kvl, int32_t batch,
                const int32_t* d_seq_len, const int32_t* d_accept_len, const int32_t* d_path, int32_t width,
                const int32_t* d_status, void* stream) {
  int rc = check_config(cfg);
  if (rc) return rc;
  if (!d_kv || !d_seq_len || !d_accept_len || !d_path) return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  if (batch < 1 || batch > LSV_MAX_BATCH) return fail(LSV_ERR_INVALID_ARG, "batch %d not in [1, %d]", batch, LSV_MAX_BATCH);
  if (width < 1 || width > LSV_MAX_SEQ_ROWS)
    return fail(LSV_ERR_INVALID_ARG, "width %d not in [1, %d]", width, (int)LSV_MAX_SEQ_ROWS);
  const lsv::Shape s = lsv::shape_of(cfg);
  if ((rc = check_kv(s, kvl)) != LSV_OK) return rc;
  return hip_rc(lsv::launch_commit_tree(s, d_kv, kvl, batch, d_seq_len, d_accept_len, d_path, width, d_status,
                                        (hipStream_t)stream),
                "commit_tree");
}
}  // namespace

int lsv_commit_tree(const lsv_model_config* cfg, void* d_kv, int32_t capacity, int32_t batch, const int32_t* d_seq_len,
                    const int32_t* d_accept_len, const int32_t* d_path, int32_t width, const int32_t* d_status,
                    void* stream) {
  return commit_tree(cfg, d_kv, slab_kv(capacity), batch, d_seq_len, d_accept_len, d_path, width, d_status, stream);
}

int lsv_commit_tree_paged(const lsv_model_config* cfg, void* d_kv_pool, int32_t n_pages, const int32_t* d_page_table,
                          int32_t max_pages, int32_t batch, const int32_t* d_seq_len, const int32_t* d_accept_len,
                          const int32_t* d_path, int32_t width, const int32_t* d_status, void* stream) {
  if (!d_page_table) return fail(LSV_ERR_INVALID_ARG, "NULL page table");
  return commit_tree(cfg, d_kv_pool, paged_kv(d_page_table, max_pages, n_pages), batch, d_seq_len, d_accept_len, d_path,
                     width, d_status, stream);
}

size_t lsv_accept_workspace_bytes(int32_t batch, int32_t max_rows, int32_t vocab) {
  if (batch < 1 || max_rows < 1 || vocab < 1) return 0;
  return lsv::accept_workspace_bytes(batch, max_rows, vocab);
}

int lsv_accept(int32_t mode, int32_t batch, int32_t vocab, const float* d_logits, const int32_t* d_row_offsets,
               int32_t max_rows, int32_t max_rows_per_seq, const int32_t* d_tokens, const float* d_draft_probs,
               float temperature, uint64_t seed, uint64_t round, int32_t* d_accept_len, int32_t* d_out_tokens,
               int32_t* d_seq_len, int32_t* d_status, void* d_workspace, size_t workspace_bytes, void* stream) {
  if (mode != LSV_ACC_GREEDY && mode != LSV_ACC_SAMPLE) return fail(LSV_ERR_INVALID_ARG, "bad accept mode %d", mode);
  if (batch < 1 || batch > LSV_MAX_BATCH || vocab < 1) return fail(LSV_ERR_INVALID_ARG, "bad batch or vocab");
  if (max_rows < 1 || max_rows > LSV_MAX_ROWS || max_rows_per_seq < 1 || max_rows_per_seq > LSV_MAX_SEQ_ROWS)
    return fail(LSV_ERR_INVALID_ARG, "bad max_rows %d (<= %d) / max_rows_per_seq %d (<= %d)", max_rows,
                (int)LSV_MAX_ROWS, max_rows_per_seq, (int)LSV_MAX_SEQ_ROWS);
  if (!d_logits || !d_row_offsets || !d_tokens || !d_accept_len || !d_out_tokens || !d_workspace)
    return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  if (mode == LSV_ACC_SAMPLE && (!d_draft_probs || !(temperature > 0.f) || !isfinite(temperature)))
    return fail(LSV_ERR_INVALID_ARG, "sampling needs draft probabilities and a finite temperature > 0");
  if (workspace_bytes < lsv::accept_workspace_bytes(batch, max_rows, vocab))
    return fail(LSV_ERR_INVALID_ARG, "accept workspace too small");
  int rc = lsv::launch_accept(mode, batch, vocab, d_logits, d_row_offsets, max_rows, max_rows_per_seq, d_tokens,
                              d_draft_probs, temperature, seed, round, d_accept_len, d_out_tokens, d_seq_len, d_status,
                              d_workspace, (hipStream_t)stream);
  return hip_rc(rc, "accept");
}

int lsv_accept_noalloc(int32_t mode, int32_t batch, int32_t vocab, const float* d_logits,
                       const int32_t* d_row_offsets, int32_t max_rows, int32_t max_rows_per_seq,
                       const int32_t* d_tokens, const float* d_draft_probs, float temperature, uint64_t seed,
                       uint64_t round, int32_t* d_accept_len, int32_t* d_out_tokens, int32_t* d_seq_len,
                       int32_t* d_status, void* stream) {
  if (mode != LSV_ACC_GREEDY && mode != LSV_ACC_SAMPLE) return fail(LSV_ERR_INVALID_ARG, "bad accept mode %d", mode);
  if (batch < 1 || batch > LSV_MAX_BATCH || vocab < 1) return fail(LSV_ERR_INVALID_ARG, "bad batch or vocab");
  if (max_rows < 1 || max_rows > LSV_MAX_ROWS || max_rows_per_seq < 1 || max_rows_per_seq > LSV_MAX_SEQ_ROWS)
    return fail(LSV_ERR_INVALID_ARG, "bad max_rows %d (<= %d) / max_rows_per_seq %d (<= %d)", max_rows,
                (int)LSV_MAX_ROWS, max_rows_per_seq, (int)LSV_MAX_SEQ_ROWS);
  if (!d_logits || !d_row_offsets || !d_tokens || !d_accept_len || !d_out_tokens)
    return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  if (mode == LSV_ACC_SAMPLE && (!d_draft_probs || !(temperature > 0.f) || !isfinite(temperature)))
    return fail(LSV_ERR_INVALID_ARG, "sampling needs draft probabilities and a finite temperature > 0");
  const size_t need = lsv::accept_workspace_bytes(batch, max_rows, vocab);
  if (need > lsv::kAcceptStaticBytes)
    return fail(LSV_ERR_UNSUPPORTED, "scratch of %zu bytes needed, the library's holds %zu (LSV_ACCEPT_NOALLOC_BYTES)",
                need, lsv::kAcceptStaticBytes);
  void* ws = nullptr;
  int rc = lsv::accept_scratch(&ws);
  if (rc != LSV_OK) return hip_rc(rc, "accept_noalloc scratch");
  rc = lsv::launch_accept(mode, batch, vocab, d_logits, d_row_offsets, max_rows, max_rows_per_seq, d_tokens,
                          d_draft_probs, temperature, seed, round, d_accept_len, d_out_tokens, d_seq_len, d_status, ws,
                          (hipStream_t)stream);
  return hip_rc(rc, "accept_noalloc");
}

int lsv_select_length(int32_t mode, int32_t batch, int32_t G, const float* d_conf, const double* d_cost, int32_t d_init,
                      int32_t d_max, double alpha, int32_t block_n, uint32_t flags, int32_t* d_gamma, int32_t* d_aux,
                      int32_t* d_row_offsets, int32_t* d_status, void* stream) {
  if (mode != LSV_SEL_MARGINAL && mode != LSV_SEL_EXHAUSTIVE && mode != LSV_SEL_ALG1)
    return fail(LSV_ERR_INVALID_ARG, "bad selector mode %d", mode);
  if (batch < 1 || G < 1 || G > LSV_MAX_G) return fail(LSV_ERR_INVALID_ARG, "need batch >= 1 and 1 <= G <= %d", LSV_MAX_G);
  if (d_max < 1 || d_max > G) return fail(LSV_ERR_INVALID_ARG, "need 1 <= d_max (%d) <= G (%d)", d_max, G);
  if (!d_conf || !d_gamma) return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  if (flags & ~(uint32_t)(LSV_SEL_BONUS | LSV_SEL_DRAFTED)) return fail(LSV_ERR_INVALID_ARG, "unknown flags");
  if ((flags & LSV_SEL_DRAFTED) && (mode != LSV_SEL_ALG1 || !d_aux))
    return fail(LSV_ERR_INVALID_ARG, "LSV_SEL_DRAFTED needs LSV_SEL_ALG1 and d_aux (blocks drafted)");
  if (d_row_offsets && batch > LSV_MAX_BATCH)
    return fail(LSV_ERR_INVALID_ARG, "row offsets need batch <= %d", LSV_MAX_BATCH);
  if (mode == LSV_SEL_ALG1) {
    if (block_n < 1) return fail(LSV_ERR_INVALID_ARG, "block_n must be >= 1");
    if (!(alpha > 0.0) || !(alpha <= 1.0e6)) return fail(LSV_ERR_INVALID_ARG, "alpha must be in (0, 1e6]");
  } else {
    if (!d_cost) return fail(LSV_ERR_INVALID_ARG, "cost table required");
    if (mode == LSV_SEL_MARGINAL && d_init < 1) return fail(LSV_ERR_INVALID_ARG, "d_init must be >= 1");
  }
  int rc = lsv::launch_select(mode, batch, G, d_conf, d_cost, d_init, d_max, alpha, block_n, flags, d_gamma, d_aux,
                              d_row_offsets, d_status, (hipStream_t)stream);
  return hip_rc(rc, "select");
}

int lsv_select_joint(int32_t batch, int32_t G, const float* d_conf, const double* d_cost, int32_t d_max, uint32_t flags,
                     int32_t* d_gamma, int32_t* d_total, int32_t* d_row_offsets, int32_t* d_status, void* stream) {
  if (batch < 1 || batch > LSV_MAX_BATCH) return fail(LSV_ERR_INVALID_ARG, "need 1 <= batch <= %d", LSV_MAX_BATCH);
  if (G < 1 || G > LSV_MAX_G) return fail(LSV_ERR_INVALID_ARG, "need 1 <= G <= %d", LSV_MAX_G);
  if (d_max < 1 || d_max > G) return fail(LSV_ERR_INVALID_ARG, "need 1 <= d_max (%d) <= G (%d)", d_max, G);
  if (flags & ~(uint32_t)LSV_SEL_BONUS) return fail(LSV_ERR_INVALID_ARG, "unknown flags");
  if (!d_conf || !d_cost || !d_gamma) return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  return hip_rc(lsv::launch_select_joint(batch, G, d_conf, d_cost, d_max, flags, d_gamma, d_total, d_row_offsets,
                                         d_status, (hipStream_t)stream),
                "select_joint");
}

int lsv_next_length_g4(int32_t batch, const int32_t* d_gamma, const int32_t* d_accept_len, const int32_t* d_status,
                       int32_t d_min, int32_t d_max, int32_t* d_gamma_next, int32_t* d_row_offsets, int32_t* d_err,
                       void* stream) {
  if (batch < 1) return fail(LSV_ERR_INVALID_ARG, "need batch >= 1");
  if (d_min < 1 || d_min > d_max || d_max > LSV_MAX_SEQ_ROWS - 1)
    return fail(LSV_ERR_INVALID_ARG, "need 1 <= d_min (%d) <= d_max (%d) <= %d", d_min, d_max, LSV_MAX_SEQ_ROWS - 1);
  if (!d_gamma || !d_accept_len || !d_gamma_next) return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  if (d_row_offsets && batch > LSV_MAX_BATCH)
    return fail(LSV_ERR_INVALID_ARG, "row offsets need batch <= %d", LSV_MAX_BATCH);
  int rc = lsv::launch_next_length_g4(batch, d_gamma, d_accept_len, d_status, d_min, d_max, d_gamma_next,
                                      d_row_offsets, d_err, (hipStream_t)stream);
  return hip_rc(rc, "next_length_g4");
}

int lsv_pack_block(int32_t batch, int32_t G, const int32_t* d_row_offsets, int32_t max_rows, const int32_t* d_roots,
                   const int32_t* d_drafts, int32_t* d_tokens, int32_t* d_status, void* stream) {
  if (batch < 1 || batch > LSV_MAX_BATCH) return fail(LSV_ERR_INVALID_ARG, "need 1 <= batch <= %d", LSV_MAX_BATCH);
  if (G < 0 || G > LSV_MAX_SEQ_ROWS - 1) return fail(LSV_ERR_INVALID_ARG, "need 0 <= G <= %d", LSV_MAX_SEQ_ROWS - 1);
  if (max_rows < 1 || max_rows > LSV_MAX_ROWS) return fail(LSV_ERR_INVALID_ARG, "need 1 <= max_rows <= %d", LSV_MAX_ROWS);
  if (!d_row_offsets || !d_roots || !d_tokens || (G > 0 && !d_drafts)) return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  return hip_rc(lsv::launch_pack_block(batch, G, d_row_offsets, max_rows, d_roots, d_drafts, d_tokens, d_status,
                                       (hipStream_t)stream),
                "pack_block");
}

int lsv_next_roots(int32_t batch, const int32_t* d_accept_len, const int32_t* d_out_tokens, int32_t width,
                   const int32_t* d_status, int32_t* d_roots, void* stream) {
  if (batch < 1) return fail(LSV_ERR_INVALID_ARG, "need batch >= 1");
  if (width < 1 || width > LSV_MAX_SEQ_ROWS) return fail(LSV_ERR_INVALID_ARG, "need 1 <= width <= %d", LSV_MAX_SEQ_ROWS);
  if (!d_accept_len || !d_out_tokens || !d_roots) return fail(LSV_ERR_INVALID_ARG, "NULL pointer");
  return hip_rc(lsv::launch_next_roots(batch, d_accept_len, d_out_tokens, width, d_status, d_roots, (hipStream_t)stream),
                "next_roots");
}

int lsv_set_timing_events(int32_t kernel, void* const* events, int32_t n_slots, uint32_t record_flags) {
  if (kernel < LSV_KERNEL_QKV || kernel > LSV_KERNEL_ATTENTION) return fail(LSV_ERR_INVALID_ARG, "bad kernel class");
  if (n_slots < 0 || n_slots > LSV_MAX_TIMING_SLOTS || (n_slots > 0 && !events))
    return fail(LSV_ERR_INVALID_ARG, "n_slots must be in [0, %d] with a non-NULL event array", LSV_MAX_TIMING_SLOTS);
  g_timing.kernel = kernel;
  g_timing.n = n_slots;
  g_timing.flags = record_flags;
  for (int i = 0; i < 2 * n_slots; ++i) g_timing.ev[i] = (hipEvent_t)events[i];
  return ok();
}

}  // extern "C"

namespace lsv {
// Events are recorded with the caller's flags (hipEventRecordExternal while capturing
// a graph).  Failures are reported through the sticky error that the surrounding
// launch checks.
static void timing_record(hipEvent_t ev, hipStream_t st) {
  const hipError_t e = hipEventRecordWithFlags(ev, st, g_timing.flags);
  if (e != hipSuccess) fail(LSV_ERR_HIP, "timing event record (flags %u): %s", g_timing.flags, hipGetErrorString(e));
}
void timing_before(int kernel, int index, hipStream_t st) {
  if (g_timing.n > 0 && kernel == g_timing.kernel && index < g_timing.n) timing_record(g_timing.ev[2 * index], st);
}
void timing_after(int kernel, int index, hipStream_t st) {
  if (g_timing.n > 0 && kernel == g_timing.kernel && index < g_timing.n) timing_record(g_timing.ev[2 * index + 1], st);
}
}  // namespace lsv
