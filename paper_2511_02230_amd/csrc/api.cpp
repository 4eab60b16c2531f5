// C ABI of the ckv library: host-side argument checks and kernel dispatch.
// Declarations and the contract of every entry point are in include/ckv.h.
#include "../../include/ckv.h"

#include <climits>
#include <cmath>
#include <unordered_set>
#include <vector>

#include "launch.hpp"

namespace {

using ckv::BatchView;
using ckv::PoolView;

// Launch grids put sequences (and, for the fp32 path, query heads) in grid
// dimensions limited to 65535 workgroups.
constexpr long long kGridYZ = 65535;

bool supported_dim(int d) { return d == 64 || d == 128 || d == 256; }
bool supported_page(int ps) { return ps == 16 || ps == 64; }
bool valid_dtype(int t) { return t == CKV_F32 || t == CKV_BF16 || t == CKV_FP8_E4M3; }
// The kernels mask keys with -inf scores and fold the scale into the
// exponent, which needs a positive, finite softmax scale.
bool valid_scale(float s) { return std::isfinite(s) && s > 0.f; }

ckv_status_t check_pool(const ckv_pool_t *p) {
  if (!p || !p->k_pages || !p->v_pages) return CKV_ERR_INVALID_ARG;
  if (p->num_pages <= 0 || p->num_kv_heads <= 0 || p->page_size <= 0 || p->head_dim <= 0)
    return CKV_ERR_INVALID_ARG;
  if (!valid_dtype(p->kv_dtype)) return CKV_ERR_INVALID_ARG;
  if (p->kv_dtype == CKV_FP8_E4M3 && (!p->k_scale || !p->v_scale)) return CKV_ERR_INVALID_ARG;
  if (!supported_dim(p->head_dim) || !supported_page(p->page_size)) return CKV_ERR_UNSUPPORTED;
  return CKV_OK;
}

// mode 0: append / prefill (uses cu_q_lens), mode 1: decode
ckv_status_t check_batch(const ckv_pool_t *p, const ckv_batch_t *b, int mode) {
  if (!b) return CKV_ERR_INVALID_ARG;
  if (b->num_seqs < 0 || b->total_q_len < 0 || b->max_q_len < 0 || b->max_ctx_len < 0)
    return CKV_ERR_INVALID_ARG;
  if (b->num_seqs == 0) return CKV_OK;
  if (b->num_seqs > kGridYZ) return CKV_ERR_UNSUPPORTED;
  if (b->max_pages_per_seq <= 0 || !b->block_table || !b->ctx_lens) return CKV_ERR_INVALID_ARG;
  const long long cap = (long long)b->max_pages_per_seq * p->page_size;
  if (mode == 0) {
    if (!b->cu_q_lens) return CKV_ERR_INVALID_ARG;
    if (b->total_q_len > (long long)b->num_seqs * b->max_q_len) return CKV_ERR_INVALID_ARG;
    if (b->max_ctx_len > cap || b->max_q_len > cap) return CKV_ERR_INVALID_ARG;
  } else {
    if (b->max_ctx_len < 1 || b->max_ctx_len > cap) return CKV_ERR_INVALID_ARG;
  }
  return CKV_OK;
}

ckv_status_t check_heads(const ckv_pool_t *p, int num_q_heads) {
  if (num_q_heads <= 0 || num_q_heads % p->num_kv_heads != 0) return CKV_ERR_INVALID_ARG;
  if (num_q_heads > kGridYZ) return CKV_ERR_UNSUPPORTED;
  return CKV_OK;
}

// Prefill grid: row tiles of the longest new turn in grid.y, and the merge
// of key partitions over total_q_len * num_q_heads rows in grid.x.
ckv_status_t check_prefill_grid(const ckv_pool_t *p, const ckv_batch_t *b, int num_q_heads) {
  const long long rows = (long long)b->max_q_len * (num_q_heads / p->num_kv_heads);
  const long long tiles = (rows + ckv::prefill_rows_per_tile() - 1) / ckv::prefill_rows_per_tile();
  if (tiles > kGridYZ) return CKV_ERR_UNSUPPORTED;
  if ((long long)b->total_q_len * num_q_heads > INT_MAX) return CKV_ERR_UNSUPPORTED;
  return CKV_OK;
}

ckv_status_t check_attn_dtypes(const ckv_pool_t *p, ckv_dtype_t q_dtype) {
  if (!valid_dtype(q_dtype)) return CKV_ERR_INVALID_ARG;
  if (q_dtype == CKV_F32 && p->kv_dtype == CKV_F32) return CKV_OK;
  if (q_dtype == CKV_BF16 && (p->kv_dtype == CKV_BF16 || p->kv_dtype == CKV_FP8_E4M3)) return CKV_OK;
  return CKV_ERR_UNSUPPORTED;
}

PoolView view(const ckv_pool_t *p) {
  PoolView v;
  v.k = p->k_pages;
  v.v = p->v_pages;
  v.k_scale = p->k_scale;
  v.v_scale = p->v_scale;
  v.num_pages = p->num_pages;
  v.h_kv = p->num_kv_heads;
  v.ps = p->page_size;
  v.d = p->head_dim;
  v.kv_dtype = p->kv_dtype;
  return v;
}

BatchView view(const ckv_batch_t *b) {
  BatchView v;
  v.num_seqs = b->num_seqs;
  v.max_pages = b->max_pages_per_seq;
  v.bt = b->block_table;
  v.ctx = b->ctx_lens;
  v.cu_q = b->cu_q_lens;
  v.total_q = b->total_q_len;
  v.max_q = b->max_q_len;
  v.max_ctx = b->max_ctx_len;
  return v;
}

ckv_status_t launched(hipError_t e) { return e == hipSuccess ? CKV_OK : CKV_ERR_LAUNCH; }

#define CKV_TRY(expr)                    \
  do {                                   \
    const ckv_status_t st_ = (expr);     \
    if (st_ != CKV_OK) return st_;       \
  } while (0)

ckv_status_t check_page_move(const ckv_pool_t *pool, const int32_t *pages, int32_t n,
                             const void *host_k, const void *host_v, const void *host_ks,
                             const void *host_vs, const void *staging, size_t staging_bytes) {
  CKV_TRY(check_pool(pool));
  if (n < 0) return CKV_ERR_INVALID_ARG;
  if (n == 0) return CKV_OK;
  if (!pages || !host_k || !host_v) return CKV_ERR_INVALID_ARG;
  if (pool->kv_dtype == CKV_FP8_E4M3 && (!host_ks || !host_vs)) return CKV_ERR_INVALID_ARG;
  if ((long long)n * ckv::page_blocks(view(pool)) > INT_MAX) return CKV_ERR_INVALID_ARG;
  if (!staging || staging_bytes < ckv::pages_staging_bytes(view(pool), n)) return CKV_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(staging) % 16 != 0) return CKV_ERR_INVALID_ARG;
  return CKV_OK;
}

}  // namespace

extern "C" {

ckv_status_t kv_append(const ckv_pool_t *pool, const ckv_batch_t *batch, const void *k_new,
                       const void *v_new, ckv_dtype_t in_dtype, hipStream_t stream) {
  CKV_TRY(check_pool(pool));
  CKV_TRY(check_batch(pool, batch, 0));
  if (!valid_dtype(in_dtype)) return CKV_ERR_INVALID_ARG;
  const bool ok = (in_dtype == CKV_F32 && pool->kv_dtype == CKV_F32) ||
                  (in_dtype == CKV_BF16 && pool->kv_dtype == CKV_BF16) ||
                  (in_dtype == CKV_BF16 && pool->kv_dtype == CKV_FP8_E4M3);
  if (!ok) return CKV_ERR_UNSUPPORTED;
  if (batch->num_seqs == 0 || batch->total_q_len == 0) return CKV_OK;
  if (!k_new || !v_new) return CKV_ERR_INVALID_ARG;
  return launched(ckv::launch_kv_append(view(pool), view(batch), k_new, v_new, in_dtype, stream));
}

size_t prefix_prefill_workspace_bytes(const ckv_pool_t *pool, const ckv_batch_t *batch,
                                      int32_t num_q_heads) {
  if (check_pool(pool) != CKV_OK || check_batch(pool, batch, 0) != CKV_OK ||
      check_heads(pool, num_q_heads) != CKV_OK)
    return 0;
  if (batch->num_seqs == 0 || batch->total_q_len == 0 || pool->kv_dtype == CKV_F32) return 0;
  if (check_prefill_grid(pool, batch, num_q_heads) != CKV_OK) return 0;
  return ckv::prefill_workspace_bytes(view(pool), view(batch), num_q_heads);
}

ckv_status_t prefix_prefill_attn(const ckv_pool_t *pool, const ckv_batch_t *batch, const void *q,
                                 ckv_dtype_t q_dtype, int32_t num_q_heads, float softmax_scale,
                                 int32_t window, void *out, void *workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  CKV_TRY(check_pool(pool));
  CKV_TRY(check_batch(pool, batch, 0));
  CKV_TRY(check_heads(pool, num_q_heads));
  CKV_TRY(check_attn_dtypes(pool, q_dtype));
  if (!valid_scale(softmax_scale) || window < 0) return CKV_ERR_INVALID_ARG;
  if (batch->num_seqs == 0 || batch->total_q_len == 0) return CKV_OK;
  if (!q || !out) return CKV_ERR_INVALID_ARG;
  CKV_TRY(check_prefill_grid(pool, batch, num_q_heads));
  if (q_dtype == CKV_F32)
    return launched(ckv::launch_attn_f32(view(pool), view(batch), static_cast<const float *>(q),
                                         num_q_heads, softmax_scale, window, false,
                                         static_cast<float *>(out), stream));
  const size_t need = ckv::prefill_workspace_bytes(view(pool), view(batch), num_q_heads);
  if (need > 0 && (!workspace || workspace_bytes < need)) return CKV_ERR_WORKSPACE;
  return launched(ckv::launch_prefill_bf16(view(pool), view(batch), q, num_q_heads, softmax_scale,
                                           window, out, workspace, stream));
}

size_t paged_decode_workspace_bytes(const ckv_pool_t *pool, const ckv_batch_t *batch,
                                    int32_t num_q_heads, int32_t kv_split_len) {
  if (check_pool(pool) != CKV_OK || check_batch(pool, batch, 1) != CKV_OK ||
      check_heads(pool, num_q_heads) != CKV_OK)
    return 0;
  if (kv_split_len < 0 || kv_split_len % 64 != 0 ||
      kv_split_len > ckv::decode_max_split_len(pool->page_size))
    return 0;
  if (batch->num_seqs == 0 || pool->kv_dtype == CKV_F32) return 0;
  return ckv::decode_workspace_bytes(view(pool), view(batch), num_q_heads, kv_split_len);
}

ckv_status_t paged_decode_attn(const ckv_pool_t *pool, const ckv_batch_t *batch, const void *q,
                               ckv_dtype_t q_dtype, int32_t num_q_heads, float softmax_scale,
                               int32_t window, int32_t kv_split_len, void *out, void *workspace,
                               size_t workspace_bytes, hipStream_t stream) {
  CKV_TRY(check_pool(pool));
  CKV_TRY(check_batch(pool, batch, 1));
  CKV_TRY(check_heads(pool, num_q_heads));
  CKV_TRY(check_attn_dtypes(pool, q_dtype));
  if (!valid_scale(softmax_scale) || window < 0) return CKV_ERR_INVALID_ARG;
  if (kv_split_len < 0 || kv_split_len % 64 != 0 ||
      kv_split_len > ckv::decode_max_split_len(pool->page_size))
    return CKV_ERR_INVALID_ARG;
  if (batch->num_seqs == 0) return CKV_OK;
  if (!q || !out) return CKV_ERR_INVALID_ARG;
  if (q_dtype == CKV_F32)
    return launched(ckv::launch_attn_f32(view(pool), view(batch), static_cast<const float *>(q),
                                         num_q_heads, softmax_scale, window, true,
                                         static_cast<float *>(out), stream));
  const size_t need = ckv::decode_workspace_bytes(view(pool), view(batch), num_q_heads, kv_split_len);
  if (need > 0 && (!workspace || workspace_bytes < need)) return CKV_ERR_WORKSPACE;
  return launched(ckv::launch_decode_bf16(view(pool), view(batch), q, num_q_heads, softmax_scale,
                                          window, kv_split_len, out, workspace, workspace_bytes,
                                          stream));
}

size_t mixed_attn_workspace_bytes(const ckv_pool_t *pool, const ckv_batch_t *prefill,
                                  const ckv_batch_t *decode, int32_t num_q_heads,
                                  int32_t kv_split_len) {
  if (check_pool(pool) != CKV_OK || check_batch(pool, prefill, 0) != CKV_OK ||
      check_batch(pool, decode, 1) != CKV_OK || check_heads(pool, num_q_heads) != CKV_OK)
    return 0;
  if (kv_split_len < 0 || kv_split_len % 64 != 0 ||
      kv_split_len > ckv::decode_max_split_len(pool->page_size))
    return 0;
  if (pool->kv_dtype == CKV_F32) return 0;
  if (prefill->num_seqs > 0 && check_prefill_grid(pool, prefill, num_q_heads) != CKV_OK) return 0;
  return ckv::mixed_workspace_bytes(view(pool), view(prefill), view(decode), num_q_heads,
                                    kv_split_len);
}

ckv_status_t mixed_attn(const ckv_pool_t *pool, const ckv_batch_t *prefill, const void *q_prefill,
                        const void *k_prefill, const void *v_prefill, void *out_prefill,
                        const ckv_batch_t *decode, const void *q_decode, const void *k_decode,
                        const void *v_decode, void *out_decode, ckv_dtype_t q_dtype,
                        int32_t num_q_heads, float softmax_scale, int32_t window,
                        int32_t kv_split_len, int32_t interleave, void *workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  CKV_TRY(check_pool(pool));
  CKV_TRY(check_batch(pool, prefill, 0));
  CKV_TRY(check_batch(pool, decode, 1));
  CKV_TRY(check_heads(pool, num_q_heads));
  CKV_TRY(check_attn_dtypes(pool, q_dtype));
  if (q_dtype != CKV_BF16) return CKV_ERR_UNSUPPORTED;
  if (!valid_scale(softmax_scale) || window < 0 || interleave < 0) return CKV_ERR_INVALID_ARG;
  if (kv_split_len < 0 || kv_split_len % 64 != 0 ||
      kv_split_len > ckv::decode_max_split_len(pool->page_size))
    return CKV_ERR_INVALID_ARG;
  const bool has_pf = prefill->num_seqs > 0 && prefill->total_q_len > 0;
  const bool has_dc = decode->num_seqs > 0;
  if (has_pf && (!q_prefill || !out_prefill)) return CKV_ERR_INVALID_ARG;
  if (has_dc && (!q_decode || !out_decode)) return CKV_ERR_INVALID_ARG;
  // fused append: both rows of a batch or neither, bf16 pools only
  if (!k_prefill != !v_prefill || !k_decode != !v_decode) return CKV_ERR_INVALID_ARG;
  if (((has_pf && k_prefill) || (has_dc && k_decode)) && pool->kv_dtype != CKV_BF16)
    return CKV_ERR_UNSUPPORTED;
  if (has_pf) CKV_TRY(check_prefill_grid(pool, prefill, num_q_heads));
  if (!has_pf && !has_dc) return CKV_OK;
  const size_t need = ckv::mixed_workspace_bytes(view(pool), view(prefill), view(decode),
                                                 num_q_heads, kv_split_len);
  if (need > 0 && (!workspace || workspace_bytes < need)) return CKV_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return CKV_ERR_INVALID_ARG;
  return launched(ckv::launch_mixed(view(pool), view(prefill), q_prefill, k_prefill, v_prefill,
                                    out_prefill, view(decode), q_decode, k_decode, v_decode,
                                    out_decode, num_q_heads, softmax_scale, window, kv_split_len,
                                    interleave, workspace, stream));
}

ckv_status_t paged_decode_attn_noalloc(const ckv_pool_t *pool, const ckv_batch_t *batch,
                                       const void *q, ckv_dtype_t q_dtype, int32_t num_q_heads,
                                       float softmax_scale, int32_t window, int32_t kv_split_len,
                                       void *out, hipStream_t stream) {
  CKV_TRY(check_pool(pool));
  CKV_TRY(check_batch(pool, batch, 1));
  CKV_TRY(check_heads(pool, num_q_heads));
  CKV_TRY(check_attn_dtypes(pool, q_dtype));
  if (!valid_scale(softmax_scale) || window < 0) return CKV_ERR_INVALID_ARG;
  if (kv_split_len < 0 || kv_split_len % 64 != 0 ||
      kv_split_len > ckv::decode_max_split_len(pool->page_size))
    return CKV_ERR_INVALID_ARG;
  if (batch->num_seqs == 0) return CKV_OK;
  if (!q || !out) return CKV_ERR_INVALID_ARG;
  if (q_dtype == CKV_F32)  // the fp32 path keeps no partials
    return launched(ckv::launch_attn_f32(view(pool), view(batch), static_cast<const float *>(q),
                                         num_q_heads, softmax_scale, window, true,
                                         static_cast<float *>(out), stream));
  const size_t need = ckv::decode_workspace_bytes(view(pool), view(batch), num_q_heads, kv_split_len);
  if (need > CKV_DECODE_SCRATCH_BYTES) return CKV_ERR_WORKSPACE;
  void *ws = nullptr;
  if (need > 0 && ckv::decode_scratch(&ws) != hipSuccess) return CKV_ERR_LAUNCH;
  return launched(ckv::launch_decode_bf16(view(pool), view(batch), q, num_q_heads, softmax_scale,
                                          window, kv_split_len, out, ws, need, stream));
}

size_t kv_pages_staging_bytes(const ckv_pool_t *pool, int32_t num_moved) {
  if (check_pool(pool) != CKV_OK || num_moved <= 0) return 0;
  return ckv::pages_staging_bytes(view(pool), num_moved);
}

ckv_status_t kv_pages_reload(const ckv_pool_t *pool, const int32_t *pages, int32_t num_moved,
                             const void *host_k, const void *host_v, const float *host_k_scale,
                             const float *host_v_scale, void *staging, size_t staging_bytes,
                             hipStream_t stream) {
  CKV_TRY(check_page_move(pool, pages, num_moved, host_k, host_v, host_k_scale, host_v_scale,
                          staging, staging_bytes));
  if (num_moved == 0) return CKV_OK;
  return launched(ckv::launch_pages_reload(view(pool), host_k, host_v, host_k_scale, host_v_scale,
                                           pages, num_moved, staging, stream));
}

ckv_status_t kv_pages_offload(const ckv_pool_t *pool, const int32_t *pages, int32_t num_moved,
                              void *host_k, void *host_v, float *host_k_scale,
                              float *host_v_scale, void *staging, size_t staging_bytes,
                              hipStream_t stream) {
  CKV_TRY(check_page_move(pool, pages, num_moved, host_k, host_v, host_k_scale, host_v_scale,
                          staging, staging_bytes));
  if (num_moved == 0) return CKV_OK;
  return launched(ckv::launch_pages_offload(view(pool), pages, num_moved, host_k, host_v,
                                            host_k_scale, host_v_scale, staging, stream));
}

ckv_status_t ckv_validate_batch(const ckv_pool_t *pool, int32_t num_seqs, int32_t max_pages_per_seq,
                                const int32_t *bt, const int32_t *ctx, const int32_t *cu,
                                int32_t max_q_len, int32_t max_ctx_len, int32_t mode,
                                int32_t distinct_pages) {
  if (!pool || pool->num_pages <= 0 || pool->page_size <= 0) return CKV_ERR_INVALID_ARG;
  if (num_seqs < 0 || (mode != 0 && mode != 1)) return CKV_ERR_INVALID_ARG;
  if (num_seqs == 0) return CKV_OK;
  if (!bt || !ctx || max_pages_per_seq <= 0 || (mode == 0 && !cu)) return CKV_ERR_INVALID_ARG;
  if (mode == 0 && cu[0] != 0) return CKV_ERR_INVALID_ARG;
  std::unordered_set<int32_t> seen;
  const int ps = pool->page_size;
  for (int b = 0; b < num_seqs; ++b) {
    long long end;
    if (mode == 0) {
      const long long n = (long long)cu[b + 1] - cu[b];
      if (n < 0 || n > max_q_len || ctx[b] < 0 || ctx[b] > max_ctx_len) return CKV_ERR_INVALID_ARG;
      end = ctx[b] + n;  // positions 0 .. end-1 are read or written
    } else {
      if (ctx[b] < 1 || ctx[b] > max_ctx_len) return CKV_ERR_INVALID_ARG;
      end = ctx[b];
    }
    const long long pages = (end + ps - 1) / ps;
    if (pages > max_pages_per_seq) return CKV_ERR_INVALID_ARG;
    for (long long k = 0; k < pages; ++k) {
      const int32_t pg = bt[(size_t)b * max_pages_per_seq + k];
      if (pg < 0 || pg >= pool->num_pages) return CKV_ERR_INVALID_ARG;
      if (distinct_pages && !seen.insert(pg).second) return CKV_ERR_INVALID_ARG;
    }
  }
  return CKV_OK;
}

const char *ckv_status_string(ckv_status_t status) {
  switch (status) {
    case CKV_OK:
      return "CKV_OK";
    case CKV_ERR_INVALID_ARG:
      return "CKV_ERR_INVALID_ARG: a pointer, size or bound is invalid";
    case CKV_ERR_UNSUPPORTED:
      return "CKV_ERR_UNSUPPORTED: no kernel for this dtype / head_dim / page_size";
    case CKV_ERR_WORKSPACE:
      return "CKV_ERR_WORKSPACE: workspace missing or too small";
    case CKV_ERR_LAUNCH:
      return "CKV_ERR_LAUNCH: kernel launch or copy failed";
  }
  return "unknown ckv status";
}

int32_t ckv_version(void) { return 100; }

}  // extern "C"
