// Internal launcher interface between the C ABI (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ckv {

struct PoolView {
  void *k, *v;
  const float *k_scale, *v_scale;
  int32_t num_pages, h_kv, ps, d;
  int kv_dtype;  // ckv_dtype_t
};

struct BatchView {
  int32_t num_seqs, max_pages;
  const int32_t *bt, *ctx, *cu_q;
  int32_t total_q, max_q, max_ctx;
};

hipError_t launch_kv_append(const PoolView &p, const BatchView &b, const void *k_new,
                            const void *v_new, int in_dtype, hipStream_t s);

hipError_t launch_attn_f32(const PoolView &p, const BatchView &b, const float *q, int h_q,
                           float scale, int window, bool decode, float *out, hipStream_t s);

size_t prefill_workspace_bytes(const PoolView &p, const BatchView &b, int h_q);
int prefill_rows_per_tile();  // query rows (token x head of a group) per prefill workgroup
hipError_t launch_prefill_bf16(const PoolView &p, const BatchView &b, const void *q, int h_q,
                               float scale, int window, void *out, void *ws, hipStream_t s);

size_t decode_workspace_bytes(const PoolView &p, const BatchView &b, int h_q, int split_len);
int decode_split_len(const PoolView &p, const BatchView &b, int h_q, int requested);
int decode_max_split_len(int page_size);
hipError_t launch_decode_bf16(const PoolView &p, const BatchView &b, const void *q, int h_q,
                              float scale, int window, int split_len, void *out, void *ws,
                              size_t ws_bytes, hipStream_t s);

// Prefill over one batch and decode over another in one launch (plus the
// merges of split keys); results equal the two separate launches bit for bit
// at the same decode partition length (mixed_split_len resolves 0).
// interleave: groups of eight workgroups per run of one kind (0 = library
// choice).  k_pf / v_pf and k_dc / v_dc (bf16 pools; null = already in the
// pool): the new rows the launch appends itself.
int mixed_split_len(const PoolView &p, const BatchView &db, int h_q, int requested);
size_t mixed_workspace_bytes(const PoolView &p, const BatchView &pb, const BatchView &db, int h_q,
                             int split_len);
hipError_t launch_mixed(const PoolView &p, const BatchView &pb, const void *q_pf, const void *k_pf,
                        const void *v_pf, void *out_pf, const BatchView &db, const void *q_dc,
                        const void *k_dc, const void *v_dc, void *out_dc, int h_q, float scale,
                        int window, int split_len, int interleave, void *ws, hipStream_t s);

// Device address of the allocation-free decode's scratch on the current
// device (CKV_DECODE_SCRATCH_BYTES bytes), looked up on first use.
hipError_t decode_scratch(void **ptr);

int page_bytes(const PoolView &p);
int page_blocks(const PoolView &p);
size_t pages_staging_bytes(const PoolView &p, int n);
hipError_t launch_pages_reload(const PoolView &p, const void *host_k, const void *host_v,
                               const float *host_ks, const float *host_vs, const int32_t *pages,
                               int n, void *staging, hipStream_t s);
hipError_t launch_pages_offload(const PoolView &p, const int32_t *pages, int n, void *host_k,
                                void *host_v, float *host_ks, float *host_vs, void *staging,
                                hipStream_t s);

}  // namespace ckv
