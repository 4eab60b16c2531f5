/*
 * ckv.h -- paged KV-cache hot path for multi-turn agent serving on MI355X
 * (gfx950): append new-turn K/V into a paged pool, prefix-reuse prefill
 * attention, paged decode attention, and whole-page moves between the pool
 * and host memory (offload on eviction, reload on a TTL miss).
 *
 * Why this path exists: Continuum (arXiv 2511.02230) keeps a tool-calling
 * request's KV blocks resident in GPU memory for a time-to-live instead of
 * freeing them when the request finishes (Sec. 5.2, "Request Pinning"), so
 * the program's next turn finds its prefix's pages still in the pool and only
 * the new tokens (tool output + next prompt) need prefilling (Sec. 1;
 * Sec. 5.2, "Offline Profile", on pages that stay resident and need no
 * recomputation).  The paper serves on a paged-attention engine (Sec. 7,
 * "LLM Inference Systems"); the three calls below are that engine's GPU work
 * for a retained-prefix turn.  The paper states no attention formula; the one
 * used is scaled dot-product softmax attention with grouped KV heads.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every pointer argument is a HIP device pointer owned by the caller,
 *    except the ckv_pool_t / ckv_batch_t structs themselves (host memory,
 *    read during the call only) and the host_* buffers of kv_pages_reload /
 *    kv_pages_offload.  The library keeps no state, never allocates or frees
 *    memory and never synchronizes; all work is enqueued on `stream` (0 = the
 *    null stream).  Calls are re-entrant.
 *  - Pool layout: K and V are each [num_pages][num_kv_heads][page_size]
 *    [head_dim], row-major, element type kv_dtype.  For CKV_FP8_E4M3 each
 *    (page, kv head) has an fp32 scale in k_scale / v_scale
 *    [num_pages][num_kv_heads]; a stored code c represents e4m3(c) * scale.
 *  - Sequence b's token at absolute position j lives in physical page
 *    block_table[b * max_pages_per_seq + j / page_size], slot j % page_size.
 *  - Packed rows: the new-turn rows of sequence b are rows
 *    cu_q_lens[b] .. cu_q_lens[b+1]-1 of q / k_new / v_new / out, row t of
 *    sequence b being its token at absolute position ctx_lens[b] + t.
 *  - Query head h reads KV head h / (num_q_heads / num_kv_heads).
 *  - Visibility: the query at absolute position i sees key j iff j <= i and,
 *    when window > 0, i - j < window (exactly `window` keys, itself included).
 *  - Device-side contents are the caller's contract: page ids must lie in
 *    [0, num_pages) and every addressed position inside the sequence's
 *    table; cu_q_lens must be non-decreasing with cu_q_lens[0] = 0 and
 *    cu_q_lens[num_seqs] = total_q_len; per-sequence lengths must not exceed
 *    the host-side bounds max_q_len / max_ctx_len.  Violations are undefined
 *    behaviour (out-of-bounds device accesses); ckv_validate_batch checks
 *    host copies of these arrays.
 *  - softmax_scale must be positive and finite (the attention calls return
 *    CKV_ERR_INVALID_ARG otherwise): the kernels remove masked keys with
 *    -inf scores and fold the scale into the exponent.
 *  - Host-side argument errors return CKV_ERR_INVALID_ARG, combinations
 *    without a kernel return CKV_ERR_UNSUPPORTED, a too-small workspace
 *    returns CKV_ERR_WORKSPACE; nothing is launched in those cases.  A failed
 *    launch returns CKV_ERR_LAUNCH.
 *
 * Supported combinations: (q, pool) dtypes (F32, F32), (BF16, BF16) and
 * (BF16, FP8_E4M3); head_dim in {64, 128, 256}; page_size in {16, 64};
 * num_q_heads a multiple of num_kv_heads.  Size limits (launch grids):
 * num_seqs <= 65535 and num_q_heads <= 65535; for prefix_prefill_attn also
 * ceil(max_q_len * num_q_heads / num_kv_heads / 128) <= 65535 and
 * total_q_len * num_q_heads < 2^31.  Beyond them a call returns
 * CKV_ERR_UNSUPPORTED and launches nothing.
 */
#ifndef CKV_H
#define CKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CKV_OK = 0,
  CKV_ERR_INVALID_ARG = 1,
  CKV_ERR_UNSUPPORTED = 2,
  CKV_ERR_WORKSPACE = 3,
  CKV_ERR_LAUNCH = 4
} ckv_status_t;

typedef enum {
  CKV_F32 = 0,
  CKV_BF16 = 1,
  CKV_FP8_E4M3 = 2 /* OCP E4M3FN: bias 7, max 448, no inf, NaN = S.1111.111 */
} ckv_dtype_t;

/* The paged KV pool: pages retained between turns (Sec. 5.2 pins them). */
typedef struct {
  void *k_pages;        /* [num_pages][num_kv_heads][page_size][head_dim] */
  void *v_pages;        /* same layout */
  const float *k_scale; /* [num_pages][num_kv_heads], FP8 only, else NULL */
  const float *v_scale; /* same */
  int32_t num_pages;
  int32_t num_kv_heads;
  int32_t page_size;
  int32_t head_dim;
  ckv_dtype_t kv_dtype;
} ckv_pool_t;

/* One launch's sequences: block tables and context/query lengths. */
typedef struct {
  int32_t num_seqs;
  int32_t max_pages_per_seq;   /* row stride of block_table */
  const int32_t *block_table;  /* [num_seqs][max_pages_per_seq] physical page ids */
  const int32_t *ctx_lens;     /* [num_seqs] append / prefill: tokens resident before
                                  this call (the retained prefix P_b);
                                  decode: context length c_b >= 1, the query being
                                  the token at position c_b - 1 */
  const int32_t *cu_q_lens;    /* [num_seqs + 1] packed row offsets (append / prefill);
                                  ignored by decode (one row per sequence) */
  int32_t total_q_len;         /* host copy of cu_q_lens[num_seqs]; decode: num_seqs */
  int32_t max_q_len;           /* host upper bound of cu_q_lens[b+1] - cu_q_lens[b] */
  int32_t max_ctx_len;         /* host upper bound of ctx_lens[b] */
} ckv_batch_t;

/*
 * kv_append -- write the new turn's keys and values into the pool.
 * Serves Sec. 1 (a tool's output is appended to the request's context and a
 * new inference step starts) and Sec. 5.2, "Request Pinning" (the finished
 * step's KV blocks are kept, so the next turn's tokens land in the pages
 * after the retained prefix).  The paper prints no formula for this write;
 * it is the paged-pool write of the paged-attention engine it runs on
 * (Sec. 7).
 * For every sequence b and row t < n_b: position j = ctx_lens[b] + t; for each
 * KV head h, K[page(j)][h][j % page_size][:] = enc(k_new[cu_q_lens[b] + t][h][:]),
 * likewise V.  No other pool byte changes.
 *   k_new, v_new: [total_q_len][num_kv_heads][head_dim], element type in_dtype.
 *   enc: bit copy when in_dtype == kv_dtype (F32 or BF16); for BF16 -> FP8_E4M3,
 *        r = x / scale[page][h] in IEEE binary32 (round to nearest even), clamped
 *        to [-448, 448], rounded to nearest-even E4M3FN (-0 -> 0x80).  NaN inputs
 *        give a NaN code.  The scales are inputs (the caller's policy).
 * Rows of different sequences must address distinct slots.
 */
ckv_status_t kv_append(const ckv_pool_t *pool, const ckv_batch_t *batch,
                       const void *k_new, const void *v_new, ckv_dtype_t in_dtype,
                       hipStream_t stream);

/*
 * prefix_prefill_attn -- causal attention of the new-turn queries over the
 * retained prefix plus the new turn itself (call kv_append first).
 * Serves Sec. 1 (the prefill stage: a turn whose prefix was evicted must
 * recompute it, one whose prefix is retained prefills only its new tokens)
 * and Sec. 5.2, "Offline Profile" (prefill time against context length,
 * pages still resident needing no recomputation).  The paper defines no
 * attention formula; the one below is scaled dot-product softmax attention
 * with grouped KV heads and a bottom-right causal mask.
 * For row t of sequence b (position i = ctx_lens[b] + t) and query head h:
 *   out[row][h][:] = sum_{j visible} e^{s_j - m} V_j / sum_{j visible} e^{s_j - m},
 *   s_j = softmax_scale * <q[row][h][:], K_j>, m = max_j s_j,
 * K_j, V_j being KV head h / G of position j read through the block table.
 *   q, out: [total_q_len][num_q_heads][head_dim]; out has q_dtype.
 *   Softmax and accumulation are fp32; BF16 products run on MFMA in bf16.
 *   workspace: at least prefix_prefill_workspace_bytes(...) bytes, device
 *   memory owned by the caller and free for the duration of the call.  It is
 *   0 when the batch's row tiles make at least four waves of workgroups on the
 *   GPU, or when no key partitioning would cut the waves per unit of work by
 *   3 %; otherwise each tile's keys are split into partitions (>= 2048 keys,
 *   at most 32) whose fp32 partials land there before a merge
 *   (total_q_len * num_q_heads * partitions * (head_dim + 2) * 4 bytes).
 *   Too small a workspace returns CKV_ERR_WORKSPACE and launches nothing.
 */
ckv_status_t prefix_prefill_attn(const ckv_pool_t *pool, const ckv_batch_t *batch,
                                 const void *q, ckv_dtype_t q_dtype, int32_t num_q_heads,
                                 float softmax_scale, int32_t window, void *out,
                                 void *workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/*
 * paged_decode_attn -- one query per sequence at position c_b - 1 over its
 * c_b = ctx_lens[b] tokens (its own K/V already appended).  Same formula.
 * Serves Sec. 1 (the decoding stage, which reads a request's whole KV cache
 * for every generated token while the cache stays in GPU memory); the
 * paper gives no formula for it either.
 *   q, out: [num_seqs][num_q_heads][head_dim]; out has q_dtype.
 *   kv_split_len: keys per split-K partition (0 = library choice, else a
 *   positive multiple of 64, at most 256 * page_size).  Partitions are fixed
 *   by logical positions only, so results do not depend on physical page
 *   placement.
 *   workspace: at least paged_decode_workspace_bytes(...) bytes.
 */
ckv_status_t paged_decode_attn(const ckv_pool_t *pool, const ckv_batch_t *batch,
                               const void *q, ckv_dtype_t q_dtype, int32_t num_q_heads,
                               float softmax_scale, int32_t window, int32_t kv_split_len,
                               void *out, void *workspace, size_t workspace_bytes,
                               hipStream_t stream);

/*
 * mixed_attn -- prefix_prefill_attn over `prefill` and paged_decode_attn over
 * `decode` in one kernel launch (followed by the small merges of split keys
 * when either needs them), for a serving step whose batch mixes
 * prefix-reuse prefills with decodes: the paper's engine runs such steps
 * with chunked prefill (Sec. 6.1, "Setup"), and the time a turn spends in
 * prefill is the cost its TTL weighs (Sec. 4.1; Sec. 5.2, "Offline
 * Profile").  The prefill's work is bound by the matrix cores and the
 * decode's by HBM; one grid holding both lets decode partitions stream
 * beside prefill row tiles.
 * Results are those of the two separate calls, bit for bit (same work
 * items, same key partitions), with the same argument rules; `prefill`
 * follows prefix_prefill_attn's batch conventions and `decode`
 * paged_decode_attn's.  Either batch may be empty (num_seqs 0).
 *   k_prefill / v_prefill, k_decode / v_decode: the new K and V rows, or
 *   both NULL when kv_append has already put them in the pool.  Given, the
 *   launch appends them itself (the append fused into the attention: each
 *   row is written into its pool slot by one work item, and the work items
 *   that need it read it from these rows), leaving the pool and the outputs
 *   exactly as kv_append followed by this call.  Prefill rows are
 *   [total_q_len][H_kv][D] as for kv_append (ctx_lens = P_b, the tokens
 *   before the turn); decode rows are [num_seqs][H_kv][D], the token at
 *   position ctx_lens[b] - 1 (ctx_lens counts it, as in paged_decode_attn).
 *   bf16 pools only (bf16 rows): an fp8 pool returns CKV_ERR_UNSUPPORTED,
 *   since every work item reading a new key would have to encode it again.
 *   One of a pair NULL returns CKV_ERR_INVALID_ARG.  The rows must not
 *   alias the pool, and the two batches must not share the pool slots the
 *   appended rows go to.
 *   q_dtype: CKV_BF16 (bf16 or fp8 pools); other types return
 *   CKV_ERR_UNSUPPORTED.
 *   kv_split_len: the decode's partition length, as for paged_decode_attn;
 *   0 = paged_decode_attn's own choice capped at 2048 keys (finer decode
 *   work interleaves better with the prefill's), so the decode output
 *   equals paged_decode_attn's at that length.
 *   interleave: the grid alternates runs of `interleave` groups of eight
 *   prefill workgroups with runs of as many decode groups (0 = the library's
 *   choice: three fills of the GPU).  It changes timing only, never
 *   results; negative values return CKV_ERR_INVALID_ARG.
 *   workspace: at least mixed_attn_workspace_bytes(...) bytes, 256-byte
 *   aligned (the prefill's partials, then the decode's).
 */
ckv_status_t mixed_attn(const ckv_pool_t *pool, const ckv_batch_t *prefill, const void *q_prefill,
                        const void *k_prefill, const void *v_prefill, void *out_prefill,
                        const ckv_batch_t *decode, const void *q_decode, const void *k_decode,
                        const void *v_decode, void *out_decode, ckv_dtype_t q_dtype,
                        int32_t num_q_heads, float softmax_scale, int32_t window,
                        int32_t kv_split_len, int32_t interleave, void *workspace,
                        size_t workspace_bytes, hipStream_t stream);
size_t mixed_attn_workspace_bytes(const ckv_pool_t *pool, const ckv_batch_t *prefill,
                                  const ckv_batch_t *decode, int32_t num_q_heads,
                                  int32_t kv_split_len);

/*
 * paged_decode_attn_noalloc -- paged_decode_attn without a workspace, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  Same arguments,
 * kernels and results as paged_decode_attn (bit for bit, for the same
 * kv_split_len), minus workspace / workspace_bytes: the split-K partials go
 * to a scratch array of CKV_DECODE_SCRATCH_BYTES bytes that the library
 * keeps in each GPU's memory from its first use on that GPU until the
 * process ends (the stream must belong to the current device).  The call
 * allocates and frees nothing.
 *   Returns CKV_ERR_WORKSPACE, launching nothing, when the partials would
 *   exceed the scratch (paged_decode_workspace_bytes(...) >
 *   CKV_DECODE_SCRATCH_BYTES); a longer kv_split_len needs fewer of them.
 *   CKV_ERR_LAUNCH if the scratch address cannot be obtained.
 *   Every call on one GPU shares that GPU's scratch: calls whose work
 *   overlaps on the GPU (concurrent streams, or threads) race and must be
 *   serialized by the caller.  A call needs no cleared scratch: each
 *   partition writes its partial before the merge reads it.
 */
#define CKV_DECODE_SCRATCH_BYTES ((size_t)64 << 20)
ckv_status_t paged_decode_attn_noalloc(const ckv_pool_t *pool, const ckv_batch_t *batch,
                                       const void *q, ckv_dtype_t q_dtype, int32_t num_q_heads,
                                       float softmax_scale, int32_t window, int32_t kv_split_len,
                                       void *out, hipStream_t stream);

/* Workspace sizes in bytes for the calls above (0 when none is needed).
 * Return 0 as well for invalid arguments, which the calls then reject. */
size_t prefix_prefill_workspace_bytes(const ckv_pool_t *pool, const ckv_batch_t *batch,
                                      int32_t num_q_heads);
size_t paged_decode_workspace_bytes(const ckv_pool_t *pool, const ckv_batch_t *batch,
                                    int32_t num_q_heads, int32_t kv_split_len);

/*
 * kv_pages_offload / kv_pages_reload -- copy whole pool pages to host memory
 * and back, bit for bit: K and V pages and, for FP8_E4M3 pools, their
 * per-(page, head) scales.  With CPU offloading on, an evicted request's KV
 * cache goes to host memory and a later turn that finds it gone reloads it
 * instead of re-running prefill (Sec. 1; Sec. 3.2); the time this takes is
 * one of the two readings of Prefill-Reload(r) in the cost model (Sec. 4.1),
 * and the host-link throughput it runs at is the first quantity of the
 * offline profile (Sec. 5.2, "Offline Profile", item (1)).
 *   pages: DEVICE int32 [num_moved], pool page ids; host page i corresponds to
 *     pool page pages[i] (e.g. the first ceil(c / page_size) entries of a
 *     sequence's block-table row).  Ids outside [0, num_pages) are skipped:
 *     the pool is never touched outside its pages, and offload leaves that
 *     host page's contents unspecified.  Reload ids must be distinct (a
 *     repeated id leaves that pool page's contents unspecified).
 *   host_k, host_v: HOST memory, [num_moved][num_kv_heads][page_size]
 *     [head_dim] in kv_dtype, dense.  host_k_scale, host_v_scale: HOST fp32
 *     [num_moved][num_kv_heads], FP8_E4M3 pools only (may be NULL otherwise).
 *     Memory from hipHostMalloc (pinned) is copied asynchronously at host-link
 *     rate; pageable memory is accepted, but HIP then copies through its own
 *     bounce buffers and the call may block the calling thread.
 *   staging: device memory, 16-byte aligned, at least
 *     kv_pages_staging_bytes(pool, num_moved) bytes (the moved pages, dense),
 *     owned by the caller and free until the stream has passed the call.
 * Reload: host -> staging by hipMemcpyAsync, then a kernel scatters staging
 * page i into pool page pages[i].  Offload: a kernel gathers pool page
 * pages[i] into staging page i, then hipMemcpyAsync copies staging -> host.
 * Staging holds K pages, V pages, K scales, V scales back to back; host
 * buffers that are adjacent in that same order (host_v == host_k + K bytes,
 * and so on) move as one copy, which saves a copy's fixed cost on small
 * moves.
 * Pool pages not named in `pages` are untouched.  The host buffers may be
 * reused (reload) or read (offload) once the stream has passed the call.
 * Errors: CKV_ERR_INVALID_ARG for a NULL or unaligned pointer, num_moved < 0
 * or a move too large for one launch; CKV_ERR_WORKSPACE for a missing or
 * small staging buffer; CKV_ERR_LAUNCH when a copy or the kernel fails to
 * enqueue.  num_moved == 0 does nothing.
 */
ckv_status_t kv_pages_reload(const ckv_pool_t *pool, const int32_t *pages, int32_t num_moved,
                             const void *host_k, const void *host_v,
                             const float *host_k_scale, const float *host_v_scale,
                             void *staging, size_t staging_bytes, hipStream_t stream);
ckv_status_t kv_pages_offload(const ckv_pool_t *pool, const int32_t *pages, int32_t num_moved,
                              void *host_k, void *host_v, float *host_k_scale,
                              float *host_v_scale, void *staging, size_t staging_bytes,
                              hipStream_t stream);

/* Staging bytes for moving num_moved pages of `pool`:
 * 2 * num_moved * num_kv_heads * page_size * head_dim * sizeof(kv_dtype),
 * plus 2 * num_moved * num_kv_heads * 4 for FP8_E4M3.  0 for invalid
 * arguments or num_moved <= 0. */
size_t kv_pages_staging_bytes(const ckv_pool_t *pool, int32_t num_moved);

/*
 * ckv_validate_batch -- host-side check of the device-side contract, on HOST
 * copies of block_table (num_seqs * max_pages_per_seq entries), ctx_lens and
 * cu_q_lens (NULL for decode).  mode 0 = append/prefill (positions up to
 * ctx_lens[b] + n_b - 1 must be mapped), mode 1 = decode (up to ctx_lens[b] - 1,
 * ctx_lens[b] >= 1).  Checks page ids in range, lengths within the host bounds
 * and the table, and distinct pages across sequences when distinct_pages != 0.
 * Returns CKV_OK or CKV_ERR_INVALID_ARG.  Pure host code; needs no GPU.
 */
ckv_status_t ckv_validate_batch(const ckv_pool_t *pool, int32_t num_seqs,
                                int32_t max_pages_per_seq, const int32_t *block_table_host,
                                const int32_t *ctx_lens_host, const int32_t *cu_q_lens_host,
                                int32_t max_q_len, int32_t max_ctx_len, int32_t mode,
                                int32_t distinct_pages);

/* Human-readable name of a status code (static storage). */
const char *ckv_status_string(ckv_status_t status);

/* Library version as major * 10000 + minor * 100 + patch. */
int32_t ckv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CKV_H */
