// paged_decode_attn for bf16 queries over a bf16 or fp8-E4M3 paged pool:
// the decode kernel (one single-wave workgroup per work item, see
// decode_impl.hpp), the merge of the split-K partitions, and the host-side
// launch.
#include <algorithm>
#include <mutex>

#include "../../include/ckv.h"
#include "args.hpp"

namespace ckv {
namespace {

using namespace dc;

template <int D, bool FP8, int PS>
__global__ __launch_bounds__(64) void decode_kernel(DecodeArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds_[DCfg<D, FP8, PS>::LDS];
  decode_item<D, FP8, PS>(a, as_lds(lds_), blockIdx.x, blockIdx.y, blockIdx.z);
}

// Merge the partitions of one (sequence, query head):
// w_s = l_s 2^(m_s - M), out = sum_s w_s o_s / sum_s w_s  (m in log2 units).
template <int D>
__global__ __launch_bounds__(64) void combine_kernel(DecodeArgs a) {
  const int h = blockIdx.x;
  const int b = blockIdx.y;
  const int c = a.ctx[b];
  const int lo = a.window > 0 ? max(0, c - a.window) : 0;
  const int nsplit = (c - lo + a.split_len - 1) / a.split_len;
  if (nsplit <= 1) return;
  const size_t base = ((size_t)b * a.h_q + h) * a.max_splits;
  float M = kNegInf;
  for (int s = 0; s < nsplit; ++s) M = fmaxf(M, a.part_ml[(base + s) * 2]);
  float acc[D / 64];
#pragma unroll
  for (int k = 0; k < D / 64; ++k) acc[k] = 0.f;
  float wsum = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const float ms = a.part_ml[(base + s) * 2];
    const float ls = a.part_ml[(base + s) * 2 + 1];
    const float w = ms == kNegInf ? 0.f : ls * fast_exp2(ms - M);
    wsum += w;
    const float *po = a.part_o + (base + s) * D;
#pragma unroll
    for (int k = 0; k < D / 64; ++k) acc[k] = fmaf(w, po[threadIdx.x + 64 * k], acc[k]);
  }
  const float inv = 1.f / wsum;
  uint16_t *orow = a.out + ((size_t)b * a.h_q + h) * D;
#pragma unroll
  for (int k = 0; k < D / 64; ++k) {
    const uint32_t pk = pack_bf16x2(acc[k] * inv, 0.f);
    orow[threadIdx.x + 64 * k] = (uint16_t)(pk & 0xffffu);
  }
}

// grid.x counts splits and is padded to an odd number (the padded split
// exits at once): workgroups are dealt to the 8 XCDs round-robin in linear
// order, so with a split count that is a multiple of 8 split s of every
// (sequence, head) would land on XCD s mod 8, and the low splits, which every
// sequence has, would pile onto the same XCDs (measured: power-of-two split
// lengths ran up to 45 % slower at Llama-70B).  An odd stride rotates them.
template <int D, bool FP8>
hipError_t launch(const DecodeArgs &a, int ps, int num_seqs, hipStream_t s) {
  dim3 grid((unsigned)(a.max_splits | 1), a.h_kv * a.head_chunks, num_seqs);
  if (ps == 16)
    hipLaunchKernelGGL((decode_kernel<D, FP8, 16>), grid, dim3(64), 0, s, a);
  else
    hipLaunchKernelGGL((decode_kernel<D, FP8, 64>), grid, dim3(64), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.max_splits <= 1) return e;
  return launch_decode_merge(a, D, num_seqs, s);
}

}  // namespace

// partitions are kept to at most 256 pages (bounds the partial buffers)
int decode_max_split_len(int page_size) { return 256 * page_size; }

// Partition length for `keys` keys per sequence, at least `floor`.
static int split_len_for(const PoolView &p, const BatchView &b, int h_q, long long keys, int floor) {
  const int group = h_q / p.h_kv;
  const int head_chunks = (group + 15) / 16;
  const long long items = (long long)b.num_seqs * p.h_kv * head_chunks;
  // about 8192 work items of 128-wide heads; a 256-wide head moves twice the
  // bytes per key, so half as many of its partitions make the same work
  const long long target = p.d >= 256 ? 4096 : 8192;
  long long want = (target + items - 1) / std::max<long long>(items, 1);
  want = std::min<long long>(std::max<long long>(want, 1), 256);
  long long len = (keys + want - 1) / want;
  len = ((len + 255) / 256) * 256;
  len = std::max<long long>(len, floor);
  return (int)std::min<long long>(len, decode_max_split_len(p.ps));
}

int decode_split_len(const PoolView &p, const BatchView &b, int h_q, int requested) {
  if (requested > 0) return requested;
  return split_len_for(p, b, h_q, b.max_ctx, 512);
}

size_t decode_workspace_bytes(const PoolView &p, const BatchView &b, int h_q, int split_len) {
  const int L = decode_split_len(p, b, h_q, split_len);
  const long long splits = (b.max_ctx + L - 1) / L;
  if (splits <= 1) return 0;
  return (size_t)b.num_seqs * h_q * splits * (p.d + 2) * sizeof(float);
}

hipError_t launch_decode_merge(const DecodeArgs &a, int d, int num_seqs, hipStream_t s) {
  const dim3 grid(a.h_q, num_seqs);
  switch (d) {
    case 64: hipLaunchKernelGGL((combine_kernel<64>), grid, dim3(64), 0, s, a); break;
    case 128: hipLaunchKernelGGL((combine_kernel<128>), grid, dim3(64), 0, s, a); break;
    case 256: hipLaunchKernelGGL((combine_kernel<256>), grid, dim3(64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

void decode_args(const PoolView &p, const BatchView &b, const void *q, int h_q, float scale,
                 int window, int split_len, void *out, void *ws, DecodeArgs &a) {
  a.q = static_cast<const uint16_t *>(q);
  a.out = static_cast<uint16_t *>(out);
  a.k = static_cast<const uint8_t *>(p.k);
  a.v = static_cast<const uint8_t *>(p.v);
  a.k_scale = p.k_scale;
  a.v_scale = p.v_scale;
  a.bt = b.bt;
  a.ctx = b.ctx;
  a.max_pages = b.max_pages;
  a.k_new = a.v_new = nullptr;  // no fused append
  a.h_q = h_q;
  a.h_kv = p.h_kv;
  a.group = h_q / p.h_kv;
  a.scale_log2 = scale * kLog2e;
  a.window = window;
  a.split_len = decode_split_len(p, b, h_q, split_len);
  a.max_splits = (int)((b.max_ctx + a.split_len - 1) / a.split_len);
  if (a.max_splits < 1) a.max_splits = 1;
  if (split_len == 0 && window > 0 && window < b.max_ctx) {
    // a sliding window sees at most `window` keys: size the partitions for
    // that (down to 256 keys: a 1024-key window then still spreads over four
    // workgroups), as long as the partials still fit the workspace sized above
    const int lw = split_len_for(p, b, h_q, window, 256);
    const int sw = (window + lw - 1) / lw;
    if (sw <= a.max_splits) {
      a.split_len = lw;
      a.max_splits = sw;
    }
  }
  a.head_chunks = (a.group + 15) / 16;
  float *w = static_cast<float *>(ws);
  const size_t n_o = (size_t)b.num_seqs * h_q * a.max_splits * p.d;
  a.part_o = a.max_splits > 1 ? w : nullptr;
  a.part_ml = a.max_splits > 1 ? w + n_o : nullptr;
}

hipError_t launch_decode_bf16(const PoolView &p, const BatchView &b, const void *q, int h_q,
                              float scale, int window, int split_len, void *out, void *ws,
                              size_t ws_bytes, hipStream_t s) {
  if (b.num_seqs == 0) return hipSuccess;
  DecodeArgs a;
  decode_args(p, b, q, h_q, scale, window, split_len, out, ws, a);
  (void)ws_bytes;
  const bool fp8 = p.kv_dtype == 2;
  switch (p.d) {
    case 64:
      return fp8 ? launch<64, true>(a, p.ps, b.num_seqs, s) : launch<64, false>(a, p.ps, b.num_seqs, s);
    case 128:
      return fp8 ? launch<128, true>(a, p.ps, b.num_seqs, s) : launch<128, false>(a, p.ps, b.num_seqs, s);
    case 256:
      return fp8 ? launch<256, true>(a, p.ps, b.num_seqs, s) : launch<256, false>(a, p.ps, b.num_seqs, s);
  }
  return hipErrorInvalidValue;
}

// ------------------------------------------------- allocation-free decode
// The split-K partials of paged_decode_attn_noalloc live in this file-scope
// device array instead of a caller workspace.  Each GPU the library runs on
// holds its own copy until the process ends; every call on a GPU shares it.
// On the host, `scratch` names a host-side stand-in, never the device copy:
// host code uses only the device address that hipGetSymbolAddress returns,
// looked up once per device (with that device current) and kept here.
namespace {
__device__ __align__(256) uint8_t scratch[CKV_DECODE_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_dev[kMaxDevices];  // device address of `scratch` per device
}  // namespace

hipError_t decode_scratch(void **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_dev[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    scratch_dev[dev] = p;
  }
  *ptr = scratch_dev[dev];
  return hipSuccess;
}

}  // namespace ckv
