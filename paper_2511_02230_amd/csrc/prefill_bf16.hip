// prefix_prefill_attn for bf16 queries over a bf16 or fp8-E4M3 paged pool:
// the prefill kernel (one workgroup per row tile, see prefill_impl.hpp), the
// merge of key partitions, and the host-side launch.
#include <algorithm>

#include "args.hpp"

namespace ckv {
namespace {

using namespace pf;

template <int D, int BN, bool FP8, int PS>
__global__ __launch_bounds__(kThreads, D >= 256 ? 1 : 2) void prefill_kernel(PrefillArgs a) {
  // K ring (2 stages), V ring (2 stages), fp8: widened K and V blocks
  __shared__ __attribute__((aligned(1024))) uint8_t lds_[Cfg<D, BN, FP8, PS>::LDS];
  // grid (H_kv * splits, tiles, B): workgroups are dealt to the XCDs
  // round-robin in linear order, so with 8 KV heads every row tile of one
  // (sequence, KV head) lands on the same XCD, next to its neighbours in
  // time, and the tiles streaming the same K/V share that XCD's L2
  prefill_tile<D, BN, FP8, PS>(a, as_lds(lds_), blockIdx.x, blockIdx.y, blockIdx.z);
}

// Merge the key partitions of one (token, head) row:
// w_s = l_s 2^(m_s - M), out = sum_s w_s o_s / sum_s w_s  (m in log2 units).
template <int D>
__global__ __launch_bounds__(64) void combine_kernel(PrefillArgs a) {
  const size_t row = blockIdx.x;
  const size_t base = row * a.splits;
  float M = kNegInf;
  for (int s = 0; s < a.splits; ++s) M = fmaxf(M, a.part_ml[(base + s) * 2]);
  float acc[D / 64];
#pragma unroll
  for (int k = 0; k < D / 64; ++k) acc[k] = 0.f;
  float wsum = 0.f;
  for (int s = 0; s < a.splits; ++s) {
    const float ms = a.part_ml[(base + s) * 2];
    const float ls = a.part_ml[(base + s) * 2 + 1];
    const float w = ms == kNegInf ? 0.f : ls * fast_exp2(ms - M);
    wsum += w;
    if (w == 0.f) continue;  // empty partition: its o was never written
    const float *po = a.part_o + (base + s) * D;
#pragma unroll
    for (int k = 0; k < D / 64; ++k) acc[k] = fmaf(w, po[threadIdx.x + 64 * k], acc[k]);
  }
  const float inv = 1.f / wsum;
  uint16_t *orow = a.out + row * D;
#pragma unroll
  for (int k = 0; k < D / 64; ++k) {
    const uint32_t pk = pack_bf16x2(acc[k] * inv, 0.f);
    orow[threadIdx.x + 64 * k] = (uint16_t)(pk & 0xffffu);
  }
}

template <int D, int BN, bool FP8>
hipError_t launch(const PrefillArgs &a, int ps, int h_kv, int num_seqs, int total_q, hipStream_t s) {
  dim3 grid(h_kv * a.splits, a.tiles, num_seqs);
  if (ps == 16)
    hipLaunchKernelGGL((prefill_kernel<D, BN, FP8, 16>), grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((prefill_kernel<D, BN, FP8, 64>), grid, dim3(kThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits <= 1) return e;
  return launch_prefill_merge(a, D, total_q, s);
}

// Keys per block of the kernel instantiated for (D, fp8).
int prefill_block_keys(int d, bool fp8) { return d >= 256 && fp8 ? 32 : 64; }

}  // namespace

int prefill_rows_per_tile() { return kRows; }

// Key partitions per row tile (small batches only; see below).
void prefill_splits(const PoolView &p, const BatchView &b, int h_q, int *splits, int *split_len) {
  const int group = h_q / p.h_kv;
  const long long tiles = ((long long)b.max_q * group + kRows - 1) / kRows;
  const long long items = tiles * p.h_kv * b.num_seqs;
  const long long slots = (p.d >= 256 ? 1 : 2) * 256;
  const long long max_kv = (long long)b.max_ctx + b.max_q;
  const int bn = prefill_block_keys(p.d, p.kv_dtype == 2);
  // Each split costs every row an fp32 (D + 2)-float partial, written and
  // read back by the merge, which a short key range does not repay: at least
  // 2048 keys per partition, at most 32 partitions.  Among those, take the
  // count with the fewest workgroup waves per unit of work (ties and gains
  // under 3 % to fewer partitions): 128 tiles on 512 slots take 4, 384 take
  // 4 (3 full waves instead of one 3/4-full wave of 4x longer ones), 768
  // take 2 (3 waves instead of 2, each half as long).  Batches of 4 waves or
  // more keep one partition.
  long long s = 1;
  if (items > 0 && items < 4 * slots) {
    const long long smax = std::min<long long>(32, (max_kv + 2047) / 2048);
    double best = (double)((items + slots - 1) / slots);
    for (long long c = 2; c <= smax; ++c) {
      const double w = (double)((items * c + slots - 1) / slots) / (double)c;
      if (w < 0.97 * best) {
        best = w;
        s = c;
      }
    }
  }
  long long len = (max_kv + s - 1) / s;
  len = (len + bn - 1) / bn * bn;
  if (len < bn) len = bn;
  *split_len = (int)len;
  *splits = (int)((max_kv + len - 1) / len);
  if (*splits < 1) *splits = 1;
}

size_t prefill_workspace_bytes(const PoolView &p, const BatchView &b, int h_q) {
  int splits, len;
  prefill_splits(p, b, h_q, &splits, &len);
  if (splits <= 1) return 0;
  return (size_t)b.total_q * h_q * splits * (p.d + 2) * sizeof(float);
}

hipError_t launch_prefill_merge(const PrefillArgs &a, int d, int total_q, hipStream_t s) {
  const dim3 grid((unsigned)total_q * a.h_q);
  switch (d) {
    case 64: hipLaunchKernelGGL((combine_kernel<64>), grid, dim3(64), 0, s, a); break;
    case 128: hipLaunchKernelGGL((combine_kernel<128>), grid, dim3(64), 0, s, a); break;
    case 256: hipLaunchKernelGGL((combine_kernel<256>), grid, dim3(64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t prefill_args(const PoolView &p, const BatchView &b, const void *q, int h_q, float scale,
                        int window, void *out, void *ws, PrefillArgs &a) {
  a.q = static_cast<const uint16_t *>(q);
  a.out = static_cast<uint16_t *>(out);
  a.k = static_cast<const uint8_t *>(p.k);
  a.v = static_cast<const uint8_t *>(p.v);
  a.k_scale = p.k_scale;
  a.v_scale = p.v_scale;
  a.bt = b.bt;
  a.ctx = b.ctx;
  a.cu = b.cu_q;
  a.k_new = a.v_new = nullptr;  // no fused append
  a.num_seqs = b.num_seqs;
  a.max_pages = b.max_pages;
  a.h_q = h_q;
  a.h_kv = p.h_kv;
  a.group = h_q / p.h_kv;
  a.scale_log2 = scale * kLog2e;
  a.window = window;
  const long long rows = (long long)b.max_q * a.group;
  a.tiles = (int)((rows + kRows - 1) / kRows);
  if (a.tiles > 65535) return hipErrorInvalidConfiguration;  // grid.y limit
  prefill_splits(p, b, h_q, &a.splits, &a.split_len);
  float *w = static_cast<float *>(ws);
  a.part_o = a.splits > 1 ? w : nullptr;
  a.part_ml = a.splits > 1 ? w + (size_t)b.total_q * h_q * a.splits * p.d : nullptr;
  return hipSuccess;
}

hipError_t launch_prefill_bf16(const PoolView &p, const BatchView &b, const void *q, int h_q,
                               float scale, int window, void *out, void *ws, hipStream_t s) {
  if (b.num_seqs == 0 || b.max_q == 0 || b.total_q == 0) return hipSuccess;
  PrefillArgs a;
  const hipError_t e = prefill_args(p, b, q, h_q, scale, window, out, ws, a);
  if (e != hipSuccess) return e;
  const bool fp8 = p.kv_dtype == 2;
  const int tq = b.total_q;
  switch (p.d) {
    case 64:
      return fp8 ? launch<64, 64, true>(a, p.ps, p.h_kv, b.num_seqs, tq, s)
                 : launch<64, 64, false>(a, p.ps, p.h_kv, b.num_seqs, tq, s);
    case 128:
      return fp8 ? launch<128, 64, true>(a, p.ps, p.h_kv, b.num_seqs, tq, s)
                 : launch<128, 64, false>(a, p.ps, p.h_kv, b.num_seqs, tq, s);
    case 256:
      return fp8 ? launch<256, 32, true>(a, p.ps, p.h_kv, b.num_seqs, tq, s)
                 : launch<256, 64, false>(a, p.ps, p.h_kv, b.num_seqs, tq, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace ckv
