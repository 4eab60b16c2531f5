// kv_append: scatter the new turn's K/V rows into their pool slots through
// the block table (bit copy, or bf16 -> fp8 E4M3FN with a per-(page, head)
// scale).  HBM-bound: each 16-byte input chunk is read once and written once.
#include "common.hpp"
#include "launch.hpp"

namespace ckv {
namespace {

struct AppendArgs {
  const uint8_t *k_new, *v_new;
  uint8_t *k_pool, *v_pool;
  const float *k_scale, *v_scale;
  const int32_t *bt, *ctx, *cu;
  int32_t max_pages, h, ps;
  int32_t units;       // 16-byte input chunks per (token, head) row
  int32_t in_row, out_row;  // bytes per (token, head) row in the input / pool
  int32_t tok_per_block;
  // log2 of units, h and ps when all three are powers of two (else -1): the
  // chunk index then splits by shifts and masks instead of divisions
  int32_t lg_units, lg_h, lg_ps;
};

// Quantize 8 bf16 values (one 16-byte chunk) to 8 E4M3FN codes:
// r = x / s (IEEE binary32 division), clamp to +-448, round to nearest even.
__device__ __forceinline__ u32x2 quantize8(u32x4 x, float s) {
  float f[8];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    f[2 * w] = bf16_lo(x[w]);
    f[2 * w + 1] = bf16_hi(x[w]);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float r = f[i] / s;
    float c = fminf(fmaxf(r, -448.0f), 448.0f);
    f[i] = (r != r) ? r : c;
  }
  u32x2 out;
  int w0 = __builtin_amdgcn_cvt_pk_fp8_f32(f[0], f[1], 0, false);
  w0 = __builtin_amdgcn_cvt_pk_fp8_f32(f[2], f[3], w0, true);
  int w1 = __builtin_amdgcn_cvt_pk_fp8_f32(f[4], f[5], 0, false);
  w1 = __builtin_amdgcn_cvt_pk_fp8_f32(f[6], f[7], w1, true);
  out.x = (uint32_t)w0;
  out.y = (uint32_t)w1;
  return out;
}

// Chunk u of a block's rows -> token (relative to t0), K (0) or V (1),
// head and 16-byte chunk: u = ((t * 2 + kv) * h + hh) * units + c.  POW2:
// units, h and ps are powers of two (shifts and masks instead of divisions).
template <bool POW2>
__device__ __forceinline__ void split_unit(const AppendArgs &a, int u, int &t, int &kv, int &hh, int &c) {
  if constexpr (POW2) {
    const int lu = a.lg_units, lh = a.lg_h;
    c = u & (a.units - 1);
    hh = (u >> lu) & (a.h - 1);
    kv = (u >> (lu + lh)) & 1;
    t = u >> (lu + lh + 1);
  } else {
    const int per_kv = a.h * a.units;
    t = u / (2 * per_kv);
    int r = u - t * 2 * per_kv;
    kv = r / per_kv;
    r -= kv * per_kv;
    hh = r / a.units;
    c = r - hh * a.units;
  }
}

// Grid: x = token chunks of one sequence, y = sequence.  Each thread moves
// 16-byte chunks; consecutive threads cover consecutive chunks of a row, and
// a (token, head) row is contiguous both in the packed input and in its page.
// A thread takes its chunks NB at a time: all loads (and page ids, then the
// fp8 scales) first, then the stores, so the batch costs one round trip to
// memory rather than one per chunk.  V addresses are K addresses plus the
// V - K distance: a per-lane choice between the two pointer arguments would
// be compiled as loads from the argument segment.
template <bool FP8, bool POW2>
__device__ __forceinline__ void append_block(const AppendArgs &a, int q0, int t0, int P, int total,
                                             const int32_t *bt) {
  constexpr int NB = 4;
  const ptrdiff_t in_vk = a.v_new - a.k_new;
  const ptrdiff_t pool_vk = a.v_pool - a.k_pool;
  const ptrdiff_t sc_vk = FP8 ? a.v_scale - a.k_scale : 0;
  for (int u0 = threadIdx.x; u0 < total; u0 += NB * blockDim.x) {
    u32x4 x[NB];
    int pg[NB], t[NB], kv[NB], hh[NB], c[NB];
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      const int u = u0 + k * blockDim.x;
      if (u < total) {
        split_unit<POW2>(a, u, t[k], kv[k], hh[k], c[k]);
        t[k] += t0;
        const int pos = P + t[k];
        pg[k] = bt[POW2 ? pos >> a.lg_ps : pos / a.ps];
        x[k] = ld<u32x4>(a.k_new + (kv[k] ? in_vk : 0) + ((size_t)(q0 + t[k]) * a.h + hh[k]) * a.in_row + c[k] * 16);
      }
    }
    float sc[NB];
    if constexpr (FP8) {
#pragma unroll
      for (int k = 0; k < NB; ++k)
        if (u0 + k * (int)blockDim.x < total) sc[k] = (a.k_scale + (kv[k] ? sc_vk : 0))[(size_t)pg[k] * a.h + hh[k]];
    }
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      if (u0 + k * (int)blockDim.x < total) {
        const int pos = P + t[k];
        const int slot = POW2 ? pos & (a.ps - 1) : pos - (pos / a.ps) * a.ps;
        uint8_t *dst = a.k_pool + (kv[k] ? pool_vk : 0) + (((size_t)pg[k] * a.h + hh[k]) * a.ps + slot) * a.out_row;
        if constexpr (!FP8)
          st<u32x4>(dst + c[k] * 16, x[k]);
        else
          st<u32x2>(dst + c[k] * 8, quantize8(x[k], sc[k]));
      }
    }
  }
}

template <bool FP8>
__global__ __launch_bounds__(256) void kv_append_kernel(AppendArgs a) {
  const int b = blockIdx.y;
  const int q0 = a.cu[b];
  const int n = a.cu[b + 1] - q0;
  const int t0 = blockIdx.x * a.tok_per_block;
  if (t0 >= n) return;
  const int P = a.ctx[b];
  const int tcount = min(a.tok_per_block, n - t0);
  const int total = tcount * 2 * a.h * a.units;
  const int32_t *bt = a.bt + (size_t)b * a.max_pages;
  if (a.lg_units >= 0)
    append_block<FP8, true>(a, q0, t0, P, total, bt);
  else
    append_block<FP8, false>(a, q0, t0, P, total, bt);
}

}  // namespace

hipError_t launch_kv_append(const PoolView &p, const BatchView &b, const void *k_new,
                            const void *v_new, int in_dtype, hipStream_t s) {
  if (b.num_seqs == 0 || b.max_q == 0 || b.total_q == 0) return hipSuccess;
  const int e_in = in_dtype == 0 ? 4 : 2;
  const bool fp8 = p.kv_dtype == 2;
  const int e_out = p.kv_dtype == 0 ? 4 : (p.kv_dtype == 1 ? 2 : 1);
  AppendArgs a;
  a.k_new = static_cast<const uint8_t *>(k_new);
  a.v_new = static_cast<const uint8_t *>(v_new);
  a.k_pool = static_cast<uint8_t *>(p.k);
  a.v_pool = static_cast<uint8_t *>(p.v);
  a.k_scale = p.k_scale;
  a.v_scale = p.v_scale;
  a.bt = b.bt;
  a.ctx = b.ctx;
  a.cu = b.cu_q;
  a.max_pages = b.max_pages;
  a.h = p.h_kv;
  a.ps = p.ps;
  a.in_row = p.d * e_in;
  a.out_row = p.d * e_out;
  a.units = a.in_row / 16;
  const int per_tok = 2 * p.h_kv * a.units;
  a.tok_per_block = per_tok >= 1024 ? 1 : 1024 / per_tok;
  auto lg = [](int x) {
    int l = 0;
    while ((1 << l) < x) ++l;
    return (1 << l) == x ? l : -1;
  };
  a.lg_units = lg(a.units);
  a.lg_h = lg(a.h);
  a.lg_ps = lg(a.ps);
  if (a.lg_h < 0 || a.lg_ps < 0) a.lg_units = -1;
  dim3 grid((b.max_q + a.tok_per_block - 1) / a.tok_per_block, b.num_seqs);
  if (fp8)
    hipLaunchKernelGGL(kv_append_kernel<true>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(kv_append_kernel<false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ckv
