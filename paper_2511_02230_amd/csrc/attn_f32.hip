// fp32 paged attention (queries and pool in binary32) for prefill and decode.
// One wavefront per (query row, query head): 64 keys per step, one key per
// lane for the scores, then the wave accumulates p * V with lane = head-dim
// column.  Online softmax in fp32.  Meant for small fp32 layers; the bf16 and
// fp8 pools go through the MFMA kernels.
#include "common.hpp"
#include "launch.hpp"

namespace ckv {
namespace {

struct F32Args {
  const float *q;
  float *out;
  const float *k, *v;
  const int32_t *bt, *ctx, *cu;
  int32_t max_pages, h_q, h_kv, group, ps, d;
  float scale;
  int32_t window;
  int32_t decode;
};

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// Grid: x = row of the sequence (decode: 0), y = query head, z = sequence.
__global__ __launch_bounds__(64) void attn_f32_kernel(F32Args a) {
  const int b = blockIdx.z;
  const int h = blockIdx.y;
  const int lane = threadIdx.x;
  int row, pos;
  if (a.decode) {
    row = b;
    pos = a.ctx[b] - 1;
  } else {
    const int q0 = a.cu[b];
    const int n = a.cu[b + 1] - q0;
    const int t = blockIdx.x;
    if (t >= n) return;
    row = q0 + t;
    pos = a.ctx[b] + t;
  }
  const int g = h / a.group;
  const int D = a.d;
  const int lo = a.window > 0 ? max(0, pos - a.window + 1) : 0;
  const int32_t *bt = a.bt + (size_t)b * a.max_pages;
  __shared__ float qs[256];
  const float *qrow = a.q + ((size_t)row * a.h_q + h) * D;
  for (int d = lane; d < D; d += 64) qs[d] = qrow[d];
  __syncthreads();

  float m = kNegInf, l = 0.f;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int j0 = lo; j0 <= pos; j0 += 64) {
    const int j = j0 + lane;
    float s = kNegInf;
    if (j <= pos) {
      const int page = bt[j / a.ps];
      const float *kr = a.k + (((size_t)page * a.h_kv + g) * a.ps + (j % a.ps)) * D;
      float dot = 0.f;
      for (int d = 0; d < D; ++d) dot = fmaf(qs[d], kr[d], dot);
      s = dot * a.scale;
    }
    const float m_new = fmaxf(m, wave_max(s));  // key j0 is visible, so finite
    const float p = (j <= pos) ? expf(s - m_new) : 0.f;
    const float alpha = expf(m - m_new);
    l = l * alpha + wave_sum(p);
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[k] *= alpha;
    const int cnt = min(64, pos - j0 + 1);
    for (int jj = 0; jj < cnt; ++jj) {
      const float pj = __shfl(p, jj);
      const int jp = j0 + jj;
      const int page = bt[jp / a.ps];
      const float *vr = a.v + (((size_t)page * a.h_kv + g) * a.ps + (jp % a.ps)) * D;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int d = lane + 64 * k;
        if (d < D) acc[k] = fmaf(pj, vr[d], acc[k]);
      }
    }
    m = m_new;
  }
  float *orow = a.out + ((size_t)row * a.h_q + h) * D;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int d = lane + 64 * k;
    if (d < D) orow[d] = acc[k] / l;
  }
}

}  // namespace

hipError_t launch_attn_f32(const PoolView &p, const BatchView &b, const float *q, int h_q,
                           float scale, int window, bool decode, float *out, hipStream_t s) {
  if (b.num_seqs == 0) return hipSuccess;
  if (!decode && (b.max_q == 0 || b.total_q == 0)) return hipSuccess;
  F32Args a;
  a.q = q;
  a.out = out;
  a.k = static_cast<const float *>(p.k);
  a.v = static_cast<const float *>(p.v);
  a.bt = b.bt;
  a.ctx = b.ctx;
  a.cu = b.cu_q;
  a.max_pages = b.max_pages;
  a.h_q = h_q;
  a.h_kv = p.h_kv;
  a.group = h_q / p.h_kv;
  a.ps = p.ps;
  a.d = p.d;
  a.scale = scale;
  a.window = window;
  a.decode = decode ? 1 : 0;
  dim3 grid(decode ? 1 : b.max_q, h_q, b.num_seqs);
  hipLaunchKernelGGL(attn_f32_kernel, grid, dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace ckv
