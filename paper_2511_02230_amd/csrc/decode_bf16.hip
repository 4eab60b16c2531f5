// paged_decode_attn for bf16 queries over a bf16 or fp8-E4M3 paged pool.
//
// Split-K: the context of each sequence is cut into partitions of L logical
// positions; one single-wave workgroup handles (partition, KV head, <=16
// query heads of its group, sequence) and reads every K/V byte of its range
// exactly once for all of those heads.  The heads are packed into the N
// dimension of v_mfma_f32_16x16x32_bf16 (padded to 16):
//   S^T (16 keys x 16 heads) = K (16 keys x 32 d) * Q^T, K fed straight from
//   global memory into the MFMA operand (16 contiguous bytes per lane);
//   O^T (16 d x 16 heads) += Vt (16 d x 32 keys) * P^T, V staged transposed
//   through LDS.
// Keys are fed to the first product in a permuted order (rho below) so that
// the 8 probabilities a lane holds are the 8 consecutive keys it supplies as
// the B operand of the second.  A partition writes (m, l, o) partials in
// fp32 unless it is its sequence's only one, in which case it writes the
// output; the combine kernel merges multi-partition sequences.
#include <algorithm>

#include "common.hpp"
#include "launch.hpp"

namespace ckv {
namespace {

struct DecodeArgs {
  const uint16_t *q;
  uint16_t *out;
  const uint8_t *k, *v;
  const float *k_scale, *v_scale;
  const int32_t *bt, *ctx;
  int32_t max_pages, h_q, h_kv, group, ps;
  float scale_log2;
  int32_t window;
  int32_t split_len, max_splits, head_chunks;
  float *part_o;   // [B][H_q][max_splits][D]
  float *part_ml;  // [B][H_q][max_splits][2]
};

constexpr int KB = 32;  // keys per iteration

// d offset of the 8 k-slots a lane (quarter q4) supplies at step `step` of
// the QK^T contraction.  bf16: 16 contiguous bytes per step; fp8: two
// consecutive steps read one 16-byte run of codes.
template <bool FP8>
__device__ __forceinline__ int qk_d0(int step, int q4) {
  if constexpr (FP8) return 64 * (step >> 1) + 16 * q4 + 8 * (step & 1);
  return 32 * step + 8 * q4;
}

template <int D, bool FP8>
__global__ __launch_bounds__(64) void decode_kernel(DecodeArgs a) {
  constexpr int DS = D / 32;   // QK^T k-steps
  constexpr int DT = D / 16;   // output d-tiles
  constexpr int CH = D / 8;    // 8-element chunks per row
  constexpr int EK = FP8 ? 1 : 2;
  constexpr int VROW = KB * 2;  // bytes per Vt row (32 bf16 keys)
  constexpr int VGROUPS = (KB / 4) * CH;
  constexpr int VPL = VGROUPS / 64;  // (4 keys x 8 d) groups per lane
  static_assert(VPL * 64 == VGROUPS, "V staging must tile evenly");
  __shared__ __attribute__((aligned(16))) uint8_t vt[D * VROW];

  const int split = blockIdx.x;
  const int g = blockIdx.y / a.head_chunks;
  const int hc = blockIdx.y - g * a.head_chunks;
  const int b = blockIdx.z;
  const int c = a.ctx[b];
  const int L = a.split_len;
  const int nsplit = (c + L - 1) / L;
  if (split >= nsplit) return;
  const int lo = a.window > 0 ? max(0, c - a.window) : 0;
  const int kbeg = max(lo, split * L);
  const int kend = min(c, (split + 1) * L);
  const int32_t *bt = a.bt + (size_t)b * a.max_pages;

  const int lane = threadIdx.x;
  const int col = lane & 15, q4 = lane >> 4;
  const int head = hc * 16 + col;
  const bool hvalid = head < a.group;
  const int qh = g * a.group + (hvalid ? head : 0);
  const size_t qoff = ((size_t)b * a.h_q + qh) * D;

  bf16x8 qf[DS];
#pragma unroll
  for (int s = 0; s < DS; ++s) {
    u32x4 x = {0u, 0u, 0u, 0u};
    if (hvalid) x = ld<u32x4>(a.q + qoff + qk_d0<FP8>(s, q4));
    qf[s] = as_bf16x8(x);
  }

  const size_t head_stride = (size_t)a.ps * D * EK;
  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{};
  float m = kNegInf, l = 0.f;

  for (int k0 = kbeg - (kbeg % KB); k0 < kend; k0 += KB) {
    // ---- S^T tiles: row m of tile tt is key rho(m) = 8(m/4) + 4tt + m%4
    f32x4 s[2];
    float ksc[2], vsc[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int kp = k0 + 8 * (col >> 2) + 4 * tt + (col & 3);
      const bool kv = kp >= kbeg && kp < kend;
      const uint8_t *row = nullptr;
      if (kv) row = a.k + ((size_t)bt[kp / a.ps] * a.h_kv + g) * head_stride + (size_t)(kp % a.ps) * D * EK;
      s[tt] = f32x4{};
      if constexpr (FP8) {
#pragma unroll
        for (int s2 = 0; s2 < DS; s2 += 2) {
          u32x4 x = {0u, 0u, 0u, 0u};
          if (kv) x = ld<u32x4>(row + qk_d0<true>(s2, q4));
          const u32x2 a0 = fp8x4_to_bf16x4(x.x), a1 = fp8x4_to_bf16x4(x.y);
          const u32x2 b0 = fp8x4_to_bf16x4(x.z), b1 = fp8x4_to_bf16x4(x.w);
          s[tt] = mfma16x16x32(as_bf16x8(u32x4{a0.x, a0.y, a1.x, a1.y}), qf[s2], s[tt]);
          s[tt] = mfma16x16x32(as_bf16x8(u32x4{b0.x, b0.y, b1.x, b1.y}), qf[s2 + 1], s[tt]);
        }
      } else {
#pragma unroll
        for (int st_ = 0; st_ < DS; ++st_) {
          u32x4 x = {0u, 0u, 0u, 0u};
          if (kv) x = ld<u32x4>(row + 2 * qk_d0<false>(st_, q4));
          s[tt] = mfma16x16x32(as_bf16x8(x), qf[st_], s[tt]);
        }
      }
      // the 4 keys this lane receives for tile tt: k0 + 8 q4 + 4 tt + j
      const int kg = k0 + 8 * q4 + 4 * tt;
      ksc[tt] = a.scale_log2;
      vsc[tt] = 1.f;
      if constexpr (FP8) {
        float sk = 0.f, sv = 0.f;
        if (kg < kend) {
          const size_t idx = (size_t)bt[kg / a.ps] * a.h_kv + g;
          sk = a.k_scale[idx];
          sv = a.v_scale[idx];
        }
        ksc[tt] = a.scale_log2 * sk;
        vsc[tt] = sv;
      }
    }

    // ---- stage V transposed: Vt[d][key], 16-byte chunks swizzled by d
    __syncthreads();
#pragma unroll
    for (int r = 0; r < VPL; ++r) {
      const int id = lane + 64 * r;
      const int kg = id / CH, cc = id % CH;
      u32x4 row4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int kp = k0 + 4 * kg + e;
        u32x4 x = {0u, 0u, 0u, 0u};
        if (kp >= kbeg && kp < kend) {
          const uint8_t *src = a.v + ((size_t)bt[kp / a.ps] * a.h_kv + g) * head_stride +
                               (size_t)(kp % a.ps) * D * EK + cc * 8 * EK;
          if constexpr (FP8) {
            const u32x2 y = ld<u32x2>(src);
            const u32x2 lo2 = fp8x4_to_bf16x4(y.x), hi2 = fp8x4_to_bf16x4(y.y);
            x = u32x4{lo2.x, lo2.y, hi2.x, hi2.y};
          } else {
            x = ld<u32x4>(src);
          }
        }
        row4[e] = x;
      }
      const int kchunk = kg >> 1, hv = kg & 1;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const u32x2 even = {pack_lo16(row4[0][w], row4[1][w]), pack_lo16(row4[2][w], row4[3][w])};
        const u32x2 odd = {pack_hi16(row4[0][w], row4[1][w]), pack_hi16(row4[2][w], row4[3][w])};
        const int d0 = 8 * cc + 2 * w;
        st<u32x2>(vt + d0 * VROW + ((kchunk ^ ((d0 >> 1) & 3)) << 4) + 8 * hv, even);
        st<u32x2>(vt + (d0 + 1) * VROW + ((kchunk ^ (((d0 + 1) >> 1) & 3)) << 4) + 8 * hv, odd);
      }
    }

    // ---- scale, mask, online softmax (lane = one head, 8 keys per block)
    float mx = kNegInf;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kp = k0 + 8 * q4 + 4 * tt + j;
        float x = s[tt][j] * ksc[tt];
        x = (kp >= kbeg && kp < kend) ? x : kNegInf;
        s[tt][j] = x;
        mx = fmaxf(mx, x);
      }
    }
    mx = fmaxf(mx, shfl_xor(mx, 16));
    mx = fmaxf(mx, shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx);
    const float m_use = m_new == kNegInf ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    m = m_new;
    l *= alpha;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
    float p[8];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float e = fast_exp2(s[tt][j] - m_use);
        l += e;
        p[4 * tt + j] = FP8 ? e * vsc[tt] : e;
      }
    }
    const u32x4 pb = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                      pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
    __syncthreads();
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int d = 16 * dt + col;
      const u32x4 vx = ld<u32x4>(vt + d * VROW + ((q4 ^ ((d >> 1) & 3)) << 4));
      o[dt] = mfma16x16x32(as_bf16x8(vx), as_bf16x8(pb), o[dt]);
    }
  }

  l += shfl_xor(l, 16);
  l += shfl_xor(l, 32);
  if (!hvalid) return;
  // lane holds head `qh`, d = 16 dt + 4 q4 + 0..3
  if (nsplit == 1) {
    const float inv = 1.f / l;
    uint16_t *orow = a.out + qoff;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const u32x2 w = {pack_bf16x2(o[dt][0] * inv, o[dt][1] * inv),
                       pack_bf16x2(o[dt][2] * inv, o[dt][3] * inv)};
      st<u32x2>(orow + 16 * dt + 4 * q4, w);
    }
    return;
  }
  const size_t pidx = ((size_t)b * a.h_q + qh) * a.max_splits + split;
  const float inv = l > 0.f ? 1.f / l : 0.f;
  float *po = a.part_o + pidx * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) st<f32x4>(po + 16 * dt + 4 * q4, o[dt] * inv);
  if (q4 == 0) st<f32x2>(a.part_ml + pidx * 2, f32x2{m, l});
}

// Merge the partitions of one (sequence, query head):
// w_s = l_s 2^(m_s - M), out = sum_s w_s o_s / sum_s w_s  (m in log2 units).
template <int D>
__global__ __launch_bounds__(64) void combine_kernel(DecodeArgs a) {
  const int h = blockIdx.x;
  const int b = blockIdx.y;
  const int c = a.ctx[b];
  const int nsplit = (c + a.split_len - 1) / a.split_len;
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

template <int D, bool FP8>
hipError_t launch(const DecodeArgs &a, int num_seqs, hipStream_t s) {
  dim3 grid(a.max_splits, a.h_kv * a.head_chunks, num_seqs);
  hipLaunchKernelGGL((decode_kernel<D, FP8>), grid, dim3(64), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.max_splits <= 1) return e;
  hipLaunchKernelGGL((combine_kernel<D>), dim3(a.h_q, num_seqs), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace

int decode_split_len(const PoolView &p, const BatchView &b, int h_q, int requested) {
  if (requested > 0) return requested;
  const int group = h_q / p.h_kv;
  const int head_chunks = (group + 15) / 16;
  const long long items = (long long)b.num_seqs * p.h_kv * head_chunks;
  long long want = (16384 + items - 1) / std::max<long long>(items, 1);
  want = std::min<long long>(std::max<long long>(want, 1), 256);
  long long len = (b.max_ctx + want - 1) / want;
  len = ((len + 63) / 64) * 64;
  return (int)std::max<long long>(len, 256);
}

size_t decode_workspace_bytes(const PoolView &p, const BatchView &b, int h_q, int split_len) {
  const int L = decode_split_len(p, b, h_q, split_len);
  const long long splits = (b.max_ctx + L - 1) / L;
  if (splits <= 1) return 0;
  return (size_t)b.num_seqs * h_q * splits * (p.d + 2) * sizeof(float);
}

hipError_t launch_decode_bf16(const PoolView &p, const BatchView &b, const void *q, int h_q,
                              float scale, int window, int split_len, void *out, void *ws,
                              size_t ws_bytes, hipStream_t s) {
  if (b.num_seqs == 0) return hipSuccess;
  DecodeArgs a;
  a.q = static_cast<const uint16_t *>(q);
  a.out = static_cast<uint16_t *>(out);
  a.k = static_cast<const uint8_t *>(p.k);
  a.v = static_cast<const uint8_t *>(p.v);
  a.k_scale = p.k_scale;
  a.v_scale = p.v_scale;
  a.bt = b.bt;
  a.ctx = b.ctx;
  a.max_pages = b.max_pages;
  a.h_q = h_q;
  a.h_kv = p.h_kv;
  a.group = h_q / p.h_kv;
  a.ps = p.ps;
  a.scale_log2 = scale * kLog2e;
  a.window = window;
  a.split_len = decode_split_len(p, b, h_q, split_len);
  a.max_splits = (int)((b.max_ctx + a.split_len - 1) / a.split_len);
  if (a.max_splits < 1) a.max_splits = 1;
  a.head_chunks = (a.group + 15) / 16;
  float *w = static_cast<float *>(ws);
  const size_t n_o = (size_t)b.num_seqs * h_q * a.max_splits * p.d;
  a.part_o = a.max_splits > 1 ? w : nullptr;
  a.part_ml = a.max_splits > 1 ? w + n_o : nullptr;
  (void)ws_bytes;
  const bool fp8 = p.kv_dtype == 2;
  switch (p.d) {
    case 64:
      return fp8 ? launch<64, true>(a, b.num_seqs, s) : launch<64, false>(a, b.num_seqs, s);
    case 128:
      return fp8 ? launch<128, true>(a, b.num_seqs, s) : launch<128, false>(a, b.num_seqs, s);
    case 256:
      return fp8 ? launch<256, true>(a, b.num_seqs, s) : launch<256, false>(a, b.num_seqs, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace ckv
