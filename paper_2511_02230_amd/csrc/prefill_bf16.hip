// prefix_prefill_attn for bf16 queries over a bf16 or fp8-E4M3 paged pool.
//
// Work item: one workgroup (4 waves) = 128 consecutive "rows" of one
// (sequence, KV head), a row being a (new-turn token, query head of the
// group) pair flattened as R = t * G + hh.  Packing the G query heads of a
// KV head into the M dimension lets every K/V byte staged in LDS serve all
// of them and keeps the causal diagonal narrow (128 / G tokens per tile).
//
// Per block of BN keys (read through the block table):
//   * K rows are staged row-major in LDS (16-byte chunks XOR-swizzled by key),
//     V is staged transposed (Vt[d][key], chunks swizzled by d) so both MFMA
//     operands are read with 16-byte LDS loads; fp8 codes are widened to bf16
//     (exactly) on the way in.
//   * Each wave computes S^T = K Q^T for its 32 rows with
//     v_mfma_f32_32x32x16_bf16: the wave's lane owns one query row (a column
//     of S^T), so row max / row sum are in-lane except for one exchange
//     between the two half-waves.  K rows are fed to the MFMA in a permuted
//     order (pi below) chosen so that the probabilities a lane holds are
//     exactly the 8 consecutive keys it must supply as the B operand of
//     O^T += Vt P^T: no shuffles between the two products.
//   * Online softmax in fp32 (base-2 exponentials, log2(e) folded into the
//     scale); masking only on blocks that straddle the causal diagonal or
//     the window edge.
// The next block's global loads are issued before the current block's
// MFMAs (register prefetch); LDS is single-buffered.
#include "common.hpp"
#include "launch.hpp"

namespace ckv {
namespace {

struct PrefillArgs {
  const uint16_t *q;
  uint16_t *out;
  const uint8_t *k, *v;
  const float *k_scale, *v_scale;
  const int32_t *bt, *ctx, *cu;
  int32_t max_pages, h_q, h_kv, group, ps;
  float scale_log2;  // softmax_scale * log2(e)
  int32_t window;
  int32_t tiles;     // grid.x: max row tiles of a sequence
};

constexpr int kRows = 128;  // rows per workgroup
constexpr int kThreads = 256;

// Row m of a 32-key S^T tile holds key pi(m) of the tile.  With
// m = 8i + 4h + j the lane that receives row m (half h, element 4i + j)
// gets key 16(i/2) + 8h + 4(i%2) + j, so elements 8s..8s+7 of a lane are
// keys 16s + 8h + 0..7.
__device__ __forceinline__ int pi_row(int m) {
  const int i = m >> 3, h = (m >> 2) & 1, j = m & 3;
  return 16 * (i >> 1) + 8 * h + 4 * (i & 1) + j;
}

template <int D, int BN, bool FP8>
struct Cfg {
  static constexpr int CH = D / 8;                       // 16-byte bf16 chunks per K row
  static constexpr int KSW = (CH < 16 ? CH : 16) - 1;    // K chunk swizzle mask
  static constexpr int NKC = BN / 8;                     // 16-byte key chunks per Vt row
  static constexpr int VSW = NKC - 1;                    // Vt chunk swizzle mask
  static constexpr int K_BYTES = BN * D * 2;
  static constexpr int LDS = 2 * K_BYTES;
  static constexpr int KPT = BN * CH / kThreads;         // K chunks per thread
  static constexpr int VGROUPS = (BN / 4) * CH;          // (4 keys x 8 d) groups
  static constexpr int VPT = (VGROUPS + kThreads - 1) / kThreads;
  static constexpr int NT = BN / 32;                     // S^T tiles per block
  static constexpr int DS = D / 16;                      // QK^T k-steps
  static constexpr int DT = D / 32;                      // output d-tiles
  static constexpr int EK = FP8 ? 1 : 2;                 // pool bytes per element
  static_assert(KPT * kThreads == BN * CH, "K staging must tile evenly");
};

__device__ __forceinline__ int k_off(int key, int chunk, int row_bytes, int ksw) {
  return key * row_bytes + ((chunk ^ (key & ksw)) << 4);
}
__device__ __forceinline__ int vt_off(int d, int kchunk, int row_bytes, int vsw) {
  return d * row_bytes + ((kchunk ^ ((d >> 1) & vsw)) << 4);
}

template <int D, int BN, bool FP8>
struct Stage {
  using C = Cfg<D, BN, FP8>;
  // bf16 pool: 16-byte chunks; fp8 pool: 8-byte code chunks (low half used)
  u32x4 k[C::KPT];
  u32x4 v[C::VPT][4];
};

template <int D, int BN, bool FP8>
__device__ __forceinline__ void load_block(Stage<D, BN, FP8> &sg, const PrefillArgs &a,
                                           const int32_t *bt, int g, int kbase, int kv_end) {
  using C = Cfg<D, BN, FP8>;
  const int tid = threadIdx.x;
  const size_t head_stride = (size_t)a.ps * D * C::EK;
#pragma unroll
  for (int r = 0; r < C::KPT; ++r) {
    const int id = tid + r * kThreads;
    const int key = id / C::CH, c = id % C::CH;
    const int kp = kbase + key;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (kp < kv_end) {
      const int page = bt[kp / a.ps];
      const uint8_t *src = a.k + ((size_t)page * a.h_kv + g) * head_stride +
                           (size_t)(kp % a.ps) * D * C::EK + c * 8 * C::EK;
      if constexpr (FP8) {
        const u32x2 y = ld<u32x2>(src);
        x.x = y.x;
        x.y = y.y;
      } else {
        x = ld<u32x4>(src);
      }
    }
    sg.k[r] = x;
  }
#pragma unroll
  for (int r = 0; r < C::VPT; ++r) {
    const int id = tid + r * kThreads;
    if (id < C::VGROUPS) {
      const int kg = id / C::CH, c = id % C::CH;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int kp = kbase + 4 * kg + e;
        u32x4 x = {0u, 0u, 0u, 0u};
        if (kp < kv_end) {
          const int page = bt[kp / a.ps];
          const uint8_t *src = a.v + ((size_t)page * a.h_kv + g) * head_stride +
                               (size_t)(kp % a.ps) * D * C::EK + c * 8 * C::EK;
          if constexpr (FP8) {
            const u32x2 y = ld<u32x2>(src);
            x.x = y.x;
            x.y = y.y;
          } else {
            x = ld<u32x4>(src);
          }
        }
        sg.v[r][e] = x;
      }
    }
  }
}

template <int D, int BN, bool FP8>
__device__ __forceinline__ void store_block(const Stage<D, BN, FP8> &sg, uint8_t *lds) {
  using C = Cfg<D, BN, FP8>;
  const int tid = threadIdx.x;
  uint8_t *klds = lds;
  uint8_t *vlds = lds + C::K_BYTES;
#pragma unroll
  for (int r = 0; r < C::KPT; ++r) {
    const int id = tid + r * kThreads;
    const int key = id / C::CH, c = id % C::CH;
    u32x4 x = sg.k[r];
    if constexpr (FP8) {
      const u32x2 lo = fp8x4_to_bf16x4(x.x), hi = fp8x4_to_bf16x4(x.y);
      x = u32x4{lo.x, lo.y, hi.x, hi.y};
    }
    st<u32x4>(klds + k_off(key, c, D * 2, C::KSW), x);
  }
#pragma unroll
  for (int r = 0; r < C::VPT; ++r) {
    const int id = tid + r * kThreads;
    if (id < C::VGROUPS) {
      const int kg = id / C::CH, c = id % C::CH;
      u32x4 row[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        row[e] = sg.v[r][e];
        if constexpr (FP8) {
          const u32x2 lo = fp8x4_to_bf16x4(row[e].x), hi = fp8x4_to_bf16x4(row[e].y);
          row[e] = u32x4{lo.x, lo.y, hi.x, hi.y};
        }
      }
      // transpose: d = 8c + 2w + half takes element (w, half) of each key row
      const int kchunk = kg >> 1, hv = kg & 1;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const u32x2 even = {pack_lo16(row[0][w], row[1][w]), pack_lo16(row[2][w], row[3][w])};
        const u32x2 odd = {pack_hi16(row[0][w], row[1][w]), pack_hi16(row[2][w], row[3][w])};
        const int d0 = 8 * c + 2 * w;
        st<u32x2>(vlds + vt_off(d0, kchunk, BN * 2, C::VSW) + 8 * hv, even);
        st<u32x2>(vlds + vt_off(d0 + 1, kchunk, BN * 2, C::VSW) + 8 * hv, odd);
      }
    }
  }
}

template <int D, int BN, bool FP8>
__global__ __launch_bounds__(kThreads, D >= 256 ? 1 : 2) void prefill_kernel(PrefillArgs a) {
  using C = Cfg<D, BN, FP8>;
  __shared__ __attribute__((aligned(16))) uint8_t lds[C::LDS];

  const int tile = a.tiles - 1 - (int)blockIdx.x;  // later (costlier) tiles first
  const int g = blockIdx.y;
  const int b = blockIdx.z;
  const int q0 = a.cu[b];
  const int n = a.cu[b + 1] - q0;
  const int G = a.group;
  const int rows = n * G;
  const int R0 = tile * kRows;
  if (R0 >= rows) return;
  const int P = a.ctx[b];
  const int32_t *bt = a.bt + (size_t)b * a.max_pages;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int half = lane >> 5, col = lane & 31;
  const int R = R0 + wave * 32 + col;
  const bool rvalid = R < rows;
  const int t = rvalid ? R / G : 0;
  const int hh = rvalid ? R - t * G : 0;
  const int ipos = rvalid ? P + t : -1;
  const size_t qrow = ((size_t)(q0 + t) * a.h_q + (size_t)g * G + hh) * D;

  bf16x8 qf[C::DS];
#pragma unroll
  for (int s = 0; s < C::DS; ++s) {
    u32x4 x = {0u, 0u, 0u, 0u};
    if (rvalid) x = ld<u32x4>(a.q + qrow + 16 * s + 8 * half);
    qf[s] = as_bf16x8(x);
  }

  const int t_first = R0 / G;
  const int t_last = min(n - 1, (R0 + kRows - 1) / G);
  const int i_min = P + t_first, i_max = P + t_last;
  const int kv_end = i_max + 1;
  const int W = a.window;
  const int kv_begin = W > 0 ? max(0, i_min - W + 1) : 0;
  const int kb_begin = kv_begin / BN;
  const int kb_end = (kv_end + BN - 1) / BN;

  f32x16 o[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) o[dt] = f32x16{};
  float m = kNegInf, l = 0.f;

  uint8_t *klds = lds;
  uint8_t *vlds = lds + C::K_BYTES;
  Stage<D, BN, FP8> stage;
  load_block<D, BN, FP8>(stage, a, bt, g, kb_begin * BN, kv_end);

  for (int kb = kb_begin; kb < kb_end; ++kb) {
    const int kbase = kb * BN;
    __syncthreads();
    store_block<D, BN, FP8>(stage, lds);
    __syncthreads();
    if (kb + 1 < kb_end) load_block<D, BN, FP8>(stage, a, bt, g, kbase + BN, kv_end);

    // ---- S^T = K Q^T, one 32-key tile at a time
    f32x16 s[C::NT];
#pragma unroll
    for (int tt = 0; tt < C::NT; ++tt) {
      s[tt] = f32x16{};
      const int key = 32 * tt + pi_row(col);
#pragma unroll
      for (int ds = 0; ds < C::DS; ++ds) {
        const u32x4 kx = ld<u32x4>(klds + k_off(key, 2 * ds + half, D * 2, C::KSW));
        s[tt] = mfma32x32x16(as_bf16x8(kx), qf[ds], s[tt]);
      }
    }

    // ---- scale (fp8: times the page-head K scale), mask, row max
    float ksc[C::NT * 2], vsc[C::NT * 2];  // per 16-key group
#pragma unroll
    for (int q = 0; q < C::NT * 2; ++q) {
      ksc[q] = a.scale_log2;
      vsc[q] = 1.f;
      if constexpr (FP8) {
        const int kp = kbase + 16 * q;
        float sk = 0.f, sv = 0.f;
        if (kp < kv_end) {
          const size_t idx = (size_t)bt[kp / a.ps] * a.h_kv + g;
          sk = a.k_scale[idx];
          sv = a.v_scale[idx];
        }
        ksc[q] = a.scale_log2 * sk;
        vsc[q] = sv;
      }
    }
    const bool full = (kbase + BN - 1 <= i_min) && (W <= 0 || i_max - kbase < W);
    float mx = kNegInf;
#pragma unroll
    for (int tt = 0; tt < C::NT; ++tt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int grp = 2 * tt + (e >> 3);
        float x = s[tt][e] * ksc[grp];
        if (!full) {
          const int i = e >> 2, j = e & 3;
          const int kp = kbase + 32 * tt + 16 * (i >> 1) + 8 * half + 4 * (i & 1) + j;
          const bool vis = kp <= ipos && (W <= 0 || ipos - kp < W);
          x = vis ? x : kNegInf;
        }
        s[tt][e] = x;
        mx = fmaxf(mx, x);
      }
    }
    mx = fmaxf(mx, shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx);
    const float m_use = m_new == kNegInf ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    m = m_new;
    l *= alpha;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) o[dt] *= alpha;

    // ---- P = exp2(x - m); O^T += Vt P^T
#pragma unroll
    for (int tt = 0; tt < C::NT; ++tt) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        float p[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          p[e] = fast_exp2(s[tt][8 * ks + e] - m_use);
          l += p[e];
          if constexpr (FP8) p[e] *= vsc[2 * tt + ks];
        }
        const u32x4 pb = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                          pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
        const int kchunk = 4 * tt + 2 * ks + half;
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt) {
          const u32x4 vx = ld<u32x4>(vlds + vt_off(32 * dt + col, kchunk, BN * 2, C::VSW));
          o[dt] = mfma32x32x16(as_bf16x8(vx), as_bf16x8(pb), o[dt]);
        }
      }
    }
  }

  // ---- normalize and store this lane's row: d = 32 dt + 8 i + 4 half + 0..3
  l += shfl_xor(l, 32);
  if (!rvalid) return;
  const float inv = 1.f / l;
  uint16_t *orow = a.out + qrow;
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u32x2 w = {pack_bf16x2(o[dt][4 * i] * inv, o[dt][4 * i + 1] * inv),
                       pack_bf16x2(o[dt][4 * i + 2] * inv, o[dt][4 * i + 3] * inv)};
      st<u32x2>(orow + 32 * dt + 8 * i + 4 * half, w);
    }
  }
}

template <int D, int BN, bool FP8>
hipError_t launch(const PrefillArgs &a, int h_kv, int num_seqs, hipStream_t s) {
  dim3 grid(a.tiles, h_kv, num_seqs);
  hipLaunchKernelGGL((prefill_kernel<D, BN, FP8>), grid, dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_prefill_bf16(const PoolView &p, const BatchView &b, const void *q, int h_q,
                               float scale, int window, void *out, hipStream_t s) {
  if (b.num_seqs == 0 || b.max_q == 0 || b.total_q == 0) return hipSuccess;
  PrefillArgs a;
  a.q = static_cast<const uint16_t *>(q);
  a.out = static_cast<uint16_t *>(out);
  a.k = static_cast<const uint8_t *>(p.k);
  a.v = static_cast<const uint8_t *>(p.v);
  a.k_scale = p.k_scale;
  a.v_scale = p.v_scale;
  a.bt = b.bt;
  a.ctx = b.ctx;
  a.cu = b.cu_q;
  a.max_pages = b.max_pages;
  a.h_q = h_q;
  a.h_kv = p.h_kv;
  a.group = h_q / p.h_kv;
  a.ps = p.ps;
  a.scale_log2 = scale * kLog2e;
  a.window = window;
  const long long rows = (long long)b.max_q * a.group;
  a.tiles = (int)((rows + kRows - 1) / kRows);
  const bool fp8 = p.kv_dtype == 2;
  switch (p.d) {
    case 64:
      return fp8 ? launch<64, 64, true>(a, p.h_kv, b.num_seqs, s)
                 : launch<64, 64, false>(a, p.h_kv, b.num_seqs, s);
    case 128:
      return fp8 ? launch<128, 64, true>(a, p.h_kv, b.num_seqs, s)
                 : launch<128, 64, false>(a, p.h_kv, b.num_seqs, s);
    case 256:
      return fp8 ? launch<256, 32, true>(a, p.h_kv, b.num_seqs, s)
                 : launch<256, 32, false>(a, p.h_kv, b.num_seqs, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace ckv
