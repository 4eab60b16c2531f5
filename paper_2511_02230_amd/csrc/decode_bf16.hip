// paged_decode_attn for bf16 queries over a bf16 or fp8-E4M3 paged pool.
//
// Split-K: the visible context [lo, c) of each sequence (lo = c - window for
// a sliding window, else 0) is cut into partitions of L positions; one
// single-wave workgroup handles (partition, KV head, <=16 query heads of its
// group, sequence) and reads every K/V byte of its range exactly once for all
// of those heads.
//
// Per 16-key tile (always inside one page):
//   * K rows go straight from HBM into VGPRs, already in the A-operand layout
//     of v_mfma_f32_16x16x32_bf16: lane l fetches 16 contiguous bytes of key
//     row l % 16 at byte 16 (l / 16) + 64 i, so a tile costs one scalar page
//     base, one fixed per-lane offset and immediate offsets.
//   * V rows go from HBM into a two-stage LDS ring with
//     global_load_lds_dwordx4 (the lane -> address map XOR-swizzles the
//     rows); V^T operands are read back with ds_read_b64_tr_b16.  The V
//     loads are non-temporal: each byte is read once, and the hint was
//     measured to lift decode by 7-10 % (K, loaded into VGPRs, measured
//     slower with it).
//   * S^T (16 keys x 16 heads) = K Q^T; lane l then holds the scores of head
//     l % 16 for keys 4 (l / 16) + 0..3, which is exactly its B operand of
//     O^T (16 d x 16 heads) += V^T (16 d x 16 keys) P^T on
//     v_mfma_f32_16x16x16_bf16.
// Blocks of KB keys (one or two tiles) are double-buffered: block j + 1 is in
// flight while block j is computed.  Online softmax in fp32, base-2, with the
// running maximum moved only when it grows by more than 2^8.  fp8 K codes are
// widened in registers; fp8 V blocks are widened once into a bf16 LDS block.
// A partition writes (m, l, o) partials in fp32 unless it is its sequence's
// only one, in which case it writes the output; the combine kernel merges
// the rest.
#include <algorithm>
#include <mutex>

#include "../../include/ckv.h"
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
  int32_t max_pages, h_q, h_kv, group;
  float scale_log2;
  int32_t window;
  int32_t split_len, max_splits, head_chunks;
  float *part_o;   // [B][H_q][max_splits][D]
  float *part_ml;  // [B][H_q][max_splits][2]
};

constexpr float kRescaleSlack = 8.0f;  // log2 units: defer rescaling below 2^8

template <int D, bool FP8, int PS>
struct DCfg {
  static constexpr int KB = D >= 256 ? 16 : 32;   // keys per block
  static constexpr int NT = KB / 16;              // 16-key tiles per block
  static constexpr int RAW_ROW = FP8 ? D : 2 * D; // pool bytes per key row
  static constexpr int ROW = 2 * D;               // bf16 bytes per row in LDS
  static constexpr int RCH = RAW_ROW / 16;        // 16-byte chunks per pool row
  static constexpr int CH = D / 8;                // 16-byte chunks per bf16 row
  static constexpr int KLD = RAW_ROW / 64;        // 16-byte K loads per lane per tile
  static constexpr int RPD = 1024 / RAW_ROW;      // rows per 1-KB V load
  static constexpr int VLD = 16 / RPD;            // V loads per tile
  static constexpr int VRAW = KB * RAW_ROW;       // raw V bytes per block
  static constexpr int DS = D / 32;               // QK^T k-steps
  static constexpr int DT = D / 16;               // output d-tiles
  static_assert(PS % 16 == 0, "tiles never straddle a page");
  static_assert(RPD >= 1 && VLD >= 1, "whole 1-KB loads per tile");
};

// d offset of the 8 k-slots a lane (quarter g) supplies at QK^T step `step`.
// bf16: 16 contiguous bytes per step; fp8: one 16-byte run of codes feeds
// two consecutive steps.
template <bool FP8>
__device__ __forceinline__ int qk_d0(int step, int g) {
  if constexpr (FP8) return 64 * (step >> 1) + 16 * g + 8 * (step & 1);
  return 32 * step + 8 * g;
}

// XOR swizzle (in 16-byte chunks) of bf16 V rows in LDS.  A wave-wide
// transposed read covers 16 consecutive rows x one 32-byte chunk pair;
// shifting row r's pairs by 2 (r & 7) spreads them over 8 pair positions.
template <int CH>
__device__ __forceinline__ int vswz(int row) {
  return (2 * (row & 7)) & (CH - 1);
}

// Registers of one block's K tiles (raw pool bytes, MFMA A-operand layout).
template <class C>
struct KRegs {
  u32x4 r[C::NT][C::KLD];
};

// Everything a block issue / compute needs that is fixed per workgroup.
template <class C>
struct DState {
  const int32_t *bt;
  size_t head_off, page_stride;
  int kbeg, kend, kb0, nblk;
  uint32_t koff;                 // per-lane K offset within a tile
  uint32_t voff[C::VLD];         // per-lane V offset of each 1-KB load (bf16: swizzled)
};

// Issue the K loads (into kr) and the V loads (into stage) of the block at
// kbase.  Rows at or beyond kend are redirected to row kend - 1 (finite data
// in a resident page; the mask removes them).
template <class C, int PS, bool FP8>
__device__ __forceinline__ void issue_block(const DecodeArgs &a, const DState<C> &S, int kbase,
                                            KRegs<C> &kr, lds_u8 *stage) {
  const int lane = threadIdx.x;
  const bool whole = kbase + C::KB <= S.kend;
#pragma unroll
  for (int tt = 0; tt < C::NT; ++tt) {
    const int t0 = kbase + 16 * tt;
    const int kp = min(t0, S.kend - 1);  // a key of the tile's page
    const int pg = ldc(S.bt, __builtin_amdgcn_readfirstlane(kp / PS));
    const size_t pbase = (size_t)pg * S.page_stride + S.head_off;
    const uint8_t *kpage = a.k + pbase;
    const uint8_t *vpage = a.v + pbase;
    lds_u8 *vdst = stage + tt * 16 * C::RAW_ROW;
    if (whole) {
      const uint8_t *kt = kpage + (size_t)(t0 % PS) * C::RAW_ROW;
#pragma unroll
      for (int i = 0; i < C::KLD; ++i) kr.r[tt][i] = ld<u32x4>(kt + S.koff + 64 * i);
      const uint8_t *vt = vpage + (size_t)(t0 % PS) * C::RAW_ROW;
#pragma unroll
      for (int r = 0; r < C::VLD; ++r) dma16_sv<true>(vt, S.voff[r], vdst + r * 1024);
    } else {
      const int row0 = kp - kp % PS;  // first key of the page
      const int mk = min(t0 + (lane & 15), S.kend - 1) - row0;
      const uint32_t ko = (uint32_t)(mk * C::RAW_ROW + 16 * (lane >> 4));
#pragma unroll
      for (int i = 0; i < C::KLD; ++i) kr.r[tt][i] = ld<u32x4>(kpage + ko + 64 * i);
#pragma unroll
      for (int r = 0; r < C::VLD; ++r) {
        const int rr = r * C::RPD + lane / C::RCH;  // row within the tile
        const int mv = min(t0 + rr, S.kend - 1) - row0;
        const int slot = lane % C::RCH;
        const int chunk = FP8 ? slot : slot ^ vswz<C::CH>(rr);
        dma16_sv<true>(vpage, (uint32_t)(mv * C::RAW_ROW + 16 * chunk), vdst + r * 1024);
      }
    }
  }
}

// Compute one block: S^T, mask, online softmax, O^T += V^T P^T.
template <class C, int PS, bool FP8>
__device__ __forceinline__ void compute_block(const DecodeArgs &a, const DState<C> &S, int kbase,
                                              const KRegs<C> &kr, const lds_u8 *stage,
                                              lds_u8 *vwide, const bf16x8 (&qf)[C::DS],
                                              f32x4 (&o)[C::DT], float &m, float &l, int g) {
  const int lane = threadIdx.x;
  const int q4 = lane >> 4, li = lane & 15;

  const lds_u8 *vb = stage;
  if constexpr (FP8) {
    // widen the block's V codes into bf16 rows (swizzled like a bf16 block)
#pragma unroll
    for (int it = 0; it < C::VRAW / 1024; ++it) {
      const int id = lane + 64 * it;
      const int row = id / C::RCH, cc = id % C::RCH;
      const u32x4 x = lds_ld16(stage + row * C::RAW_ROW + cc * 16);
      const u32x2 a0 = fp8x4_to_bf16x4(x.x), a1 = fp8x4_to_bf16x4(x.y);
      const u32x2 b0 = fp8x4_to_bf16x4(x.z), b1 = fp8x4_to_bf16x4(x.w);
      lds_u8 *dst = vwide + row * C::ROW;
      const int sw = vswz<C::CH>(row);
      lds_st16(dst + (((2 * cc) ^ sw) << 4), u32x4{a0.x, a0.y, a1.x, a1.y});
      lds_st16(dst + (((2 * cc + 1) ^ sw) << 4), u32x4{b0.x, b0.y, b1.x, b1.y});
    }
    vb = vwide;
  }

  // ---- S^T tiles: lane holds head li, keys 16 tt + 4 q4 + 0..3
  f32x4 s[C::NT];
  float ksc[C::NT], vsc[C::NT];
#pragma unroll
  for (int tt = 0; tt < C::NT; ++tt) {
    s[tt] = f32x4{};
#pragma unroll
    for (int i = 0; i < C::KLD; ++i) {
      const u32x4 x = kr.r[tt][i];
      if constexpr (FP8) {
        const u32x2 a0 = fp8x4_to_bf16x4(x.x), a1 = fp8x4_to_bf16x4(x.y);
        const u32x2 b0 = fp8x4_to_bf16x4(x.z), b1 = fp8x4_to_bf16x4(x.w);
        s[tt] = mfma16x16x32(as_bf16x8(u32x4{a0.x, a0.y, a1.x, a1.y}), qf[2 * i], s[tt]);
        s[tt] = mfma16x16x32(as_bf16x8(u32x4{b0.x, b0.y, b1.x, b1.y}), qf[2 * i + 1], s[tt]);
      } else {
        s[tt] = mfma16x16x32(as_bf16x8(x), qf[i], s[tt]);
      }
    }
    ksc[tt] = a.scale_log2;
    vsc[tt] = 1.f;
    if constexpr (FP8) {
      const int kp = min(kbase + 16 * tt, S.kend - 1);
      const int idx = ldc(S.bt, __builtin_amdgcn_readfirstlane(kp / PS)) * a.h_kv + g;
      ksc[tt] = a.scale_log2 * ldc(a.k_scale, idx);
      vsc[tt] = ldc(a.v_scale, idx);
    }
  }

  // ---- scale, mask, block maximum (log2 units)
  const bool edge = kbase < S.kbeg || kbase + C::KB > S.kend;
  float mx = kNegInf;
#pragma unroll
  for (int tt = 0; tt < C::NT; ++tt) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float x = s[tt][j] * ksc[tt];
      if (edge) {
        const int kp = kbase + 16 * tt + 4 * q4 + j;
        x = (kp >= S.kbeg && kp < S.kend) ? x : kNegInf;
      }
      s[tt][j] = x;
      mx = fmaxf(mx, x);
    }
  }
  {
    const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    mx = fmaxf(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
    const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    mx = fmaxf(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
  }
  const bool bump = mx > m + kRescaleSlack;
  if (__builtin_amdgcn_ballot_w64(bump)) {
    const float alpha = bump ? fast_exp2(m - mx) : 1.f;
    m = bump ? mx : m;
    l *= alpha;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) o[dt] *= alpha;
  }
  const float m_use = m == kNegInf ? 0.f : m;

  // ---- P (bf16) and O^T += V^T P^T, one 16-key tile at a time.  The row
  // sum adds the weights the MFMA multiplies: the bf16 probabilities, or for
  // fp8 the bf16 values of P v_scale divided by v_scale (a value scale of 0,
  // or one so small or large that P v_scale flushes or overflows, keeps the
  // fp32 probabilities instead).
#pragma unroll
  for (int tt = 0; tt < C::NT; ++tt) {
    float p[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) p[j] = fast_exp2(s[tt][j] - m_use);
    float praw = 0.f;
    if constexpr (FP8) {
      praw = (p[0] + p[1]) + (p[2] + p[3]);
#pragma unroll
      for (int j = 0; j < 4; ++j) p[j] *= vsc[tt];
    }
    const u32x2 pb = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3])};
    if constexpr (FP8) {
      const bool vs_ok = (vsc[tt] >= 0x1p-100f) & (vsc[tt] <= 0x1p100f);
      l = vs_ok ? __builtin_fmaf(add_bf16x2(pb.y, add_bf16x2(pb.x, 0.f)), __builtin_amdgcn_rcpf(vsc[tt]), l)
                : l + praw;
    } else {
      l = add_bf16x2(pb.y, add_bf16x2(pb.x, l));
    }
    // lane li of group q4 addresses key 4 q4 + li / 4 of the tile, columns
    // 16 dt + 4 (li % 4) .. +3
    const int row = 16 * tt + 4 * q4 + (li >> 2);
    const lds_u8 *vr = vb + row * C::ROW;
    const int sw = vswz<C::CH>(row);
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) {
      const int byte = 2 * (16 * dt + 4 * (li & 3));
      const u32x2 vx = ds_read_tr16(vr + (((byte >> 4) ^ sw) << 4) + (byte & 15));
      o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, vx),
                                                         __builtin_bit_cast(i16x4, pb), o[dt], 0, 0, 0);
    }
  }
}

// Wait for everything this wave has in flight (the K registers and V stage
// of the next block to compute, and LDS reads of the stage about to be
// refilled), then make the compiler's own wait for the K registers land here
// as well.
template <class C>
__device__ __forceinline__ void block_ready(const KRegs<C> &kr) {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int tt = 0; tt < C::NT; ++tt)
#pragma unroll
    for (int i = 0; i < C::KLD; ++i) asm volatile("" ::"v"(kr.r[tt][i]));
}

template <int D, bool FP8, int PS>
__global__ __launch_bounds__(64) void decode_kernel(DecodeArgs a) {
  using C = DCfg<D, FP8, PS>;
  // two V stages (+ the widened bf16 block for fp8), one LDS object so that
  // nothing is lost to padding
  __shared__ __attribute__((aligned(1024))) uint8_t lds_[2 * C::VRAW + (FP8 ? C::KB * C::ROW : 0)];
  lds_u8 *const st0 = as_lds(lds_);
  lds_u8 *const st1 = st0 + C::VRAW;
  lds_u8 *const vwide = st0 + 2 * C::VRAW;  // fp8 only

  const int split = blockIdx.x;
  const int g = blockIdx.y / a.head_chunks;
  const int hc = blockIdx.y - g * a.head_chunks;
  const int b = blockIdx.z;
  const int c = a.ctx[b];
  const int lo = a.window > 0 ? max(0, c - a.window) : 0;
  const int L = a.split_len;
  const int nsplit = (c - lo + L - 1) / L;
  if (split >= nsplit) return;

  const int lane = threadIdx.x;
  const int li = lane & 15, q4 = lane >> 4;
  const int head = hc * 16 + li;
  const bool hvalid = head < a.group;
  const int qh = g * a.group + (hvalid ? head : 0);
  const size_t qoff = ((size_t)b * a.h_q + qh) * D;

  DState<C> S;
  S.bt = a.bt + (size_t)b * a.max_pages;
  S.head_off = (size_t)g * PS * C::RAW_ROW;
  S.page_stride = (size_t)a.h_kv * PS * C::RAW_ROW;
  S.kbeg = lo + split * L;
  S.kend = min(c, S.kbeg + L);
  S.kb0 = S.kbeg - S.kbeg % C::KB;
  S.nblk = (S.kend - S.kb0 + C::KB - 1) / C::KB;
  S.koff = (uint32_t)(li * C::RAW_ROW + 16 * q4);
#pragma unroll
  for (int r = 0; r < C::VLD; ++r) {
    const int rr = r * C::RPD + lane / C::RCH;
    const int slot = lane % C::RCH;
    const int chunk = FP8 ? slot : slot ^ vswz<C::CH>(rr);
    S.voff[r] = (uint32_t)(rr * C::RAW_ROW + 16 * chunk);
  }

  KRegs<C> k0, k1;
  issue_block<C, PS, FP8>(a, S, S.kb0, k0, st0);

  bf16x8 qf[C::DS];
#pragma unroll
  for (int s = 0; s < C::DS; ++s) {
    u32x4 x = {0u, 0u, 0u, 0u};
    if (hvalid) x = ld<u32x4>(a.q + qoff + qk_d0<FP8>(s, q4));
    qf[s] = as_bf16x8(x);
  }
  f32x4 o[C::DT];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) o[dt] = f32x4{};
  float m = kNegInf, l = 0.f;

  for (int j = 0; j < S.nblk; j += 2) {
    const int kbase = S.kb0 + j * C::KB;
    block_ready<C>(k0);
    if (j + 1 < S.nblk) issue_block<C, PS, FP8>(a, S, kbase + C::KB, k1, st1);
    compute_block<C, PS, FP8>(a, S, kbase, k0, st0, vwide, qf, o, m, l, g);
    if (j + 1 < S.nblk) {
      block_ready<C>(k1);
      if (j + 2 < S.nblk) issue_block<C, PS, FP8>(a, S, kbase + 2 * C::KB, k0, st0);
      compute_block<C, PS, FP8>(a, S, kbase + C::KB, k1, st1, vwide, qf, o, m, l, g);
    }
  }

  {
    const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(l), __float_as_uint(l), false, false);
    l = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
    const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l), false, false);
    l = __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
  }
  if (!hvalid) return;
  // lane holds head `qh`, d = 16 dt + 4 q4 + 0..3
  if (nsplit == 1) {
    const float inv = 1.f / l;
    uint16_t *orow = a.out + qoff;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) {
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
  for (int dt = 0; dt < C::DT; ++dt) st<f32x4>(po + 16 * dt + 4 * q4, o[dt] * inv);
  if (q4 == 0) st<f32x2>(a.part_ml + pidx * 2, f32x2{m, l});
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
  hipLaunchKernelGGL((combine_kernel<D>), dim3(a.h_q, num_seqs), dim3(64), 0, s, a);
  return hipGetLastError();
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
