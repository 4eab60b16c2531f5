// paged_decode_attn for bf16 queries over a bf16 or fp8-E4M3 paged pool:
// the device code of one work item (one wave), shared by the decode kernel
// and the mixed prefill + decode kernel.
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
#pragma once

#include "common.hpp"

namespace ckv {
namespace dc {

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
  // fused append (bf16 pools, DCfg::AP): each sequence's new token's K and V
  // rows [B][H_kv][D], the last context position c - 1; the kernel writes
  // them into their pool slots and reads that key from here
  const uint8_t *k_new, *v_new;
};

constexpr float kRescaleSlack = 8.0f;  // log2 units: defer rescaling below 2^8

// Lane within the wave (a decode item is one wave's work).  WAVES: waves
// per workgroup of the calling kernel (one for the decode kernel itself,
// where the thread index is the lane).
template <int WAVES>
__device__ __forceinline__ int lane_id() {
  if constexpr (WAVES == 1) return threadIdx.x;
  return threadIdx.x & 63;
}

template <int D, bool FP8, int PS, bool APPEND = false>
struct DCfg {
  static constexpr bool AP = APPEND;              // fused append (bf16 pools)
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
  // two V stages (+ the widened bf16 block for fp8), one LDS object so that
  // nothing is lost to padding
  static constexpr int LDS = 2 * VRAW + (FP8 ? KB * ROW : 0);
  static_assert(PS % 16 == 0, "tiles never straddle a page");
  static_assert(RPD >= 1 && VLD >= 1, "whole 1-KB loads per tile");
  static_assert(!(AP && FP8), "the fused append writes bf16 rows");
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
  int cnew;                      // fused append: position of the new token (else -1)
  const uint8_t *nk, *nv;        // fused append: its K and V rows (head g)
};

// Issue the K loads (into kr) and the V loads (into stage) of the block at
// kbase.  Rows at or beyond kend are redirected to row kend - 1 (finite data
// in a resident page; the mask removes them).
template <class C, int PS, bool FP8, int WAVES>
__device__ __forceinline__ void issue_block(const DecodeArgs &a, const DState<C> &S, int kbase,
                                            KRegs<C> &kr, lds_u8 *stage) {
  const int lane = lane_id<WAVES>();
  if constexpr (C::AP) {
    if (S.cnew >= 0 && kbase + C::KB > S.cnew) {
      // the block of the new token: its row comes from the input, the
      // others (and clamped rows below it) from their page
#pragma unroll
      for (int tt = 0; tt < C::NT; ++tt) {
        const int t0 = kbase + 16 * tt;
        const int kp = min(t0, S.kend - 1);
        const int pg = ldc(S.bt, __builtin_amdgcn_readfirstlane(kp / PS));
        const size_t pbase = (size_t)pg * S.page_stride + S.head_off;
        const int row0 = kp - kp % PS;
        const int mk = min(t0 + (lane & 15), S.kend - 1);
#pragma unroll
        for (int i = 0; i < C::KLD; ++i) {
          const uint32_t co = (uint32_t)(16 * (lane >> 4) + 64 * i);
          kr.r[tt][i] = ld<u32x4>(mk == S.cnew ? S.nk + co : a.k + pbase + (size_t)(mk - row0) * C::RAW_ROW + co);
        }
        lds_u8 *vdst = stage + tt * 16 * C::RAW_ROW;
#pragma unroll
        for (int r = 0; r < C::VLD; ++r) {
          const int rr = r * C::RPD + lane / C::RCH;
          const int mv = min(t0 + rr, S.kend - 1);
          const uint32_t co = (uint32_t)(16 * ((lane % C::RCH) ^ vswz<C::CH>(rr)));
          dma16(mv == S.cnew ? S.nv + co : a.v + pbase + (size_t)(mv - row0) * C::RAW_ROW + co, vdst + r * 1024);
        }
      }
      return;
    }
  }
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
template <class C, int PS, bool FP8, int WAVES>
__device__ __forceinline__ void compute_block(const DecodeArgs &a, const DState<C> &S, int kbase,
                                              const KRegs<C> &kr, const lds_u8 *stage,
                                              lds_u8 *vwide, const bf16x8 (&qf)[C::DS],
                                              f32x4 (&o)[C::DT], float &m, float &l, int g) {
  const int lane = lane_id<WAVES>();
  const int q4 = lane >> 4, li = lane & 15;

  const lds_u8 *vb = stage;
  if constexpr (FP8) {
    // widen the block's V codes into bf16 rows (swizzled like a bf16 block):
    // each lane turns 8 codes into one 16-byte chunk, so every 8 and 16
    // consecutive lanes store to distinct 16-byte bank groups
#pragma unroll
    for (int it = 0; it < C::KB * C::ROW / 1024; ++it) {
      const int id = lane + 64 * it;
      const int row = id / C::CH, cc = id % C::CH;
      const u32x4 w = fp8x8_to_bf16x8(lds_ld8(stage + row * C::RAW_ROW + cc * 8));
      lds_st16(vwide + row * C::ROW + ((cc ^ vswz<C::CH>(row)) << 4), w);
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

// One work item, run by one wave: partition `split` of the KV head and
// head chunk `hy` (hy = head_chunks * g + chunk) of sequence `b`.  `lds`
// holds DCfg::LDS bytes for this wave alone, 1024-aligned.
// AP: fused append (DecodeArgs::k_new / v_new).
template <int D, bool FP8, int PS, int WAVES = 1, bool AP = false>
__device__ __forceinline__ void decode_item(const DecodeArgs &a, lds_u8 *lds, int split, int hy, int b) {
  using C = DCfg<D, FP8, PS, AP>;
  lds_u8 *const st0 = lds;
  lds_u8 *const st1 = st0 + C::VRAW;
  lds_u8 *const vwide = st0 + 2 * C::VRAW;  // fp8 only

    const int g = hy / a.head_chunks;
  const int hc = hy - g * a.head_chunks;
    const int c = a.ctx[b];
  const int lo = a.window > 0 ? max(0, c - a.window) : 0;
  const int L = a.split_len;
  const int nsplit = (c - lo + L - 1) / L;
  if (split >= nsplit) return;

  const int lane = lane_id<WAVES>();
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
  // Fused append: the new token (position c - 1) is read from the input by
  // the partition that holds it, whose first head chunk also writes its K
  // and V rows into the pool slot (lanes 0 .. 2 CH - 1, one 16-byte chunk
  // each).  No work item reads that slot.
  S.cnew = -1;
  u32x4 apx{};
  uint8_t *apdst = nullptr;
  if constexpr (AP) {
    S.nk = a.k_new + ((size_t)b * a.h_kv + g) * C::ROW;
    S.nv = a.v_new + ((size_t)b * a.h_kv + g) * C::ROW;
    if (split == nsplit - 1) {
      S.cnew = c - 1;
      if (hc == 0 && lane < 2 * C::CH) {
        // V = K address plus the V - K distance (a per-lane choice between
        // two pointers would index a copy of the arguments in scratch)
        const int kv = lane / C::CH, cc = lane % C::CH;
        apx = ld<u32x4>(S.nk + (kv ? S.nv - S.nk : 0) + 16 * cc);
        const int pg = S.bt[(c - 1) / PS];
        apdst = const_cast<uint8_t *>(a.k) + (kv ? a.v - a.k : 0) + (size_t)pg * S.page_stride + S.head_off +
                (size_t)((c - 1) % PS) * C::RAW_ROW + 16 * cc;
      }
    }
  }

  KRegs<C> k0, k1;
  issue_block<C, PS, FP8, WAVES>(a, S, S.kb0, k0, st0);

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
    if constexpr (AP) {
      if (j == 0 && apdst) st<u32x4>(apdst, apx);
    }
    if (j + 1 < S.nblk) issue_block<C, PS, FP8, WAVES>(a, S, kbase + C::KB, k1, st1);
    compute_block<C, PS, FP8, WAVES>(a, S, kbase, k0, st0, vwide, qf, o, m, l, g);
    if (j + 1 < S.nblk) {
      block_ready<C>(k1);
      if (j + 2 < S.nblk) issue_block<C, PS, FP8, WAVES>(a, S, kbase + 2 * C::KB, k0, st0);
      compute_block<C, PS, FP8, WAVES>(a, S, kbase + C::KB, k1, st1, vwide, qf, o, m, l, g);
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

}  // namespace dc
}  // namespace ckv
