// prefix_prefill_attn for bf16 queries over a bf16 or fp8-E4M3 paged pool:
// the device code of one row tile (work item), shared by the prefill kernel
// and the mixed prefill + decode kernel.
//
// Work item: one workgroup (4 waves) = 128 consecutive "rows" of one
// (sequence, KV head), a row being a (new-turn token, query head of the
// group) pair flattened as R = t * G + hh.  Packing the G query heads of a
// KV head into the M dimension lets every K/V byte staged in LDS serve all
// of them and keeps the causal diagonal narrow (128 / G tokens per tile).
//
// Data movement, per block of BN keys read through the block table:
//   * K and V rows go from HBM straight into an NS-stage LDS ring with
//     global_load_lds_dwordx4 (no register staging): a wave-uniform base
//     (page, head, first row; scalar arithmetic) plus a per-lane offset
//     fixed for the whole kernel, which also XOR-swizzles the ring.  One
//     barrier per block; loads for block j + NS - 1 are issued while block j
//     is computed, in one burst after the barrier (head_dim 256: in three
//     parts spread over the step, as one wave per SIMD has no partner wave
//     to cover the burst).
//   * fp8 pools stay raw in LDS.  Each wave widens the codes of its own
//     operands in registers (exactly: every E4M3 value is a bf16 value): K
//     16 codes per read (two k-steps; Q is loaded in the matching order of
//     d), V^T 8 codes per ds_read_b64_tr_b8 (8 keys of one column).  There
//     is no widening pass and no second barrier, and the operand reads move
//     half the LDS bytes of the bf16 path.
// Math, per wave of 32 rows:
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (Q stays in registers).  The
//     lane that owns a query row holds a column of S^T, so the row max / row
//     sum are in-lane plus one exchange between the half-waves.  K rows are
//     fed in a permuted order (pi) so that the probabilities a lane holds are
//     exactly the 8 consecutive keys it supplies as the B operand of
//     O^T += V^T P^T; V^T operands come from row-major V in LDS through
//     ds_read_b64_tr_b16 (4 keys x 16 columns transposed per 16 lanes).
//   * Online softmax in fp32 with base-2 exponentials; the row sum adds the
//     bf16 probabilities the MFMA consumes, two at a time.  The reference
//     maximum only moves (and O is rescaled) when a block's maximum exceeds
//     it by more than 2^8, which leaves the result unchanged but skips most
//     rescales.  The exponentials are taken first, one FMA (scale and
//     reference folded) and one exp per score, and the row maximum is
//     reduced only when the block's row sum shows that it may move.  fp8
//     pools take the same lazy way with the key scale in the FMA and the
//     value scale in the exponent's addend.
//     Masking only on blocks that straddle the causal diagonal or the window
//     edge.
#pragma once

#include "common.hpp"

namespace ckv {
namespace pf {

struct PrefillArgs {
  const uint16_t *q;
  uint16_t *out;
  const uint8_t *k, *v;
  const float *k_scale, *v_scale;
  const int32_t *bt, *ctx, *cu;
  int32_t num_seqs, max_pages, h_q, h_kv, group;
  float scale_log2;  // softmax_scale * log2(e)
  int32_t window;
  int32_t tiles;      // grid.y: max row tiles of a sequence
  int32_t splits;     // key partitions per row tile (grid.x = H_kv * splits)
  int32_t split_len;  // keys per partition (a multiple of the block size)
  float *part_o;      // splits > 1: [total_q * H_q][splits][D] fp32
  float *part_ml;     // splits > 1: [total_q * H_q][splits][2] (m, l)
  // fused append (bf16 pools, Cfg::AP): the new turn's K and V rows
  // [total_q][H_kv][D]; the kernel writes them into their pool slots and
  // reads the new keys from here instead of from the pool
  const uint8_t *k_new, *v_new;
};

constexpr int kRows = 128;  // rows per workgroup
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kRescaleSlack = 8.0f;  // log2 units: defer rescaling below 2^8

// Row m of a 32-key S^T tile holds key pi(m) of the tile.  With
// m = 8i + 4h + j the lane that receives row m (half h, element 4i + j)
// gets key 16(i/2) + 8h + 4(i%2) + j, so elements 8s..8s+7 of a lane are
// keys 16s + 8h + 0..7.
__device__ __forceinline__ int pi_row(int m) {
  const int i = m >> 3, h = (m >> 2) & 1, j = m & 3;
  return 16 * (i >> 1) + 8 * h + 4 * (i & 1) + j;
}

template <int D, int BN, bool FP8, int PS, bool APPEND = false>
struct Cfg {
  static constexpr bool AP = APPEND;                   // fused append (bf16 pools)
  static constexpr int ROW = D * 2;                    // bf16 bytes per key row in LDS
  static constexpr int CH = D / 8;                     // 16-byte chunks per bf16 row
  static constexpr int BN_ = BN;                       // keys per block
  static constexpr bool F8 = FP8;                      // raw fp8 rows in LDS
  static constexpr int BLK = BN * ROW;                 // bf16 bytes of one K (or V) block
  static constexpr int RAW_ROW = FP8 ? D : D * 2;      // pool bytes per key row
  static constexpr int RCH = RAW_ROW / 16;             // 16-byte chunks per pool row
  static constexpr int RAW_BLK = BN * RAW_ROW;         // pool bytes of one block
  static constexpr int DPW = RAW_BLK / 2 / 1024;       // 1-KB loads per wave per block
  static constexpr int RPD = 1024 / RAW_ROW;           // rows per load
  static constexpr int NT = BN / 32;                   // S^T tiles per block
  static constexpr int DS = D / 16;                    // QK^T k-steps
  static constexpr int DT = D / 32;                    // output d-tiles
  static constexpr int NQK = NT * DS;                  // QK^T MFMAs per block
  // Chunks in which a wave issues its loads of a step.  At head_dim 256 (one
  // wave per SIMD) no partner wave covers the stall of a burst of 16 loads,
  // so a third goes out after the barrier, a third after the first S^T half
  // and the rest inside PV; with two waves per SIMD one burst is faster.
  static constexpr int SPREAD = (D >= 256 && !FP8) ? 3 : 1;
  // two-stage K ring + two-stage V ring
  static constexpr int LDS = 4 * RAW_BLK;
  static_assert(RAW_BLK % 2048 == 0, "each wave issues whole 1-KB loads");
  static_assert(PS % RPD == 0, "a load never straddles a page");
  // two workgroups per CU below head_dim 256; one (as the registers allow) above
  static_assert(LDS <= (D >= 256 ? 160 : 80) * 1024, "LDS budget");
  static_assert(!(AP && FP8), "the fused append writes bf16 rows");
};

// XOR swizzles of the 16-byte chunk index within a bf16 row.
//  K: the 16 keys read together by one S^T operand load (16 lanes) differ in
//     their low 4 bits, so key & 15 spreads them over 16 chunk slots.
//  V: a transposed read covers 4 consecutive keys x 2 chunks per 16 lanes;
//     shifting each key's chunk pair by 4 * (key & 3) keeps them apart.
template <int CH>
__device__ __forceinline__ int swz_k(int key) { return key & ((CH < 16 ? CH : 16) - 1); }
template <int CH>
__device__ __forceinline__ int swz_v(int key) { return (4 * (key & 3)) & (CH - 1); }

// XOR swizzles of the 16-byte chunk index within a raw fp8 row (RCH chunks).
//  K: a lane reads 16 codes (two k-steps) of key pi(col); the 8 keys of each
//     8-lane group (pi of 0-7 or 8-15 within 16) and the even and the odd
//     keys among 16 lanes land on distinct chunks.
//  V: a transposed 8-bit read covers 8 consecutive keys x two 8-byte runs
//     per 16 lanes; shifting key k's chunks by k & 7 spreads them over all
//     sixteen 8-byte bank groups of a 128-byte row.
template <int RCH>
__device__ __forceinline__ int swz8_k(int key) { return (((key >> 1) ^ ((key & 1) << 1)) & 7) & (RCH - 1); }
template <int RCH>
__device__ __forceinline__ int swz8_v(int key) { return key & 7 & (RCH - 1); }

// Workgroup barrier without a memory fence: LDS reads of this wave are
// complete (lgkmcnt 0) and the compiler may not move memory accesses across.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Load plan: wave w fills half h = w & 1 of tensor t = w >> 1 (0 = K, 1 = V)
// of each block, i.e. rows h BN/2 .. h BN/2 + BN/2 - 1, with DPW wave-wide
// 1-KB loads of RPD rows each.  Those rows span NPW pages (DPP loads each),
// so a block costs the wave NPW page-table reads and NPW scalar bases; the
// per-lane part of every load's address is fixed for the whole kernel.
// Per-lane byte offset of load i, relative to the scalar base of its page
// (the page's first row covered by this wave).  Lane l lands in LDS slot l of
// the load (row l / RCH, chunk slot l % RCH) and fetches the chunk that the
// swizzle assigns to that slot.
template <class C, int PS, bool FP8>
__device__ __forceinline__ void lane_offsets(uint32_t (&loff)[C::DPW]) {
  constexpr int HROWS = C::RAW_BLK / 2 / C::RAW_ROW;
  constexpr int NPW = HROWS > PS ? HROWS / PS : 1;
  constexpr int DPP = C::DPW / NPW;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int t = wave >> 1, h = wave & 1;
#pragma unroll
  for (int i = 0; i < C::DPW; ++i) {
    const int row = h * HROWS + i * C::RPD + lane / C::RCH;  // row within the block
    const int slot = lane % C::RCH;
    const int chunk = FP8 ? slot ^ (t == 0 ? swz8_k<C::RCH>(row) : swz8_v<C::RCH>(row))
                          : slot ^ (t == 0 ? swz_k<C::CH>(row) : swz_v<C::CH>(row));
    loff[i] = (uint32_t)(((i % DPP) * C::RPD + lane / C::RCH) * C::RAW_ROW + chunk * 16);
  }
}

// Page ids of the NPW pages this wave loads for the block at kbase (scalar
// loads through the constant address space).  Pages are looked up by the
// first row the wave covers in them, clamped to kv_end - 1.
template <class C, int PS>
__device__ __forceinline__ void block_pages(const int32_t *bt, int kbase, int kv_end, int (&pg)[C::DPW]) {
  constexpr int HROWS = C::RAW_BLK / 2 / C::RAW_ROW;
  constexpr int NPW = HROWS > PS ? HROWS / PS : 1;
  const int h = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) & 1;
#pragma unroll
  for (int p = 0; p < NPW; ++p) {
    const int key = min(kbase + h * HROWS + p * PS, kv_end - 1);
    pg[p] = ldc(bt, (int)((uint32_t)key / PS));
  }
}

// Issue this wave's loads [LO, HI) (of DPW) of one block of its tensor into a
// ring stage; the whole block by default.  Rows at or beyond
// kv_end (last block only) are redirected to row kv_end - 1: valid, finite
// data in the same page as the load's first row (or that row's page), which
// the causal mask removes.
//
// With the fused append (C::AP), keys at or beyond `pnew` (the new turn) are
// read from the caller's rows at `nsrc` (this wave's tensor, the sequence's
// first new token, KV head g; consecutive tokens H_kv rows apart) through
// per-lane addresses, on the blocks that hold any.
template <class C, int PS, bool FP8, int LO = 0, int HI = C::DPW>
__device__ __forceinline__ void issue_block(const PrefillArgs &a, const int32_t *bt, int g, int kbase,
                                            int kv_end, const int (&pg)[C::DPW],
                                            const uint32_t (&loff)[C::DPW], lds_u8 *ring_stage,
                                            int pnew = 0, const uint8_t *nsrc = nullptr) {
  constexpr int HROWS = C::RAW_BLK / 2 / C::RAW_ROW;
  constexpr int NPW = HROWS > PS ? HROWS / PS : 1;
  constexpr int DPP = C::DPW / NPW;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t = wave >> 1, h = wave & 1;
  const uint8_t *tens = t == 0 ? a.k : a.v;
  const size_t page_stride = (size_t)a.h_kv * PS * C::RAW_ROW;
  const size_t head_off = (size_t)g * PS * C::RAW_ROW;
  lds_u8 *wdst = ring_stage + h * (C::RAW_BLK / 2);
  if constexpr (C::AP) {
    if (kbase + C::BN_ > pnew) {
      // load i covers rows of page pg[i / DPP] (looked up by its first row,
      // clamped); rows past kv_end repeat row kv_end - 1, a new-turn row, so
      // every pool row read here lies in that page
      const int lane = threadIdx.x & 63;
      const size_t nstride = (size_t)a.h_kv * C::RAW_ROW;
#pragma unroll
      for (int i = LO; i < HI; ++i) {
        const int r0 = kbase + h * HROWS + i * C::RPD;
        const int kp = min(r0 + lane / C::RCH, kv_end - 1);
        const uint32_t co = loff[i] % C::RAW_ROW;
        const uint8_t *src =
            kp >= pnew ? nsrc + (size_t)(kp - pnew) * nstride + co
                       : tens + (size_t)pg[i / DPP] * page_stride + head_off + (size_t)(kp % PS) * C::RAW_ROW + co;
        dma16(src, wdst + i * 1024);
      }
      return;
    }
  }
  if (kbase + C::BN_ <= kv_end) {
#pragma unroll
    for (int p = 0; p < NPW; ++p) {
      const int key = kbase + h * HROWS + p * PS;
      const uint8_t *base =
          tens + (size_t)pg[p] * page_stride + head_off + (size_t)((uint32_t)key % PS) * C::RAW_ROW;
#pragma unroll
      for (int i = p * DPP; i < (p + 1) * DPP; ++i)
        if (i >= LO && i < HI) dma16_sv(base, loff[i], wdst + i * 1024);
    }
  } else {
    // last block: per-load page of its first row (clamped), per-lane clamp
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = LO; i < HI; ++i) {
      const int kf = min(kbase + h * HROWS + i * C::RPD, kv_end - 1);
      const int pgi = ldc(bt, (int)((uint32_t)kf / PS));
      const uint8_t *base = tens + (size_t)pgi * page_stride + head_off;
      const int kp = min(kbase + h * HROWS + i * C::RPD + lane / C::RCH, kv_end - 1);
      const uint32_t voff = (uint32_t)((kp % PS) * C::RAW_ROW) + (loff[i] % C::RAW_ROW);
      dma16_sv(base, voff, wdst + i * 1024);
    }
  }
}


// Exchange between lane l and lane l ^ 32 (the two halves of a wave).
__device__ __forceinline__ float half_swap_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_swap_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Per-workgroup state that the block loop carries.
template <class C>
struct Tile {
  bf16x8 qf[C::DS];
  f32x16 o[C::DT];
  float m, l;
  int pg[C::DPW];          // page ids of the block being issued
  uint32_t loff[C::DPW];   // per-lane load offsets
  int kb_iss;              // first key of the block being issued (-1: none)
  lds_u8 *dst_iss;         // its ring stage
  int g, t, ipos, i_min, i_max, kv_end, kb_begin, nblk, half, col, gq, li;
  int pnew;                // fused append: first new-turn position
  const uint8_t *nsrc;     // fused append: this wave's tensor's new rows
  // per-lane LDS byte offsets within a bf16 block: V^T reads of output tile
  // dt (keys 8 (gq / 2) + li / 4, plus 32 tt + 16 ks and 4 for the second
  // read) and K reads of k-step ds (key pi(col), plus 32 tt).  The swizzles
  // depend on key & 15 (K) and key & 3 (V) only, so the tt / ks parts are
  // plain immediates and the loop does no address arithmetic.
  int offv[C::DT], offk[C::DS];
};

template <class C>
__device__ __forceinline__ void lds_offsets(Tile<C> &T) {
  if constexpr (C::F8) {
    // K: the 16 codes of k-steps 2p, 2p+1 of key pi(col) (chunk 2p + half);
    // V^T: group lane 2m + h names key 8 (gq / 2) + m, columns
    // 32 dt + 16 (gq & 1) + 8 h .. + 7 (chunk 2 dt + (gq & 1), run h)
    const int key = pi_row(T.col);
#pragma unroll
    for (int p = 0; p < C::DS / 2; ++p)
      T.offk[p] = key * C::RAW_ROW + (((2 * p + T.half) ^ swz8_k<C::RCH>(key)) << 4);
    const int vkey = 8 * (T.gq >> 1) + (T.li >> 1);
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
      T.offv[dt] = vkey * C::RAW_ROW + (((2 * dt + (T.gq & 1)) ^ swz8_v<C::RCH>(vkey)) << 4) + 8 * (T.li & 1);
    return;
  }
  const int key0 = 8 * (T.gq >> 1) + (T.li >> 2);
  const int dsub = 16 * (T.gq & 1) + 4 * (T.li & 3);
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) {
    const int byte = 2 * (32 * dt + dsub);
    T.offv[dt] = key0 * C::ROW + (((byte >> 4) ^ swz_v<C::CH>(key0)) << 4) + (byte & 15);
  }
  const int key = pi_row(T.col);
#pragma unroll
  for (int ds = 0; ds < C::DS; ++ds)
    T.offk[ds] = key * C::ROW + (((2 * ds + T.half) ^ swz_k<C::CH>(key)) << 4);
}

// Part P (0 or 1) of S^T = K Q^T for one block: k-steps [P DS/2, (P+1) DS/2)
// of every tile, so that each half can be scheduled against a different
// stretch of the previous block's softmax and holds NT independent
// accumulation chains.  Row m of tile tt is key 32 tt + pi(m).
template <class C, int P>
__device__ __forceinline__ void qk_part(const lds_u8 *kb, const Tile<C> &T, f32x16 (&s)[C::NT]) {
  if constexpr (C::F8) {
    // one 16-code read per tile feeds k-steps 2p and 2p + 1
#pragma unroll
    for (int pp = 0; pp < C::DS / 4; ++pp) {
      const int p = P * (C::DS / 4) + pp;
      u32x4 x[C::NT];
#pragma unroll
      for (int tt = 0; tt < C::NT; ++tt) x[tt] = lds_ld16(kb + T.offk[p] + 32 * tt * C::RAW_ROW);
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int tt = 0; tt < C::NT; ++tt) {
          if (p == 0 && e == 0) s[tt] = f32x16{};
          const u32x4 w = fp8x8_to_bf16x8(e ? u32x2{x[tt].z, x[tt].w} : u32x2{x[tt].x, x[tt].y});
          s[tt] = mfma32x32x16(as_bf16x8(w), T.qf[2 * p + e], s[tt]);
        }
    }
    return;
  }
#pragma unroll
  for (int n = 0; n < C::NQK / 2; ++n) {
    const int tt = n % C::NT, ds = P * (C::DS / 2) + n / C::NT;
    if (ds == 0) s[tt] = f32x16{};
    const u32x4 kx = lds_ld16(kb + T.offk[ds] + 32 * tt * C::ROW);
    s[tt] = mfma32x32x16(as_bf16x8(kx), T.qf[ds], s[tt]);
  }
}

// fp8 scales of block j's 16-key slices (key scale times the softmax scale
// in log2 units, and the value scale) and the causal / window mask of its
// scores (the mask only on blocks that straddle the diagonal or the window
// edge).  The scores stay unscaled.
template <class C, int PS, bool FP8>
__device__ __forceinline__ void scale_mask(const PrefillArgs &a, const int32_t *bt, const Tile<C> &T,
                                           int j, f32x16 (&s)[C::NT], float (&ksc)[C::NT * 2],
                                           float (&vsc)[C::NT * 2]) {
  constexpr int BN = C::BN_;
  const int kbase = (T.kb_begin + j) * BN;
  const int half = T.half;
  if constexpr (FP8) {
#pragma unroll
    for (int q = 0; q < C::NT * 2; ++q) {
      const int kp = min(kbase + 16 * q, T.kv_end - 1);
      const int idx = ldc(bt, (int)((uint32_t)kp / PS)) * a.h_kv + T.g;
      ksc[q] = a.scale_log2 * ldc(a.k_scale, idx);
      vsc[q] = ldc(a.v_scale, idx);
    }
  }
  const int W = a.window;
  const bool full = (kbase + BN - 1 <= T.i_min) && (W <= 0 || T.i_max - kbase < W);
  if (!full) {
#pragma unroll
    for (int tt = 0; tt < C::NT; ++tt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = e >> 2, jj = e & 3;
        const int kp = kbase + 32 * tt + 16 * (i >> 1) + 8 * half + 4 * (i & 1) + jj;
        const bool vis = (kp <= T.ipos) & ((W <= 0) | (T.ipos - kp < W));
        s[tt][e] = vis ? s[tt][e] : kNegInf;
      }
    }
  }
}

// Row maximum of block j's scores in log2 units (both halves of the wave),
// and the lazy move of the reference maximum: only when the block's maximum
// exceeds it by more than the slack; O and l are then rescaled.
template <class C, bool FP8>
__device__ __forceinline__ void bump_max(const PrefillArgs &a, Tile<C> &T, const f32x16 (&s)[C::NT]) {
  float mx = kNegInf;
#pragma unroll
  for (int tt = 0; tt < C::NT; ++tt)
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[tt][e]);
  if constexpr (!FP8) mx *= a.scale_log2;  // scores stay unscaled until the exp
  mx = half_swap_max(mx);
  const bool bump = mx > T.m + kRescaleSlack;
  if (__builtin_amdgcn_ballot_w64(bump)) {
    // lanes that keep their reference scale by 1 (their m may still be -inf
    // when every key so far was masked); a first bump from -inf scales by 0
    const float alpha = bump ? fast_exp2(T.m - mx) : 1.f;
    T.m = bump ? mx : T.m;
    T.l *= alpha;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) T.o[dt] *= alpha;
  }
}

// O^T += V^T P^T for one 16-key slice (tile tt, half ks) of block j with the
// packed bf16 probabilities pb of that slice.  Transposed V reads: 16-lane
// group gq covers columns 16(gq&1) + 0..15 of a 32-column tile and keys
// key0 .. key0+3 (key0+4 .. +7 on the second read, same swizzle); lane li of
// the group addresses key key0 + li/4, columns 4(li%4) .. +3.
template <class C>
__device__ __forceinline__ void pv_slice(Tile<C> &T, const lds_u8 *vb, int tt, int ks, const u32x4 &pb) {
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) {
    u32x4 vx;
    if constexpr (C::F8) {
      // 8 keys of one column, widened in registers
      vx = fp8x8_to_bf16x8(ds_read_tr8(vb + T.offv[dt] + (32 * tt + 16 * ks) * C::RAW_ROW));
    } else {
      const lds_u8 *r0 = vb + T.offv[dt] + (32 * tt + 16 * ks) * C::ROW;
      const u32x2 lo = ds_read_tr16(r0);
      const u32x2 hi = ds_read_tr16(r0 + 4 * C::ROW);
      vx = u32x4{lo.x, lo.y, hi.x, hi.y};
    }
    T.o[dt] = mfma32x32x16(as_bf16x8(vx), as_bf16x8(pb), T.o[dt]);
  }
}

// bf16 pools: the block's probabilities P = exp2(scale * s - m), packed to
// bf16, and this lane's part of the block's row sum (the bf16 values the MFMA
// consumes, two at a time).
template <class C>
__device__ __forceinline__ float exp_block(const f32x16 (&s)[C::NT], float scale, float m,
                                           u32x4 (&pb)[C::NT * 2]) {
  float lb = 0.f;
#pragma unroll
  for (int q = 0; q < C::NT * 2; ++q) {
    float p[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) p[e] = fast_exp2(__builtin_fmaf(s[q >> 1][8 * (q & 1) + e], scale, -m));
    pb[q] = u32x4{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]),
                  pack_bf16x2(p[6], p[7])};
    lb = add_bf16x2(pb[q].x, lb);
    lb = add_bf16x2(pb[q].y, lb);
    lb = add_bf16x2(pb[q].z, lb);
    lb = add_bf16x2(pb[q].w, lb);
  }
  return lb;
}

// Loads [K DPW / SPREAD, (K + 1) DPW / SPREAD) of the block this wave issues
// at this step (chunk 0 right after the barrier, the rest spread over the
// step's MFMAs).
template <class C, int PS, bool FP8, int K>
__device__ __forceinline__ void issue_chunk(const PrefillArgs &a, const int32_t *bt, const Tile<C> &T) {
  if constexpr (K >= 1 && K < C::SPREAD) {
    if (T.kb_iss >= 0)
      issue_block<C, PS, FP8, K * C::DPW / C::SPREAD, (K + 1) * C::DPW / C::SPREAD>(
          a, bt, T.g, T.kb_iss, T.kv_end, T.pg, T.loff, T.dst_iss, T.pnew, T.nsrc);
  }
}

// Softmax of block j (scores s after scale_mask) and O^T += V^T P^T with V
// of block j (bf16 layout at vb).  The two halves of the next block's S^T
// are issued around the exponentials.
//
// bf16 pools skip the row maximum on most blocks: the exponentials are taken
// against the current reference maximum first.  Every probability is at most
// the block's row sum, so a sum of at most 2^slack (on both halves) shows
// that no score rose more than the slack above the reference, the case in
// which the maximum would not move anyway.  Otherwise (a larger or
// non-finite sum, e.g. while a row has seen no key and its reference is
// -inf) the block is redone the reduced way: row maximum, possible move of
// the reference with the rescale of O and l, exponentials again.  The
// reference maximum therefore follows the same rule as on the reduced path,
// block by block.  fp8 pools do the same with the key scale as the FMA's
// multiplier and the value scale in its addend.
template <class C, int PS, bool FP8>
__device__ __forceinline__ void softmax_pv(const PrefillArgs &a, const int32_t *bt, Tile<C> &T, f32x16 (&s)[C::NT],
                                           const float (&ksc)[C::NT * 2], const float (&vsc)[C::NT * 2],
                                           const lds_u8 *vb, const lds_u8 *kb_next, f32x16 (&s_next)[C::NT]) {
  __builtin_amdgcn_s_setprio(1);
  if constexpr (!FP8) {
    constexpr float kSlackSum = 256.f;  // 2^kRescaleSlack
    static_assert(kRescaleSlack == 8.0f, "kSlackSum is 2^kRescaleSlack");
    u32x4 pb[C::NT * 2];
    qk_part<C, 0>(kb_next, T, s_next);
    issue_chunk<C, PS, FP8, 1>(a, bt, T);
    float lb = exp_block<C>(s, a.scale_log2, T.m, pb);
    // second half of the next block's S^T, independent of the softmax
    qk_part<C, 1>(kb_next, T, s_next);
    if (__builtin_amdgcn_ballot_w64(!(lb <= kSlackSum) | (T.m == kNegInf))) {
      bump_max<C, FP8>(a, T, s);
      lb = exp_block<C>(s, a.scale_log2, T.m == kNegInf ? 0.f : T.m, pb);
    }
    T.l += lb;
#pragma unroll
    for (int q = 0; q < C::NT * 2; ++q) {
      pv_slice<C>(T, vb, q >> 1, q & 1, pb[q]);
      if (q == 1) issue_chunk<C, PS, FP8, 2>(a, bt, T);
    }
  } else {
    constexpr float kSlackSum = 256.f;  // 2^kRescaleSlack
    // The value scale rides in the exponent: P v_scale = exp2(k_scale scale s
    // - m + log2 v_scale), one FMA and one exp per score; the slice's row
    // sum divided by v_scale is its part of l.  Needs a positive, finite key
    // scale and a value scale within 2^-100 .. 2^100, so that the slice sums
    // neither flush nor overflow (a page of zeros has scale 0: such blocks
    // take the reduced way).
    bool pos = true;
    float bias[C::NT * 2], ivs[C::NT * 2];
#pragma unroll
    for (int q = 0; q < C::NT * 2; ++q) {
      pos &= (ksc[q] > 0.f) & (ksc[q] <= 3.0e38f) & (vsc[q] >= 0x1p-100f) & (vsc[q] <= 0x1p100f);
      bias[q] = __builtin_amdgcn_logf(vsc[q]) - T.m;
      ivs[q] = __builtin_amdgcn_rcpf(vsc[q]);
    }
    u32x4 pb[C::NT * 2];
    qk_part<C, 0>(kb_next, T, s_next);
    float lb = 0.f;
#pragma unroll
    for (int q = 0; q < C::NT * 2; ++q) {
      float p[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) p[e] = fast_exp2(__builtin_fmaf(s[q >> 1][8 * (q & 1) + e], ksc[q], bias[q]));
      pb[q] = u32x4{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]),
                    pack_bf16x2(p[6], p[7])};
      float ss = add_bf16x2(pb[q].x, 0.f);
      ss = add_bf16x2(pb[q].y, ss);
      ss = add_bf16x2(pb[q].z, ss);
      ss = add_bf16x2(pb[q].w, ss);
      lb = __builtin_fmaf(ss, ivs[q], lb);
    }
    // second half of the next block's S^T, independent of the softmax
    qk_part<C, 1>(kb_next, T, s_next);
    if (!pos || __builtin_amdgcn_ballot_w64(!(lb <= kSlackSum) | (T.m == kNegInf))) {
      // reduced way: scaled scores (masked ones stay -inf), row maximum,
      // P = exp2(k_scale scale s - m) v_scale.  The row sum adds the bf16
      // values of P v_scale divided by v_scale, the weights the MFMA
      // multiplies, unless the value scale is outside 2^-100 .. 2^100 (0 for
      // a page of zeros): then the fp32 probabilities
#pragma unroll
      for (int q = 0; q < C::NT * 2; ++q)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = s[q >> 1][8 * (q & 1) + e];
          s[q >> 1][8 * (q & 1) + e] = x == kNegInf ? kNegInf : x * ksc[q];
        }
      bump_max<C, FP8>(a, T, s);
      const float m_use = T.m == kNegInf ? 0.f : T.m;
      lb = 0.f;
#pragma unroll
      for (int q = 0; q < C::NT * 2; ++q) {
        float p[8], praw = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          p[e] = fast_exp2(s[q >> 1][8 * (q & 1) + e] - m_use);
          praw += p[e];
          p[e] *= vsc[q];
        }
        pb[q] = u32x4{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]),
                      pack_bf16x2(p[6], p[7])};
        float ss = add_bf16x2(pb[q].x, 0.f);
        ss = add_bf16x2(pb[q].y, ss);
        ss = add_bf16x2(pb[q].z, ss);
        ss = add_bf16x2(pb[q].w, ss);
        const bool vs_ok = (vsc[q] >= 0x1p-100f) & (vsc[q] <= 0x1p100f);
        lb = vs_ok ? __builtin_fmaf(ss, ivs[q], lb) : lb + praw;
      }
    }
    T.l += lb;
#pragma unroll
    for (int q = 0; q < C::NT * 2; ++q) pv_slice<C>(T, vb, q >> 1, q & 1, pb[q]);
  }
  __builtin_amdgcn_s_setprio(0);
}

// The K ring holds K of blocks j+1 and j+2 while step j runs, the V ring V
// of blocks j and j+1.  Stage of block b: b & 1 in both rings.
template <class C>
struct Rings {
  lds_u8 *k, *v;
  __device__ __forceinline__ lds_u8 *kst(int b) const { return k + (b & 1) * C::RAW_BLK; }
  __device__ __forceinline__ lds_u8 *vst(int b) const { return v + (b & 1) * C::RAW_BLK; }
};

// Loads issued at step j (j = -1 is the prologue): K of block j+2 by waves 0
// and 1, V of block j+1 by waves 2 and 3.  Page ids resolve while the wave
// waits for the previous step's loads.
template <class C, int PS, bool FP8, int U, bool ALL = false>
__device__ __forceinline__ void wait_and_issue(const PrefillArgs &a, const int32_t *bt, Tile<C> &T,
                                               int j, const Rings<C> &R) {
  constexpr int BN = C::BN_;
  const int bi = j + 2 - T.t;  // block whose tensor-t half this wave loads
  const bool iss = bi < T.nblk;
  const int kb_iss = (T.kb_begin + bi) * BN;
  if (iss) block_pages<C, PS>(bt, kb_iss, T.kv_end, T.pg);
  wait_vmcnt<0>();
  lds_barrier();
  // stage of block bi: (j + 2) & 1 = U for K, (j + 1) & 1 = U ^ 1 for V
  lds_u8 *dst = T.t == 0 ? R.k + U * C::RAW_BLK : R.v + (U ^ 1) * C::RAW_BLK;
  if constexpr (C::SPREAD > 1) {
    T.kb_iss = iss ? kb_iss : -1;
    T.dst_iss = dst;
  }
  if (iss) {
    if constexpr (ALL || C::SPREAD == 1)
      issue_block<C, PS, FP8>(a, bt, T.g, kb_iss, T.kv_end, T.pg, T.loff, dst, T.pnew, T.nsrc);
    else
      issue_block<C, PS, FP8, 0, C::DPW / C::SPREAD>(a, bt, T.g, kb_iss, T.kv_end, T.pg, T.loff, dst,
                                                     T.pnew, T.nsrc);
  }
}

// Step j: K of block j+1 and V of block j are resident after the barrier;
// S^T of block j+1 is computed around block j's softmax, then O^T for
// block j.  U = j & 1 (compile time, so every stage address folds).
template <class C, int PS, bool FP8, int U>
__device__ __forceinline__ void step(const PrefillArgs &a, const int32_t *bt, Tile<C> &T, int j,
                                     f32x16 (&s_cur)[C::NT], f32x16 (&s_nxt)[C::NT], const Rings<C> &R) {
  wait_and_issue<C, PS, FP8, U>(a, bt, T, j, R);
  const lds_u8 *kb = R.k + (U ^ 1) * C::RAW_BLK;  // K of block j+1
  const lds_u8 *vb = R.v + U * C::RAW_BLK;        // V of block j
  float ksc[C::NT * 2], vsc[C::NT * 2];
  scale_mask<C, PS, FP8>(a, bt, T, j, s_cur, ksc, vsc);
  // (past the last block this reads a stale K stage; the result is unused)
  softmax_pv<C, PS, FP8>(a, bt, T, s_cur, ksc, vsc, vb, kb, s_nxt);
}

// Fused append: the new K and V rows that one workgroup writes into the
// pool, in units of one 16-byte chunk: unit u is chunk u % CH of the K
// ((u / CH) & 1 == 0) or V row of token tok_lo + u / (2 CH), KV head g.
// Each thread moves up to NAP units per batch (all loads, then all stores),
// held in vector values rather than arrays.  K and V addresses are the K
// address plus a
// per-lane multiple of the V - K distance: a per-lane choice between two
// pointer members would be compiled as a load from a dynamically indexed
// copy of this struct in scratch memory.
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));
template <class C, int PS>
struct AppendRows {
  static constexpr int NAP = C::CH >= 32 ? 2 : 4;  // head_dim 256: registers are scarce
  const uint8_t *src_k;          // K row of token 0 of the sequence, head g
  uint8_t *dst_k;                // K pool, head g of page 0
  ptrdiff_t src_vk, dst_vk;      // V minus K addresses (input, pool)
  const int32_t *bt;
  int tok_lo, pos0, units, stride;  // stride: bytes between tokens in the input

  __device__ __forceinline__ void load(int u0, u32x16 &x, u32x4 &pg) const {
#pragma unroll
    for (int k = 0; k < NAP; ++k) {
      const int u = u0 + (int)threadIdx.x + k * kThreads;
      if (u < units) {
        const int tok = tok_lo + u / (2 * C::CH), kv = (u / C::CH) & 1, c = u % C::CH;
        const u32x4 v = ld<u32x4>(src_k + (kv ? src_vk : 0) + (size_t)tok * stride + 16 * c);
        x[4 * k] = v.x;
        x[4 * k + 1] = v.y;
        x[4 * k + 2] = v.z;
        x[4 * k + 3] = v.w;
        pg[k] = (uint32_t)bt[(pos0 + tok) / PS];
      }
    }
  }
  __device__ __forceinline__ void store(int u0, const u32x16 &x, const u32x4 &pg) const {
    const size_t page_stride = (size_t)stride / C::ROW * PS * C::ROW;  // H_kv * PS rows
#pragma unroll
    for (int k = 0; k < NAP; ++k) {
      const int u = u0 + (int)threadIdx.x + k * kThreads;
      if (u < units) {
        const int tok = tok_lo + u / (2 * C::CH), kv = (u / C::CH) & 1, c = u % C::CH;
        const int pos = pos0 + tok;
        st<u32x4>(dst_k + (kv ? dst_vk : 0) + (size_t)pg[k] * page_stride + (size_t)(pos % PS) * C::ROW + 16 * c,
                  u32x4{x[4 * k], x[4 * k + 1], x[4 * k + 2], x[4 * k + 3]});
      }
    }
  }
  // units [u0, units), batch by batch
  __device__ __forceinline__ void copy_from(int u0) const {
    for (; u0 < units; u0 += NAP * kThreads) {
      u32x16 x{};
      u32x4 pg{};
      load(u0, x, pg);
      store(u0, x, pg);
    }
  }
};

// One work item: row tile `tile_rev` (counted from the last) of the
// sequence of cost rank `rank`, KV head and key partition from `hx`
// (hx = H_kv * split + g).  `lds` holds Cfg::LDS bytes, 1024-aligned.
// AP: fused append (PrefillArgs::k_new / v_new).
template <int D, int BN, bool FP8, int PS, bool AP = false>
__device__ __forceinline__ void prefill_tile(const PrefillArgs &a, lds_u8 *lds, int hx, int tile_rev,
                                             int rank) {
  using C = Cfg<D, BN, FP8, PS, AP>;
  Rings<C> R;
  R.k = lds;
  R.v = R.k + 2 * C::RAW_BLK;

  // hx = H_kv * split + g (KV head fastest); with splits > 1 each item
  // covers one key partition
  const int g = hx % a.h_kv;
  const int split = hx / a.h_kv;
  const int tile = a.tiles - 1 - tile_rev;  // later (costlier) tiles first
  // `rank` orders sequences by decreasing per-tile cost (retained prefix
  // plus new turn), so the longest tiles are dealt out first and the short
  // ones fill the tail
  __shared__ int rank_cost[kThreads];
  __shared__ int rank_seq;
  int b = rank;
  if (a.num_seqs <= kThreads) {
    const int nb = a.num_seqs, tid = threadIdx.x;
    if (tid < nb) rank_cost[tid] = a.ctx[tid] + (a.cu[tid + 1] - a.cu[tid]);
    __syncthreads();
    if (tid < nb) {
      const int c = rank_cost[tid];
      int r = 0;
      for (int o = 0; o < nb; ++o) {
        const int co = rank_cost[o];
        r += (co > c) | ((co == c) & (o < tid));
      }
      if (r == rank) rank_seq = tid;
    }
    __syncthreads();
    b = __builtin_amdgcn_readfirstlane(rank_seq);
  }
  const int q0 = a.cu[b];
  const int n = a.cu[b + 1] - q0;
  const int G = a.group;
  const int rows = n * G;
  const int R0 = tile * kRows;
  if (R0 >= rows) return;
  const int P = a.ctx[b];
  const int32_t *bt = a.bt + (size_t)b * a.max_pages;

  Tile<C> T;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  T.half = lane >> 5;
  T.col = lane & 31;
  T.gq = lane >> 4;
  T.li = lane & 15;
  lds_offsets<C>(T);
  T.g = g;
  T.t = __builtin_amdgcn_readfirstlane(wave >> 1);
  const int Rw = R0 + wave * 32 + T.col;
  const bool rvalid = Rw < rows;
  const int t = rvalid ? Rw / G : 0;
  const int hh = rvalid ? Rw - t * G : 0;
  T.ipos = rvalid ? P + t : -1;
  const size_t qrow = ((size_t)(q0 + t) * a.h_q + (size_t)g * G + hh) * D;

  // workgroup-uniform bounds, pinned to scalar registers (the integer
  // divisions would otherwise leave them in vector registers and drag the
  // whole load-address computation onto the VALU)
  const int t_first = __builtin_amdgcn_readfirstlane(R0 / G);
  const int t_last = __builtin_amdgcn_readfirstlane(min(n - 1, (R0 + kRows - 1) / G));
  T.i_min = P + t_first;
  T.i_max = P + t_last;
  T.kv_end = T.i_max + 1;
  const int W = a.window;
  const int kv_begin = W > 0 ? max(0, T.i_min - W + 1) : 0;
  // this workgroup's keys: the tile's visible range, cut to its partition
  // (partitions are whole blocks, so every key lands in exactly one)
  const int part_lo = split * a.split_len, part_hi = part_lo + a.split_len;
  T.kb_begin = max(kv_begin, part_lo) / BN;
  const int kb_end = (min(T.kv_end, part_hi) + BN - 1) / BN;
  T.nblk = kb_end - T.kb_begin;
  // Fused append: keys from P on come from the input rows, and partition
  // 0's workgroup writes the rows of the tokens whose first row t G lies in
  // this tile (every token has exactly one such tile).  No workgroup reads
  // the pool slots written here, so nothing orders the workgroups.
  AppendRows<C, PS> ap;
  T.pnew = 0;
  T.nsrc = nullptr;
  if constexpr (AP) {
    T.pnew = P;
    const size_t in_stride = (size_t)a.h_kv * C::ROW;
    const size_t row0 = ((size_t)q0 * a.h_kv + g) * C::ROW;
    ap.src_k = a.k_new + row0;
    ap.src_vk = a.v_new - a.k_new;
    T.nsrc = (T.t == 0 ? a.k_new : a.v_new) + row0;
    ap.dst_k = const_cast<uint8_t *>(a.k) + (size_t)g * PS * C::ROW;
    ap.dst_vk = a.v - a.k;
    ap.bt = bt;
    ap.pos0 = P;
    ap.stride = (int)in_stride;
    ap.tok_lo = __builtin_amdgcn_readfirstlane((R0 + G - 1) / G);
    const int tok_hi = min(n, (R0 + kRows + G - 1) / G);
    ap.units = split == 0 ? max(0, tok_hi - ap.tok_lo) * 2 * C::CH : 0;
    if (T.nblk <= 0) ap.copy_from(0);
  }
  const size_t prow = (size_t)(q0 + t) * a.h_q + (size_t)g * G + hh;  // (token, head) row
  if (T.nblk <= 0) {
    // an empty partition: weight 0 in the merge
    if (rvalid && T.half == 0) {
      const size_t pi = prow * a.splits + split;
      st<f32x2>(a.part_ml + pi * 2, f32x2{kNegInf, 0.f});
    }
    return;
  }

  lane_offsets<C, PS, FP8>(T.loff);
  // prologue: K of block 0, then K of block 1 and V of block 0 while S^T of
  // block 0 is computed
  if (T.t == 0) {
    block_pages<C, PS>(bt, T.kb_begin * BN, T.kv_end, T.pg);
    issue_block<C, PS, FP8>(a, bt, g, T.kb_begin * BN, T.kv_end, T.pg, T.loff, R.k, T.pnew, T.nsrc);
  }
  // fused append: the first batch of rows is loaded beside Q and stored
  // once the prologue's loads have landed
  u32x16 apx{};
  u32x4 appg{};
  if constexpr (AP) ap.load(0, apx, appg);
  // k-step s takes d = 16 s + 8 half + 0..7; fp8 pools pair the steps so
  // that one 16-code K read feeds two: d = 32 (s / 2) + 16 half + 8 (s % 2)
#pragma unroll
  for (int s = 0; s < C::DS; ++s) {
    const int d0 = FP8 ? 32 * (s >> 1) + 16 * T.half + 8 * (s & 1) : 16 * s + 8 * T.half;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (rvalid) x = ld<u32x4>(a.q + qrow + d0);
    T.qf[s] = as_bf16x8(x);
  }
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) T.o[dt] = f32x16{};
  T.m = kNegInf;
  T.l = 0.f;

  f32x16 sA[C::NT], sB[C::NT];
  wait_and_issue<C, PS, FP8, 1, true>(a, bt, T, -1, R);  // U = (-1) & 1
  if constexpr (AP) {
    ap.store(0, apx, appg);
    // tiles that own more rows than one batch (few query heads per KV head)
    ap.copy_from(AppendRows<C, PS>::NAP * kThreads);
  }
  qk_part<C, 0>(R.k, T, sA);
  qk_part<C, 1>(R.k, T, sA);

  for (int j0 = 0; j0 < T.nblk; j0 += 2) {
    step<C, PS, FP8, 0>(a, bt, T, j0, sA, sB, R);
    if (j0 + 1 < T.nblk) step<C, PS, FP8, 1>(a, bt, T, j0 + 1, sB, sA, R);
  }

  // ---- normalize and store this lane's row: d = 32 dt + 8 i + 4 half + 0..3
  const float l = half_swap_sum(T.l);
  if (!rvalid) return;
  if (a.splits > 1) {
    // partial of this partition: (m, l) and o / l, merged by combine_kernel
    const size_t pi = prow * a.splits + split;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    float *po = a.part_o + pi * D;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        st<f32x4>(po + 32 * dt + 8 * i + 4 * T.half,
                  f32x4{T.o[dt][4 * i] * inv, T.o[dt][4 * i + 1] * inv, T.o[dt][4 * i + 2] * inv,
                        T.o[dt][4 * i + 3] * inv});
    if (T.half == 0) st<f32x2>(a.part_ml + pi * 2, f32x2{T.m, l});
    return;
  }
  const float inv = 1.f / l;
  uint16_t *orow = a.out + qrow;
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u32x2 w = {pack_bf16x2(T.o[dt][4 * i] * inv, T.o[dt][4 * i + 1] * inv),
                       pack_bf16x2(T.o[dt][4 * i + 2] * inv, T.o[dt][4 * i + 3] * inv)};
      st<u32x2>(orow + 32 * dt + 8 * i + 4 * T.half, w);
    }
  }
}

}  // namespace pf
}  // namespace ckv
