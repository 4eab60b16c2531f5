// prefix_prefill_attn for bf16 queries over a bf16 or fp8-E4M3 paged pool.
//
// Work item: one workgroup (4 waves) = 128 consecutive "rows" of one
// (sequence, KV head), a row being a (new-turn token, query head of the
// group) pair flattened as R = t * G + hh.  Packing the G query heads of a
// KV head into the M dimension lets every K/V byte staged in LDS serve all
// of them and keeps the causal diagonal narrow (128 / G tokens per tile).
//
// Data movement, per block of BN keys read through the block table:
//   * K and V rows go from HBM straight into an NS-stage LDS ring with
//     global_load_lds_dwordx4 (no register staging); the lane -> address map
//     of each load permutes 16-byte chunks so that the ring is XOR-swizzled.
//     One barrier per block; loads for block j + NS - 1 are issued while
//     block j is computed.
//   * fp8 pools are loaded raw, then widened to bf16 (exactly) once per
//     workgroup into a bf16 block with the same layout.
// Math, per wave of 32 rows:
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (Q stays in registers).  The
//     lane that owns a query row holds a column of S^T, so the row max / row
//     sum are in-lane plus one exchange between the half-waves.  K rows are
//     fed in a permuted order (pi) so that the probabilities a lane holds are
//     exactly the 8 consecutive keys it supplies as the B operand of
//     O^T += V^T P^T; V^T operands come from row-major V in LDS through
//     ds_read_b64_tr_b16 (4 keys x 16 columns transposed per 16 lanes).
//   * Online softmax in fp32 with base-2 exponentials; the running maximum
//     is only moved (and O rescaled) when it grows by more than 2^8, which
//     leaves the result unchanged but skips most rescales.  Masking only on
//     blocks that straddle the causal diagonal or the window edge.
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

template <int D, int BN, int NS, bool FP8>
struct Cfg {
  static constexpr int ROW = D * 2;                    // bf16 bytes per key row in LDS
  static constexpr int CH = D / 8;                     // 16-byte chunks per bf16 row
  static constexpr int BLK = BN * ROW;                 // bf16 bytes of one K (or V) block
  static constexpr int RAW_ROW = FP8 ? D : D * 2;      // pool bytes per key row
  static constexpr int RAW_BLK = BN * RAW_ROW;         // pool bytes of one block
  static constexpr int STAGE = 2 * RAW_BLK;            // K + V, raw
  static constexpr int LDS = NS * STAGE + (FP8 ? 2 * BLK : 0);
  static constexpr int DMA_PER_TENSOR = RAW_BLK / 1024;  // 1 KB per wave-wide load
  static constexpr int DMA_PER_WAVE = 2 * DMA_PER_TENSOR / kWaves;
  static constexpr int ROWS_PER_DMA = 1024 / RAW_ROW;
  static constexpr int NT = BN / 32;                   // S^T tiles per block
  static constexpr int DS = D / 16;                    // QK^T k-steps
  static constexpr int DT = D / 32;                    // output d-tiles
  static_assert((2 * DMA_PER_TENSOR) % kWaves == 0, "each wave issues whole loads");
  static_assert(LDS <= 160 * 1024, "LDS budget");
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

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4_t;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4_t;

__device__ __forceinline__ u32x2 ds_read_tr16(const uint8_t *p) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(p));
  return __builtin_bit_cast(u32x2, v);
}
__device__ __forceinline__ u32x4 lds_ld16(const uint8_t *p) { return *(const lds_u32x4_t *)(p); }
__device__ __forceinline__ void lds_st16(uint8_t *p, u32x4 v) { *(lds_u32x4_t *)(p) = v; }

// Read-only tables (block table, fp8 scales) are read through the constant
// address space so that wave-uniform lookups become scalar loads.
template <typename T>
__device__ __forceinline__ T ldc(const T *p, int i) {
  return ((const __attribute__((address_space(4))) T *)(p))[i];
}

// One wave-wide 16-byte-per-lane load from global memory straight into LDS:
// lane l's 16 bytes land at lds_base + 16 l.  Issued as inline assembly so
// that the compiler does not track it; the kernel orders these loads itself
// (s_waitcnt vmcnt + barrier before the data is read, barrier before a stage
// is overwritten).
__device__ __forceinline__ void dma16(const void *g, uint8_t *lds_wave_base) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t *)(lds_wave_base));
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(m0) : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier without a memory fence: LDS reads of this wave are
// complete (lgkmcnt 0) and the compiler may not move memory accesses across.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Page id (physical page of the first row) of each wave-wide load this wave
// issues for the block starting at kbase.  All rows of one load share a page
// (page_size is a multiple of ROWS_PER_DMA); the lookups are scalar loads.
template <int D, int BN, int NS, bool FP8>
__device__ __forceinline__ void block_pages(const int32_t *bt, int ps, int kbase, int kv_end,
                                            int (&pg)[Cfg<D, BN, NS, FP8>::DMA_PER_WAVE]) {
  using C = Cfg<D, BN, NS, FP8>;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
  for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
    const int idx = wave * C::DMA_PER_WAVE + i;
    const int r = idx % C::DMA_PER_TENSOR;
    const int kp0 = min(kbase + r * C::ROWS_PER_DMA, kv_end - 1);
    pg[i] = ldc(bt, __builtin_amdgcn_readfirstlane(kp0 / ps));
  }
}

// Issue this wave's share of the loads of one K/V block into an LDS stage.
// Rows at or beyond kv_end are redirected to row kv_end - 1 (valid, finite
// data that the causal mask removes).
template <int D, int BN, int NS, bool FP8>
__device__ __forceinline__ void issue_block(const PrefillArgs &a, int g, int kbase, int kv_end,
                                            const int (&pg)[Cfg<D, BN, NS, FP8>::DMA_PER_WAVE],
                                            uint8_t *stage) {
  using C = Cfg<D, BN, NS, FP8>;
  constexpr int RCH = C::RAW_ROW / 16;  // 16-byte chunks per pool row
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const size_t head_off = (size_t)g * a.ps * C::RAW_ROW;
  const size_t page_stride = (size_t)a.h_kv * a.ps * C::RAW_ROW;
#pragma unroll
  for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
    const int idx = wave * C::DMA_PER_WAVE + i;  // 0 .. 2*DMA_PER_TENSOR-1
    const int tensor = idx / C::DMA_PER_TENSOR;  // 0 = K, 1 = V
    const int r = idx % C::DMA_PER_TENSOR;
    const int row = r * C::ROWS_PER_DMA + lane / RCH;
    const int slot = lane % RCH;
    const int kp = min(kbase + row, kv_end - 1);
    int chunk = slot;
    if constexpr (!FP8) chunk = slot ^ (tensor == 0 ? swz_k<C::CH>(row) : swz_v<C::CH>(row));
    const uint8_t *base = tensor == 0 ? a.k : a.v;
    const uint8_t *src = base + (size_t)pg[i] * page_stride + head_off +
                         (size_t)(kp % a.ps) * C::RAW_ROW + chunk * 16;
    dma16(src, stage + tensor * C::RAW_BLK + r * 1024);
  }
}

// fp8: widen one raw stage into the bf16 K/V blocks (same layout as bf16).
template <int D, int BN, int NS, bool FP8>
__device__ __forceinline__ void widen_block(const uint8_t *stage, uint8_t *k16, uint8_t *v16) {
  using C = Cfg<D, BN, NS, FP8>;
  constexpr int RAW_CH = C::RAW_ROW / 16;  // 16-code chunks per raw row
  constexpr int TOTAL = 2 * BN * RAW_CH;
  static_assert(TOTAL % kThreads == 0, "widening must tile evenly");
#pragma unroll
  for (int it = 0; it < TOTAL / kThreads; ++it) {
    const int id = threadIdx.x + it * kThreads;
    const int tensor = id / (BN * RAW_CH);
    const int rem = id % (BN * RAW_CH);
    const int row = rem / RAW_CH, c = rem % RAW_CH;
    const u32x4 x = lds_ld16(stage + tensor * C::RAW_BLK + row * C::RAW_ROW + c * 16);
    const u32x2 a0 = fp8x4_to_bf16x4(x.x), a1 = fp8x4_to_bf16x4(x.y);
    const u32x2 b0 = fp8x4_to_bf16x4(x.z), b1 = fp8x4_to_bf16x4(x.w);
    uint8_t *dst = (tensor == 0 ? k16 : v16) + row * C::ROW;
    const int sw = tensor == 0 ? swz_k<C::CH>(row) : swz_v<C::CH>(row);
    lds_st16(dst + (((2 * c) ^ sw) << 4), u32x4{a0.x, a0.y, a1.x, a1.y});
    lds_st16(dst + (((2 * c + 1) ^ sw) << 4), u32x4{b0.x, b0.y, b1.x, b1.y});
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
template <int D, int BN, int NS, bool FP8>
struct Tile {
  using C = Cfg<D, BN, NS, FP8>;
  bf16x8 qf[C::DS];
  f32x16 o[C::DT];
  float m, l;
  int pg[C::DMA_PER_WAVE];  // page ids of the next block to issue
  int g, ipos, i_min, i_max, kv_end, kb_begin, nblk, half, col, gq, li;
};

// One block of BN keys: wait for its loads, barrier, issue the loads NS-1
// blocks ahead, then S^T, softmax and O^T for this block.  U is the stage
// of block j (compile time, so each stage is its own LDS object and the
// compiler can tell the in-flight loads apart from the reads).
template <int D, int BN, int NS, bool FP8, int U>
__device__ __forceinline__ void block_step(const PrefillArgs &a, const int32_t *bt, Tile<D, BN, NS, FP8> &T,
                                           int j, uint8_t *const (&stages)[3], uint8_t *k16,
                                           uint8_t *v16) {
  using C = Cfg<D, BN, NS, FP8>;
  const int kbase = (T.kb_begin + j) * BN;
  if constexpr (NS >= 3) {
    if (j + 1 < T.nblk) wait_vmcnt<C::DMA_PER_WAVE>();
    else wait_vmcnt<0>();
  } else {
    wait_vmcnt<0>();
  }
  lds_barrier();
  if (j + NS - 1 < T.nblk) {
    issue_block<D, BN, NS, FP8>(a, T.g, kbase + (NS - 1) * BN, T.kv_end, T.pg, stages[(U + NS - 1) % NS]);
    if (j + NS < T.nblk) block_pages<D, BN, NS, FP8>(bt, a.ps, kbase + NS * BN, T.kv_end, T.pg);
  }
  const uint8_t *kb;
  const uint8_t *vb;
  if constexpr (FP8) {
    widen_block<D, BN, NS, FP8>(stages[U], k16, v16);
    lds_barrier();
    kb = k16;
    vb = v16;
  } else {
    kb = stages[U];
    vb = kb + C::BLK;
  }
  const int half = T.half, col = T.col;

  // ---- S^T = K Q^T, one 32-key tile at a time
  f32x16 s[C::NT];
#pragma unroll
  for (int tt = 0; tt < C::NT; ++tt) {
    s[tt] = f32x16{};
    const int key = 32 * tt + pi_row(col);
    const uint8_t *krow = kb + key * C::ROW;
    const int sw = swz_k<C::CH>(key);
#pragma unroll
    for (int ds = 0; ds < C::DS; ++ds) {
      const u32x4 kx = lds_ld16(krow + (((2 * ds + half) ^ sw) << 4));
      s[tt] = mfma32x32x16(as_bf16x8(kx), T.qf[ds], s[tt]);
    }
  }

  // ---- scale (fp8: times the page-head K scale), mask, row max
  float ksc[C::NT * 2], vsc[C::NT * 2];  // per 16-key group
#pragma unroll
  for (int q = 0; q < C::NT * 2; ++q) {
    ksc[q] = a.scale_log2;
    vsc[q] = 1.f;
    if constexpr (FP8) {
      const int kp = min(kbase + 16 * q, T.kv_end - 1);
      const int idx = ldc(bt, __builtin_amdgcn_readfirstlane(kp / a.ps)) * a.h_kv + T.g;
      ksc[q] = a.scale_log2 * ldc(a.k_scale, idx);
      vsc[q] = ldc(a.v_scale, idx);
    }
  }
  const int W = a.window;
  const bool full = (kbase + BN - 1 <= T.i_min) && (W <= 0 || T.i_max - kbase < W);
  float mx = kNegInf;
#pragma unroll
  for (int tt = 0; tt < C::NT; ++tt) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int grp = 2 * tt + (e >> 3);
      float x = s[tt][e] * ksc[grp];
      if (!full) {
        const int i = e >> 2, jj = e & 3;
        const int kp = kbase + 32 * tt + 16 * (i >> 1) + 8 * half + 4 * (i & 1) + jj;
        const bool vis = kp <= T.ipos && (W <= 0 || T.ipos - kp < W);
        x = vis ? x : kNegInf;
      }
      s[tt][e] = x;
      mx = fmaxf(mx, x);
    }
  }
  mx = half_swap_max(mx);
  // move the reference maximum only when it grows by more than the slack
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
  const float m_use = T.m == kNegInf ? 0.f : T.m;

  // ---- P = exp2(x - m); O^T += V^T P^T
#pragma unroll
  for (int tt = 0; tt < C::NT; ++tt) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      float p[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = fast_exp2(s[tt][8 * ks + e] - m_use);
        T.l += p[e];
        if constexpr (FP8) p[e] *= vsc[2 * tt + ks];
      }
      const u32x4 pb = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                        pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
      // transposed V reads: 16-lane group gq covers columns 16(gq&1) + 0..15
      // of a 32-column tile and keys key0 .. key0+3 (key0+4 .. +7 on the
      // second read); lane li of the group addresses key key0 + li/4,
      // columns 4(li%4) .. +3.
      const int key0 = 32 * tt + 16 * ks + 8 * (T.gq >> 1) + (T.li >> 2);
      const int dsub = 16 * (T.gq & 1) + 4 * (T.li & 3);
      const uint8_t *r0 = vb + key0 * C::ROW;
      const uint8_t *r1 = r0 + 4 * C::ROW;
      const int sw0 = swz_v<C::CH>(key0), sw1 = swz_v<C::CH>(key0 + 4);
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) {
        const int byte = 2 * (32 * dt + dsub);
        const int cidx = byte >> 4, within = byte & 15;
        const u32x2 lo = ds_read_tr16(r0 + ((cidx ^ sw0) << 4) + within);
        const u32x2 hi = ds_read_tr16(r1 + ((cidx ^ sw1) << 4) + within);
        const u32x4 vx = {lo.x, lo.y, hi.x, hi.y};
        T.o[dt] = mfma32x32x16(as_bf16x8(vx), as_bf16x8(pb), T.o[dt]);
      }
    }
  }
}

template <int D, int BN, int NS, bool FP8>
__global__ __launch_bounds__(kThreads, D >= 256 ? 1 : 2) void prefill_kernel(PrefillArgs a) {
  using C = Cfg<D, BN, NS, FP8>;
  static_assert(NS == 2 || NS == 3, "two or three stages");
  // one LDS object per ring stage (see block_step)
  __shared__ __attribute__((aligned(1024))) uint8_t st0[C::STAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t st1[C::STAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t st2[NS >= 3 ? C::STAGE : 16];
  __shared__ __attribute__((aligned(1024))) uint8_t cvt[FP8 ? 2 * C::BLK : 16];
  uint8_t *const stages[3] = {st0, st1, st2};

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

  Tile<D, BN, NS, FP8> T;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  T.half = lane >> 5;
  T.col = lane & 31;
  T.gq = lane >> 4;
  T.li = lane & 15;
  T.g = g;
  const int R = R0 + wave * 32 + T.col;
  const bool rvalid = R < rows;
  const int t = rvalid ? R / G : 0;
  const int hh = rvalid ? R - t * G : 0;
  T.ipos = rvalid ? P + t : -1;
  const size_t qrow = ((size_t)(q0 + t) * a.h_q + (size_t)g * G + hh) * D;

  const int t_first = R0 / G;
  const int t_last = min(n - 1, (R0 + kRows - 1) / G);
  T.i_min = P + t_first;
  T.i_max = P + t_last;
  T.kv_end = T.i_max + 1;
  const int W = a.window;
  const int kv_begin = W > 0 ? max(0, T.i_min - W + 1) : 0;
  T.kb_begin = kv_begin / BN;
  const int kb_end = (T.kv_end + BN - 1) / BN;
  T.nblk = kb_end - T.kb_begin;

  // prologue: the first NS-1 blocks in flight before anything else
#pragma unroll
  for (int s = 0; s < NS - 1; ++s) {
    if (s < T.nblk) {
      block_pages<D, BN, NS, FP8>(bt, a.ps, (T.kb_begin + s) * BN, T.kv_end, T.pg);
      issue_block<D, BN, NS, FP8>(a, g, (T.kb_begin + s) * BN, T.kv_end, T.pg, stages[s]);
    }
  }
  if (NS - 1 < T.nblk) block_pages<D, BN, NS, FP8>(bt, a.ps, (T.kb_begin + NS - 1) * BN, T.kv_end, T.pg);

#pragma unroll
  for (int s = 0; s < C::DS; ++s) {
    u32x4 x = {0u, 0u, 0u, 0u};
    if (rvalid) x = ld<u32x4>(a.q + qrow + 16 * s + 8 * T.half);
    T.qf[s] = as_bf16x8(x);
  }
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt) T.o[dt] = f32x16{};
  T.m = kNegInf;
  T.l = 0.f;

  uint8_t *k16 = cvt;  // fp8 only
  uint8_t *v16 = cvt + (FP8 ? C::BLK : 0);
  for (int j0 = 0; j0 < T.nblk; j0 += NS) {
    block_step<D, BN, NS, FP8, 0>(a, bt, T, j0, stages, k16, v16);
    if (j0 + 1 < T.nblk) block_step<D, BN, NS, FP8, 1>(a, bt, T, j0 + 1, stages, k16, v16);
    if constexpr (NS >= 3)
      if (j0 + 2 < T.nblk) block_step<D, BN, NS, FP8, 2>(a, bt, T, j0 + 2, stages, k16, v16);
  }

  // ---- normalize and store this lane's row: d = 32 dt + 8 i + 4 half + 0..3
  const float l = half_swap_sum(T.l);
  if (!rvalid) return;
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

template <int D, int BN, int NS, bool FP8>
hipError_t launch(const PrefillArgs &a, int h_kv, int num_seqs, hipStream_t s) {
  dim3 grid(a.tiles, h_kv, num_seqs);
  hipLaunchKernelGGL((prefill_kernel<D, BN, NS, FP8>), grid, dim3(kThreads), 0, s, a);
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
      return fp8 ? launch<64, 64, 2, true>(a, p.h_kv, b.num_seqs, s)
                 : launch<64, 64, 2, false>(a, p.h_kv, b.num_seqs, s);
    case 128:
      return fp8 ? launch<128, 64, 2, true>(a, p.h_kv, b.num_seqs, s)
                 : launch<128, 64, 2, false>(a, p.h_kv, b.num_seqs, s);
    case 256:
      return fp8 ? launch<256, 32, 2, true>(a, p.h_kv, b.num_seqs, s)
                 : launch<256, 32, 2, false>(a, p.h_kv, b.num_seqs, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace ckv
