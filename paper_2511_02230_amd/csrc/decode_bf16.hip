// paged_decode_attn for bf16 queries over a bf16 or fp8-E4M3 paged pool.
//
// Split-K: the context of each sequence is cut into partitions of L logical
// positions; one single-wave workgroup handles (partition, KV head, <=16
// query heads of its group, sequence) and reads every K/V byte of its range
// exactly once for all of those heads.
//
// Data movement: blocks of KB keys stream from the pool into an NS-stage LDS
// ring with global_load_lds_dwordx4 (lane -> address map XOR-swizzles the
// ring), NS-1 blocks ahead of the one being computed.  The ring belongs to
// one wave, so ordering needs only s_waitcnt, no barriers.
// Math: the heads are packed into the N dimension of
// v_mfma_f32_16x16x32_bf16 (padded to 16):
//   S^T (16 keys x 16 heads) = K (16 keys x 32 d) * Q^T,
//   O^T (16 d x 16 heads)   += V^T (16 d x 32 keys) * P^T,
// K rows are fed in a permuted order (rho) so that the 8 probabilities a lane
// holds are the 8 consecutive keys it supplies as the B operand of the
// second product; V^T operands come from row-major V through
// ds_read_b64_tr_b16.  fp8 K codes are widened in registers after the LDS
// read; fp8 V blocks are widened once into a bf16 block.  A partition writes
// (m, l, o) partials in fp32 unless it is its sequence's only one, in which
// case it writes the output; the combine kernel merges the rest.
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

constexpr float kRescaleSlack = 8.0f;  // log2 units: defer rescaling below 2^8

template <int D, bool FP8, int KB, int NS>
struct DCfg {
  static constexpr int ROW = D * 2;                // bf16 bytes per row
  static constexpr int CH = D / 8;                 // 16-byte bf16 chunks per row
  static constexpr int RAW_ROW = FP8 ? D : D * 2;  // pool bytes per row
  static constexpr int RAW_BLK = KB * RAW_ROW;
  static constexpr int STAGE = 2 * RAW_BLK;
  static constexpr int DMA_PER_TENSOR = RAW_BLK / 1024;
  static constexpr int ROWS_PER_DMA = 1024 / RAW_ROW;
  static constexpr int DMA_PER_BLOCK = 2 * DMA_PER_TENSOR;
  static constexpr int NT = KB / 16;  // S^T tiles per block
  static constexpr int DS = D / 32;   // QK^T k-steps
  static constexpr int DT = D / 16;   // output d-tiles
  static_assert(KB % 32 == 0, "blocks of whole 32-key MFMA steps");
  static_assert(DMA_PER_BLOCK * (NS - 1) < 64, "vmcnt range");
};

// d offset of the 8 k-slots a lane (quarter q4) supplies at step `step` of
// the QK^T contraction.  bf16: 16 contiguous bytes per step; fp8: two
// consecutive steps read one 16-byte run of codes.
template <bool FP8>
__device__ __forceinline__ int qk_d0(int step, int q4) {
  if constexpr (FP8) return 64 * (step >> 1) + 16 * q4 + 8 * (step & 1);
  return 32 * step + 8 * q4;
}

// XOR swizzles of the 16-byte chunk index within a row (bf16 rows; fp8 raw
// rows use the K one on their 16-code chunks).
//  K: one operand load reads, per 16 lanes, keys {0..3, 8..11, 16..19,
//     24..27} (+4) of a 32-key step at one chunk: (key & 3) | ((key >> 3) & 3) << 2
//     gives them 16 different slots.
//  V: a transposed read covers 4 consecutive keys x 2 chunks per 16 lanes and
//     two groups 8 keys apart share a pass.
template <int CH>
__device__ __forceinline__ int dswz_k(int key) {
  return ((key & 3) | (((key >> 3) & 3) << 2)) & (CH - 1);
}
template <int CH>
__device__ __forceinline__ int dswz_v(int key) {
  return (((key & 3) << 2) | (((key >> 3) & 1) << 1)) & (CH - 1);
}

// Per-lane byte offset (relative to the first row of load r of tensor t,
// 0 = K, 1 = V) of the 16 bytes this lane fetches: lane l lands in LDS slot
// l of the load and fetches the chunk the swizzle assigns to that slot.
template <class C, bool FP8>
__device__ __forceinline__ uint32_t d_lane_offset(int t, int r) {
  constexpr int RCH = C::RAW_ROW / 16;
  const int lane = threadIdx.x;
  const int row = r * C::ROWS_PER_DMA + lane / RCH;
  const int slot = lane % RCH;
  const int chunk = slot ^ (t == 0 ? dswz_k<RCH>(row) : (FP8 ? 0 : dswz_v<C::CH>(row)));
  return (uint32_t)((lane / RCH) * C::RAW_ROW + chunk * 16);
}

// Page of each load of the block at kbase (clamped into [kbeg, kend)),
// scalar loads through the constant address space.
template <class C, int PS>
__device__ __forceinline__ void d_block_pages(const int32_t *bt, int kbase, int kbeg, int kend,
                                              int (&pg)[C::DMA_PER_TENSOR]) {
#pragma unroll
  for (int r = 0; r < C::DMA_PER_TENSOR; ++r) {
    const int kp0 = min(max(kbase + r * C::ROWS_PER_DMA, kbeg), kend - 1);
    pg[r] = ldc(bt, __builtin_amdgcn_readfirstlane(kp0 / PS));
  }
}

// All loads of one block (K then V) into a ring stage.  Keys outside
// [kbeg, kend) (first or last block of a partition) are redirected to a key
// of the range in the same page: finite data that the mask removes.
template <class C, int PS, bool FP8>
__device__ __forceinline__ void d_issue_block(const DecodeArgs &a, int g, int kbase, int kbeg, int kend,
                                              const int (&pg)[C::DMA_PER_TENSOR], lds_u8 *stage) {
  constexpr int RCH = C::RAW_ROW / 16;
  const int lane = threadIdx.x;
  const size_t head_off = (size_t)g * PS * C::RAW_ROW;
  const size_t page_stride = (size_t)a.h_kv * PS * C::RAW_ROW;
  const bool inner = kbase >= kbeg && kbase + C::DMA_PER_TENSOR * C::ROWS_PER_DMA <= kend;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
#pragma unroll
    for (int r = 0; r < C::DMA_PER_TENSOR; ++r) {
      const int kp0 = kbase + r * C::ROWS_PER_DMA;
      const uint8_t *page_base = (t == 0 ? a.k : a.v) + (size_t)pg[r] * page_stride + head_off;
      lds_u8 *dst = stage + t * C::RAW_BLK + r * 1024;
      const uint32_t loff = d_lane_offset<C, FP8>(t, r);
      if (inner) {
        dma16_sv(page_base + (size_t)(kp0 % PS) * C::RAW_ROW, loff, dst);
      } else {
        const int kp = min(max(kp0 + lane / RCH, kbeg), kend - 1);
        dma16_sv(page_base, (uint32_t)((kp % PS) * C::RAW_ROW) + loff % C::RAW_ROW, dst);
      }
    }
  }
}

template <int D, bool FP8, int KB, int NS, int PS>
__global__ __launch_bounds__(64) void decode_kernel(DecodeArgs a) {
  using C = DCfg<D, FP8, KB, NS>;
  static_assert(NS >= 2 && NS <= 4, "ring depth");
  // the ring is written only by the (untracked) LDS loads of this wave; the
  // compiler barriers after each wait keep LDS reads behind the waits
  __shared__ __attribute__((aligned(1024))) uint8_t ring_[NS * C::STAGE];
  __shared__ __attribute__((aligned(1024))) uint8_t vwide_[FP8 ? KB * C::ROW : 16];
  lds_u8 *const ring = as_lds(ring_);
  lds_u8 *const vwide = as_lds(vwide_);

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

  const int kb0 = kbeg - (kbeg % KB);
  const int nblk = kbeg < kend ? (kend - kb0 + KB - 1) / KB : 0;
  int pg[C::DMA_PER_TENSOR];
#pragma unroll
  for (int s = 0; s < NS - 1; ++s) {
    if (s < nblk) {
      d_block_pages<C, PS>(bt, kb0 + s * KB, kbeg, kend, pg);
      d_issue_block<C, PS, FP8>(a, g, kb0 + s * KB, kbeg, kend, pg, ring + s * C::STAGE);
    }
  }

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

  for (int j = 0; j < nblk; ++j) {
    const int kbase = kb0 + j * KB;
    // page ids of the block issued below: the scalar loads resolve while
    // this wave waits for block j
    const bool issue = j + NS - 1 < nblk;
    if (issue) d_block_pages<C, PS>(bt, kbase + (NS - 1) * KB, kbeg, kend, pg);
    // this block's loads are done once at most min(NS-2, later blocks)
    // blocks' worth of loads are still outstanding
    const int later = min(NS - 2, nblk - 1 - j);
    if constexpr (NS >= 4) {
      if (later >= 2) wait_vmcnt<2 * C::DMA_PER_BLOCK>();
      else if (later == 1) wait_vmcnt<C::DMA_PER_BLOCK>();
      else wait_vmcnt<0>();
    } else if constexpr (NS == 3) {
      if (later >= 1) wait_vmcnt<C::DMA_PER_BLOCK>();
      else wait_vmcnt<0>();
    } else {
      wait_vmcnt<0>();
    }
    asm volatile("" ::: "memory");
    if (issue)
      d_issue_block<C, PS, FP8>(a, g, kbase + (NS - 1) * KB, kbeg, kend, pg,
                                ring + ((j + NS - 1) % NS) * C::STAGE);
    const lds_u8 *kblk = ring + (j % NS) * C::STAGE;
    const lds_u8 *vblk = kblk + C::RAW_BLK;
    if constexpr (FP8) {
      // widen V codes to bf16 rows (same swizzle as a bf16 V block)
      constexpr int RCH = C::RAW_ROW / 16;
#pragma unroll
      for (int it = 0; it < KB * RCH / 64; ++it) {
        const int id = lane + 64 * it;
        const int row = id / RCH, cc = id % RCH;
        const u32x4 x = lds_ld16(vblk + row * C::RAW_ROW + cc * 16);
        const u32x2 a0 = fp8x4_to_bf16x4(x.x), a1 = fp8x4_to_bf16x4(x.y);
        const u32x2 b0 = fp8x4_to_bf16x4(x.z), b1 = fp8x4_to_bf16x4(x.w);
        lds_u8 *dst = vwide + row * C::ROW;
        const int sw = dswz_v<C::CH>(row);
        lds_st16(dst + (((2 * cc) ^ sw) << 4), u32x4{a0.x, a0.y, a1.x, a1.y});
        lds_st16(dst + (((2 * cc + 1) ^ sw) << 4), u32x4{b0.x, b0.y, b1.x, b1.y});
      }
      vblk = vwide;
    }

    // fp8 scales of the block's 16-key spans (uniform lookups); a lane's
    // 4-key group 32 kk + 8 q4 + 4 tt lies in span 2 kk + q4 / 2
    float ksp[KB / 16], vsp[KB / 16];
    if constexpr (FP8) {
#pragma unroll
      for (int sp = 0; sp < KB / 16; ++sp) {
        const int kp = min(max(kbase + 16 * sp, kbeg), kend - 1);
        const int idx = ldc(bt, __builtin_amdgcn_readfirstlane(kp / PS)) * a.h_kv + g;
        ksp[sp] = a.scale_log2 * ldc(a.k_scale, idx);
        vsp[sp] = ldc(a.v_scale, idx);
      }
    }
#pragma unroll
    for (int kk = 0; kk < KB / 32; ++kk) {
      // ---- S^T tiles: row m of tile tt is key rho(m) = 8(m/4) + 4tt + m%4
      f32x4 s[2];
      float ksc[2], vsc[2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        const int key = 32 * kk + 8 * (col >> 2) + 4 * tt + (col & 3);
        s[tt] = f32x4{};
        if constexpr (FP8) {
          const lds_u8 *krow = kblk + key * C::RAW_ROW;
          const int sw = dswz_k<C::RAW_ROW / 16>(key);
#pragma unroll
          for (int s2 = 0; s2 < C::DS; s2 += 2) {
            const int cc = qk_d0<true>(s2, q4) / 16;
            const u32x4 x = lds_ld16(krow + ((cc ^ sw) << 4));
            const u32x2 a0 = fp8x4_to_bf16x4(x.x), a1 = fp8x4_to_bf16x4(x.y);
            const u32x2 b0 = fp8x4_to_bf16x4(x.z), b1 = fp8x4_to_bf16x4(x.w);
            s[tt] = mfma16x16x32(as_bf16x8(u32x4{a0.x, a0.y, a1.x, a1.y}), qf[s2], s[tt]);
            s[tt] = mfma16x16x32(as_bf16x8(u32x4{b0.x, b0.y, b1.x, b1.y}), qf[s2 + 1], s[tt]);
          }
        } else {
          const lds_u8 *krow = kblk + key * C::ROW;
          const int sw = dswz_k<C::CH>(key);
#pragma unroll
          for (int st_ = 0; st_ < C::DS; ++st_) {
            const int cc = qk_d0<false>(st_, q4) / 8;
            const u32x4 x = lds_ld16(krow + ((cc ^ sw) << 4));
            s[tt] = mfma16x16x32(as_bf16x8(x), qf[st_], s[tt]);
          }
        }
        // the 4 keys this lane receives for tile tt: kbase + 32kk + 8 q4 + 4 tt + j
        ksc[tt] = a.scale_log2;
        vsc[tt] = 1.f;
        if constexpr (FP8) {
          const int hi = q4 >> 1;  // span 2 kk + hi
          ksc[tt] = hi ? ksp[2 * kk + 1] : ksp[2 * kk];
          vsc[tt] = hi ? vsp[2 * kk + 1] : vsp[2 * kk];
        }
      }

      // ---- scale, mask, online softmax (lane = one head, 8 keys per step)
      float mx = kNegInf;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int kp = kbase + 32 * kk + 8 * q4 + 4 * tt + jj;
          float x = s[tt][jj] * ksc[tt];
          x = (kp >= kbeg && kp < kend) ? x : kNegInf;
          s[tt][jj] = x;
          mx = fmaxf(mx, x);
        }
      }
      mx = fmaxf(mx, shfl_xor(mx, 16));
      mx = fmaxf(mx, shfl_xor(mx, 32));
      const bool bump = mx > m + kRescaleSlack;
      if (__builtin_amdgcn_ballot_w64(bump)) {
        const float alpha = bump ? fast_exp2(m - mx) : 1.f;
        m = bump ? mx : m;
        l *= alpha;
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt) o[dt] *= alpha;
      }
      const float m_use = m == kNegInf ? 0.f : m;
      float p[8];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const float e = fast_exp2(s[tt][jj] - m_use);
          l += e;
          p[4 * tt + jj] = FP8 ? e * vsc[tt] : e;
        }
      }
      const u32x4 pb = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                        pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
      // ---- O^T += V^T P^T: 16-lane group q4 supplies keys 8 q4 + 0..7;
      // lane li of the group addresses key 8 q4 + li/4 (+4), columns 4(li%4)..
      const int key0 = 32 * kk + 8 * q4 + (col >> 2);
      const lds_u8 *r0 = vblk + key0 * C::ROW;
      const lds_u8 *r1 = r0 + 4 * C::ROW;
      const int sw0 = dswz_v<C::CH>(key0), sw1 = dswz_v<C::CH>(key0 + 4);
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) {
        const int byte = 2 * (16 * dt + 4 * (col & 3));
        const int cidx = byte >> 4, within = byte & 15;
        const u32x2 lo2 = ds_read_tr16(r0 + ((cidx ^ sw0) << 4) + within);
        const u32x2 hi2 = ds_read_tr16(r1 + ((cidx ^ sw1) << 4) + within);
        o[dt] = mfma16x16x32(as_bf16x8(u32x4{lo2.x, lo2.y, hi2.x, hi2.y}), as_bf16x8(pb), o[dt]);
      }
    }
    asm volatile("" ::: "memory");
  }

  l += shfl_xor(l, 16);
  l += shfl_xor(l, 32);
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
  constexpr int KB = FP8 ? 64 : 32;
  constexpr int NS = D >= 256 ? 2 : 4;
  if (a.ps == 16)
    hipLaunchKernelGGL((decode_kernel<D, FP8, KB, NS, 16>), grid, dim3(64), 0, s, a);
  else
    hipLaunchKernelGGL((decode_kernel<D, FP8, KB, NS, 64>), grid, dim3(64), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.max_splits <= 1) return e;
  hipLaunchKernelGGL((combine_kernel<D>), dim3(a.h_q, num_seqs), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace

// partitions are kept to at most 256 pages (bounds the partial buffers)
int decode_max_split_len(int page_size) { return 256 * page_size; }

int decode_split_len(const PoolView &p, const BatchView &b, int h_q, int requested) {
  if (requested > 0) return requested;
  const int group = h_q / p.h_kv;
  const int head_chunks = (group + 15) / 16;
  const long long items = (long long)b.num_seqs * p.h_kv * head_chunks;
  long long want = (16384 + items - 1) / std::max<long long>(items, 1);
  want = std::min<long long>(std::max<long long>(want, 1), 256);
  long long len = (b.max_ctx + want - 1) / want;
  len = ((len + 63) / 64) * 64;
  len = std::max<long long>(len, 256);
  return (int)std::min<long long>(len, decode_max_split_len(p.ps));
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
