// prefix_prefill_attn and paged_decode_attn over two batches in one launch.
//
// A serving step that mixes prefix-reuse prefills with decodes (the batch
// of a chunked-prefill engine) has an MFMA-bound part and an HBM-bound part.
// Run back to back, each leaves the other's resource idle; here one grid
// holds both kinds of work item, so decode partitions stream K/V on CUs
// beside prefill row tiles that keep the matrix cores busy.
//
// Work items are exactly those of the two separate kernels (prefill_impl.hpp:
// one row tile of one KV head per 4-wave workgroup; decode_impl.hpp: one
// split-K partition of one KV head per wave, four per workgroup), with the
// same key partitions, so the outputs are bit-identical to the separate
// calls with the same decode partition length.
//
// The grid is dealt out in groups of 8 workgroups: workgroups go to the 8
// XCDs round-robin, so a prefill group keeps KV head g of consecutive tiles
// on XCD g, as the prefill kernel's own grid does.  Groups alternate in runs
// of `half` prefill groups and `half` decode groups.  Within an XCD
// workgroups fill the CUs round-robin, and a CU holds two (head_dim <= 128),
// so runs of 32 put one prefill and one decode workgroup on every CU of the
// first fill; longer runs (the default is three fills) start every CU on
// prefill tiles and let decode workgroups take the slots that finishing
// tiles free.  Measured at the Llama-3.1-70B step (one process, 20 reps):
// 9.2-9.5 ms for runs of 96-192 groups against 9.9-10.1 ms for the two
// kernels back to back; runs of 32 gave 9.4-9.8.  A batch whose decode is a
// small part of the work runs all prefill groups first (see launch_mixed).
#include <algorithm>

#include "args.hpp"

namespace ckv {
namespace {

struct MixedLayout {
  int32_t pf_items, pf_x, pf_y;  // prefill items = pf_x * pf_y * B (x: H_kv * splits, y: tiles)
  int32_t dc_items, dc_x, dc_y;  // decode items = dc_x * dc_y * B (x: padded splits, y: H_kv * chunks)
  int32_t pf_groups, dc_groups;  // groups of 8 workgroups
  int32_t half;                  // groups per run (runs alternate prefill, decode)
};

// Decode groups among group positions [0, i): in periods of 2 half
// positions the second half are decode groups, capped by the decode groups
// there are; past the last prefill group every position is a decode group.
// Non-decreasing in steps of 0 or 1 and reaching dc_groups at position
// pf_groups + dc_groups, so every group of either kind gets one position.
__device__ __forceinline__ int dc_before(const MixedLayout &m, int i) {
  const int h = m.half;
  long long pat = (long long)h * (i / (2LL * h)) + max(0LL, i % (2LL * h) - h);
  pat = max(pat, (long long)i - m.pf_groups);
  return (int)min(pat, (long long)m.dc_groups);
}

// AP: fused append (bf16 pools): the prefill batch's new turn and the
// decode batch's new tokens are written into the pool by this launch, and
// read from the input rows by its work items (PrefillArgs / DecodeArgs
// k_new, v_new; either pair may be null).
template <int D, int BN, bool FP8, int PS, bool AP>
__global__ __launch_bounds__(pf::kThreads, D >= 256 ? 1 : 2) void mixed_kernel(pf::PrefillArgs pa,
                                                                               dc::DecodeArgs da,
                                                                               MixedLayout m) {
  using PC = pf::Cfg<D, BN, FP8, PS>;
  using DC = dc::DCfg<D, FP8, PS>;
  constexpr int kWaves = pf::kThreads / 64;
  constexpr int LDS = PC::LDS > kWaves * DC::LDS ? PC::LDS : kWaves * DC::LDS;
  __shared__ __attribute__((aligned(1024))) uint8_t lds_[LDS];

  const int grp = (int)blockIdx.x >> 3, r = (int)blockIdx.x & 7;
  // decode groups before position grp, and whether grp holds one
  const int before = dc_before(m, grp);
  const bool is_dc = dc_before(m, grp + 1) > before;
  if (is_dc) {
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int d = (before * 8 + r) * kWaves + wave;
    if (d >= m.dc_items) return;
    const int split = d % m.dc_x;
    const int rest = d / m.dc_x;
    if (AP && da.k_new)
      dc::decode_item<D, FP8, PS, kWaves, AP>(da, as_lds(lds_) + wave * DC::LDS, split, rest % m.dc_y,
                                              rest / m.dc_y);
    else
      dc::decode_item<D, FP8, PS, kWaves>(da, as_lds(lds_) + wave * DC::LDS, split, rest % m.dc_y,
                                          rest / m.dc_y);
  } else {
    const int p = (grp - before) * 8 + r;
    if (p >= m.pf_items) return;
    const int rest = p / m.pf_x;
    if (AP && pa.k_new)
      pf::prefill_tile<D, BN, FP8, PS, AP>(pa, as_lds(lds_), p % m.pf_x, rest % m.pf_y, rest / m.pf_y);
    else
      pf::prefill_tile<D, BN, FP8, PS>(pa, as_lds(lds_), p % m.pf_x, rest % m.pf_y, rest / m.pf_y);
  }
}

template <int D, int BN, bool FP8, bool AP = false>
hipError_t launch(const pf::PrefillArgs &pa, const dc::DecodeArgs &da, const MixedLayout &m, int ps,
                  hipStream_t s) {
  const dim3 grid((unsigned)(8 * (m.pf_groups + m.dc_groups)));
  if (ps == 16)
    hipLaunchKernelGGL((mixed_kernel<D, BN, FP8, 16, AP>), grid, dim3(pf::kThreads), 0, s, pa, da, m);
  else
    hipLaunchKernelGGL((mixed_kernel<D, BN, FP8, 64, AP>), grid, dim3(pf::kThreads), 0, s, pa, da, m);
  return hipGetLastError();
}

}  // namespace

int mixed_split_len(const PoolView &p, const BatchView &db, int h_q, int requested) {
  if (requested > 0) return requested;
  // finer decode partitions interleave better with the prefill's tiles
  return std::min(decode_split_len(p, db, h_q, 0), 2048);
}

size_t mixed_workspace_bytes(const PoolView &p, const BatchView &pb, const BatchView &db, int h_q,
                             int split_len) {
  const size_t a = prefill_workspace_bytes(p, pb, h_q);
  const size_t b = db.num_seqs > 0 ? decode_workspace_bytes(p, db, h_q, mixed_split_len(p, db, h_q, split_len)) : 0;
  return (a + 255) / 256 * 256 + b;
}

hipError_t launch_mixed(const PoolView &p, const BatchView &pb, const void *q_pf, const void *k_pf,
                        const void *v_pf, void *out_pf, const BatchView &db, const void *q_dc,
                        const void *k_dc, const void *v_dc, void *out_dc, int h_q, float scale,
                        int window, int split_len, int interleave, void *ws, hipStream_t s) {
  const bool has_pf = pb.num_seqs > 0 && pb.max_q > 0 && pb.total_q > 0;
  const bool has_dc = db.num_seqs > 0;
  uint8_t *w = static_cast<uint8_t *>(ws);
  const size_t pf_ws = (prefill_workspace_bytes(p, pb, h_q) + 255) / 256 * 256;
  pf::PrefillArgs pa{};
  dc::DecodeArgs da{};
  MixedLayout m{};
  if (has_pf) {
    const hipError_t e = prefill_args(p, pb, q_pf, h_q, scale, window, out_pf, w, pa);
    if (e != hipSuccess) return e;
    pa.k_new = static_cast<const uint8_t *>(k_pf);
    pa.v_new = static_cast<const uint8_t *>(v_pf);
    m.pf_x = p.h_kv * pa.splits;
    m.pf_y = pa.tiles;
    m.pf_items = m.pf_x * m.pf_y * pb.num_seqs;
  }
  if (has_dc) {
    decode_args(p, db, q_dc, h_q, scale, window, mixed_split_len(p, db, h_q, split_len), out_dc,
                w + pf_ws, da);
    da.k_new = static_cast<const uint8_t *>(k_dc);
    da.v_new = static_cast<const uint8_t *>(v_dc);
    m.dc_x = da.max_splits | 1;  // the decode kernel's odd split stride
    m.dc_y = p.h_kv * da.head_chunks;
    m.dc_items = m.dc_x * m.dc_y * db.num_seqs;
  }
  constexpr int kWaves = pf::kThreads / 64;
  m.pf_groups = (m.pf_items + 7) / 8;
  m.dc_groups = (m.dc_items + 8 * kWaves - 1) / (8 * kWaves);
  const long long total = (long long)m.pf_groups + m.dc_groups;
  if (total == 0) return hipSuccess;
  if (8 * total > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  // Default runs: three fills of the GPU (256 CUs, two workgroups per CU
  // below head_dim 256) in groups of eight workgroups.  When the decode is a
  // small part of the step (its bytes at ~6.5 TB/s under 5 % of the prefill's
  // flops at ~1.1 PFLOP/s, both from the host-side bounds), all prefill
  // groups go first and the decode only fills the prefill's tail: at
  // GLM-4.5 (2 ms of decode in a 270 ms step) interleaving cost more than it
  // saved (272.1 ms prefill-first, 273.1 in runs of 192, 272.9 back to back).
  if (interleave > 0) {
    m.half = interleave;
  } else {
    const double e_kv = p.kv_dtype == 2 ? 1.0 : 2.0;
    const double pf_s = has_pf ? 4.0 * p.d * h_q * pb.total_q * ((double)pb.max_ctx + pb.max_q) / 1.1e15 : 0.0;
    const double dc_s = has_dc ? (double)db.num_seqs * db.max_ctx * p.h_kv * p.d * 2.0 * e_kv / 6.5e12 : 0.0;
    m.half = dc_s < 0.05 * pf_s ? 0x3fffffff : 3 * (p.d >= 256 ? 1 : 2) * 256 / 8;
  }
  const bool fp8 = p.kv_dtype == 2;
  const bool ap = (has_pf && k_pf) || (has_dc && k_dc);
  if (ap && fp8) return hipErrorInvalidValue;  // rejected by the caller's checks
  if (!has_pf) pa.k_new = pa.v_new = nullptr;
  if (!has_dc) da.k_new = da.v_new = nullptr;
  hipError_t e = hipErrorInvalidValue;
  switch (p.d) {
    case 64:
      e = fp8 ? launch<64, 64, true>(pa, da, m, p.ps, s)
              : (ap ? launch<64, 64, false, true>(pa, da, m, p.ps, s) : launch<64, 64, false>(pa, da, m, p.ps, s));
      break;
    case 128:
      e = fp8 ? launch<128, 64, true>(pa, da, m, p.ps, s)
              : (ap ? launch<128, 64, false, true>(pa, da, m, p.ps, s)
                    : launch<128, 64, false>(pa, da, m, p.ps, s));
      break;
    case 256:
      e = fp8 ? launch<256, 32, true>(pa, da, m, p.ps, s)
              : (ap ? launch<256, 64, false, true>(pa, da, m, p.ps, s)
                    : launch<256, 64, false>(pa, da, m, p.ps, s));
      break;
  }
  if (e != hipSuccess) return e;
  if (has_pf && pa.splits > 1) {
    e = launch_prefill_merge(pa, p.d, pb.total_q, s);
    if (e != hipSuccess) return e;
  }
  if (has_dc && da.max_splits > 1) e = launch_decode_merge(da, p.d, db.num_seqs, s);
  return e;
}

}  // namespace ckv
