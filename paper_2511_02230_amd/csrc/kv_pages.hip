// Whole-page moves between the pool and a dense staging area: the device
// half of offloading KV pages to host memory and reloading them after a
// TTL miss.  A pool page is one contiguous [num_kv_heads][page_size]
// [head_dim] block, so a page move is a straight copy; fp8 pools move their
// per-(page, head) scales with it.  HBM-bound; the host copies around these
// kernels (hipMemcpyAsync) are bound by the host link.
#include "common.hpp"
#include "launch.hpp"

namespace ckv {
namespace {

constexpr int kPageThreads = 256;

struct PageArgs {
  uint8_t *k_pool, *v_pool;
  float *k_scale, *v_scale;  // fp8 pools only
  uint8_t *st_k, *st_v;      // staging: num pages x page_bytes each
  float *st_ks, *st_vs;      // staging scales: num pages x H_kv each (fp8)
  const int32_t *pages;      // pool page of staging page i
  int32_t pool_pages, page_bytes, h_kv, blocks_per_page;
};

// TO_POOL: staging page i -> pool page pages[i]; else the reverse.  Page ids
// outside [0, pool_pages) are skipped (the pool is never written outside).
template <bool TO_POOL>
__global__ __launch_bounds__(kPageThreads) void page_copy_kernel(PageArgs a) {
  const int i = blockIdx.x / a.blocks_per_page, part = blockIdx.x % a.blocks_per_page;
  const int p = a.pages[i];
  if (p < 0 || p >= a.pool_pages) return;
  const size_t pool_off = (size_t)p * a.page_bytes, st_off = (size_t)i * a.page_bytes;
  const int chunks = a.page_bytes / 16;  // page_bytes is a multiple of 16
  for (int c = part * kPageThreads + threadIdx.x; c < chunks; c += a.blocks_per_page * kPageThreads) {
    if (TO_POOL) {
      st<u32x4>(a.k_pool + pool_off + 16 * c, ld<u32x4>(a.st_k + st_off + 16 * c));
      st<u32x4>(a.v_pool + pool_off + 16 * c, ld<u32x4>(a.st_v + st_off + 16 * c));
    } else {
      st<u32x4>(a.st_k + st_off + 16 * c, ld<u32x4>(a.k_pool + pool_off + 16 * c));
      st<u32x4>(a.st_v + st_off + 16 * c, ld<u32x4>(a.v_pool + pool_off + 16 * c));
    }
  }
  if (a.k_scale && part == 0) {
    for (int h = threadIdx.x; h < a.h_kv; h += kPageThreads) {
      if (TO_POOL) {
        a.k_scale[(size_t)p * a.h_kv + h] = a.st_ks[(size_t)i * a.h_kv + h];
        a.v_scale[(size_t)p * a.h_kv + h] = a.st_vs[(size_t)i * a.h_kv + h];
      } else {
        a.st_ks[(size_t)i * a.h_kv + h] = a.k_scale[(size_t)p * a.h_kv + h];
        a.st_vs[(size_t)i * a.h_kv + h] = a.v_scale[(size_t)p * a.h_kv + h];
      }
    }
  }
}

PageArgs page_args(const PoolView &p, const int32_t *pages, int n, void *staging) {
  PageArgs a;
  a.k_pool = static_cast<uint8_t *>(p.k);
  a.v_pool = static_cast<uint8_t *>(p.v);
  const bool fp8 = p.kv_dtype == 2;
  a.k_scale = fp8 ? const_cast<float *>(p.k_scale) : nullptr;
  a.v_scale = fp8 ? const_cast<float *>(p.v_scale) : nullptr;
  a.page_bytes = page_bytes(p);
  uint8_t *s = static_cast<uint8_t *>(staging);
  a.st_k = s;
  a.st_v = s + (size_t)n * a.page_bytes;
  a.st_ks = fp8 ? reinterpret_cast<float *>(s + 2 * (size_t)n * a.page_bytes) : nullptr;
  a.st_vs = fp8 ? a.st_ks + (size_t)n * p.h_kv : nullptr;
  a.pages = pages;
  a.pool_pages = p.num_pages;
  a.h_kv = p.h_kv;
  a.blocks_per_page = page_blocks(p);
  return a;
}

template <bool TO_POOL>
hipError_t launch_copy(const PageArgs &a, int n, hipStream_t s) {
  const dim3 grid((unsigned)n * a.blocks_per_page);
  hipLaunchKernelGGL((page_copy_kernel<TO_POOL>), grid, dim3(kPageThreads), 0, s, a);
  return hipGetLastError();
}

// Host <-> staging copies.  Staging holds [K pages][V pages][K scales]
// [V scales] back to back; host segments that are also adjacent in host
// memory (e.g. one buffer holding all four) go as one copy, since each copy
// carries a fixed setup cost that dominates small moves.
hipError_t host_copies(const PageArgs &a, int n, int h_kv, const void *const host[4], bool to_dev,
                       hipStream_t s) {
  const size_t bytes = (size_t)n * a.page_bytes, sbytes = (size_t)n * h_kv * sizeof(float);
  const int segs = a.k_scale ? 4 : 2;
  uint8_t *stg = a.st_k;
  size_t len[4] = {bytes, bytes, sbytes, sbytes};
  size_t off = 0;
  for (int i = 0; i < segs;) {
    const uint8_t *h0 = static_cast<const uint8_t *>(host[i]);
    size_t run = len[i];
    int j = i + 1;
    while (j < segs && static_cast<const uint8_t *>(host[j]) == h0 + run) run += len[j++];
    const hipError_t e =
        to_dev ? hipMemcpyAsync(stg + off, h0, run, hipMemcpyHostToDevice, s)
               : hipMemcpyAsync(const_cast<uint8_t *>(h0), stg + off, run, hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) return e;
    off += run;
    i = j;
  }
  return hipSuccess;
}

}  // namespace

int page_bytes(const PoolView &p) {
  const int e = p.kv_dtype == 0 ? 4 : (p.kv_dtype == 1 ? 2 : 1);
  return p.h_kv * p.ps * p.d * e;
}

int page_blocks(const PoolView &p) { return (page_bytes(p) / 16 + kPageThreads - 1) / kPageThreads; }

size_t pages_staging_bytes(const PoolView &p, int n) {
  size_t b = 2 * (size_t)n * page_bytes(p);
  if (p.kv_dtype == 2) b += 2 * (size_t)n * p.h_kv * sizeof(float);
  return b;
}

hipError_t launch_pages_reload(const PoolView &p, const void *host_k, const void *host_v,
                               const float *host_ks, const float *host_vs, const int32_t *pages,
                               int n, void *staging, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const PageArgs a = page_args(p, pages, n, staging);
  const void *host[4] = {host_k, host_v, host_ks, host_vs};
  const hipError_t e = host_copies(a, n, p.h_kv, host, true, s);
  if (e != hipSuccess) return e;
  return launch_copy<true>(a, n, s);
}

hipError_t launch_pages_offload(const PoolView &p, const int32_t *pages, int n, void *host_k,
                                void *host_v, float *host_ks, float *host_vs, void *staging,
                                hipStream_t s) {
  if (n == 0) return hipSuccess;
  const PageArgs a = page_args(p, pages, n, staging);
  const hipError_t e = launch_copy<false>(a, n, s);
  if (e != hipSuccess) return e;
  const void *host[4] = {host_k, host_v, host_ks, host_vs};
  return host_copies(a, n, p.h_kv, host, false, s);
}

}  // namespace ckv
