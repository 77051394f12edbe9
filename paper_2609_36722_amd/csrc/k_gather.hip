// K1: paged artifact pool -- store and block-table gather (bit-exact copies).
//
// Pools with one layout: the HBM pool and, optionally, a host pool in pinned
// host memory (the paper keeps artifact caches in CPU RAM and copies them to
// the GPU per request, inside the timed region, appendix A.2) and a staging
// pool in HBM.  The gather kernel reads host pages over the host link
// directly, or, after bulk copies moved them into the staging pool,
// from there (a block-table entry's flag bits say which pool).
// Pool layout: [n_layers][pool_pages][2 (K, V)][n_kv][16 tokens][128] bf16, so
// one page of one layer is a contiguous 2 * n_kv * 4 KiB block and each
// (K|V, head) slab of it is 4 KiB.  Request cache layout:
// [n_layers][2][n_kv][cache_rows][128].
//
// Gather: one workgroup of 256 threads moves one (K|V, head) slab of one
// layer for a run of kGatherRun consecutive block-table entries: thread t
// owns row t / 16 and 16-byte chunk t % 16 of the slab in each entry, so a
// workgroup reads kGatherRun 4 KiB spans and writes them to one cache plane,
// where consecutive entries' rows follow each other.  Measured on gfx950 for
// the 9.66 GB of the 36-layer 32k-token cache: one workgroup per page (all 16
// slabs, 16 writes 9 MB apart) 1.89 ms, runs of 4 entries 1.52-1.55 ms (66
// VGPRs), single entries 1.50 ms (8 VGPRs); runs of 8 are slower.  With 8
// VGPRs the gather's waves also fit beside the attention kernel's (two waves
// of 240 VGPRs per SIMD leave 32), so per-layer gathers on a second stream
// hide better: 36-layer steps 22.22 -> 22.06 ms (32k cached tokens), 8.02 ->
// 7.82 ms (17.7k), 3.32 -> 3.26 ms (8k) against runs of 4.  Loads and stores
// are streaming (non-temporal: every byte is touched once).  The block-table
// entries are wave-uniform and live in scalar registers.  The store kernel
// keeps one workgroup per page.

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace attuner {

namespace {

constexpr int kSlabBatch = 8;

ATTUNER_VIOLATION_WORD(g_violations_gather, read_violations_gather_impl)

__global__ __launch_bounds__(256) void store_pages_kernel(const u32x4* __restrict__ k, const u32x4* __restrict__ v,
                                                          int n_tokens, const int32_t* __restrict__ pages,
                                                          u32x4* __restrict__ pool, int64_t pool_pages, int n_kv) {
  const int pi = blockIdx.x;      // page index within the artifact
  const int layer = blockIdx.y;
  const int page = pages[pi];
  if constexpr (kChecked) {
    if (page < 0 || page >= pool_pages) {
      if (threadIdx.x == 0) ATTUNER_VIOLATE(g_violations_gather, kViolStorePage);
      return;
    }
  }
  const int rr = threadIdx.x >> 4;
  const int chunk = threadIdx.x & 15;
  const int tok = pi * kPageTokens + rr;
  const bool valid = tok < n_tokens;
  const int n_slab = 2 * n_kv;
  for (int s0 = 0; s0 < n_slab; s0 += kSlabBatch) {
    u32x4 buf[kSlabBatch];
#pragma unroll
    for (int i = 0; i < kSlabBatch; ++i) {
      const int s = s0 + i;
      buf[i] = u32x4{0u, 0u, 0u, 0u};
      if (s < n_slab && valid) {
        const int c = s / n_kv, g = s % n_kv;
        const u32x4* src = c ? v : k;
        buf[i] = src[(((int64_t)layer * n_kv + g) * n_tokens + tok) * 16 + chunk];
      }
    }
#pragma unroll
    for (int i = 0; i < kSlabBatch; ++i) {
      const int s = s0 + i;
      if (s < n_slab) {
        const int64_t slab = ((int64_t)layer * pool_pages + page) * n_slab + s;
        pool[(slab * kPageTokens + rr) * 16 + chunk] = buf[i];
      }
    }
  }
}

constexpr int kGatherRun = 1;  // block-table entries per gather workgroup

__global__ __launch_bounds__(256) void gather_kernel(const int4* __restrict__ table, int64_t n_entries,
                                                     const u32x4* __restrict__ dev_pool, int64_t dev_pages,
                                                     const u32x4* __restrict__ host_pool, int64_t host_pages,
                                                     const u32x4* __restrict__ stage_pool, int64_t stage_pages,
                                                     int n_kv, u32x4* __restrict__ req_kv, int64_t cache_rows,
                                                     int layer_begin) {
  const int n_slab = 2 * n_kv;
  const int64_t e0 = (int64_t)blockIdx.x * kGatherRun;
  const int s = (int)(blockIdx.y % n_slab);  // slab s = c * n_kv + g
  const int layer = layer_begin + (int)(blockIdx.y / n_slab);
  const int rr = threadIdx.x >> 4;
  const int chunk = threadIdx.x & 15;
  // slab s of layer l is cache plane (l * 2 + c) * n_kv + g
  const int64_t plane = (int64_t)layer * n_slab + s;
  int4 ent[kGatherRun];  // {page, n_valid, dst_row, request}
  u32x4 buf[kGatherRun];
#pragma unroll
  for (int i = 0; i < kGatherRun; ++i) {
    ent[i] = e0 + i < n_entries ? table[e0 + i] : int4{0, 0, 0, 0};
    if constexpr (kChecked) {
      const bool rows_ok = ent[i].y >= 0 && ent[i].y <= kPageTokens && ent[i].z >= 0 &&
                           (int64_t)ent[i].z + ent[i].y <= cache_rows;
      const bool staged_ = (ent[i].x & kStagePageFlag) != 0, host_ = (ent[i].x & kHostPageFlag) != 0;
      const u32x4* pool_ = staged_ ? stage_pool : host_ ? host_pool : dev_pool;
      const int64_t pages_ = pool_ == nullptr ? 0 : staged_ ? stage_pages : host_ ? host_pages : dev_pages;
      const bool page_ok = ent[i].x >= 0 && (int64_t)(ent[i].x & kPageIdMask) < pages_;
      if (ent[i].y != 0 && (!rows_ok || !page_ok)) {
        if (threadIdx.x == 0) ATTUNER_VIOLATE(g_violations_gather, rows_ok ? kViolGatherPage : kViolGatherRows);
        ent[i].y = 0;  // neither read nor write this entry
      }
    }
    if (rr < ent[i].y) {
      const bool host = (ent[i].x & kHostPageFlag) != 0;
      const bool staged = (ent[i].x & kStagePageFlag) != 0;
      const u32x4* __restrict__ pool = staged ? stage_pool : host ? host_pool : dev_pool;
      const int64_t pool_pages = staged ? stage_pages : host ? host_pages : dev_pages;
      const int64_t src = ((int64_t)layer * pool_pages + (ent[i].x & kPageIdMask)) * n_slab + s;
      buf[i] = __builtin_nontemporal_load(pool + (src * kPageTokens + rr) * 16 + chunk);
    }
  }
#pragma unroll
  for (int i = 0; i < kGatherRun; ++i)
    if (rr < ent[i].y)
      __builtin_nontemporal_store(buf[i], req_kv + (plane * cache_rows + ent[i].z + rr) * 16 + chunk);
}

}  // namespace

hipError_t read_violations_gather(unsigned int* bits, bool reset) { return read_violations_gather_impl(bits, reset); }

hipError_t launch_store_pages(const uint16_t* k, const uint16_t* v, int n_tokens, const int32_t* pages_dev,
                              int n_pages, uint16_t* pool, int64_t pool_pages, int n_layers, int n_kv,
                              hipStream_t stream) {
  if (n_pages == 0) return hipSuccess;
  dim3 grid(n_pages, n_layers);
  ATTUNER_LAUNCH("store_pages_kernel", store_pages_kernel, grid, dim3(256), stream, reinterpret_cast<const u32x4*>(k),
                     reinterpret_cast<const u32x4*>(v), n_tokens, pages_dev, reinterpret_cast<u32x4*>(pool),
                     pool_pages, n_kv);
  return hipGetLastError();
}

hipError_t launch_gather(const int32_t* table_dev, int64_t n_entries, const uint16_t* pool, int64_t pool_pages,
                         const uint16_t* host_pool, int64_t host_pages, const uint16_t* stage_pool,
                         int64_t stage_pages, int layer_begin, int n_layers, int n_kv, uint16_t* req_kv,
                         int64_t cache_rows, hipStream_t stream) {
  if (n_entries == 0 || n_layers == 0) return hipSuccess;
  const int64_t runs = (n_entries + kGatherRun - 1) / kGatherRun;
  if (runs > INT32_MAX) return hipErrorInvalidValue;
  // grid.y = layers x slabs, at most 65535 per launch
  const int per_launch = std::max(1, 65535 / (2 * n_kv));
  for (int l0 = 0; l0 < n_layers; l0 += per_launch) {
    const int nl = std::min(per_launch, n_layers - l0);
    dim3 grid(static_cast<unsigned>(runs), static_cast<unsigned>(nl * 2 * n_kv));
    ATTUNER_LAUNCH("gather_kernel", gather_kernel, grid, dim3(256), stream, reinterpret_cast<const int4*>(table_dev),
                   n_entries, reinterpret_cast<const u32x4*>(pool), pool_pages,
                   reinterpret_cast<const u32x4*>(host_pool), host_pages,
                   reinterpret_cast<const u32x4*>(stage_pool), stage_pages, n_kv, reinterpret_cast<u32x4*>(req_kv),
                   cache_rows, layer_begin + l0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace attuner
