// offsets.hip -- CSR offsets of a sampled block (Sec. 5: the compression
// engine's CSR-style ind_ptr): an exclusive scan of per-destination counts.
#include "scan.h"

namespace fast {

struct InCounts {
  const int32_t* c;
  __device__ uint32_t operator()(int64_t i) const { return uint32_t(c[i]); }
};
struct OutOffsets {
  int32_t* off;
  __device__ void operator()(int64_t i, uint32_t prefix, uint32_t) const { off[i] = int32_t(prefix); }
};

// Several blocks in one pair of launches: the scan tiles of block b are
// [t0[b], t0[b+1]) of the grid; each tile reduces its counts, then adds up
// the tile sums before it within its own block (as the few-tiles plan of the
// single-block scan does) and writes that block's offsets.
constexpr int OFF_MAX_BATCH = 8;
struct OffBatch {
  int nb;
  const int32_t* counts[OFF_MAX_BATCH];
  int32_t* off[OFF_MAX_BATCH];
  int64_t n[OFF_MAX_BATCH];
  int64_t t0[OFF_MAX_BATCH + 1];   // first tile of each block; t0[nb] = all tiles
};

__device__ __forceinline__ int batch_block(const OffBatch& B, int64_t t) {
  int b = 0;
#pragma unroll
  for (int k = 1; k < OFF_MAX_BATCH; ++k)
    if (k < B.nb && t >= B.t0[k]) b = k;
  return b;
}

__global__ void __launch_bounds__(SCAN_THREADS) k_off_batch_reduce(OffBatch B, uint32_t* tsum) {
  __shared__ uint32_t lds4[4];
  const int64_t t = blockIdx.x;
  const int b = batch_block(B, t);
  const int64_t base = (t - B.t0[b]) * SCAN_TILE, n = B.n[b];
  const int32_t* c = B.counts[b];
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int64_t i = base + k * SCAN_THREADS + threadIdx.x;
    if (i < n) s += uint32_t(c[i]);
  }
  uint32_t total;
  block_exclusive_scan(s, lds4, total);
  if (threadIdx.x == 0) tsum[t] = total;
}

__global__ void __launch_bounds__(SCAN_THREADS) k_off_batch_down(OffBatch B, const uint32_t* tsum) {
  __shared__ uint32_t lds4[4];
  const int64_t t = blockIdx.x;
  const int b = batch_block(B, t);
  uint32_t part = 0;
  for (int64_t j = B.t0[b] + threadIdx.x; j < t; j += SCAN_THREADS) part += tsum[j];
  uint32_t tile_base;
  block_exclusive_scan(part, lds4, tile_base);   // block-wide sum of the parts
  uint32_t total;
  scan_tile_down(InCounts{B.counts[b]}, B.n[b], (t - B.t0[b]) * SCAN_TILE, tile_base,
                 OutOffsets{B.off[b]}, lds4, total);
  if (threadIdx.x == 0) {
    if (t == B.t0[b + 1] - 1) B.off[b][B.n[b]] = int32_t(tile_base + total);   // the block's E
    if (t == 0) {                     // blocks without counts: offsets = {0}
      for (int k = 0; k < B.nb; ++k)
        if (B.n[k] == 0) B.off[k][0] = 0;
    }
  }
}

}  // namespace fast

using namespace fast;

extern "C" size_t fast_csr_offsets_workspace(int64_t n) {
  return n < 0 ? 0 : scan_workspace(n);
}

extern "C" fast_status_t fast_csr_offsets(const int32_t* counts, int64_t n, int32_t* offsets,
                                          void* ws, size_t ws_bytes, fast_stream_t stream) {
  if (n < 0) return fail(FAST_ERR_INVALID_ARG, "fast_csr_offsets: n = %lld < 0", (long long)n);
  if (n >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "fast_csr_offsets: n >= 2^31");
  if (!offsets) return fail(FAST_ERR_INVALID_ARG, "fast_csr_offsets: offsets is NULL");
  if (n > 0 && !counts) return fail(FAST_ERR_INVALID_ARG, "fast_csr_offsets: counts is NULL");
  if (!ws || ws_bytes < scan_workspace(n))
    return fail(FAST_ERR_WORKSPACE, "fast_csr_offsets: workspace %zu < %zu bytes", ws_bytes,
                scan_workspace(n));
  hipError_t e = scan_launch(InCounts{counts}, OutOffsets{offsets}, n, ws, nullptr, offsets + n,
                             static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "fast_csr_offsets: %s", hipGetErrorString(e));
  return ok();
}

// Batched form: the workspace holds either the batch's tile sums or, when a
// block has too many tiles for the one-pair plan (or there are more than
// OFF_MAX_BATCH blocks), the largest single-block workspace (the blocks then
// run one after another).
static bool batch_one_pair(int nblocks, const int64_t* n) {
  if (nblocks > OFF_MAX_BATCH) return false;
  int64_t tiles = 0;
  for (int b = 0; b < nblocks; ++b) {
    if (scan_tiles(n[b]) > SCAN_FEW_TILES) return false;
    tiles += scan_tiles(n[b]);
  }
  return tiles > 0;
}

extern "C" size_t fast_csr_offsets_batched_workspace(int nblocks, const int64_t* n) {
  if (nblocks < 0 || (nblocks > 0 && !n)) return 0;
  size_t single = 256, tiles = 0;
  for (int b = 0; b < nblocks; ++b) {
    if (n[b] < 0) return 0;
    const size_t w = scan_workspace(n[b]);
    single = w > single ? w : single;
    tiles += size_t(scan_tiles(n[b]));
  }
  const size_t pair = align_up(tiles * sizeof(uint32_t), 256);
  return pair > single ? pair : single;
}

extern "C" fast_status_t fast_csr_offsets_batched(int nblocks, const int32_t* const* counts,
                                                  const int64_t* n, int32_t* const* offsets,
                                                  void* ws, size_t ws_bytes, fast_stream_t stream) {
  const char* fn = "fast_csr_offsets_batched";
  if (nblocks < 0) return fail(FAST_ERR_INVALID_ARG, "%s: nblocks = %d < 0", fn, nblocks);
  if (nblocks == 0) return ok();
  if (!counts || !n || !offsets) return fail(FAST_ERR_INVALID_ARG, "%s: NULL host array", fn);
  for (int b = 0; b < nblocks; ++b) {
    if (n[b] < 0) return fail(FAST_ERR_INVALID_ARG, "%s: n[%d] = %lld < 0", fn, b, (long long)n[b]);
    if (n[b] >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: n[%d] >= 2^31", fn, b);
    if (!offsets[b]) return fail(FAST_ERR_INVALID_ARG, "%s: offsets[%d] is NULL", fn, b);
    if (n[b] > 0 && !counts[b]) return fail(FAST_ERR_INVALID_ARG, "%s: counts[%d] is NULL", fn, b);
  }
  const size_t need = fast_csr_offsets_batched_workspace(nblocks, n);
  if (!ws || ws_bytes < need)
    return fail(FAST_ERR_WORKSPACE, "%s: workspace %zu < %zu bytes", fn, ws_bytes, need);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (!batch_one_pair(nblocks, n)) {
    for (int b = 0; b < nblocks; ++b) {
      const hipError_t e = scan_launch(InCounts{counts[b]}, OutOffsets{offsets[b]}, n[b], ws, nullptr,
                                       offsets[b] + n[b], st);
      if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
    }
    return ok();
  }
  OffBatch B = {};
  B.nb = nblocks;
  int64_t t = 0;
  for (int b = 0; b < nblocks; ++b) {
    B.counts[b] = counts[b];
    B.off[b] = offsets[b];
    B.n[b] = n[b];
    B.t0[b] = t;
    t += scan_tiles(n[b]);
  }
  B.t0[nblocks] = t;
  uint32_t* tsum = static_cast<uint32_t*>(ws);
  hipLaunchKernelGGL(k_off_batch_reduce, dim3(uint32_t(t)), dim3(SCAN_THREADS), 0, st, B, tsum);
  hipLaunchKernelGGL(k_off_batch_down, dim3(uint32_t(t)), dim3(SCAN_THREADS), 0, st, B,
                     static_cast<const uint32_t*>(tsum));
  return check_launch(fn);
}
