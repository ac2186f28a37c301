// scan.h -- device-wide exclusive scan over uint32 (default) or uint64 items
// (per-tile reduce, one-block scan of the tile sums, per-tile down-sweep; up
// to 2048 tiles the down-sweep adds up the preceding tile sums itself and the
// middle launch is skipped).  Item producers and prefix consumers are
// functors, so callers fuse their own load (counts, bitmap popcounts, miss
// flags) and store (offsets, word ranks, compaction scatter) into the scan's
// two passes over the data.  A uint64 item can carry two 32-bit counters that are scanned
// together (high and low word), as long as neither total reaches 2^32.
#pragma once

#include "common.h"

namespace fast {

constexpr int SCAN_THREADS = 256;
constexpr int SCAN_ITEMS = 8;
constexpr int SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;

inline int64_t scan_tiles(int64_t n) { return (n + SCAN_TILE - 1) / SCAN_TILE; }
// Workspace of one scan over n items of type T: the tile sums plus the total.
template <typename T = uint32_t>
inline size_t scan_workspace(int64_t n) {
  return align_up(size_t(scan_tiles(n) + 1) * sizeof(T), 256);
}

// Exclusive prefix of a 256-thread block; returns the thread's exclusive
// prefix and writes the block total.  Uses 4 items of LDS.
template <typename T>
__device__ __forceinline__ T block_exclusive_scan(T x, T* lds4, T& total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  T inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    T y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  if (lane == 63) lds4[wid] = inc;
  __syncthreads();
  T before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < SCAN_THREADS / 64; ++w) {
    T v = lds4[w];
    before += (w < wid) ? v : T(0);
    tot += v;
  }
  __syncthreads();
  total = tot;
  return before + inc - x;
}

template <class In, typename T = uint32_t>
__global__ void __launch_bounds__(SCAN_THREADS) k_scan_reduce(In in, int64_t n, T* tsum) {
  __shared__ T lds4[4];
  const int64_t base = int64_t(blockIdx.x) * SCAN_TILE;
  T s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int64_t i = base + k * SCAN_THREADS + threadIdx.x;
    if (i < n) s += in(i);
  }
  T total;
  block_exclusive_scan(s, lds4, total);
  if (threadIdx.x == 0) tsum[blockIdx.x] = total;
}

// One 256-thread block scans the nt tile sums in place (exclusive) and
// stores the grand total at tsum[nt] and into the optional outputs.  The
// sums are walked SCAN_TILE at a time (coalesced loads through LDS, then
// SCAN_ITEMS consecutive sums per thread), so a scan of 10^8 items needs
// about 50 block-wide steps here.
template <typename T = uint32_t>
__global__ void __launch_bounds__(SCAN_THREADS) k_scan_top(T* tsum, int64_t nt,
                                                           int64_t* total_i64,
                                                           int32_t* total_i32) {
  __shared__ T tile[SCAN_TILE + SCAN_TILE / 32];
  __shared__ T lds4[4];
  T carry = 0;
  for (int64_t b0 = 0; b0 < nt; b0 += SCAN_TILE) {
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
      const int j = k * SCAN_THREADS + threadIdx.x;
      const int64_t i = b0 + j;
      tile[j + (j >> 5)] = (i < nt) ? tsum[i] : T(0);
    }
    __syncthreads();
    T v[SCAN_ITEMS], s = 0;
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
      const int j = threadIdx.x * SCAN_ITEMS + k;
      v[k] = tile[j + (j >> 5)];
      s += v[k];
    }
    T total;
    T run = carry + block_exclusive_scan(s, lds4, total);
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
      const int j = threadIdx.x * SCAN_ITEMS + k;
      tile[j + (j >> 5)] = run;
      run += v[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
      const int j = k * SCAN_THREADS + threadIdx.x;
      const int64_t i = b0 + j;
      if (i < nt) tsum[i] = tile[j + (j >> 5)];
    }
    carry += total;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    tsum[nt] = carry;
    if (total_i64) *total_i64 = int64_t(carry);
    if (total_i32) *total_i32 = int32_t(carry);
  }
}

// Down-sweep: the tile's items are loaded striped (coalesced) into LDS, each
// thread scans SCAN_ITEMS consecutive items, and the exclusive prefixes
// replace the items in LDS (plus the running total after the last item), so
// that `out` is called in striped order too -- neighbouring lanes write
// neighbouring outputs (offsets, ranks, slot maps) -- with each item's value
// recovered as the difference of consecutive prefixes.  The tile's base is
// tsum[tile] after the one-block scan of the tile sums, or, with SUM_PREV
// (few tiles), the sum of the unscanned tile sums before it, added up by the
// tile's own workgroup; the last tile then also stores the grand total.
// The down-sweep of one tile: items [base, base + SCAN_TILE) (those below n)
// from their prefix tile_base; returns the tile's sum in `total`.  Every
// thread of the workgroup must call it.
template <class In, class Out, typename T>
__device__ __forceinline__ void scan_tile_down(In in, int64_t n, int64_t base, T tile_base, Out out,
                                               T* lds4, T& total_out) {
  constexpr int PAD_END = SCAN_TILE + SCAN_TILE / 32;
  __shared__ T tile[PAD_END + 1];
  // striped, coalesced load into LDS (padded every 32 words against bank conflicts)
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int j = k * SCAN_THREADS + threadIdx.x;
    const int64_t i = base + j;
    tile[j + (j >> 5)] = (i < n) ? in(i) : T(0);
  }
  __syncthreads();
  T v[SCAN_ITEMS], s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int j = threadIdx.x * SCAN_ITEMS + k;
    v[k] = tile[j + (j >> 5)];
    s += v[k];
  }
  T total;
  // (the block scan's barriers also order every read of tile above before
  // the writes below)
  T run = block_exclusive_scan(s, lds4, total) + tile_base;
  total_out = total;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int j = threadIdx.x * SCAN_ITEMS + k;
    tile[j + (j >> 5)] = run;
    run += v[k];
  }
  if (threadIdx.x == SCAN_THREADS - 1) tile[PAD_END] = run;
  __syncthreads();
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int j = k * SCAN_THREADS + threadIdx.x;
    const int64_t i = base + j;
    const int j1 = j + 1;
    const T p0 = tile[j + (j >> 5)];
    const T p1 = j1 < SCAN_TILE ? tile[j1 + (j1 >> 5)] : tile[PAD_END];
    if (i < n) out(i, p0, T(p1 - p0));
  }
}

template <class In, class Out, typename T = uint32_t, bool SUM_PREV = false>
__global__ void __launch_bounds__(SCAN_THREADS) k_scan_down(In in, int64_t n,
                                                            const T* tsum, Out out,
                                                            int64_t* total_i64, int32_t* total_i32) {
  __shared__ T lds4[4];
  T tile_base;
  if constexpr (SUM_PREV) {
    T part = 0;
    for (int64_t t = threadIdx.x; t < int64_t(blockIdx.x); t += SCAN_THREADS) part += tsum[t];
    block_exclusive_scan(part, lds4, tile_base);   // block-wide sum of the parts
  } else {
    tile_base = tsum[blockIdx.x];
  }
  T total;
  scan_tile_down(in, n, int64_t(blockIdx.x) * SCAN_TILE, tile_base, out, lds4, total);
  if constexpr (SUM_PREV) {
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) {
      if (total_i64) *total_i64 = int64_t(tile_base + total);
      if (total_i32) *total_i32 = int32_t(tile_base + total);
    }
  }
}

// Enqueues the launches: per-tile reduce, then either (at most
// SCAN_FEW_TILES tiles) the down-sweep in which every tile adds up the tile
// sums before it, or the one-block scan of the tile sums and the down-sweep.
// ws must hold scan_workspace<T>(n) bytes.  total_i64 / total_i32 (device,
// optional) receive the sum of all items.
constexpr int64_t SCAN_FEW_TILES = 2048;

// The launches after the per-tile reduce, for a scan whose tile sums are
// already in ws (tsum[t] = the sum of items [t SCAN_TILE, (t+1) SCAN_TILE)),
// written by k_scan_reduce or by a caller's kernel that produces the items.
template <class In, class Out, typename T = uint32_t>
hipError_t scan_finish_launch(In in, Out out, int64_t n, void* ws, int64_t* total_i64,
                              int32_t* total_i32, hipStream_t st) {
  T* tsum = static_cast<T*>(ws);
  const int64_t nt = scan_tiles(n);
  if (nt > 0 && nt <= SCAN_FEW_TILES) {
    hipLaunchKernelGGL((k_scan_down<In, Out, T, true>), dim3(uint32_t(nt)), dim3(SCAN_THREADS), 0, st,
                       in, n, tsum, out, total_i64, total_i32);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_scan_top<T>, dim3(1), dim3(SCAN_THREADS), 0, st, tsum, nt, total_i64,
                     total_i32);
  if (nt > 0) {
    hipLaunchKernelGGL((k_scan_down<In, Out, T, false>), dim3(uint32_t(nt)), dim3(SCAN_THREADS), 0, st,
                       in, n, tsum, out, static_cast<int64_t*>(nullptr), static_cast<int32_t*>(nullptr));
  }
  return hipGetLastError();
}

template <class In, class Out, typename T = uint32_t>
hipError_t scan_launch(In in, Out out, int64_t n, void* ws, int64_t* total_i64,
                       int32_t* total_i32, hipStream_t st) {
  const int64_t nt = scan_tiles(n);
  if (nt > 0) {
    hipLaunchKernelGGL((k_scan_reduce<In, T>), dim3(uint32_t(nt)), dim3(SCAN_THREADS), 0, st, in, n,
                       static_cast<T*>(ws));
  }
  return scan_finish_launch<In, Out, T>(in, out, n, ws, total_i64, total_i32, st);
}

}  // namespace fast
