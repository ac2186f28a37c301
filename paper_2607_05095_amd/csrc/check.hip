// check.hip -- contract check of a sampled temporal subgraph: counts the ways
// a CSR block (Sec. 4.3 CSR layout, Sec. 5 ind_ptr) breaks the data contract
// every other operator assumes.  Read-only over the subgraph; every offset is
// clamped before it addresses an edge array.
#include "common.h"

namespace fast {

constexpr int CK_THREADS = 256;
constexpr int CK_WAVES = CK_THREADS / 64;
constexpr int CK_MAX_BLOCKS = 2048;

__global__ void __launch_bounds__(64) k_check_zero(int64_t* v) {
  if (threadIdx.x < 5) v[threadIdx.x] = 0;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

__device__ __forceinline__ void flush(int64_t* dst, uint64_t c) {
  c = wave_sum_u64(c);
  if ((threadIdx.x & 63) == 0 && c != 0)
    atomicAdd(reinterpret_cast<unsigned long long*>(dst), (unsigned long long)c);
}

// Thread-per-element passes for [0], [2], [3]; wave-per-destination pass for
// [4]; one thread for [1].  The dt pass visits each monotone segment's edges,
// clamped to [0, E): its cost is E for well-formed offsets.
__global__ void __launch_bounds__(CK_THREADS) k_check(const int32_t* __restrict__ off, int64_t N,
                                                      int64_t E, const int64_t* __restrict__ src,
                                                      int64_t src_bound,
                                                      const int64_t* __restrict__ eid,
                                                      int64_t edge_bound,
                                                      const float* __restrict__ et,
                                                      const float* __restrict__ dt,
                                                      int64_t* __restrict__ viol) {
  const int64_t tid = int64_t(blockIdx.x) * CK_THREADS + threadIdx.x;
  const int64_t nthr = int64_t(gridDim.x) * CK_THREADS;
  uint64_t c0 = 0, c2 = 0, c3 = 0, c4 = 0;
  for (int64_t v = tid; v < N; v += nthr) c0 += off[v + 1] < off[v];
  if (src || eid)
    for (int64_t e = tid; e < E; e += nthr) {
      if (src) {
        const int64_t s = src[e];
        c2 += (s < 0) | (s >= src_bound);
      }
      if (eid) {
        const int64_t s = eid[e];
        c3 += (s < 0) | (s >= edge_bound);
      }
    }
  if (et && dt) {
    const int lane = threadIdx.x & 63;
    const int64_t wave = int64_t(blockIdx.x) * CK_WAVES + (threadIdx.x >> 6);
    const int64_t nwave = int64_t(gridDim.x) * CK_WAVES;
    for (int64_t v = wave; v < N; v += nwave) {
      const int64_t a = off[v], b = off[v + 1];
      if (b < a) continue;
      const int64_t lo = clamp64(a, 0, E), hi = clamp64(b, 0, E);
      const float tv = dt[v];
      for (int64_t e = lo + lane; e < hi; e += 64) c4 += et[e] > tv;
    }
  }
  flush(viol + 0, c0);
  flush(viol + 2, c2);
  flush(viol + 3, c3);
  flush(viol + 4, c4);
  if (tid == 0) {
    const uint64_t c1 = uint64_t(off[0] != 0) + uint64_t(int64_t(off[N]) != E);
    if (c1) atomicAdd(reinterpret_cast<unsigned long long*>(viol + 1), (unsigned long long)c1);
  }
}

}  // namespace fast

using namespace fast;

extern "C" fast_status_t fast_check_tcsr(const fast_tcsr_t* g, int64_t src_bound,
                                         int64_t edge_bound, int64_t* violations,
                                         fast_stream_t stream) {
  static const char* fn = "fast_check_tcsr";
  if (!g) return fail(FAST_ERR_INVALID_ARG, "%s: g is NULL", fn);
  const int64_t N = g->num_dst, E = g->num_edges;
  if (N < 0 || E < 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: N = %lld, E = %lld", fn, (long long)N, (long long)E);
  if (N >= (int64_t(1) << 31) || E >= (int64_t(1) << 31))
    return fail(FAST_ERR_UNSUPPORTED, "%s: N or E >= 2^31", fn);
  if (!g->dst_offsets) return fail(FAST_ERR_INVALID_ARG, "%s: dst_offsets is NULL", fn);
  if (!violations) return fail(FAST_ERR_INVALID_ARG, "%s: violations is NULL", fn);
  if (g->src_ids && src_bound < 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: src_bound = %lld < 0", fn, (long long)src_bound);
  if (g->edge_ids && edge_bound < 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: edge_bound = %lld < 0", fn, (long long)edge_bound);
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(k_check_zero, dim3(1), dim3(64), 0, st, violations);
  const int64_t work = N > E ? N : E;
  int64_t nb = (work + CK_THREADS - 1) / CK_THREADS;
  if (nb < 1) nb = 1;
  if (nb > CK_MAX_BLOCKS) nb = CK_MAX_BLOCKS;
  hipLaunchKernelGGL(k_check, dim3(uint32_t(nb)), dim3(CK_THREADS), 0, st, g->dst_offsets, N, E,
                     g->src_ids, src_bound, g->edge_ids, edge_bound, g->edge_t, g->dst_t,
                     violations);
  return check_launch(fn);
}
