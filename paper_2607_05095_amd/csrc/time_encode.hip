// time_encode.hip -- TGAT time features (Sec. 6.1, random Fourier features):
//   te[e, j] = cos(fmaf(omega[j], dst_t[v] - edge_t[e], phi[j])),  e in segment v.
//
// The op writes E*d_t values from 8 bytes of input per edge, so it is bound by
// HBM writes and by the cosine.  A workgroup owns TE_SEGS consecutive
// destination segments: it loads their offsets and times into LDS with one
// coalesced access, then walks the segments' edges in tiles of rows: each
// row finds its segment by a short binary search in LDS and stages dt in LDS,
// and the [rows, d_t] tile is streamed out with 16-byte stores.
//
// The argument reaches |omega*dt| ~ 1e4 rad, where the hardware cosine
// (argument in revolutions, no range reduction worth the name) would lose
// the 1e-5 target on its own, and the device library's general cosf costs
// most of the op's time.  cos_rr below first reduces exactly: a Cody-Waite
// reduction (W. J. Cody and W. Waite, "Software Manual for the Elementary
// Functions", 1980) x = k*2pi + r with 2pi split into two fp32 parts D1 + D2
// (four times the fp32 roundings of pi/2 and of what remained of it, derived
// exactly from Machin's formula for pi; the third part would change r by
// less than 1e-10 for |x| <= 2^16), each step one fused multiply-add, so
// |r| <= pi carries about 2.5e-7 absolute error.  r/(2 pi), a value within
// half a revolution, goes to v_cos_f32, whose worst-case absolute error
// measured 3e-7 against fp64 below one revolution on MI355X.  Arguments
// beyond 2^16 take the library cosf.
#include "common.h"

namespace fast {

// 8 segments per workgroup (about 80-160 rows at the sampled fan-outs)
// measured fastest inside the training step for both fp32 rows of 100 and
// bf16 rows of 128 (32 segments: 0.202 / 0.276 ms, 8: 0.197 / 0.246 ms for
// the layer-1 blocks of the two large workloads); 1-4 pay the workgroup's
// serial offsets -> times -> stores latency too often.
#ifndef FAST_TE_SEGS
#define FAST_TE_SEGS 8
#endif
#ifndef FAST_TE_PASSES
#define FAST_TE_PASSES 25
#endif
constexpr int TE_THREADS = 256;
constexpr int TE_SEGS = FAST_TE_SEGS;    // destination segments per workgroup
constexpr int TE_TILE_MAX = 256;         // rows staged per tile (at most)
constexpr int TE_PASSES = FAST_TE_PASSES;  // row passes per tile

// Branch-free: valid (within 6e-7 absolute) for |x| <= 2^16, finite beyond.
__device__ __forceinline__ float cos_rr(float x) {
  const float D1 = 0x1.921fb6p+2f, D2 = -0x1.777a5cp-23f;   // 2pi = D1 + D2 + O(2^-47)
  const float INV_TWO_PI = 0x1.45f306p-3f;
  const float k = rintf(x * INV_TWO_PI);
  float r = fmaf(-k, D1, x);
  r = fmaf(-k, D2, r);
  return __builtin_amdgcn_cosf(r * INV_TWO_PI);
}

// Large arguments (|x| > 2^16, or not finite) take the library cosf.
__device__ __forceinline__ bool cos_cw_ok(float x) { return fabsf(x) <= 65536.f; }

// A bf16 row is checked once: every |fmaf(om, dt, ph)| of its columns is at
// most fmaf(max |om|, |dt|, max |ph|) up to one rounding, so a bound of 65000
// keeps them all inside cos_rr's range.
constexpr float TE_ROW_LIMIT = 65000.f;

// Workgroup `wg` of one block: segments [wg TE_SEGS, (wg + 1) TE_SEGS).
// Thread t owns the column chunk t % cpr of rows t / cpr, t / cpr + rpp, ...
// (rpp = rows per pass), so omega and phi of its columns stay in registers.
template <typename TO, int VEC, bool NT>
__device__ __forceinline__ void te_segments(
    int64_t wg, const int32_t* __restrict__ off, int64_t N, int64_t E,
    const float* __restrict__ dst_t, const float* __restrict__ edge_t,
    const float* __restrict__ omega, const float* __restrict__ phi, int d_t,
    TO* __restrict__ te) {
  __shared__ int64_t s_off[TE_SEGS + 1];
  __shared__ float s_tdst[TE_SEGS];
  __shared__ float s_dt[TE_TILE_MAX];
  const int64_t s0 = wg * TE_SEGS;
  const int ns = int(N - s0 < TE_SEGS ? N - s0 : TE_SEGS);
  if (threadIdx.x <= ns) s_off[threadIdx.x] = clamp64(off[s0 + threadIdx.x], 0, E);
  if (threadIdx.x < ns) s_tdst[threadIdx.x] = dst_t[s0 + threadIdx.x];
  __syncthreads();
  const int64_t r0 = s_off[0], r1 = s_off[ns];

  const int cpr = d_t / VEC;                       // vector chunks per row
  const bool narrow = cpr <= TE_THREADS;
  const int rpp = narrow ? TE_THREADS / cpr : 1;   // rows per pass
  const int rsub = narrow ? int(threadIdx.x) / cpr : 0;
  const int c0 = narrow ? int(threadIdx.x) - rsub * cpr : int(threadIdx.x);
  const int tile = rpp * TE_PASSES < TE_TILE_MAX ? rpp * TE_PASSES : (TE_TILE_MAX / rpp) * rpp;
  float om[VEC], ph[VEC], om_max = 0.f, ph_max = 0.f;
  if (narrow && rsub < rpp) {
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
      om[k] = omega[c0 * VEC + k];
      ph[k] = phi[c0 * VEC + k];
      om_max = fmaxf(om_max, fabsf(om[k]));
      ph_max = fmaxf(ph_max, fabsf(ph[k]));
    }
  }
  for (int64_t t0 = r0; t0 < r1; t0 += tile) {
    const int nrows = int(r1 - t0 < tile ? r1 - t0 : tile);
    if (threadIdx.x < nrows) {
      const int64_t e = t0 + threadIdx.x;
      int lo = 0, hi = ns - 1;          // last local segment with s_off <= e
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_off[mid] <= e) lo = mid; else hi = mid - 1;
      }
      s_dt[threadIdx.x] = s_tdst[lo] - edge_t[e];
    }
    __syncthreads();
    if (narrow) {
      if (rsub < rpp) {
        for (int row = rsub; row < nrows; row += rpp) {
          const float dt = s_dt[row];
          float o[VEC];
          if constexpr (sizeof(TO) == 2) {
            // bf16 rows are ALU-bound (twice the elements per byte written):
            // one range check per row.  Not-less-than also sends a NaN bound
            // (a NaN time) to the checked path.
            if (__builtin_expect(!(fmaf(om_max, fabsf(dt), ph_max) <= TE_ROW_LIMIT), 0)) {
#pragma unroll
              for (int k = 0; k < VEC; ++k) {
                const float x = fmaf(om[k], dt, ph[k]);
                o[k] = cos_cw_ok(x) ? cos_rr(x) : cosf(x);
              }
            } else {
#pragma unroll
              for (int k = 0; k < VEC; ++k) o[k] = cos_rr(fmaf(om[k], dt, ph[k]));
            }
          } else {
            // fp32 rows are bound by the stores: a compare per element and a
            // rare fix-up, with no branch in the row loop, measured faster
            float x[VEC];
            bool big = false;
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
              x[k] = fmaf(om[k], dt, ph[k]);
              o[k] = cos_rr(x[k]);
              big |= !cos_cw_ok(x[k]);
            }
            if (__builtin_expect(big, 0)) {
#pragma unroll
              for (int k = 0; k < VEC; ++k)
                if (!cos_cw_ok(x[k])) o[k] = cosf(x[k]);
            }
          }
          StreamIO<TO, VEC, NT>::store(te + (t0 + row) * d_t + c0 * VEC, o);
        }
      }
    } else {                            // very wide rows: stride over the columns
      for (int row = 0; row < nrows; ++row) {
        const float dt = s_dt[row];
        for (int c = c0; c < cpr; c += TE_THREADS) {
          float o[VEC];
#pragma unroll
          for (int k = 0; k < VEC; ++k) {
            const float x = fmaf(omega[c * VEC + k], dt, phi[c * VEC + k]);
            o[k] = cos_cw_ok(x) ? cos_rr(x) : cosf(x);
          }
          StreamIO<TO, VEC, NT>::store(te + (t0 + row) * d_t + c * VEC, o);
        }
      }
    }
    __syncthreads();
  }
}

template <typename TO, int VEC, bool NT>
__global__ void __launch_bounds__(TE_THREADS) k_time_encode(
    const int32_t* __restrict__ off, int64_t N, int64_t E, const float* __restrict__ dst_t,
    const float* __restrict__ edge_t, const float* __restrict__ omega,
    const float* __restrict__ phi, int d_t, TO* __restrict__ te) {
  te_segments<TO, VEC, NT>(blockIdx.x, off, N, E, dst_t, edge_t, omega, phi, d_t, te);
}

// Several blocks (the layer blocks of one batch) in one launch: workgroups
// [w0[b], w0[b+1]) encode block b.
constexpr int TE_MAX_BATCH = 8;
struct TeBatch {
  int nb;
  const int32_t* off[TE_MAX_BATCH];
  int64_t N[TE_MAX_BATCH], E[TE_MAX_BATCH];
  const float* dst_t[TE_MAX_BATCH];
  const float* edge_t[TE_MAX_BATCH];
  void* te[TE_MAX_BATCH];
  int64_t w0[TE_MAX_BATCH + 1];
};

template <typename TO, int VEC, bool NT>
__global__ void __launch_bounds__(TE_THREADS) k_time_encode_batch(TeBatch B,
                                                                  const float* __restrict__ omega,
                                                                  const float* __restrict__ phi,
                                                                  int d_t) {
  const int64_t w = blockIdx.x;
  int b = 0;
#pragma unroll
  for (int k = 1; k < TE_MAX_BATCH; ++k)
    if (k < B.nb && w >= B.w0[k]) b = k;
  te_segments<TO, VEC, NT>(w - B.w0[b], B.off[b], B.N[b], B.E[b], B.dst_t[b], B.edge_t[b], omega,
                           phi, d_t, static_cast<TO*>(B.te[b]));
}

template <typename TO, int VEC>
static void launch_te_batch(const TeBatch& B, const float* omega, const float* phi, int d_t,
                            bool nt, hipStream_t st) {
  const uint32_t grid = uint32_t(B.w0[B.nb]);
  if (nt)
    hipLaunchKernelGGL((k_time_encode_batch<TO, VEC, true>), dim3(grid), dim3(TE_THREADS), 0, st, B,
                       omega, phi, d_t);
  else
    hipLaunchKernelGGL((k_time_encode_batch<TO, VEC, false>), dim3(grid), dim3(TE_THREADS), 0, st, B,
                       omega, phi, d_t);
}

template <typename TO, int VEC>
static void launch_te(const fast_tcsr_t* g, const float* omega, const float* phi, int d_t,
                      void* te, hipStream_t st) {
  const int64_t nb = (g->num_dst + TE_SEGS - 1) / TE_SEGS;
  // streaming stores only when each output row covers whole cache lines
#ifdef FAST_TE_FORCE_NT
  const bool nt = true;
#else
  const bool nt = (size_t(d_t) * sizeof(TO)) % CACHE_LINE == 0 && aligned(te, CACHE_LINE);
#endif
  if (nt)
    hipLaunchKernelGGL((k_time_encode<TO, VEC, true>), dim3(uint32_t(nb)), dim3(TE_THREADS), 0, st,
                       g->dst_offsets, g->num_dst, g->num_edges, g->dst_t, g->edge_t, omega, phi,
                       d_t, static_cast<TO*>(te));
  else
    hipLaunchKernelGGL((k_time_encode<TO, VEC, false>), dim3(uint32_t(nb)), dim3(TE_THREADS), 0, st,
                       g->dst_offsets, g->num_dst, g->num_edges, g->dst_t, g->edge_t, omega, phi,
                       d_t, static_cast<TO*>(te));
}

}  // namespace fast

using namespace fast;

// Argument checks of one block; *work is set when the block has edges.
static fast_status_t te_check(const char* fn, const fast_tcsr_t* g, const float* omega,
                              const float* phi, int d_t, const void* te, fast_dtype_t te_dtype,
                              bool* work) {
  *work = false;
  if (!g) return fail(FAST_ERR_INVALID_ARG, "%s: graph is NULL", fn);
  if (g->num_dst < 0 || g->num_edges < 0) return fail(FAST_ERR_INVALID_ARG, "%s: negative size", fn);
  if (g->num_edges >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: E >= 2^31", fn);
  if (d_t <= 0) return fail(FAST_ERR_INVALID_ARG, "%s: d_t = %d <= 0", fn, d_t);
  if (te_dtype != FAST_F32 && te_dtype != FAST_BF16) return fail(FAST_ERR_INVALID_ARG, "%s: bad dtype", fn);
  if (g->num_dst == 0 && g->num_edges > 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: E > 0 edges but no destination", fn);
  if (g->num_edges == 0) return FAST_OK;
  if (!g->dst_offsets || !g->dst_t || !g->edge_t || !omega || !phi || !te)
    return fail(FAST_ERR_INVALID_ARG, "%s: NULL dst_offsets/dst_t/edge_t/omega/phi/te", fn);
  if (int64_t(d_t) * g->num_edges >= (int64_t(1) << 40))
    return fail(FAST_ERR_UNSUPPORTED, "%s: output too large", fn);
  *work = true;
  return FAST_OK;
}

// Widest vector (elements per thread access) that every output allows, or 0.
static int te_vec(fast_dtype_t te_dtype, int d_t, const void* const* te, int n) {
  auto all = [&](size_t a) {
    for (int k = 0; k < n; ++k)
      if (te[k] && !aligned(te[k], a)) return false;
    return true;
  };
  if (te_dtype == FAST_F32) {
    if (d_t % 4 == 0 && all(16)) return 4;
    if (d_t % 2 == 0 && all(8)) return 2;
    return all(4) ? 1 : 0;
  }
  if (d_t % 8 == 0 && all(16)) return 8;
  if (d_t % 4 == 0 && all(8)) return 4;
  if (d_t % 2 == 0 && all(4)) return 2;
  return all(2) ? 1 : 0;
}

extern "C" fast_status_t fast_time_encode_batched(int nblocks, const fast_tcsr_t* const* g,
                                                  const float* omega, const float* phi, int d_t,
                                                  void* const* te, fast_dtype_t te_dtype,
                                                  fast_stream_t stream) {
  const char* fn = "fast_time_encode_batched";
  if (nblocks < 0) return fail(FAST_ERR_INVALID_ARG, "%s: nblocks = %d < 0", fn, nblocks);
  if (nblocks == 0) return ok();
  if (!g || !te) return fail(FAST_ERR_INVALID_ARG, "%s: NULL host array", fn);
  TeBatch B = {};
  const void* outs[TE_MAX_BATCH];
  hipStream_t st = static_cast<hipStream_t>(stream);
  bool launched = false;
  for (int b0 = 0; b0 < nblocks; b0 += TE_MAX_BATCH) {   // at most TE_MAX_BATCH blocks per launch
    B = {};
    int64_t w = 0;
    for (int b = b0; b < nblocks && b < b0 + TE_MAX_BATCH; ++b) {
      bool work = false;
      const fast_status_t s = te_check(fn, g[b], omega, phi, d_t, te[b], te_dtype, &work);
      if (s != FAST_OK) return s;
      if (!work) continue;
      const int k = B.nb++;
      B.off[k] = g[b]->dst_offsets;
      B.N[k] = g[b]->num_dst;
      B.E[k] = g[b]->num_edges;
      B.dst_t[k] = g[b]->dst_t;
      B.edge_t[k] = g[b]->edge_t;
      B.te[k] = te[b];
      B.w0[k] = w;
      outs[k] = te[b];
      w += (g[b]->num_dst + TE_SEGS - 1) / TE_SEGS;
    }
    if (B.nb == 0) continue;
    B.w0[B.nb] = w;
    const int vec = te_vec(te_dtype, d_t, outs, B.nb);
    if (vec == 0)
      return fail(FAST_ERR_UNSUPPORTED, "%s: te is not %d-byte aligned", fn,
                  te_dtype == FAST_F32 ? 4 : 2);
    // streaming stores only when each output row covers whole cache lines
    const size_t esz = te_dtype == FAST_F32 ? 4 : 2;
    bool nt = (size_t(d_t) * esz) % CACHE_LINE == 0;
    for (int k = 0; k < B.nb; ++k) nt = nt && aligned(B.te[k], CACHE_LINE);
    launched = true;
    if (te_dtype == FAST_F32) {
      if (vec == 4) launch_te_batch<float, 4>(B, omega, phi, d_t, nt, st);
      else if (vec == 2) launch_te_batch<float, 2>(B, omega, phi, d_t, nt, st);
      else launch_te_batch<float, 1>(B, omega, phi, d_t, nt, st);
    } else {
      if (vec == 8) launch_te_batch<uint16_t, 8>(B, omega, phi, d_t, nt, st);
      else if (vec == 4) launch_te_batch<uint16_t, 4>(B, omega, phi, d_t, nt, st);
      else if (vec == 2) launch_te_batch<uint16_t, 2>(B, omega, phi, d_t, nt, st);
      else launch_te_batch<uint16_t, 1>(B, omega, phi, d_t, nt, st);
    }
  }
  return launched ? check_launch(fn) : ok();   // no block with edges: no HIP call
}

extern "C" fast_status_t fast_time_encode(const fast_tcsr_t* g, const float* omega,
                                          const float* phi, int d_t, void* te,
                                          fast_dtype_t te_dtype, fast_stream_t stream) {
  const char* fn = "fast_time_encode";
  bool work = false;
  const fast_status_t s = te_check(fn, g, omega, phi, d_t, te, te_dtype, &work);
  if (s != FAST_OK) return s;
  if (!work) return ok();
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (te_dtype == FAST_F32) {
    if (d_t % 4 == 0 && aligned(te, 16)) launch_te<float, 4>(g, omega, phi, d_t, te, st);
    else if (d_t % 2 == 0 && aligned(te, 8)) launch_te<float, 2>(g, omega, phi, d_t, te, st);
    else if (aligned(te, 4)) launch_te<float, 1>(g, omega, phi, d_t, te, st);
    else return fail(FAST_ERR_UNSUPPORTED, "%s: te is not 4-byte aligned", fn);
  } else {
    if (d_t % 8 == 0 && aligned(te, 16)) launch_te<uint16_t, 8>(g, omega, phi, d_t, te, st);
    else if (d_t % 4 == 0 && aligned(te, 8)) launch_te<uint16_t, 4>(g, omega, phi, d_t, te, st);
    else if (d_t % 2 == 0 && aligned(te, 4)) launch_te<uint16_t, 2>(g, omega, phi, d_t, te, st);
    else if (aligned(te, 2)) launch_te<uint16_t, 1>(g, omega, phi, d_t, te, st);
    else return fail(FAST_ERR_UNSUPPORTED, "%s: te is not 2-byte aligned", fn);
  }
  return check_launch(fn);
}
