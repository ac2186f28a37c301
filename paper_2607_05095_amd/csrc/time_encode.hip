// time_encode.hip -- TGAT time features (Sec. 6.1, random Fourier features):
//   te[e, j] = cos(fmaf(omega[j], dst_t[v] - edge_t[e], phi[j])),  e in segment v.
//
// The op writes E*d_t values from 8 bytes of input per edge, so it is bound by
// HBM writes and by the cosine.  A workgroup owns TE_ROWS consecutive edges:
// it locates their segments with two binary searches over the offsets (one
// per block end) and a short search per row inside that range, stages the
// per-edge dt in LDS, and then streams the [TE_ROWS, d_t] tile out with
// 16-byte stores.  The cosine is the accurate device-library cosf (its
// argument reaches |omega*dt| ~ 1e4 rad, where a hardware sine without a
// full range reduction would lose the 1e-5 target).
#include "common.h"

namespace fast {

constexpr int TE_THREADS = 256;
constexpr int TE_ROWS = 64;

// Largest s in [lo, hi] with off[s] <= e (the segment holding edge e).
__device__ __forceinline__ int64_t seg_of(const int32_t* __restrict__ off, int64_t e,
                                          int64_t lo, int64_t hi) {
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (int64_t(off[mid]) <= e) lo = mid; else hi = mid - 1;
  }
  return lo;
}

template <typename TO, int VEC>
__global__ void __launch_bounds__(TE_THREADS) k_time_encode(
    const int32_t* __restrict__ off, int64_t N, int64_t E, const float* __restrict__ dst_t,
    const float* __restrict__ edge_t, const float* __restrict__ omega,
    const float* __restrict__ phi, int d_t, TO* __restrict__ te) {
  __shared__ float s_dt[TE_ROWS];
  __shared__ int64_t s_rng[2];
  const int64_t r0 = int64_t(blockIdx.x) * TE_ROWS;
  const int nrows = int(E - r0 < TE_ROWS ? E - r0 : TE_ROWS);
  if (threadIdx.x < 2) {
    const int64_t e = r0 + (threadIdx.x == 0 ? 0 : nrows - 1);
    s_rng[threadIdx.x] = seg_of(off, e, 0, N - 1);
  }
  __syncthreads();
  if (threadIdx.x < nrows) {
    const int64_t e = r0 + threadIdx.x;
    const int64_t s = seg_of(off, e, s_rng[0], s_rng[1] < s_rng[0] ? s_rng[0] : s_rng[1]);
    s_dt[threadIdx.x] = dst_t[s] - edge_t[e];
  }
  __syncthreads();
  const int cpr = d_t / VEC;
  const int total = nrows * cpr;
  for (int idx = threadIdx.x; idx < total; idx += TE_THREADS) {
    const int row = idx / cpr;
    const int c = idx - row * cpr;
    const float dt = s_dt[row];
    float o[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
      const int j = c * VEC + k;
      o[k] = cosf(fmaf(omega[j], dt, phi[j]));
    }
    VecIO<TO, VEC>::store(te + (r0 + row) * d_t + c * VEC, o);
  }
}

template <typename TO, int VEC>
static void launch_te(const fast_tcsr_t* g, const float* omega, const float* phi, int d_t,
                      void* te, hipStream_t st) {
  const int64_t nb = (g->num_edges + TE_ROWS - 1) / TE_ROWS;
  hipLaunchKernelGGL((k_time_encode<TO, VEC>), dim3(uint32_t(nb)), dim3(TE_THREADS), 0, st,
                     g->dst_offsets, g->num_dst, g->num_edges, g->dst_t, g->edge_t, omega, phi,
                     d_t, static_cast<TO*>(te));
}

}  // namespace fast

using namespace fast;

extern "C" fast_status_t fast_time_encode(const fast_tcsr_t* g, const float* omega,
                                          const float* phi, int d_t, void* te,
                                          fast_dtype_t te_dtype, fast_stream_t stream) {
  const char* fn = "fast_time_encode";
  if (!g) return fail(FAST_ERR_INVALID_ARG, "%s: graph is NULL", fn);
  if (g->num_dst < 0 || g->num_edges < 0) return fail(FAST_ERR_INVALID_ARG, "%s: negative size", fn);
  if (g->num_edges >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: E >= 2^31", fn);
  if (d_t <= 0) return fail(FAST_ERR_INVALID_ARG, "%s: d_t = %d <= 0", fn, d_t);
  if (te_dtype != FAST_F32 && te_dtype != FAST_BF16) return fail(FAST_ERR_INVALID_ARG, "%s: bad dtype", fn);
  if (g->num_dst == 0 && g->num_edges > 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: E > 0 edges but no destination", fn);
  if (g->num_edges == 0) return ok();
  if (!g->dst_offsets || !g->dst_t || !g->edge_t || !omega || !phi || !te)
    return fail(FAST_ERR_INVALID_ARG, "%s: NULL dst_offsets/dst_t/edge_t/omega/phi/te", fn);
  if (int64_t(d_t) * g->num_edges >= (int64_t(1) << 40))
    return fail(FAST_ERR_UNSUPPORTED, "%s: output too large", fn);
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
