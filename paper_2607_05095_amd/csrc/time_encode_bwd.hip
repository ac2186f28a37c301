// time_encode_bwd.hip -- backward of the TGAT time features (Sec. 6.1; the
// frequencies and phases of the time encoder are trained with the model):
//   a_ej      = fmaf(omega[j], dt_e, phi[j])            (the forward's argument)
//   dphi[j]   = sum_e dte[e,j] * (-sin a_ej)
//   domega[j] = sum_e dte[e,j] * (-sin a_ej) * dt_e
//
// Each output is a sum over every edge of the block (millions of terms of
// both signs).  An fp32 sine (a few ulp per term) leaves the sum of a column
// that nearly cancels with a relative error far above 1e-5, so the sine is
// evaluated in fp64 on the exact fp32 argument and every product and sum is
// fp64: a two-part Cody-Waite reduction by pi (x = k*pi + r, |r| <= pi/2; pi
// split into its fp64 rounding and the fp64 rounding of the remainder, each
// step one fused multiply-add) and the Taylor series of sin(r)/r in r^2
// through r^14, whose truncation error is below 6e-12 for |r| <= pi/2.
// Arguments beyond 2^30 rad (or not finite) take the library sine in a cold
// second pass of the workgroups that met one.
//
// Determinism: the reduction order depends only on N and d_t.  A workgroup
// owns the segment groups b, b + nblk, b + 2*nblk, ... (TB_SEGS segments
// each, nblk = min(groups, TB_MAX_BLOCKS)); each thread accumulates its
// column chunk over its rows in a fixed order, the row lanes are added in
// lane order through LDS, and a second kernel adds the per-workgroup partials
// in a fixed tree.  Repeated calls give bitwise-identical results.
#include "common.h"

namespace fast {

constexpr int TB_THREADS = 256;
constexpr int TB_SEGS = 32;          // destination segments per group
constexpr int TB_TILE_MAX = 256;     // rows staged per tile
constexpr int TB_MAX_BLOCKS = 2048;  // 8 workgroups per CU
constexpr int TB_MAX_VEC = 8;

__host__ __device__ inline int64_t tb_groups(int64_t N) { return (N + TB_SEGS - 1) / TB_SEGS; }
__host__ __device__ inline int64_t tb_blocks(int64_t N) {
  const int64_t g = tb_groups(N);
  return g < TB_MAX_BLOCKS ? g : TB_MAX_BLOCKS;
}

// sin(x) for an fp32 x with |x| <= 2^30, in fp64, returned as (-1)^k sin r
// where x = k*pi + r: the value is sin(r), and bit 31 of `flip` is set when
// k is odd (sin x = -sin r).  k comes from the magic-number rounding
// fma(x, 1/pi, 1.5*2^52), whose low word holds k in two's complement.  For
// |x| <= 2^30, k <= 2^29: k * PI_HI is exact inside the first fma and
// k * (pi - PI_HI - PI_LO) stays below 1e-24, so r carries an absolute error
// of about 1e-16.
__device__ __forceinline__ double sin_reduced(float xf, uint32_t& flip) {
  const double x = double(xf);
  const double PI_HI = 0x1.921fb54442d18p+1, PI_LO = 0x1.1a62633145c07p-53;
  const double INV_PI = 0x1.45f306dc9c883p-2, MAGIC = 0x1.8p52;
  const double t = fma(x, INV_PI, MAGIC);
  const double k = t - MAGIC;
  flip = uint32_t(__double2loint(t)) << 31;
  double r = fma(-k, PI_HI, x);
  r = fma(-k, PI_LO, r);
  const double r2 = r * r;
  double p = -0x1.ae7f3e733b81fp-41;          // -1/15!
  p = fma(p, r2, 0x1.6124613a86d09p-33);      //  1/13!
  p = fma(p, r2, -0x1.ae64567f544e4p-26);     // -1/11!
  p = fma(p, r2, 0x1.71de3a556c734p-19);      //  1/9!
  p = fma(p, r2, -0x1.a01a01a01a01ap-13);     // -1/7!
  p = fma(p, r2, 0x1.1111111111111p-7);       //  1/5!
  p = fma(p, r2, -0x1.5555555555555p-3);      // -1/3!
  return fma(r * r2, p, r);                   // r + r^3 * (...)
}

// Arguments beyond this (or not finite) are left to the library sine, called
// out of line so that its registers do not weigh on the streaming loop.
__device__ __forceinline__ bool sin_reduced_ok(float x) { return fabsf(x) <= 0x1p30f; }
__device__ __attribute__((noinline)) double sin_library(double x) { return sin(x); }

// Grid: tb_blocks(N) workgroups.  Thread t owns the column chunk t % cpr of
// the rows t / cpr, t / cpr + rpp, ... of every tile, as in the forward.
// partial: [2 * d_t][nblk] fp64 (domega rows first, then dphi).
template <typename TG, int VEC, bool NT>
__global__ void __launch_bounds__(TB_THREADS) k_time_encode_bwd(
    const int32_t* __restrict__ off, int64_t N, int64_t E, const float* __restrict__ dst_t,
    const float* __restrict__ edge_t, const float* __restrict__ omega,
    const float* __restrict__ phi, int d_t, const TG* __restrict__ dte,
    double* __restrict__ partial) {
  __shared__ int64_t s_off[TB_SEGS + 1];
  __shared__ float s_tdst[TB_SEGS];
  __shared__ float s_dt[TB_TILE_MAX];
  __shared__ double s_red[TB_THREADS * VEC * 2];

  const int64_t ngroups = tb_groups(N), nblk = tb_blocks(N);
  const int cpr = d_t / VEC;               // vector chunks per row (<= TB_THREADS)
  const int rpp = TB_THREADS / cpr;        // rows per pass
  const int rsub = int(threadIdx.x) / cpr;
  const int c0 = int(threadIdx.x) - rsub * cpr;
  const bool active = rsub < rpp;
  const int tile = (TB_TILE_MAX / rpp) * rpp;

  float om[VEC], ph[VEC];
  double acc_w[VEC], acc_p[VEC];
  bool big = false;                        // an argument beyond the reduction's range
#pragma unroll
  for (int k = 0; k < VEC; ++k) {
    om[k] = active ? omega[c0 * VEC + k] : 0.f;
    ph[k] = active ? phi[c0 * VEC + k] : 0.f;
    acc_w[k] = 0.0;
    acc_p[k] = 0.0;
  }

  for (int64_t grp = blockIdx.x; grp < ngroups; grp += nblk) {
    const int64_t s0 = grp * TB_SEGS;
    const int ns = int(N - s0 < TB_SEGS ? N - s0 : TB_SEGS);
    if (threadIdx.x <= ns) s_off[threadIdx.x] = clamp64(off[s0 + threadIdx.x], 0, E);
    if (threadIdx.x < ns) s_tdst[threadIdx.x] = dst_t[s0 + threadIdx.x];
    __syncthreads();
    const int64_t r0 = s_off[0], r1 = s_off[ns] > r0 ? s_off[ns] : r0;
    for (int64_t t0 = r0; t0 < r1; t0 += tile) {
      const int nrows = int(r1 - t0 < tile ? r1 - t0 : tile);
      if (threadIdx.x < nrows) {
        const int64_t e = t0 + threadIdx.x;
        int lo = 0, hi = ns - 1;           // last local segment with s_off <= e
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (s_off[mid] <= e) lo = mid; else hi = mid - 1;
        }
        s_dt[threadIdx.x] = s_tdst[lo] - edge_t[e];
      }
      __syncthreads();
      if (active) {
        for (int row = rsub; row < nrows; row += rpp) {
          const float dt = s_dt[row];
          Raw<TG, VEC> raw;
          raw.template load<NT>(dte + (t0 + row) * d_t + c0 * VEC);
          float g[VEC];
          raw.unpack(g);
#pragma unroll
          for (int k = 0; k < VEC; ++k) {
            const float x = fmaf(om[k], dt, ph[k]);
            uint32_t flip;
            const double s = sin_reduced(x, flip);
            const bool ok = sin_reduced_ok(x);
            big |= !ok;
            // -g * sin x, the sign folded into g; 0 for an argument left to
            // the cold pass
            const float gn = ok ? __uint_as_float(__float_as_uint(g[k]) ^ flip ^ 0x80000000u) : 0.f;
            const double gs = double(gn) * s;
            acc_p[k] += gs;
            acc_w[k] = fma(gs, double(dt), acc_w[k]);
          }
        }
      }
      __syncthreads();
    }
  }

  // Cold pass, only in a workgroup that met an argument beyond 2^30 rad (or
  // not finite): the same rows again, adding just those elements with the
  // library sine.  The order stays a fixed function of the inputs.
  if (__syncthreads_or(big)) {
    for (int64_t grp = blockIdx.x; grp < ngroups; grp += nblk) {
      const int64_t s0 = grp * TB_SEGS;
      const int ns = int(N - s0 < TB_SEGS ? N - s0 : TB_SEGS);
      if (threadIdx.x <= ns) s_off[threadIdx.x] = clamp64(off[s0 + threadIdx.x], 0, E);
      if (threadIdx.x < ns) s_tdst[threadIdx.x] = dst_t[s0 + threadIdx.x];
      __syncthreads();
      const int64_t r0 = s_off[0], r1 = s_off[ns] > r0 ? s_off[ns] : r0;
      for (int64_t t0 = r0; t0 < r1; t0 += tile) {
        const int nrows = int(r1 - t0 < tile ? r1 - t0 : tile);
        if (threadIdx.x < nrows) {
          const int64_t e = t0 + threadIdx.x;
          int lo = 0, hi = ns - 1;
          while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_off[mid] <= e) lo = mid; else hi = mid - 1;
          }
          s_dt[threadIdx.x] = s_tdst[lo] - edge_t[e];
        }
        __syncthreads();
        if (active && big) {
          for (int row = rsub; row < nrows; row += rpp) {
            const float dt = s_dt[row];
            Raw<TG, VEC> raw;
            raw.template load<false>(dte + (t0 + row) * d_t + c0 * VEC);
            float g[VEC];
            raw.unpack(g);
            for (int k = 0; k < VEC; ++k) {
              const float x = fmaf(om[k], dt, ph[k]);
              if (!sin_reduced_ok(x)) {
                const double gs = -double(g[k]) * sin_library(double(x));
                acc_p[k] += gs;
                acc_w[k] = fma(gs, double(dt), acc_w[k]);
              }
            }
          }
        }
        __syncthreads();
      }
    }
  }

  // row lanes of one column chunk, added in lane order
  if (active) {
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
      s_red[(rsub * d_t + c0 * VEC + k) * 2 + 0] = acc_w[k];
      s_red[(rsub * d_t + c0 * VEC + k) * 2 + 1] = acc_p[k];
    }
  }
  __syncthreads();
  for (int j = threadIdx.x; j < d_t; j += TB_THREADS) {
    double w = 0.0, p = 0.0;
    for (int r = 0; r < rpp; ++r) {
      w += s_red[(r * d_t + j) * 2 + 0];
      p += s_red[(r * d_t + j) * 2 + 1];
    }
    partial[int64_t(j) * nblk + blockIdx.x] = w;
    partial[int64_t(d_t + j) * nblk + blockIdx.x] = p;
  }
}

// One workgroup per output value: out[j] for j < d_t is domega, then dphi.
// Strided fp64 partial sums per thread, then a fixed LDS tree.
__global__ void __launch_bounds__(TB_THREADS) k_time_encode_bwd_final(
    const double* __restrict__ partial, int64_t nblk, int d_t, float* __restrict__ domega,
    float* __restrict__ dphi) {
  __shared__ double s[TB_THREADS];
  const int row = blockIdx.x;
  double acc = 0.0;
  for (int64_t b = threadIdx.x; b < nblk; b += TB_THREADS) acc += partial[row * nblk + b];
  s[threadIdx.x] = acc;
  __syncthreads();
  for (int w = TB_THREADS / 2; w > 0; w >>= 1) {
    if (int(threadIdx.x) < w) s[threadIdx.x] += s[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    if (row < d_t) domega[row] = float(s[0]);
    else dphi[row - d_t] = float(s[0]);
  }
}

template <typename TG, int VEC>
static void launch_tb(const fast_tcsr_t* g, const float* omega, const float* phi, int d_t,
                      const void* dte, double* partial, hipStream_t st) {
  const int64_t nb = tb_blocks(g->num_dst);
  const bool nt = (size_t(d_t) * sizeof(TG)) % CACHE_LINE == 0 && aligned(dte, CACHE_LINE);
  if (nt)
    hipLaunchKernelGGL((k_time_encode_bwd<TG, VEC, true>), dim3(uint32_t(nb)), dim3(TB_THREADS),
                       0, st, g->dst_offsets, g->num_dst, g->num_edges, g->dst_t, g->edge_t,
                       omega, phi, d_t, static_cast<const TG*>(dte), partial);
  else
    hipLaunchKernelGGL((k_time_encode_bwd<TG, VEC, false>), dim3(uint32_t(nb)), dim3(TB_THREADS),
                       0, st, g->dst_offsets, g->num_dst, g->num_edges, g->dst_t, g->edge_t,
                       omega, phi, d_t, static_cast<const TG*>(dte), partial);
}

// Widest vector of VEC elements that divides d_t, keeps the row's chunks
// within one workgroup and matches the pointer's alignment; 0 if none.
static int pick_vec(int d_t, int esz, const void* p) {
  for (int v = TB_MAX_VEC; v >= 1; v >>= 1) {
    if (v * esz > 16) continue;
    if (d_t % v == 0 && d_t / v <= TB_THREADS && aligned(p, size_t(v) * esz)) return v;
  }
  return 0;
}

}  // namespace fast

using namespace fast;

extern "C" size_t fast_time_encode_bwd_workspace(int64_t num_dst, int d_t) {
  if (num_dst < 0 || d_t <= 0) return 0;
  return align_up(size_t(2) * size_t(d_t) * size_t(tb_blocks(num_dst)) * sizeof(double), 256) + 256;
}

extern "C" fast_status_t fast_time_encode_bwd(const fast_tcsr_t* g, const float* omega,
                                              const float* phi, int d_t, const void* dte,
                                              fast_dtype_t dte_dtype, float* domega, float* dphi,
                                              void* ws, size_t ws_bytes, fast_stream_t stream) {
  const char* fn = "fast_time_encode_bwd";
  if (!g) return fail(FAST_ERR_INVALID_ARG, "%s: graph is NULL", fn);
  if (g->num_dst < 0 || g->num_edges < 0) return fail(FAST_ERR_INVALID_ARG, "%s: negative size", fn);
  if (g->num_edges >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: E >= 2^31", fn);
  if (d_t <= 0) return fail(FAST_ERR_INVALID_ARG, "%s: d_t = %d <= 0", fn, d_t);
  if (dte_dtype != FAST_F32 && dte_dtype != FAST_BF16) return fail(FAST_ERR_INVALID_ARG, "%s: bad dtype", fn);
  if (g->num_dst == 0 && g->num_edges > 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: E > 0 edges but no destination", fn);
  if (!domega || !dphi) return fail(FAST_ERR_INVALID_ARG, "%s: NULL domega/dphi", fn);
  if (!aligned(domega, 4) || !aligned(dphi, 4))
    return fail(FAST_ERR_UNSUPPORTED, "%s: domega/dphi not 4-byte aligned", fn);
  const size_t need = fast_time_encode_bwd_workspace(g->num_dst, d_t);
  if (!ws || ws_bytes < need)
    return fail(FAST_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu", fn, ws_bytes, need);
  if (!aligned(ws, 8)) return fail(FAST_ERR_UNSUPPORTED, "%s: workspace not 8-byte aligned", fn);
  const int esz = elem_size(dte_dtype);
  int vec = 1;
  if (g->num_edges > 0) {
    if (!g->dst_offsets || !g->dst_t || !g->edge_t || !omega || !phi || !dte)
      return fail(FAST_ERR_INVALID_ARG, "%s: NULL dst_offsets/dst_t/edge_t/omega/phi/dte", fn);
    vec = pick_vec(d_t, esz, dte);
    if (vec == 0)
      return fail(FAST_ERR_UNSUPPORTED,
                  "%s: d_t = %d needs more than %d vector chunks per row, or dte is misaligned",
                  fn, d_t, TB_THREADS);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  double* partial = static_cast<double*>(ws);
  int64_t nblk = 0;
  if (g->num_edges > 0) {
    nblk = tb_blocks(g->num_dst);
    if (dte_dtype == FAST_F32) {
      switch (vec) {
        case 4: launch_tb<float, 4>(g, omega, phi, d_t, dte, partial, st); break;
        case 2: launch_tb<float, 2>(g, omega, phi, d_t, dte, partial, st); break;
        default: launch_tb<float, 1>(g, omega, phi, d_t, dte, partial, st); break;
      }
    } else {
      switch (vec) {
        case 8: launch_tb<uint16_t, 8>(g, omega, phi, d_t, dte, partial, st); break;
        case 4: launch_tb<uint16_t, 4>(g, omega, phi, d_t, dte, partial, st); break;
        case 2: launch_tb<uint16_t, 2>(g, omega, phi, d_t, dte, partial, st); break;
        default: launch_tb<uint16_t, 1>(g, omega, phi, d_t, dte, partial, st); break;
      }
    }
  }
  // with no edges every sum is empty: the final pass writes zeros
  hipLaunchKernelGGL(k_time_encode_bwd_final, dim3(uint32_t(2 * d_t)), dim3(TB_THREADS), 0, st,
                     partial, nblk, d_t, domega, dphi);
  return check_launch(fn);
}
