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
// fp64: a one-step Cody-Waite reduction by pi (x = k*pi + r, |r| <= pi/2,
// one fused multiply-add with the fp64 rounding of pi) and an odd polynomial
// of degree 11 for sin(r), whose coefficients were fitted near-minimax
// (Lawson's iteratively reweighted least squares on Chebyshev nodes of
// [0, (pi/2)^2] in r^2, on the relative error of sin): its relative error is
// below 2.4e-11 on |r| <= pi/2, and the one-step reduction adds at most
// 4e-11 absolute for |x| <= 1e6.  Terms of a cancelling column need about
// 1e-8 (the 1e-5 target on a sum 1e-3 of the sum of its magnitudes).
// The range is checked once per row: a row whose bound
// fmaf(max|omega|, |dt|, max|phi|) exceeds 1e6 (or is not finite) is left
// to the library sine in a cold second pass of the workgroups that met one.
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

// sin(x) in fp64 for an fp32 x with |x| <= 1e6.  k = round(x / pi) comes
// from the magic-number rounding fma(x, 1/pi, 1.5*2^52), whose low word
// holds k in two's complement; r = x - k*pi in one fused multiply-add
// (k <= 3.2e5, so the neglected k*(pi - PI_HI) stays below 4e-11), and the
// parity of k flips the sign of r, since sin x = (-1)^k sin r = sin((-1)^k r).
__device__ __forceinline__ double sin_reduced(float xf) {
  const double x = double(xf);
  const double PI_HI = 0x1.921fb54442d18p+1;
  const double INV_PI = 0x1.45f306dc9c883p-2, MAGIC = 0x1.8p52;
  const double t = fma(x, INV_PI, MAGIC);
  const double k = t - MAGIC;
  double r = fma(-k, PI_HI, x);
  const uint32_t flip = uint32_t(__double2loint(t)) << 31;
  r = __hiloint2double(int(uint32_t(__double2hiint(r)) ^ flip), __double2loint(r));
  const double r2 = r * r;
  double p = -0x1.9a6887b9bb2dbp-26;
  p = fma(p, r2, 0x1.71708023de99ap-19);
  p = fma(p, r2, -0x1.a017d9a03cff9p-13);
  p = fma(p, r2, 0x1.11110c4a00de9p-7);
  p = fma(p, r2, -0x1.555555476965fp-3);
  return fma(r * r2, p, r);                   // r + r^3 p(r^2)
}

// A row is reduced in-line when every |fmaf(omega[j], dt, phi[j])| of its
// columns is at most 1e6 * (1 + 2^-22) < 2^20: fmaf(max|omega|, |dt|,
// max|phi|) bounds them up to two roundings.  Not-less-than sends a NaN
// bound (a NaN time) to the library path too.
constexpr float TB_ROW_LIMIT = 1.0e6f;
__device__ __forceinline__ bool tb_row_ok(float om_max, float ph_max, float dt) {
  return fmaf(om_max, fabsf(dt), ph_max) <= TB_ROW_LIMIT;
}
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

  float om[VEC], ph[VEC], om_max = 0.f, ph_max = 0.f;
  double acc_w[VEC], acc_p[VEC];
  bool big = false;                        // a row beyond the reduction's range
#pragma unroll
  for (int k = 0; k < VEC; ++k) {
    om[k] = active ? omega[c0 * VEC + k] : 0.f;
    ph[k] = active ? phi[c0 * VEC + k] : 0.f;
    om_max = fmaxf(om_max, fabsf(om[k]));
    ph_max = fmaxf(ph_max, fabsf(ph[k]));
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
          if (__builtin_expect(!tb_row_ok(om_max, ph_max, dt), 0)) {
            big = true;                    // left to the cold pass
            continue;
          }
          Raw<TG, VEC> raw;
          raw.template load<NT>(dte + (t0 + row) * d_t + c0 * VEC);
          float g[VEC];
          raw.unpack(g);
          const double dtd = double(dt);
#pragma unroll
          for (int k = 0; k < VEC; ++k) {
            // the term is -g sin x
            const double q = double(g[k]) * sin_reduced(fmaf(om[k], dt, ph[k]));
            acc_p[k] -= q;
            acc_w[k] = fma(-q, dtd, acc_w[k]);
          }
        }
      }
      __syncthreads();
    }
  }

  // Cold pass, only in a workgroup that met a row beyond the reduction's
  // range (or not finite): the same rows again, adding just those rows with
  // the library sine.  The order stays a fixed function of the inputs.
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
            if (tb_row_ok(om_max, ph_max, dt)) continue;
            Raw<TG, VEC> raw;
            raw.template load<false>(dte + (t0 + row) * d_t + c0 * VEC);
            float g[VEC];
            raw.unpack(g);
            for (int k = 0; k < VEC; ++k) {
              const float x = fmaf(om[k], dt, ph[k]);
              const double gs = -double(g[k]) * sin_library(double(x));
              acc_p[k] += gs;
              acc_w[k] = fma(gs, double(dt), acc_w[k]);
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
