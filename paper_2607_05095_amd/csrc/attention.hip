// attention.hip -- edge softmax (ESM) with per-edge multi-head logits and
// attention-weighted aggregation (AGG), forward and backward, separately and
// fused (Sec. 4.3; Eq. 1 with an attention-weighted sum as AGG).
//
// Mapping (MI355X, wave64, no MFMA: every op here is a gather/reduce whose
// arithmetic intensity is ~0.5 flop/byte, far below the vector-ALU ridge):
//   * One sub-wavefront of G = H * LPH lanes owns one destination segment
//     and walks its edges in CSR order.  Each head is a group of LPH lanes
//     (a power of two); lane l of a head holds feature chunks l, l+LPH, ...
//     of VE elements, VE*bytes <= 16, so one row of a segment is read with
//     one coalesced vector load per lane.
//   * Per-edge, per-head dot products (the logits, and in backward the
//     <dOut, V> terms) are all-reduced inside the head group with DPP row
//     operations and the gfx950 permlane swaps; no LDS, no atomics.
//   * Softmax is computed online over chunks of CH edges (one rescale per
//     chunk), so any degree works; the segment's edges are streamed once.
//   * Every destination row is produced by exactly one sub-wavefront: the
//     results are deterministic run to run (unlike the paper's edge-parallel
//     atomicAdd aggregation, which is prior art for a different GPU).
//   * Backward needs one pass over K and V: with w = exp(s - m),
//       dQ = scale/Z * (sum w c dalpha K - D * sum w c K),  D = sum w dalpha / Z
//     is accumulated while streaming, and dK, dV of the first NSAVE*CH edges
//     are written from per-edge scalars kept in registers (longer segments
//     re-read K and V for the remainder).
#include "common.h"

namespace fast {

constexpr int ATT_BLOCK = 256;
constexpr int ATT_CH = 8;      // edges per online-softmax chunk
constexpr int ATT_NSAVE = 3;   // chunks whose per-edge scalars stay in registers (bwd)

struct AttnLayout {
  int H, dh, F;   // heads, head dim, F = H*dh
  int VE;         // elements per vector access
  int CPH;        // vector chunks per head = dh / VE
  int LPH;        // lanes per head (power of two)
  int G;          // lanes per segment = H * LPH
  int SPB;        // segments per workgroup
  int block;      // workgroup size
};

struct AttnArgs {
  AttnLayout L;
  int64_t N, E;
  const int32_t* off;
  float scale, slope;
  const void* Q;
  const void* K;
  const void* V;
  const void* dO;
  const float* alpha_in;
  const float* dalpha_in;
  const float* lse_in;
  void* out;
  float* lse_out;
  void* dQ;
  void* dK;
  void* dV;
  float* alpha_out;
  float* dalpha_out;
};

template <int P>
struct LaneMap {
  int64_t seg;
  int h, l;
  int foff[P];    // element offset of chunk p inside a row
  bool cok[P];    // chunk p exists (padding lanes of a head hold zeros)
};

template <int VE, int P>
__device__ __forceinline__ bool lane_setup(const AttnArgs& a, LaneMap<P>& m) {
  const int t = threadIdx.x;
  const int sub = t / a.L.G;
  const int r = t - sub * a.L.G;
  m.h = r / a.L.LPH;
  m.l = r - m.h * a.L.LPH;
  m.seg = int64_t(xcd_tile(blockIdx.x, gridDim.x)) * a.L.SPB + sub;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const int c = m.l + p * a.L.LPH;
    m.cok[p] = c < a.L.CPH;
    m.foff[p] = m.h * a.L.dh + (m.cok[p] ? c : 0) * VE;
  }
  return sub < a.L.SPB && m.seg < a.N;
}

template <typename T, int VE, int P>
__device__ __forceinline__ void load_row(const T* __restrict__ base, int64_t row, int F,
                                         const LaneMap<P>& m, float (&x)[P][VE]) {
#pragma unroll
  for (int p = 0; p < P; ++p) {
    if (m.cok[p]) {
      VecIO<T, VE>::load(base + row * F + m.foff[p], x[p]);
    } else {
#pragma unroll
      for (int j = 0; j < VE; ++j) x[p][j] = 0.f;
    }
  }
}

template <typename T, int VE, int P>
__device__ __forceinline__ void store_row(T* __restrict__ base, int64_t row, int F,
                                          const LaneMap<P>& m, const float (&x)[P][VE]) {
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (m.cok[p]) VecIO<T, VE>::store(base + row * F + m.foff[p], x[p]);
}

template <int VE, int P>
__device__ __forceinline__ float head_dot(const float (&a)[P][VE], const float (&b)[P][VE], int lph) {
  float d = 0.f;
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) d = fmaf(a[p][j], b[p][j], d);
  return group_sum(d, lph);
}

__device__ __forceinline__ float lrelu(float pre, float slope) { return pre > 0.f ? pre : slope * pre; }
__device__ __forceinline__ float lrelu_grad(float pre, float slope) { return pre > 0.f ? 1.f : slope; }

__device__ __forceinline__ void seg_range(const AttnArgs& a, int64_t seg, int64_t& e0, int64_t& e1) {
  e0 = clamp64(a.off[seg], 0, a.E);
  e1 = clamp64(a.off[seg + 1], e0, a.E);
}

// ============================================================ fused forward
template <typename T, int VE, int P>
__global__ void __launch_bounds__(ATT_BLOCK) k_attn_fwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P>(a, m)) return;
  const int F = a.L.F, LPH = a.L.LPH;
  const T* Q = static_cast<const T*>(a.Q);
  const T* K = static_cast<const T*>(a.K);
  const T* V = static_cast<const T*>(a.V);
  float q[P][VE];
  load_row<T, VE, P>(Q, m.seg, F, m, q);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);

  float mx = -INFINITY, Z = 0.f, acc[P][VE];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) acc[p][j] = 0.f;

  for (int64_t base = e0; base < e1; base += ATT_CH) {
    float kx[ATT_CH][P][VE], vx[ATT_CH][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) {
      const int64_t e = (base + i < e1) ? base + i : e1 - 1;
      load_row<T, VE, P>(K, e, F, m, kx[i]);
      load_row<T, VE, P>(V, e, F, m, vx[i]);
    }
    float s[ATT_CH];
    float cm = -INFINITY;
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) {
      const float pre = head_dot<VE, P>(q, kx[i], LPH) * a.scale;
      s[i] = (base + i < e1) ? lrelu(pre, a.slope) : -INFINITY;
      cm = fmaxf(cm, s[i]);
    }
    const float mn = fmaxf(mx, cm);
    const float corr = expf(mx - mn);
    Z *= corr;
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int j = 0; j < VE; ++j) acc[p][j] *= corr;
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) {
      const float w = expf(s[i] - mn);
      Z += w;
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int j = 0; j < VE; ++j) acc[p][j] = fmaf(w, vx[i][p][j], acc[p][j]);
    }
    mx = mn;
  }
  const float inv = Z > 0.f ? 1.f / Z : 0.f;
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) acc[p][j] *= inv;
  store_row<T, VE, P>(static_cast<T*>(a.out), m.seg, F, m, acc);
  if (a.lse_out && m.l == 0)
    a.lse_out[m.seg * a.L.H + m.h] = Z > 0.f ? mx + logf(Z) : -INFINITY;
}

// ============================================================ fused backward
template <typename T, int VE, int P>
struct BwdState {
  float q[P][VE], go[P][VE];
  float A[P][VE], B[P][VE];   // sum w c dalpha K, sum w c K
  float mx, Z, Dn;            // running max (or lse), sum w, sum w dalpha
};

// Processes edges [base, base+CH) ∩ [.., e1): loads K, V, forms pre and
// dalpha, and folds them into the running sums.  Returns the per-edge pre
// and dalpha (invalid slots are don't-care).
template <typename T, int VE, int P>
__device__ __forceinline__ void bwd_chunk(const AttnArgs& a, const LaneMap<P>& m, int64_t base,
                                          int64_t e1, bool has_lse, BwdState<T, VE, P>& S,
                                          float (&pre)[ATT_CH], float (&da)[ATT_CH]) {
  const int F = a.L.F, LPH = a.L.LPH;
  const T* K = static_cast<const T*>(a.K);
  const T* V = static_cast<const T*>(a.V);
  float kx[ATT_CH][P][VE], vx[ATT_CH][P][VE];
#pragma unroll
  for (int i = 0; i < ATT_CH; ++i) {
    const int64_t e = (base + i < e1) ? base + i : e1 - 1;
    load_row<T, VE, P>(K, e, F, m, kx[i]);
    load_row<T, VE, P>(V, e, F, m, vx[i]);
  }
  float s[ATT_CH];
  float cm = -INFINITY;
#pragma unroll
  for (int i = 0; i < ATT_CH; ++i) {
    pre[i] = head_dot<VE, P>(S.q, kx[i], LPH) * a.scale;
    da[i] = head_dot<VE, P>(S.go, vx[i], LPH);
    s[i] = (base + i < e1) ? lrelu(pre[i], a.slope) : -INFINITY;
    cm = fmaxf(cm, s[i]);
  }
  if (!has_lse) {
    const float mn = fmaxf(S.mx, cm);
    const float corr = expf(S.mx - mn);
    S.Z *= corr;
    S.Dn *= corr;
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int j = 0; j < VE; ++j) {
        S.A[p][j] *= corr;
        S.B[p][j] *= corr;
      }
    S.mx = mn;
  }
#pragma unroll
  for (int i = 0; i < ATT_CH; ++i) {
    const float w = expf(s[i] - S.mx);
    const float wc = w * lrelu_grad(pre[i], a.slope);
    const float wcd = wc * da[i];
    S.Z += w;
    S.Dn = fmaf(w, da[i], S.Dn);
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int j = 0; j < VE; ++j) {
        S.A[p][j] = fmaf(wcd, kx[i][p][j], S.A[p][j]);
        S.B[p][j] = fmaf(wc, kx[i][p][j], S.B[p][j]);
      }
  }
}

template <typename T, int VE, int P>
__device__ __forceinline__ void bwd_emit(const AttnArgs& a, const LaneMap<P>& m, int64_t e,
                                         float pre, float da, float mx, float invZ, float D,
                                         const BwdState<T, VE, P>& S) {
  const float al = expf(lrelu(pre, a.slope) - mx) * invZ;
  const float g = al * (da - D) * lrelu_grad(pre, a.slope) * a.scale;
  float dk[P][VE], dv[P][VE];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) {
      dk[p][j] = g * S.q[p][j];
      dv[p][j] = al * S.go[p][j];
    }
  store_row<T, VE, P>(static_cast<T*>(a.dK), e, a.L.F, m, dk);
  store_row<T, VE, P>(static_cast<T*>(a.dV), e, a.L.F, m, dv);
}

template <typename T, int VE, int P>
__global__ void __launch_bounds__(ATT_BLOCK) k_attn_bwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P>(a, m)) return;
  const int F = a.L.F;
  BwdState<T, VE, P> S;
  load_row<T, VE, P>(static_cast<const T*>(a.Q), m.seg, F, m, S.q);
  load_row<T, VE, P>(static_cast<const T*>(a.dO), m.seg, F, m, S.go);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  const bool has_lse = a.lse_in != nullptr;
  S.mx = has_lse ? a.lse_in[m.seg * a.L.H + m.h] : -INFINITY;
  if (has_lse && !(S.mx > -INFINITY)) S.mx = 0.f;   // empty segment: no edges use it
  S.Z = 0.f;
  S.Dn = 0.f;
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) S.A[p][j] = S.B[p][j] = 0.f;

  // pass 1: stream K and V once
  float spre[ATT_NSAVE][ATT_CH], sda[ATT_NSAVE][ATT_CH];
#pragma unroll
  for (int c = 0; c < ATT_NSAVE; ++c) {
    const int64_t base = e0 + c * ATT_CH;
    if (base < e1) bwd_chunk<T, VE, P>(a, m, base, e1, has_lse, S, spre[c], sda[c]);
  }
  for (int64_t base = e0 + ATT_NSAVE * ATT_CH; base < e1; base += ATT_CH) {
    float tp[ATT_CH], td[ATT_CH];
    bwd_chunk<T, VE, P>(a, m, base, e1, has_lse, S, tp, td);
  }

  // dQ
  const float invZ = has_lse ? 1.f : (S.Z > 0.f ? 1.f / S.Z : 0.f);
  const float D = S.Dn * invZ;
  float dq[P][VE];
  const float f = invZ * a.scale;
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) dq[p][j] = (S.A[p][j] - D * S.B[p][j]) * f;
  store_row<T, VE, P>(static_cast<T*>(a.dQ), m.seg, F, m, dq);

  // pass 2: dK, dV from the saved scalars
#pragma unroll
  for (int c = 0; c < ATT_NSAVE; ++c) {
    const int64_t base = e0 + c * ATT_CH;
    if (base < e1) {
#pragma unroll
      for (int i = 0; i < ATT_CH; ++i)
        if (base + i < e1) bwd_emit<T, VE, P>(a, m, base + i, spre[c][i], sda[c][i], S.mx, invZ, D, S);
    }
  }
  // long segments: re-read K and V for the edges past the register window
  for (int64_t base = e0 + ATT_NSAVE * ATT_CH; base < e1; base += ATT_CH) {
    const int LPH = a.L.LPH;
    const T* K = static_cast<const T*>(a.K);
    const T* V = static_cast<const T*>(a.V);
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) {
      const int64_t e = (base + i < e1) ? base + i : e1 - 1;
      float kx[P][VE], vx[P][VE];
      load_row<T, VE, P>(K, e, F, m, kx);
      load_row<T, VE, P>(V, e, F, m, vx);
      const float pre = head_dot<VE, P>(S.q, kx, LPH) * a.scale;
      const float da = head_dot<VE, P>(S.go, vx, LPH);
      if (base + i < e1) bwd_emit<T, VE, P>(a, m, e, pre, da, S.mx, invZ, D, S);
    }
  }
}

// ============================================================ edge softmax fwd
template <typename T, int VE, int P>
__global__ void __launch_bounds__(ATT_BLOCK) k_softmax_fwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P>(a, m)) return;
  const int F = a.L.F, LPH = a.L.LPH, H = a.L.H;
  const T* K = static_cast<const T*>(a.K);
  float q[P][VE];
  load_row<T, VE, P>(static_cast<const T*>(a.Q), m.seg, F, m, q);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  float mx = -INFINITY, Z = 0.f;
  // pass 1: running max and normaliser
  for (int64_t base = e0; base < e1; base += ATT_CH) {
    float kx[ATT_CH][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i)
      load_row<T, VE, P>(K, (base + i < e1) ? base + i : e1 - 1, F, m, kx[i]);
    float s[ATT_CH], cm = -INFINITY;
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) {
      s[i] = (base + i < e1) ? lrelu(head_dot<VE, P>(q, kx[i], LPH) * a.scale, a.slope) : -INFINITY;
      cm = fmaxf(cm, s[i]);
    }
    const float mn = fmaxf(mx, cm);
    Z *= expf(mx - mn);
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) Z += expf(s[i] - mn);
    mx = mn;
  }
  const float invZ = Z > 0.f ? 1.f / Z : 0.f;
  if (a.lse_out && m.l == 0) a.lse_out[m.seg * H + m.h] = Z > 0.f ? mx + logf(Z) : -INFINITY;
  // pass 2: alpha (the segment's K rows are re-read, normally from L2)
  for (int64_t base = e0; base < e1; base += ATT_CH) {
    float kx[ATT_CH][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i)
      load_row<T, VE, P>(K, (base + i < e1) ? base + i : e1 - 1, F, m, kx[i]);
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) {
      const float s = lrelu(head_dot<VE, P>(q, kx[i], LPH) * a.scale, a.slope);
      if (base + i < e1 && m.l == 0) a.alpha_out[(base + i) * H + m.h] = expf(s - mx) * invZ;
    }
  }
}

// ============================================================ edge softmax bwd
template <typename T, int VE, int P>
__global__ void __launch_bounds__(ATT_BLOCK) k_softmax_bwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P>(a, m)) return;
  const int F = a.L.F, LPH = a.L.LPH, H = a.L.H;
  const T* K = static_cast<const T*>(a.K);
  float q[P][VE];
  load_row<T, VE, P>(static_cast<const T*>(a.Q), m.seg, F, m, q);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  float D = 0.f;
  for (int64_t e = e0; e < e1; ++e) D = fmaf(a.alpha_in[e * H + m.h], a.dalpha_in[e * H + m.h], D);
  float dq[P][VE];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) dq[p][j] = 0.f;
  for (int64_t base = e0; base < e1; base += ATT_CH) {
    float kx[ATT_CH][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i)
      load_row<T, VE, P>(K, (base + i < e1) ? base + i : e1 - 1, F, m, kx[i]);
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) {
      const int64_t e = (base + i < e1) ? base + i : e1 - 1;
      const float pre = head_dot<VE, P>(q, kx[i], LPH) * a.scale;
      const float al = a.alpha_in[e * H + m.h], da = a.dalpha_in[e * H + m.h];
      const float g = (base + i < e1) ? al * (da - D) * lrelu_grad(pre, a.slope) * a.scale : 0.f;
      float dk[P][VE];
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int j = 0; j < VE; ++j) {
          dq[p][j] = fmaf(g, kx[i][p][j], dq[p][j]);
          dk[p][j] = g * q[p][j];
        }
      if (base + i < e1) store_row<T, VE, P>(static_cast<T*>(a.dK), e, F, m, dk);
    }
  }
  store_row<T, VE, P>(static_cast<T*>(a.dQ), m.seg, F, m, dq);
}

// ============================================================ aggregation fwd
template <typename T, int VE, int P>
__global__ void __launch_bounds__(ATT_BLOCK) k_agg_fwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P>(a, m)) return;
  const int F = a.L.F, H = a.L.H;
  const T* V = static_cast<const T*>(a.V);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  float acc[P][VE];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) acc[p][j] = 0.f;
  for (int64_t base = e0; base < e1; base += ATT_CH) {
    float vx[ATT_CH][P][VE], al[ATT_CH];
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) {
      const int64_t e = (base + i < e1) ? base + i : e1 - 1;
      load_row<T, VE, P>(V, e, F, m, vx[i]);
      al[i] = (base + i < e1) ? a.alpha_in[e * H + m.h] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i)
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int j = 0; j < VE; ++j) acc[p][j] = fmaf(al[i], vx[i][p][j], acc[p][j]);
  }
  store_row<T, VE, P>(static_cast<T*>(a.out), m.seg, F, m, acc);
}

// ============================================================ aggregation bwd
template <typename T, int VE, int P>
__global__ void __launch_bounds__(ATT_BLOCK) k_agg_bwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P>(a, m)) return;
  const int F = a.L.F, LPH = a.L.LPH, H = a.L.H;
  const T* V = static_cast<const T*>(a.V);
  float go[P][VE];
  load_row<T, VE, P>(static_cast<const T*>(a.dO), m.seg, F, m, go);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  for (int64_t base = e0; base < e1; base += ATT_CH) {
    float vx[ATT_CH][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i)
      load_row<T, VE, P>(V, (base + i < e1) ? base + i : e1 - 1, F, m, vx[i]);
#pragma unroll
    for (int i = 0; i < ATT_CH; ++i) {
      const int64_t e = (base + i < e1) ? base + i : e1 - 1;
      const float da = head_dot<VE, P>(go, vx[i], LPH);
      const float al = a.alpha_in[e * H + m.h];
      float dv[P][VE];
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int j = 0; j < VE; ++j) dv[p][j] = al * go[p][j];
      if (base + i < e1) {
        if (m.l == 0) a.dalpha_out[e * H + m.h] = da;
        store_row<T, VE, P>(static_cast<T*>(a.dV), e, F, m, dv);
      }
    }
  }
}

// ============================================================ host side
enum class Op { kAttnFwd, kAttnBwd, kSoftmaxFwd, kSoftmaxBwd, kAggFwd, kAggBwd };

static int next_pow2(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Picks the vector width and lane mapping for (H, dh, dtype) given every row
// pointer the op touches (all must be aligned to the vector access).
static fast_status_t make_layout(const char* fn, int H, int dh, fast_dtype_t dt,
                                 const void* const* rows, int nrows, AttnLayout& L, int& P) {
  if (H < 1 || dh < 1) return fail(FAST_ERR_INVALID_ARG, "%s: H = %d, dh = %d", fn, H, dh);
  if (int64_t(H) * dh > 4096) return fail(FAST_ERR_UNSUPPORTED, "%s: H*dh > 4096", fn);
  const int esz = elem_size(dt);
  const int cands_f32[] = {4, 2, 1};
  const int cands_bf16[] = {8, 4, 2, 1};
  const int* cands = dt == FAST_BF16 ? cands_bf16 : cands_f32;
  const int nc = dt == FAST_BF16 ? 4 : 3;
  int VE = 1;
  for (int i = 0; i < nc; ++i) {
    const int ve = cands[i];
    if (dh % ve) continue;
    bool al = true;
    for (int k = 0; k < nrows; ++k)
      if (rows[k] && !aligned(rows[k], size_t(ve) * esz)) al = false;
    if (!al) continue;
    if (ve > 1 && dh / ve > 64) continue;
    VE = ve;
    break;
  }
  for (int k = 0; k < nrows; ++k)
    if (rows[k] && !aligned(rows[k], size_t(esz)))
      return fail(FAST_ERR_UNSUPPORTED, "%s: operand %d is not %d-byte aligned", fn, k, esz);
  const int CPH = dh / VE;
  int LPH;
  if (CPH <= 64) {
    LPH = next_pow2(CPH);
    P = 1;
  } else {
    LPH = 64;
    P = (CPH + 63) / 64;
    if (P > 4) return fail(FAST_ERR_UNSUPPORTED, "%s: dh = %d too large for this dtype", fn, dh);
    if (P == 3) P = 4;
  }
  const int G = H * LPH;
  if (G > 1024) return fail(FAST_ERR_UNSUPPORTED, "%s: H * lanes-per-head = %d > 1024", fn, G);
  L.H = H;
  L.dh = dh;
  L.F = H * dh;
  L.VE = VE;
  L.CPH = CPH;
  L.LPH = LPH;
  L.G = G;
  if (G <= ATT_BLOCK) {
    L.block = ATT_BLOCK;
    L.SPB = ATT_BLOCK / G;
  } else {
    L.block = (G + 63) / 64 * 64;
    L.SPB = 1;
  }
  return FAST_OK;
}

template <typename T, int VE, int P>
static void launch_op(Op op, const AttnArgs& a, dim3 grid, dim3 block, hipStream_t st) {
  switch (op) {
    case Op::kAttnFwd: hipLaunchKernelGGL((k_attn_fwd<T, VE, P>), grid, block, 0, st, a); break;
    case Op::kAttnBwd: hipLaunchKernelGGL((k_attn_bwd<T, VE, P>), grid, block, 0, st, a); break;
    case Op::kSoftmaxFwd: hipLaunchKernelGGL((k_softmax_fwd<T, VE, P>), grid, block, 0, st, a); break;
    case Op::kSoftmaxBwd: hipLaunchKernelGGL((k_softmax_bwd<T, VE, P>), grid, block, 0, st, a); break;
    case Op::kAggFwd: hipLaunchKernelGGL((k_agg_fwd<T, VE, P>), grid, block, 0, st, a); break;
    case Op::kAggBwd: hipLaunchKernelGGL((k_agg_bwd<T, VE, P>), grid, block, 0, st, a); break;
  }
}

template <typename T>
static bool dispatch_t(Op op, const AttnArgs& a, int P, dim3 grid, dim3 block, hipStream_t st) {
  const int VE = a.L.VE;
  if (P == 1) {
    if (VE == 1) launch_op<T, 1, 1>(op, a, grid, block, st);
    else if (VE == 2) launch_op<T, 2, 1>(op, a, grid, block, st);
    else if (VE == 4) launch_op<T, 4, 1>(op, a, grid, block, st);
    else if (VE == 8 && sizeof(T) == 2) launch_op<T, (sizeof(T) == 2 ? 8 : 4), 1>(op, a, grid, block, st);
    else return false;
  } else if (VE == 1 && P == 2) {
    launch_op<T, 1, 2>(op, a, grid, block, st);
  } else if (VE == 1 && P == 4) {
    launch_op<T, 1, 4>(op, a, grid, block, st);
  } else {
    return false;
  }
  return true;
}

static fast_status_t run_op(const char* fn, Op op, const fast_tcsr_t* g, int H, int dh,
                            fast_dtype_t dt, AttnArgs a, const void* const* rows, int nrows,
                            fast_stream_t stream) {
  if (!g) return fail(FAST_ERR_INVALID_ARG, "%s: graph is NULL", fn);
  if (g->num_dst < 0 || g->num_edges < 0) return fail(FAST_ERR_INVALID_ARG, "%s: negative size", fn);
  if (g->num_edges >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: E >= 2^31", fn);
  if (g->num_dst >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: N >= 2^31", fn);
  if (dt != FAST_F32 && dt != FAST_BF16) return fail(FAST_ERR_INVALID_ARG, "%s: bad dtype", fn);
  if (!(a.slope == a.slope) || !(a.scale == a.scale)) return fail(FAST_ERR_INVALID_ARG, "%s: NaN scale/slope", fn);
  if (g->num_dst == 0 && g->num_edges > 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: E > 0 edges but no destination", fn);
  int P = 1;
  fast_status_t s = make_layout(fn, H, dh, dt, rows, nrows, a.L, P);
  if (s != FAST_OK) return s;
  if (g->num_dst == 0) return ok();
  if (!g->dst_offsets) return fail(FAST_ERR_INVALID_ARG, "%s: dst_offsets is NULL", fn);
  a.N = g->num_dst;
  a.E = g->num_edges;
  a.off = g->dst_offsets;
  const int64_t nb = (a.N + a.L.SPB - 1) / a.L.SPB;
  const dim3 grid{uint32_t(nb)}, block{uint32_t(a.L.block)};
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool done = dt == FAST_BF16 ? dispatch_t<uint16_t>(op, a, P, grid, block, st)
                                    : dispatch_t<float>(op, a, P, grid, block, st);
  if (!done) return fail(FAST_ERR_UNSUPPORTED, "%s: no kernel for VE=%d P=%d", fn, a.L.VE, P);
  return check_launch(fn);
}

}  // namespace fast

using namespace fast;

#define FAST_NEED(ptr, fn)                                                               \
  do {                                                                                   \
    if (!(ptr)) return fail(FAST_ERR_INVALID_ARG, "%s: " #ptr " is NULL", fn);           \
  } while (0)

static bool has_work(const fast_tcsr_t* g) { return g && g->num_dst > 0; }

extern "C" fast_status_t fast_edge_attention_fwd(const fast_tcsr_t* g, int H, int dh,
                                                 fast_dtype_t dtype, const void* Q, const void* K,
                                                 const void* V, float scale, float neg_slope,
                                                 void* out, float* lse, fast_stream_t stream) {
  const char* fn = "fast_edge_attention_fwd";
  if (has_work(g)) {
    FAST_NEED(Q, fn); FAST_NEED(out, fn);
    if (g->num_edges > 0) { FAST_NEED(K, fn); FAST_NEED(V, fn); }
  }
  AttnArgs a = {};
  a.scale = scale; a.slope = neg_slope;
  a.Q = Q; a.K = K; a.V = V; a.out = out; a.lse_out = lse;
  const void* rows[] = {Q, K, V, out};
  return run_op(fn, Op::kAttnFwd, g, H, dh, dtype, a, rows, 4, stream);
}

extern "C" fast_status_t fast_edge_attention_bwd(const fast_tcsr_t* g, int H, int dh,
                                                 fast_dtype_t dtype, const void* Q, const void* K,
                                                 const void* V, float scale, float neg_slope,
                                                 const float* lse, const void* dout, void* dQ,
                                                 void* dK, void* dV, fast_stream_t stream) {
  const char* fn = "fast_edge_attention_bwd";
  if (has_work(g)) {
    FAST_NEED(Q, fn); FAST_NEED(dout, fn); FAST_NEED(dQ, fn);
    if (g->num_edges > 0) { FAST_NEED(K, fn); FAST_NEED(V, fn); FAST_NEED(dK, fn); FAST_NEED(dV, fn); }
  }
  AttnArgs a = {};
  a.scale = scale; a.slope = neg_slope;
  a.Q = Q; a.K = K; a.V = V; a.dO = dout; a.lse_in = lse; a.dQ = dQ; a.dK = dK; a.dV = dV;
  const void* rows[] = {Q, K, V, dout, dQ, dK, dV};
  return run_op(fn, Op::kAttnBwd, g, H, dh, dtype, a, rows, 7, stream);
}

extern "C" fast_status_t fast_edge_softmax_fwd(const fast_tcsr_t* g, int H, int dh,
                                               fast_dtype_t dtype, const void* Q, const void* K,
                                               float scale, float neg_slope, float* alpha,
                                               float* lse, fast_stream_t stream) {
  const char* fn = "fast_edge_softmax_fwd";
  if (has_work(g)) {
    FAST_NEED(Q, fn);
    if (g->num_edges > 0) { FAST_NEED(K, fn); FAST_NEED(alpha, fn); }
  }
  AttnArgs a = {};
  a.scale = scale; a.slope = neg_slope;
  a.Q = Q; a.K = K; a.alpha_out = alpha; a.lse_out = lse;
  const void* rows[] = {Q, K};
  return run_op(fn, Op::kSoftmaxFwd, g, H, dh, dtype, a, rows, 2, stream);
}

extern "C" fast_status_t fast_edge_softmax_bwd(const fast_tcsr_t* g, int H, int dh,
                                               fast_dtype_t dtype, const void* Q, const void* K,
                                               float scale, float neg_slope, const float* alpha,
                                               const float* dalpha, void* dQ, void* dK,
                                               fast_stream_t stream) {
  const char* fn = "fast_edge_softmax_bwd";
  if (has_work(g)) {
    FAST_NEED(Q, fn); FAST_NEED(dQ, fn);
    if (g->num_edges > 0) { FAST_NEED(K, fn); FAST_NEED(alpha, fn); FAST_NEED(dalpha, fn); FAST_NEED(dK, fn); }
  }
  AttnArgs a = {};
  a.scale = scale; a.slope = neg_slope;
  a.Q = Q; a.K = K; a.alpha_in = alpha; a.dalpha_in = dalpha; a.dQ = dQ; a.dK = dK;
  const void* rows[] = {Q, K, dQ, dK};
  return run_op(fn, Op::kSoftmaxBwd, g, H, dh, dtype, a, rows, 4, stream);
}

extern "C" fast_status_t fast_temporal_aggregate_fwd(const fast_tcsr_t* g, int H, int dh,
                                                     fast_dtype_t dtype, const float* alpha,
                                                     const void* V, void* out,
                                                     fast_stream_t stream) {
  const char* fn = "fast_temporal_aggregate_fwd";
  if (has_work(g)) {
    FAST_NEED(out, fn);
    if (g->num_edges > 0) { FAST_NEED(alpha, fn); FAST_NEED(V, fn); }
  }
  AttnArgs a = {};
  a.alpha_in = alpha; a.V = V; a.out = out;
  const void* rows[] = {V, out};
  return run_op(fn, Op::kAggFwd, g, H, dh, dtype, a, rows, 2, stream);
}

extern "C" fast_status_t fast_temporal_aggregate_bwd(const fast_tcsr_t* g, int H, int dh,
                                                     fast_dtype_t dtype, const float* alpha,
                                                     const void* V, const void* dout,
                                                     float* dalpha, void* dV,
                                                     fast_stream_t stream) {
  const char* fn = "fast_temporal_aggregate_bwd";
  if (has_work(g)) {
    FAST_NEED(dout, fn);
    if (g->num_edges > 0) { FAST_NEED(alpha, fn); FAST_NEED(V, fn); FAST_NEED(dalpha, fn); FAST_NEED(dV, fn); }
  }
  AttnArgs a = {};
  a.alpha_in = alpha; a.V = V; a.dO = dout; a.dalpha_out = dalpha; a.dV = dV;
  const void* rows[] = {V, dout, dV};
  return run_op(fn, Op::kAggBwd, g, H, dh, dtype, a, rows, 3, stream);
}
