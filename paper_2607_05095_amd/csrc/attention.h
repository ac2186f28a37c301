// attention.h -- edge softmax (ESM) with per-edge multi-head logits and
// attention-weighted aggregation (AGG), forward and backward, separately and
// fused (Sec. 4.3; Eq. 1 with an attention-weighted sum as AGG).
//
// Mapping (MI355X, wave64, no MFMA: every op here is a gather/reduce whose
// arithmetic intensity is ~0.5 flop/byte, far below the vector-ALU ridge):
//   * One sub-wavefront of G = H * LPH lanes owns one destination segment
//     and walks its edges in CSR order.  Each head is a group of LPH lanes
//     (a power of two); lane l of a head holds feature chunks l, l+LPH, ...
//     (P of them) of VE elements, VE*bytes <= 16, so a row of a segment is
//     read with P coalesced vector loads per lane.
//   * Per-edge, per-head dot products (the logits, and in backward the
//     <dOut, V> terms) are all-reduced inside the head group with DPP row
//     operations and the gfx950 permlane swaps; no LDS, no atomics.  LPH is a
//     template parameter for the common layouts, so the CH reductions of a
//     chunk are straight-line code the scheduler interleaves.
//   * Softmax is computed online over chunks of CH edges (one rescale per
//     chunk) in base 2, so any degree works and a segment is streamed once.
//     The loads of a chunk are issued back to back; slots past the segment
//     end re-read its last row (a cache hit) and are masked out.
//   * Every destination row is produced by exactly one sub-wavefront: the
//     results are deterministic run to run (unlike the paper's edge-parallel
//     atomicAdd aggregation, which is prior art for a different GPU).
//   * Backward needs one pass over K and V: with w = exp(s - m),
//       dQ = scale/Z * (sum w c dalpha K - D * sum w c K),  D = sum w dalpha / Z
//     is accumulated while streaming, and dK, dV of the first 24 edges are
//     written from per-edge scalars kept in registers (longer segments
//     re-read K and V for the remainder).
#pragma once

#include "common.h"

// Edges per chunk.  Forward: 10, the sampler's top-k fan-out (Sec. 6.1), so
// a sampled segment is one chunk and one round trip to memory.  Backward
// holds two rows per edge and twice the accumulators, so it uses shorter
// chunks (4) and keeps the per-edge scalars of the first 24 edges in registers.
#ifndef FAST_ATT_CH_FWD
#define FAST_ATT_CH_FWD 10
#endif
#ifndef FAST_ATT_CH_BWD
#define FAST_ATT_CH_BWD 4
#endif
#ifndef FAST_ATT_SAVE_EDGES
#define FAST_ATT_SAVE_EDGES 24
#endif

// Workgroup sizes: 256 threads for the forward and unfused kernels, 512 for
// the fused backward (measured faster on MI355X for the backward's mixed
// read/write stream); a segment wider than the workgroup (many heads) gets a
// 512-thread workgroup.  A segment never exceeds ATT_MAX_GROUP lanes.
#ifndef FAST_ATT_BLOCK
#define FAST_ATT_BLOCK 256
#endif
#ifndef FAST_ATT_BLOCK_BWD
#define FAST_ATT_BLOCK_BWD 512
#endif
// Occupancy target of the fused kernels in waves per SIMD (the register
// budget follows from it: 512 / waves).
#ifdef FAST_ATT_WAVES_PER_EU
#define FAST_ATT_OCC __attribute__((amdgpu_waves_per_eu(FAST_ATT_WAVES_PER_EU)))
#else
#define FAST_ATT_OCC
#endif

namespace fast {

constexpr int ATT_BLOCK = FAST_ATT_BLOCK;
constexpr int ATT_BLOCK_BWD = FAST_ATT_BLOCK_BWD;
constexpr int ATT_MAX_GROUP = 512;   // lanes per destination segment, at most
constexpr int ATT_MAX_BLOCK = 512;   // launch bound of every attention kernel
constexpr int ATT_CH_FWD = FAST_ATT_CH_FWD;
constexpr int ATT_CH_BWD = FAST_ATT_CH_BWD;
constexpr int ATT_NSAVE = (FAST_ATT_SAVE_EDGES + ATT_CH_BWD - 1) / ATT_CH_BWD;
// Every attention kernel is compiled for at most ATT_MAX_BLOCK threads per
// workgroup (its register budget follows from that bound); a larger launch
// is refused by the runtime, so the workgroup sizes may not exceed it.
static_assert(ATT_BLOCK <= ATT_MAX_BLOCK && ATT_BLOCK_BWD <= ATT_MAX_BLOCK,
              "attention workgroup size above the kernels' launch bound");
static_assert(ATT_BLOCK % 64 == 0 && ATT_BLOCK_BWD % 64 == 0 && ATT_BLOCK >= 64 &&
                  ATT_BLOCK_BWD >= 64,
              "attention workgroup size must be a whole number of waves");

struct AttnLayout {
  int H, dh, F;   // heads, head dim, F = H*dh
  int VE;         // elements per vector access
  int P;          // vector chunks per lane
  int CPH;        // vector chunks per head = dh / VE
  int LPH;        // lanes per head (power of two)
  int G;          // lanes per segment = H * LPH
  int SPB;        // segments per workgroup
  int block;      // workgroup size
  bool nt;        // streamed rows cover whole cache lines: non-temporal policy
  bool rm;        // row-major lanes (attention_rowmajor.h): lane c owns elements 4c..4c+3
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
  // row stride of K, V, dK and dV in elements for the fused operators: F for
  // separate arrays, 2F for packed K|V rows (0 on entry: F)
  int64_t ldkv;
  // indexed operands: edge e reads row kidx[e] of K and vidx[e] of V (NULL:
  // row e); an index outside [0, rows) reads the nearest row
  const int32_t* kidx;
  const int32_t* vidx;
  int64_t k_rows, v_rows;
  // indexed backward, coefficient form: per edge and head g (dK = g Q[seg])
  // and alpha (dV = alpha dOut[seg]) instead of the dK, dV rows
  float* g_out;
  float* al_out;
};

// Row of K or V read by edge e.
template <bool IDX>
__device__ __forceinline__ int64_t operand_row(const int32_t* idx, int64_t rows, int64_t e) {
  if constexpr (IDX) {
    if (idx) return clamp64(idx[e], 0, rows - 1);
  }
  return e;
}

// ------------------------------------------------------------------ lane map
template <int P>
struct LaneMap {
  int64_t seg;
  int h, l, lph;
  int foff[P];    // element offset of chunk p inside a row
  bool cok[P];    // chunk p exists (padding lanes of a head hold zeros)
};

// LPH_CT > 0: lanes per head known at compile time; 0: read from the layout.
template <int VE, int P, int LPH_CT>
__device__ __forceinline__ bool lane_setup(const AttnArgs& a, LaneMap<P>& m) {
  const int t = threadIdx.x;
  const int lph = LPH_CT > 0 ? LPH_CT : a.L.LPH;
  const int G = LPH_CT > 0 ? LPH_CT * a.L.H : a.L.G;
  const int sub = t / G;
  const int r = t - sub * G;
  m.lph = lph;
  m.h = r / lph;
  m.l = r - m.h * lph;
  m.seg = int64_t(xcd_tile(blockIdx.x, gridDim.x)) * a.L.SPB + sub;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const int c = m.l + p * lph;
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

template <typename T, int VE, int P, bool NT>
__device__ __forceinline__ void load_raw(const T* __restrict__ base, int64_t row, int F,
                                         const LaneMap<P>& m, Raw<T, VE> (&x)[P]) {
#pragma unroll
  for (int p = 0; p < P; ++p) {
    if (m.cok[p]) x[p].template load<NT>(base + row * F + m.foff[p]);
    else x[p].zero();
  }
}

template <typename T, int VE, int P>
__device__ __forceinline__ void unpack_row(const Raw<T, VE> (&r)[P], float (&x)[P][VE]) {
#pragma unroll
  for (int p = 0; p < P; ++p) r[p].unpack(x[p]);
}

template <typename T, int VE, int P>
__device__ __forceinline__ void store_row(T* __restrict__ base, int64_t row, int F,
                                          const LaneMap<P>& m, const float (&x)[P][VE]) {
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (m.cok[p]) VecIO<T, VE>::store(base + row * F + m.foff[p], x[p]);
}

template <typename T, int VE, int P, bool NT>
__device__ __forceinline__ void store_row_stream(T* __restrict__ base, int64_t row, int F,
                                                 const LaneMap<P>& m, const float (&x)[P][VE]) {
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (m.cok[p]) StreamIO<T, VE, NT>::store(base + row * F + m.foff[p], x[p]);
}

// load_row with a streaming (non-temporal) policy when NT is set.
template <typename T, int VE, int P, bool NT>
__device__ __forceinline__ void load_row_stream(const T* __restrict__ base, int64_t row, int F,
                                                const LaneMap<P>& m, float (&x)[P][VE]) {
  Raw<T, VE> r[P];
  load_raw<T, VE, P, NT>(base, row, F, m, r);
  unpack_row<T, VE, P>(r, x);
}

template <int LPH>
__device__ __forceinline__ float group_sum_ct(float x) {
  if constexpr (LPH >= 2) x += dpp_quad_xor1(x);
  if constexpr (LPH >= 4) x += dpp_quad_xor2(x);
  if constexpr (LPH >= 8) x += dpp_row_half_mirror(x);
  if constexpr (LPH >= 16) x += dpp_row_mirror(x);
  if constexpr (LPH >= 32) x = sum_rows16(x);
  if constexpr (LPH >= 64) x = sum_halves32(x);
  return x;
}

template <int VE, int P, int LPH_CT>
__device__ __forceinline__ float head_dot(const float (&a)[P][VE], const float (&b)[P][VE], int lph) {
  float d = 0.f;
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) d = fmaf(a[p][j], b[p][j], d);
  if constexpr (LPH_CT > 0) return group_sum_ct<LPH_CT>(d);
  else return group_sum(d, lph);
}

__device__ __forceinline__ float lrelu(float x, float slope) { return x > 0.f ? x : slope * x; }
// LeakyReLU' taken at the PRE-activation x (its sign picks the branch).  The
// activated value cannot stand in for x: a negative slope maps both signs of
// x to positive values.
__device__ __forceinline__ float lrelu_grad(float x, float slope) { return x > 0.f ? 1.f : slope; }
// Softmax in base 2: logits are formed as t = LReLU(pre * log2(e)) (LeakyReLU
// is positively homogeneous, so t = log2(e) * LReLU(pre), and pre * log2(e)
// has the sign of pre), and exp(s - m) = exp2(t - m2) is one v_exp_f32.
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ void seg_range(const AttnArgs& a, int64_t seg, int64_t& e0, int64_t& e1) {
  e0 = clamp64(a.off[seg], 0, a.E);
  e1 = clamp64(a.off[seg + 1], e0, a.E);
}
// Row of chunk slot i: past the segment end the last row is read again.
__device__ __forceinline__ int64_t slot_row(int64_t base, int i, int64_t e1) {
  return base + i < e1 ? base + i : e1 - 1;
}

#define FAST_ZERO(arr)                                        \
  _Pragma("unroll") for (int p_ = 0; p_ < P; ++p_)            \
      _Pragma("unroll") for (int j_ = 0; j_ < VE; ++j_) arr[p_][j_] = 0.f

// ============================================================ fused forward
template <typename T, int VE, int P, int LPH_CT, bool NT, bool IDX = false>
__global__ void __launch_bounds__(ATT_MAX_BLOCK) FAST_ATT_OCC k_attn_fwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P, LPH_CT>(a, m)) return;
  const int F = a.L.F, ld = int(a.ldkv);
  const T* K = static_cast<const T*>(a.K);
  const T* V = static_cast<const T*>(a.V);
  const float sl2 = a.scale * LOG2E;
  float q[P][VE];
  // with streaming K|V rows, Q and out stream too (large bf16 step, layer-1
  // forward 0.463 -> 0.452 ms; the backward's Q, dO and dQ measured slower
  // streamed and stay cached)
  load_row_stream<T, VE, P, NT>(static_cast<const T*>(a.Q), m.seg, F, m, q);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);

  float mx = -INFINITY, Z = 0.f, acc[P][VE];
  FAST_ZERO(acc);
  for (int64_t base = e0; base < e1; base += ATT_CH_FWD) {
    Raw<T, VE> kr[ATT_CH_FWD][P], vr[ATT_CH_FWD][P];
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i) {
      const int64_t e = slot_row(base, i, e1);
      // indexed rows are shared across segments: keep them cacheable
      load_raw<T, VE, P, NT && !IDX>(K, operand_row<IDX>(a.kidx, a.k_rows, e), ld, m, kr[i]);
      load_raw<T, VE, P, NT && !IDX>(V, operand_row<IDX>(a.vidx, a.v_rows, e), ld, m, vr[i]);
    }
    float t[ATT_CH_FWD];
    float cm = -INFINITY;
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i) {
      float kx[P][VE];
      unpack_row<T, VE, P>(kr[i], kx);
      const float ti = lrelu(head_dot<VE, P, LPH_CT>(q, kx, m.lph) * sl2, a.slope);
      t[i] = base + i < e1 ? ti : -INFINITY;
      cm = fmaxf(cm, t[i]);
    }
    const float mn = fmaxf(mx, cm);
    const float corr = exp2_hw(mx - mn);
    Z *= corr;
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int j = 0; j < VE; ++j) acc[p][j] *= corr;
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i) {
      const float w = exp2_hw(t[i] - mn);
      Z += w;
      float vx[P][VE];
      unpack_row<T, VE, P>(vr[i], vx);
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int j = 0; j < VE; ++j) acc[p][j] = fmaf(w, vx[p][j], acc[p][j]);
    }
    mx = mn;
  }
  const float inv = Z > 0.f ? 1.f / Z : 0.f;
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) acc[p][j] *= inv;
  store_row_stream<T, VE, P, NT>(static_cast<T*>(a.out), m.seg, F, m, acc);
  if (a.lse_out && m.l == 0)
    a.lse_out[m.seg * a.L.H + m.h] = Z > 0.f ? (mx + log2f(Z)) * LN2 : -INFINITY;
}

// ============================================================ fused backward
template <int VE, int P>
struct BwdState {
  float q[P][VE], go[P][VE];
  float A[P][VE], B[P][VE];   // sum w c dalpha K, sum w c K
  float mx, Z, Dn;            // reference point (running max or lse, log2 units), sum w, sum w dalpha
};

// Edges [base, min(base+CH, e1)): loads K and V, forms the pre-activation
// x = pre * log2(e), the logit t = LReLU(x) and dalpha = <dOut, V>, and folds
// them into the running sums.  Returns x (not t: LReLU' needs x's sign).
template <typename T, int VE, int P, int LPH_CT, bool NT, bool IDX>
__device__ __forceinline__ void bwd_chunk(const AttnArgs& a, const LaneMap<P>& m, int64_t base,
                                          int64_t e1, bool has_lse, float sl2,
                                          BwdState<VE, P>& S, float (&x)[ATT_CH_BWD],
                                          float (&da)[ATT_CH_BWD]) {
  const int ld = int(a.ldkv);
  const T* K = static_cast<const T*>(a.K);
  const T* V = static_cast<const T*>(a.V);
  Raw<T, VE> kr[ATT_CH_BWD][P], vr[ATT_CH_BWD][P];
#pragma unroll
  for (int i = 0; i < ATT_CH_BWD; ++i) {
    const int64_t e = slot_row(base, i, e1);
    load_raw<T, VE, P, NT && !IDX>(K, operand_row<IDX>(a.kidx, a.k_rows, e), ld, m, kr[i]);
    load_raw<T, VE, P, NT && !IDX>(V, operand_row<IDX>(a.vidx, a.v_rows, e), ld, m, vr[i]);
  }
  float t[ATT_CH_BWD], cm = -INFINITY;
#pragma unroll
  for (int i = 0; i < ATT_CH_BWD; ++i) {
    float kx[P][VE], vx[P][VE];
    unpack_row<T, VE, P>(kr[i], kx);
    unpack_row<T, VE, P>(vr[i], vx);
    x[i] = head_dot<VE, P, LPH_CT>(S.q, kx, m.lph) * sl2;
    da[i] = head_dot<VE, P, LPH_CT>(S.go, vx, m.lph);
    t[i] = base + i < e1 ? lrelu(x[i], a.slope) : -INFINITY;
    cm = fmaxf(cm, t[i]);
  }
  if (!has_lse) {
    const float mn = fmaxf(S.mx, cm);
    const float corr = exp2_hw(S.mx - mn);
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
  for (int i = 0; i < ATT_CH_BWD; ++i) {
    const float w = exp2_hw(t[i] - S.mx);       // 0 for masked slots
    const float wc = w * lrelu_grad(x[i], a.slope);
    const float wcd = wc * da[i];
    S.Z += w;
    S.Dn = fmaf(w, da[i], S.Dn);
    float kx[P][VE];
    unpack_row<T, VE, P>(kr[i], kx);
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int j = 0; j < VE; ++j) {
        S.A[p][j] = fmaf(wcd, kx[p][j], S.A[p][j]);
        S.B[p][j] = fmaf(wc, kx[p][j], S.B[p][j]);
      }
  }
}

// dK, dV of edge e from its pre-activation x (log2 units) and dalpha.
template <typename T, int VE, int P, bool NT, bool IDX>
__device__ __forceinline__ void bwd_emit(const AttnArgs& a, const LaneMap<P>& m, int64_t e, float x,
                                         float da, float invZ, float D, const BwdState<VE, P>& S) {
  const float al = exp2_hw(lrelu(x, a.slope) - S.mx) * invZ;
  const float g = al * (da - D) * lrelu_grad(x, a.slope) * a.scale;
  if constexpr (IDX) {
    if (a.g_out) {                       // the head's first lane writes its coefficients
      if (m.l == 0) {
        a.g_out[e * a.L.H + m.h] = g;
        a.al_out[e * a.L.H + m.h] = al;
      }
      return;
    }
  }
  float dk[P][VE], dv[P][VE];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) {
      dk[p][j] = g * S.q[p][j];
      dv[p][j] = al * S.go[p][j];
    }
  store_row_stream<T, VE, P, NT>(static_cast<T*>(a.dK), e, int(a.ldkv), m, dk);
  store_row_stream<T, VE, P, NT>(static_cast<T*>(a.dV), e, int(a.ldkv), m, dv);
}

template <typename T, int VE, int P, int LPH_CT, bool NT, bool IDX = false>
__global__ void __launch_bounds__(ATT_MAX_BLOCK) FAST_ATT_OCC k_attn_bwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P, LPH_CT>(a, m)) return;
  const int F = a.L.F;
  const float sl2 = a.scale * LOG2E;
  BwdState<VE, P> S;
  load_row<T, VE, P>(static_cast<const T*>(a.Q), m.seg, F, m, S.q);
  load_row<T, VE, P>(static_cast<const T*>(a.dO), m.seg, F, m, S.go);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  const bool has_lse = a.lse_in != nullptr;
  S.mx = has_lse ? a.lse_in[m.seg * a.L.H + m.h] * LOG2E : -INFINITY;
  if (has_lse && !(S.mx > -INFINITY)) S.mx = 0.f;   // empty segment: no edge reads it
  S.Z = 0.f;
  S.Dn = 0.f;
  FAST_ZERO(S.A);
  FAST_ZERO(S.B);

  // pass 1: stream K and V once; keep x and dalpha of the first NSAVE chunks
  float st[ATT_NSAVE][ATT_CH_BWD], sda[ATT_NSAVE][ATT_CH_BWD];
#pragma unroll
  for (int c = 0; c < ATT_NSAVE; ++c) {
    const int64_t base = e0 + c * ATT_CH_BWD;
    if (base < e1)
      bwd_chunk<T, VE, P, LPH_CT, NT, IDX>(a, m, base, e1, has_lse, sl2, S, st[c], sda[c]);
  }
  for (int64_t base = e0 + ATT_NSAVE * ATT_CH_BWD; base < e1; base += ATT_CH_BWD) {
    float tt[ATT_CH_BWD], td[ATT_CH_BWD];
    bwd_chunk<T, VE, P, LPH_CT, NT, IDX>(a, m, base, e1, has_lse, sl2, S, tt, td);
  }

  // dQ = scale/Z * (A - D B)
  const float invZ = has_lse ? 1.f : (S.Z > 0.f ? 1.f / S.Z : 0.f);
  const float D = S.Dn * invZ;
  const float f = invZ * a.scale;
  float dq[P][VE];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < VE; ++j) dq[p][j] = (S.A[p][j] - D * S.B[p][j]) * f;
  store_row<T, VE, P>(static_cast<T*>(a.dQ), m.seg, F, m, dq);

  // pass 2: dK, dV from the saved per-edge scalars
#pragma unroll
  for (int c = 0; c < ATT_NSAVE; ++c) {
    const int64_t base = e0 + c * ATT_CH_BWD;
#pragma unroll
    for (int i = 0; i < ATT_CH_BWD; ++i)
      if (base + i < e1) bwd_emit<T, VE, P, NT, IDX>(a, m, base + i, st[c][i], sda[c][i], invZ, D, S);
  }
  // long segments: re-read K and V for the edges past the register window
  for (int64_t base = e0 + ATT_NSAVE * ATT_CH_BWD; base < e1; base += ATT_CH_BWD) {
    float kx[ATT_CH_BWD][P][VE], vx[ATT_CH_BWD][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH_BWD; ++i) {
      const int64_t e = slot_row(base, i, e1);
      load_row<T, VE, P>(static_cast<const T*>(a.K), operand_row<IDX>(a.kidx, a.k_rows, e), int(a.ldkv), m, kx[i]);
      load_row<T, VE, P>(static_cast<const T*>(a.V), operand_row<IDX>(a.vidx, a.v_rows, e), int(a.ldkv), m, vx[i]);
    }
#pragma unroll
    for (int i = 0; i < ATT_CH_BWD; ++i) {
      const float x = head_dot<VE, P, LPH_CT>(S.q, kx[i], m.lph) * sl2;
      const float da = head_dot<VE, P, LPH_CT>(S.go, vx[i], m.lph);
      if (base + i < e1) bwd_emit<T, VE, P, NT, IDX>(a, m, base + i, x, da, invZ, D, S);
    }
  }
}

// ============================================================ edge softmax fwd
template <typename T, int VE, int P, int LPH_CT>
__global__ void __launch_bounds__(ATT_MAX_BLOCK) k_softmax_fwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P, LPH_CT>(a, m)) return;
  const int F = a.L.F, H = a.L.H;
  const T* K = static_cast<const T*>(a.K);
  const float sl2 = a.scale * LOG2E;
  float q[P][VE];
  load_row<T, VE, P>(static_cast<const T*>(a.Q), m.seg, F, m, q);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  float mx = -INFINITY, Z = 0.f;
  // pass 1: running max and normaliser
  for (int64_t base = e0; base < e1; base += ATT_CH_FWD) {
    float kx[ATT_CH_FWD][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i) load_row<T, VE, P>(K, slot_row(base, i, e1), F, m, kx[i]);
    float t[ATT_CH_FWD], cm = -INFINITY;
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i) {
      const float ti = lrelu(head_dot<VE, P, LPH_CT>(q, kx[i], m.lph) * sl2, a.slope);
      t[i] = base + i < e1 ? ti : -INFINITY;
      cm = fmaxf(cm, t[i]);
    }
    const float mn = fmaxf(mx, cm);
    Z *= exp2_hw(mx - mn);
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i) Z += exp2_hw(t[i] - mn);
    mx = mn;
  }
  const float invZ = Z > 0.f ? 1.f / Z : 0.f;
  if (a.lse_out && m.l == 0) a.lse_out[m.seg * H + m.h] = Z > 0.f ? (mx + log2f(Z)) * LN2 : -INFINITY;
  // pass 2: alpha (the segment's K rows are re-read, normally from L2)
  for (int64_t base = e0; base < e1; base += ATT_CH_FWD) {
    float kx[ATT_CH_FWD][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i) load_row<T, VE, P>(K, slot_row(base, i, e1), F, m, kx[i]);
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i) {
      const float t = lrelu(head_dot<VE, P, LPH_CT>(q, kx[i], m.lph) * sl2, a.slope);
      if (base + i < e1 && m.l == 0) a.alpha_out[(base + i) * H + m.h] = exp2_hw(t - mx) * invZ;
    }
  }
}

// ============================================================ edge softmax bwd
template <typename T, int VE, int P, int LPH_CT>
__global__ void __launch_bounds__(ATT_MAX_BLOCK) k_softmax_bwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P, LPH_CT>(a, m)) return;
  const int F = a.L.F, H = a.L.H;
  const T* K = static_cast<const T*>(a.K);
  float q[P][VE];
  load_row<T, VE, P>(static_cast<const T*>(a.Q), m.seg, F, m, q);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  float D = 0.f;
  for (int64_t e = e0; e < e1; ++e) D = fmaf(a.alpha_in[e * H + m.h], a.dalpha_in[e * H + m.h], D);
  float dq[P][VE];
  FAST_ZERO(dq);
  for (int64_t base = e0; base < e1; base += ATT_CH_BWD) {
    float kx[ATT_CH_BWD][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH_BWD; ++i) load_row<T, VE, P>(K, slot_row(base, i, e1), F, m, kx[i]);
#pragma unroll
    for (int i = 0; i < ATT_CH_BWD; ++i) {
      const int64_t e = slot_row(base, i, e1);
      const float pre = head_dot<VE, P, LPH_CT>(q, kx[i], m.lph) * a.scale;
      const float g = base + i < e1 ? a.alpha_in[e * H + m.h] * (a.dalpha_in[e * H + m.h] - D) *
                                          lrelu_grad(pre, a.slope) * a.scale
                                    : 0.f;
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
template <typename T, int VE, int P, int LPH_CT>
__global__ void __launch_bounds__(ATT_MAX_BLOCK) k_agg_fwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P, LPH_CT>(a, m)) return;
  const int F = a.L.F, H = a.L.H;
  const T* V = static_cast<const T*>(a.V);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  float acc[P][VE];
  FAST_ZERO(acc);
  for (int64_t base = e0; base < e1; base += ATT_CH_FWD) {
    float vx[ATT_CH_FWD][P][VE], al[ATT_CH_FWD];
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i) {
      const int64_t e = slot_row(base, i, e1);
      load_row<T, VE, P>(V, e, F, m, vx[i]);
      al[i] = base + i < e1 ? a.alpha_in[e * H + m.h] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < ATT_CH_FWD; ++i)
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int j = 0; j < VE; ++j) acc[p][j] = fmaf(al[i], vx[i][p][j], acc[p][j]);
  }
  store_row<T, VE, P>(static_cast<T*>(a.out), m.seg, F, m, acc);
}

// ============================================================ aggregation bwd
template <typename T, int VE, int P, int LPH_CT>
__global__ void __launch_bounds__(ATT_MAX_BLOCK) k_agg_bwd(AttnArgs a) {
  LaneMap<P> m;
  if (!lane_setup<VE, P, LPH_CT>(a, m)) return;
  const int F = a.L.F, H = a.L.H;
  const T* V = static_cast<const T*>(a.V);
  float go[P][VE];
  load_row<T, VE, P>(static_cast<const T*>(a.dO), m.seg, F, m, go);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  for (int64_t base = e0; base < e1; base += ATT_CH_BWD) {
    float vx[ATT_CH_BWD][P][VE];
#pragma unroll
    for (int i = 0; i < ATT_CH_BWD; ++i) load_row<T, VE, P>(V, slot_row(base, i, e1), F, m, vx[i]);
#pragma unroll
    for (int i = 0; i < ATT_CH_BWD; ++i) {
      const int64_t e = slot_row(base, i, e1);
      const float da = head_dot<VE, P, LPH_CT>(go, vx[i], m.lph);
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

#undef FAST_ZERO

// ============================================================ host side
enum class Op { kAttnFwd, kAttnBwd, kSoftmaxFwd, kSoftmaxBwd, kAggFwd, kAggBwd,
                kAttnFwdIdx, kAttnBwdIdx };

// Picks the vector width and lane mapping for (H, dh, dtype) given every row
// pointer the op touches (all must be aligned to the vector access), for
// workgroups of `block` threads.
fast_status_t attn_layout(const char* fn, int H, int dh, fast_dtype_t dt, const void* const* rows,
                          int nrows, int block, AttnLayout& L);

// Validates the graph and launches `op` with the chosen layout.
fast_status_t attn_run(const char* fn, Op op, const fast_tcsr_t* g, int H, int dh, fast_dtype_t dt,
                       AttnArgs a, const void* const* rows, int nrows, fast_stream_t stream);

// Kernel selection for one op family; defined in the translation unit that
// instantiates that family's kernels.  Returns false if no kernel fits.
bool attn_launch_fused(Op op, fast_dtype_t dt, const AttnArgs& a, dim3 grid, dim3 block,
                       hipStream_t st);
bool attn_launch_unfused(Op op, fast_dtype_t dt, const AttnArgs& a, dim3 grid, dim3 block,
                         hipStream_t st);
bool attn_launch_indexed(Op op, fast_dtype_t dt, const AttnArgs& a, dim3 grid, dim3 block,
                         hipStream_t st);

// Dispatch over the instantiated layouts: a fast set with compile-time lanes
// per head, and a runtime-lanes fallback for every other (VE, P).
#define FAST_ATTN_FAST_SET(X)                                                         \
  X(float, 4, 1, 8) X(float, 4, 1, 16) X(float, 4, 1, 32) X(float, 4, 2, 16)          \
  X(float, 2, 1, 32) X(float, 2, 2, 16) X(float, 2, 4, 8)                             \
  X(uint16_t, 8, 1, 4) X(uint16_t, 8, 1, 8) X(uint16_t, 8, 1, 16) X(uint16_t, 8, 2, 4) \
  X(uint16_t, 4, 1, 8) X(uint16_t, 2, 1, 32) X(uint16_t, 2, 2, 16)

#define FAST_ATTN_GENERIC_SET(X)                                              \
  X(float, 4, 1, 0) X(float, 2, 1, 0) X(float, 1, 1, 0) X(float, 1, 2, 0)     \
  X(float, 1, 4, 0) X(float, 2, 2, 0) X(float, 2, 4, 0) X(float, 4, 2, 0)     \
  X(uint16_t, 8, 1, 0) X(uint16_t, 4, 1, 0) X(uint16_t, 2, 1, 0)              \
  X(uint16_t, 1, 1, 0) X(uint16_t, 1, 2, 0) X(uint16_t, 1, 4, 0)              \
  X(uint16_t, 8, 2, 0) X(uint16_t, 4, 2, 0) X(uint16_t, 2, 2, 0) X(uint16_t, 2, 4, 0)

}  // namespace fast
