// attention_rowmajor.h -- the fused edge softmax + aggregation kernels in a
// row-major lane layout, for fp32 rows whose head dim is not a multiple of 4
// while the row width is (the 2 x 50 heads of the workloads' 100-wide rows).
//
// The head-major layout of attention.h gives every head its own lanes; with
// dh = 50 a head is 200 bytes, so the second head starts 8 bytes off a
// 16-byte boundary and the rows move as 8-byte accesses (measured on MI355X:
// 400-byte rows copy at 4.06 TB/s that way, at 4.87 TB/s as 16-byte
// accesses).  Here lane c of a G-lane group owns elements 4c .. 4c+3 of every
// row, so each row moves as one 16-byte access per lane; a lane whose four
// elements straddle two heads keeps both heads' values.  The per-head dot
// products become H all-reduces over the G lanes (DPP / permlane, no LDS),
// and every per-element weight picks its head's value.  Everything else --
// chunked online softmax in base 2, one pass over K and V in the backward,
// per-edge scalars kept in registers, one group per destination row, no
// atomics -- follows the head-major kernels.
#pragma once

#include "attention.h"

namespace fast {

// Edges per chunk (forward, backward) and edges whose backward scalars stay
// in registers (both heads' values per lane).  Measured on the 2 x 50-head,
// 10-edge segments of the big-dedup block: chunks of 5 in both directions
// and 10 saved edges beat chunks of 4 / 10 with 12 saved edges by 2-3 %.
#ifndef FAST_ATT_RM_CH_FWD
#define FAST_ATT_RM_CH_FWD 5
#endif
#ifndef FAST_ATT_RM_CH_BWD
#define FAST_ATT_RM_CH_BWD 5
#endif
#ifndef FAST_ATT_RM_SAVE_EDGES
#define FAST_ATT_RM_SAVE_EDGES 10
#endif
constexpr int RM_CH_FWD = FAST_ATT_RM_CH_FWD;
constexpr int RM_CH_BWD = FAST_ATT_RM_CH_BWD;
constexpr int ATT_RM_NSAVE = (FAST_ATT_RM_SAVE_EDGES + RM_CH_BWD - 1) / RM_CH_BWD;

template <int H>
struct RmMap {
  int64_t seg;
  int c;        // 4-element chunk of the row owned by this lane
  bool ok;      // the chunk exists (lanes past F/4 hold zeros)
  int hs[4];    // head of each of the four elements
};

// Row groups in plain block order.  Unlike the head-major kernels, these
// measured no gain from handing each XCD a contiguous range of groups
// (xcd_tile): on the packed K|V rows of the 1e7-node batch's layer-1 block
// the forward ran 0.414 -> 0.402 ms and the backward 0.800 -> 0.798 ms in
// plain order on one box, 0.816 -> 0.806 ms on another.
template <int H, int G>
__device__ __forceinline__ bool rm_setup(const AttnArgs& a, RmMap<H>& m) {
  const int t = threadIdx.x;
  const int sub = t / G;
  m.c = t - sub * G;
  m.ok = m.c < a.L.F / 4;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int h = m.ok ? (4 * m.c + k) / a.L.dh : 0;
    m.hs[k] = h < H ? h : H - 1;
  }
  m.seg = int64_t(blockIdx.x) * a.L.SPB + sub;
  return sub < a.L.SPB && m.seg < a.N;
}

template <int H>
__device__ __forceinline__ float pick(const float (&v)[H], int h) {
  float r = v[0];
#pragma unroll
  for (int j = 1; j < H; ++j) r = h == j ? v[j] : r;
  return r;
}

template <bool NT, int H>
__device__ __forceinline__ void rm_load_row(const float* __restrict__ base, int64_t row, int F,
                                            const RmMap<H>& m, float (&x)[4]) {
  if (m.ok) {
    const f32x4 v = ld_stream<f32x4, NT>(base + row * F + 4 * m.c);
    x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
  } else {
    x[0] = x[1] = x[2] = x[3] = 0.f;
  }
}

template <bool NT, int H>
__device__ __forceinline__ void rm_store_row(float* __restrict__ base, int64_t row, int F,
                                             const RmMap<H>& m, const float (&x)[4]) {
  if (m.ok) st_stream<f32x4, NT>(base + row * F + 4 * m.c, f32x4{x[0], x[1], x[2], x[3]});
}

// Per-head dot products of two rows: d[h] = sum over the row's elements of
// head h, all-reduced over the G lanes of the group.
template <int H, int G>
__device__ __forceinline__ void rm_dots(const float (&x)[4], const float (&y)[4], const RmMap<H>& m,
                                        float (&d)[H]) {
#pragma unroll
  for (int h = 0; h < H; ++h) {
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < 4; ++k) s = fmaf(m.hs[k] == h ? x[k] : 0.f, y[k], s);
    d[h] = group_sum_ct<G>(s);
  }
}

// ============================================================ fused forward
template <int H, int G, bool NT, bool IDX>
__global__ void __launch_bounds__(ATT_MAX_BLOCK) FAST_ATT_OCC k_attn_fwd_rm(AttnArgs a) {
  RmMap<H> m;
  if (!rm_setup<H, G>(a, m)) return;
  const int F = a.L.F, ld = int(a.ldkv);
  const float* K = static_cast<const float*>(a.K);
  const float* V = static_cast<const float*>(a.V);
  const float sl2 = a.scale * LOG2E;
  float q[4];
  // Q and out stream too (each row is read or written once per call): the
  // 1e7-node fp32 batch's layer-1 forward 0.430 -> 0.385 ms with both, its step
  // 1.887 -> 1.845 ms.  The HBM reads of K|V then run without the write-back
  // of out lines interleaved at random; read-only, the same access shape
  // reads at 7.0-7.3 TB/s, with 400-byte output rows stored normally at 5.6.
  rm_load_row<!IDX, H>(static_cast<const float*>(a.Q), m.seg, F, m, q);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);

  float mx[H], Z[H], acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int h = 0; h < H; ++h) {
    mx[h] = -INFINITY;
    Z[h] = 0.f;
  }
  for (int64_t base = e0; base < e1; base += RM_CH_FWD) {
    float kx[RM_CH_FWD][4], vx[RM_CH_FWD][4];
    // K and V rows stream (non-temporal) whatever NT says: the forward reads
    // them once, and alone it ran 0.422 -> 0.396 ms on packed rows of the
    // 1e7-node batch's layer-1 block.  (Indexed rows are shared by several
    // segments and stay cacheable.)
#pragma unroll
    for (int i = 0; i < RM_CH_FWD; ++i) {
      const int64_t e = slot_row(base, i, e1);
      rm_load_row<!IDX, H>(K, operand_row<IDX>(a.kidx, a.k_rows, e), ld, m, kx[i]);
      rm_load_row<!IDX, H>(V, operand_row<IDX>(a.vidx, a.v_rows, e), ld, m, vx[i]);
    }
    float t[RM_CH_FWD][H], cm[H];
#pragma unroll
    for (int h = 0; h < H; ++h) cm[h] = -INFINITY;
#pragma unroll
    for (int i = 0; i < RM_CH_FWD; ++i) {
      float d[H];
      rm_dots<H, G>(q, kx[i], m, d);
#pragma unroll
      for (int h = 0; h < H; ++h) {
        t[i][h] = base + i < e1 ? lrelu(d[h] * sl2, a.slope) : -INFINITY;
        cm[h] = fmaxf(cm[h], t[i][h]);
      }
    }
    float mn[H], corr[H];
#pragma unroll
    for (int h = 0; h < H; ++h) {
      mn[h] = fmaxf(mx[h], cm[h]);
      corr[h] = exp2_hw(mx[h] - mn[h]);
      Z[h] *= corr[h];
      mx[h] = mn[h];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[k] *= pick<H>(corr, m.hs[k]);
#pragma unroll
    for (int i = 0; i < RM_CH_FWD; ++i) {
      float w[H];
#pragma unroll
      for (int h = 0; h < H; ++h) {
        w[h] = exp2_hw(t[i][h] - mx[h]);
        Z[h] += w[h];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[k] = fmaf(pick<H>(w, m.hs[k]), vx[i][k], acc[k]);
    }
  }
  float inv[H];
#pragma unroll
  for (int h = 0; h < H; ++h) inv[h] = Z[h] > 0.f ? 1.f / Z[h] : 0.f;
#pragma unroll
  for (int k = 0; k < 4; ++k) acc[k] *= pick<H>(inv, m.hs[k]);
  rm_store_row<!IDX, H>(static_cast<float*>(a.out), m.seg, F, m, acc);
  if (a.lse_out && m.c == 0) {
#pragma unroll
    for (int h = 0; h < H; ++h)
      a.lse_out[m.seg * H + h] = Z[h] > 0.f ? (mx[h] + log2f(Z[h])) * LN2 : -INFINITY;
  }
}

// ============================================================ fused backward
template <int H>
struct RmBwdState {
  float q[4], go[4];
  float A[4], B[4];          // sum w c dalpha K, sum w c K (per element, its head's weights)
  float mx[H], Z[H], Dn[H];  // reference point (log2 units), sum w, sum w dalpha
};

template <int H, int G, bool NT, bool IDX>
__device__ __forceinline__ void rm_bwd_chunk(const AttnArgs& a, const RmMap<H>& m, int64_t base,
                                             int64_t e1, bool has_lse, float sl2,
                                             RmBwdState<H>& S, float (&x)[RM_CH_BWD][H],
                                             float (&da)[RM_CH_BWD][H]) {
  const int ld = int(a.ldkv);
  const float* K = static_cast<const float*>(a.K);
  const float* V = static_cast<const float*>(a.V);
  float kx[RM_CH_BWD][4], vx[RM_CH_BWD][4];
#pragma unroll
  for (int i = 0; i < RM_CH_BWD; ++i) {
    const int64_t e = slot_row(base, i, e1);
    rm_load_row<NT && !IDX, H>(K, operand_row<IDX>(a.kidx, a.k_rows, e), ld, m, kx[i]);
    rm_load_row<NT && !IDX, H>(V, operand_row<IDX>(a.vidx, a.v_rows, e), ld, m, vx[i]);
  }
  float t[RM_CH_BWD][H], cm[H];
#pragma unroll
  for (int h = 0; h < H; ++h) cm[h] = -INFINITY;
#pragma unroll
  for (int i = 0; i < RM_CH_BWD; ++i) {
    float d[H];
    rm_dots<H, G>(S.q, kx[i], m, d);
    rm_dots<H, G>(S.go, vx[i], m, da[i]);
#pragma unroll
    for (int h = 0; h < H; ++h) {
      x[i][h] = d[h] * sl2;
      t[i][h] = base + i < e1 ? lrelu(x[i][h], a.slope) : -INFINITY;
      cm[h] = fmaxf(cm[h], t[i][h]);
    }
  }
  if (!has_lse) {
    float corr[H];
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const float mn = fmaxf(S.mx[h], cm[h]);
      corr[h] = exp2_hw(S.mx[h] - mn);
      S.Z[h] *= corr[h];
      S.Dn[h] *= corr[h];
      S.mx[h] = mn;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float c = pick<H>(corr, m.hs[k]);
      S.A[k] *= c;
      S.B[k] *= c;
    }
  }
#pragma unroll
  for (int i = 0; i < RM_CH_BWD; ++i) {
    float wc[H], wcd[H];
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const float w = exp2_hw(t[i][h] - S.mx[h]);      // 0 for masked slots
      wc[h] = w * lrelu_grad(x[i][h], a.slope);
      wcd[h] = wc[h] * da[i][h];
      S.Z[h] += w;
      S.Dn[h] = fmaf(w, da[i][h], S.Dn[h]);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      S.A[k] = fmaf(pick<H>(wcd, m.hs[k]), kx[i][k], S.A[k]);
      S.B[k] = fmaf(pick<H>(wc, m.hs[k]), kx[i][k], S.B[k]);
    }
  }
}

// dK, dV of edge e from its pre-activations x (log2 units) and dalpha.
template <int H, bool NT, bool IDX>
__device__ __forceinline__ void rm_bwd_emit(const AttnArgs& a, const RmMap<H>& m, int64_t e,
                                            const float (&x)[H], const float (&da)[H],
                                            const float (&invZ)[H], const float (&D)[H],
                                            const RmBwdState<H>& S) {
  float al[H], g[H];
#pragma unroll
  for (int h = 0; h < H; ++h) {
    al[h] = exp2_hw(lrelu(x[h], a.slope) - S.mx[h]) * invZ[h];
    g[h] = al[h] * (da[h] - D[h]) * lrelu_grad(x[h], a.slope) * a.scale;
  }
  if constexpr (IDX) {
    if (a.g_out) {                       // every lane holds all heads' values
      if (m.c == 0) {
#pragma unroll
        for (int h = 0; h < H; ++h) {
          a.g_out[e * H + h] = g[h];
          a.al_out[e * H + h] = al[h];
        }
      }
      return;
    }
  }
  float dk[4], dv[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    dk[k] = pick<H>(g, m.hs[k]) * S.q[k];
    dv[k] = pick<H>(al, m.hs[k]) * S.go[k];
  }
  // with indexed operands the per-edge gradients are written once and read
  // back only through the occurrence lists: streamed, as are Q, dO and dQ
  // (1e7-node batch, layer-1 indexed backward 1.425 -> 1.297 ms)
  rm_store_row<NT || IDX, H>(static_cast<float*>(a.dK), e, int(a.ldkv), m, dk);
  rm_store_row<NT || IDX, H>(static_cast<float*>(a.dV), e, int(a.ldkv), m, dv);
}

template <int H, int G, bool NT, bool IDX>
__global__ void __launch_bounds__(ATT_MAX_BLOCK) FAST_ATT_OCC k_attn_bwd_rm(AttnArgs a) {
  RmMap<H> m;
  if (!rm_setup<H, G>(a, m)) return;
  const int F = a.L.F;
  const float sl2 = a.scale * LOG2E;
  RmBwdState<H> S;
  // Q, dO and dQ stream, as in the forward (that batch's step 1.845 -> 1.837 ms;
  // with indexed operands too, below)
  rm_load_row<true, H>(static_cast<const float*>(a.Q), m.seg, F, m, S.q);
  rm_load_row<true, H>(static_cast<const float*>(a.dO), m.seg, F, m, S.go);
  int64_t e0, e1;
  seg_range(a, m.seg, e0, e1);
  const bool has_lse = a.lse_in != nullptr;
#pragma unroll
  for (int h = 0; h < H; ++h) {
    S.mx[h] = has_lse ? a.lse_in[m.seg * H + h] * LOG2E : -INFINITY;
    if (has_lse && !(S.mx[h] > -INFINITY)) S.mx[h] = 0.f;   // empty segment: no edge reads it
    S.Z[h] = 0.f;
    S.Dn[h] = 0.f;
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) S.A[k] = S.B[k] = 0.f;

  // pass 1: stream K and V once; keep x and dalpha of the first chunks
  float st[ATT_RM_NSAVE][RM_CH_BWD][H], sda[ATT_RM_NSAVE][RM_CH_BWD][H];
#pragma unroll
  for (int c = 0; c < ATT_RM_NSAVE; ++c) {
    const int64_t base = e0 + c * RM_CH_BWD;
    if (base < e1) rm_bwd_chunk<H, G, NT, IDX>(a, m, base, e1, has_lse, sl2, S, st[c], sda[c]);
  }
  for (int64_t base = e0 + ATT_RM_NSAVE * RM_CH_BWD; base < e1; base += RM_CH_BWD) {
    float tt[RM_CH_BWD][H], td[RM_CH_BWD][H];
    rm_bwd_chunk<H, G, NT, IDX>(a, m, base, e1, has_lse, sl2, S, tt, td);
  }

  // dQ = scale/Z * (A - D B), per element with its head's Z and D
  float invZ[H], D[H], f[H];
#pragma unroll
  for (int h = 0; h < H; ++h) {
    invZ[h] = has_lse ? 1.f : (S.Z[h] > 0.f ? 1.f / S.Z[h] : 0.f);
    D[h] = S.Dn[h] * invZ[h];
    f[h] = invZ[h] * a.scale;
  }
  float dq[4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
    dq[k] = (S.A[k] - pick<H>(D, m.hs[k]) * S.B[k]) * pick<H>(f, m.hs[k]);
  rm_store_row<true, H>(static_cast<float*>(a.dQ), m.seg, F, m, dq);

  // pass 2: dK, dV from the saved per-edge scalars
#pragma unroll
  for (int c = 0; c < ATT_RM_NSAVE; ++c) {
    const int64_t base = e0 + c * RM_CH_BWD;
#pragma unroll
    for (int i = 0; i < RM_CH_BWD; ++i)
      if (base + i < e1) rm_bwd_emit<H, NT, IDX>(a, m, base + i, st[c][i], sda[c][i], invZ, D, S);
  }
  // long segments: re-read K and V for the edges past the register window
  for (int64_t base = e0 + ATT_RM_NSAVE * RM_CH_BWD; base < e1; base += RM_CH_BWD) {
    float kx[RM_CH_BWD][4], vx[RM_CH_BWD][4];
#pragma unroll
    for (int i = 0; i < RM_CH_BWD; ++i) {
      const int64_t e = slot_row(base, i, e1);
      rm_load_row<false, H>(static_cast<const float*>(a.K), operand_row<IDX>(a.kidx, a.k_rows, e), int(a.ldkv), m, kx[i]);
      rm_load_row<false, H>(static_cast<const float*>(a.V), operand_row<IDX>(a.vidx, a.v_rows, e), int(a.ldkv), m, vx[i]);
    }
#pragma unroll
    for (int i = 0; i < RM_CH_BWD; ++i) {
      float d[H], da[H], x[H];
      rm_dots<H, G>(S.q, kx[i], m, d);
      rm_dots<H, G>(S.go, vx[i], m, da);
#pragma unroll
      for (int h = 0; h < H; ++h) x[h] = d[h] * sl2;
      if (base + i < e1) rm_bwd_emit<H, NT, IDX>(a, m, base + i, x, da, invZ, D, S);
    }
  }
}

// Kernels exist for these head counts and group widths (G = lanes per row).
// (Four heads would keep twice the per-edge scalars and spill registers.)
#define FAST_ATTN_RM_SET(X) X(2, 32) X(2, 16) X(2, 64)

template <bool IDX>
inline bool attn_launch_rm(Op op, const AttnArgs& a, dim3 grid, dim3 block, hipStream_t st) {
  const bool fwd = op == Op::kAttnFwd || op == Op::kAttnFwdIdx;
#define FAST_TRY_RM(H_, G_)                                                                      \
  if (a.L.H == H_ && a.L.G == G_) {                                                              \
    if (fwd) {                                                                                   \
      if (a.L.nt) hipLaunchKernelGGL((k_attn_fwd_rm<H_, G_, true, IDX>), grid, block, 0, st, a);  \
      else hipLaunchKernelGGL((k_attn_fwd_rm<H_, G_, false, IDX>), grid, block, 0, st, a);        \
    } else {                                                                                     \
      if (a.L.nt) hipLaunchKernelGGL((k_attn_bwd_rm<H_, G_, true, IDX>), grid, block, 0, st, a);  \
      else hipLaunchKernelGGL((k_attn_bwd_rm<H_, G_, false, IDX>), grid, block, 0, st, a);        \
    }                                                                                            \
    return true;                                                                                 \
  }
  FAST_ATTN_RM_SET(FAST_TRY_RM)
#undef FAST_TRY_RM
  return false;
}

}  // namespace fast
