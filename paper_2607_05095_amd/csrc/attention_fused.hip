// attention_fused.hip -- fused edge softmax + aggregation forward/backward
// (Sec. 4.3 operators in one pass; alpha never reaches memory), and the
// host-side layout choice and validation shared with the unfused operators.
#include <cstdlib>
#include <type_traits>

#include "attention.h"
#include "attention_rowmajor.h"

namespace fast {

static int next_pow2(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Optional tuning override of the lanes per head (FAST_ATTN_LANES_PER_HEAD,
// a power of two <= 64), read once; 0 = use the default rule.
static int lanes_override() {
  static const int v = [] {
    const char* e = std::getenv("FAST_ATTN_LANES_PER_HEAD");
    const int x = e ? std::atoi(e) : 0;
    return (x > 0 && x <= 64 && (x & (x - 1)) == 0) ? x : 0;
  }();
  return v;
}

static bool rowmajor_enabled() {
  static const bool v = [] {
    const char* e = std::getenv("FAST_ATTN_ROWMAJOR");
    return !(e && e[0] == '0');
  }();
  return v;
}

// Kernels exist for these (vector width, chunks per lane) pairs.
static bool have_kernel(fast_dtype_t dt, int VE, int P) {
  if (P == 1) return true;
  if (VE <= 2) return P == 2 || P == 4;
  return P == 2;   // 16-byte (fp32 x4, bf16 x8) and bf16 x4 vectors
}

fast_status_t attn_layout(const char* fn, int H, int dh, fast_dtype_t dt, const void* const* rows,
                          int nrows, int block, AttnLayout& L) {
  if (H < 1 || dh < 1) return fail(FAST_ERR_INVALID_ARG, "%s: H = %d, dh = %d", fn, H, dh);
  if (int64_t(H) * dh > 4096) return fail(FAST_ERR_UNSUPPORTED, "%s: H*dh > 4096", fn);
  const int esz = elem_size(dt);
  for (int k = 0; k < nrows; ++k)
    if (rows[k] && !aligned(rows[k], size_t(esz)))
      return fail(FAST_ERR_UNSUPPORTED, "%s: operand %d is not %d-byte aligned", fn, k, esz);
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
  const int CPH = dh / VE;
  // Default: at most 16 lanes per head (fewer reduction steps and less
  // per-lane repetition of the scalar softmax work), more chunks per lane;
  // wider heads spread over up to 64 lanes with at most 4 chunks each.
  int LPH = next_pow2(CPH < 16 ? CPH : 16);
  int P = (CPH + LPH - 1) / LPH;
  if (P > 2 && VE >= 4) {          // wide vectors: keep P <= 2, widen the group instead
    LPH = next_pow2((CPH + 1) / 2);
    P = (CPH + LPH - 1) / LPH;
  }
  while (P > 4 && LPH < 64) {
    LPH *= 2;
    P = (CPH + LPH - 1) / LPH;
  }
  if (P > 4) return fail(FAST_ERR_UNSUPPORTED, "%s: dh = %d too large for this dtype", fn, dh);
  if (P == 3) P = 4;
  if (const int o = lanes_override()) {
    int p = (CPH + o - 1) / o;
    if (p == 3) p = 4;
    if (p <= 4 && have_kernel(dt, VE, p)) {
      LPH = o;
      P = p;
    }
  }
  // many heads: narrow the head groups until a segment fits ATT_MAX_GROUP lanes
  while (H * LPH > ATT_MAX_GROUP && LPH > 1) {
    LPH >>= 1;
    P = (CPH + LPH - 1) / LPH;
    if (P == 3) P = 4;
  }
  if (int64_t(H) * LPH > ATT_MAX_GROUP || P > 4 || !have_kernel(dt, VE, P))
    return fail(FAST_ERR_UNSUPPORTED, "%s: no lane layout for H = %d, dh = %d", fn, H, dh);
  L.H = H;
  L.dh = dh;
  L.F = H * dh;
  L.VE = VE;
  L.P = P;
  L.CPH = CPH;
  L.LPH = LPH;
  L.G = H * LPH;
  L.block = L.G <= block ? block : ATT_MAX_BLOCK;
  L.SPB = L.block / L.G;
  return FAST_OK;
}

fast_status_t attn_run(const char* fn, Op op, const fast_tcsr_t* g, int H, int dh, fast_dtype_t dt,
                       AttnArgs a, const void* const* rows, int nrows, fast_stream_t stream) {
  if (!g) return fail(FAST_ERR_INVALID_ARG, "%s: graph is NULL", fn);
  if (g->num_dst < 0 || g->num_edges < 0) return fail(FAST_ERR_INVALID_ARG, "%s: negative size", fn);
  if (g->num_edges >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: E >= 2^31", fn);
  if (g->num_dst >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: N >= 2^31", fn);
  if (dt != FAST_F32 && dt != FAST_BF16) return fail(FAST_ERR_INVALID_ARG, "%s: bad dtype", fn);
  if (!(a.slope == a.slope) || !(a.scale == a.scale))
    return fail(FAST_ERR_INVALID_ARG, "%s: NaN scale/slope", fn);
  if (g->num_dst == 0 && g->num_edges > 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: E > 0 edges but no destination", fn);
  const int wg = (op == Op::kAttnBwd || op == Op::kAttnBwdIdx) ? ATT_BLOCK_BWD : ATT_BLOCK;
  fast_status_t s = attn_layout(fn, H, dh, dt, rows, nrows, wg, a.L);
  if (s != FAST_OK) return s;
  // K, V, dK and dV rows: F apart (separate arrays) unless the packed entry
  // points set 2F; a stride that is a multiple of F keeps every row on the
  // vector alignment checked above
  if (a.ldkv == 0) a.ldkv = a.L.F;
  if (a.ldkv != a.L.F && !(op == Op::kAttnFwd || op == Op::kAttnBwd))
    return fail(FAST_ERR_UNSUPPORTED, "%s: strided K/V rows only in the fused operators", fn);
  if (a.ldkv % a.L.F != 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: K/V row stride %lld is not a multiple of F = %d", fn,
                (long long)a.ldkv, a.L.F);
  // fp32 rows whose heads break the 16-byte alignment (dh % 4 != 0) but whose
  // width does not (F % 4 == 0): the fused operators use row-major lanes so
  // every row moves as 16-byte accesses (FAST_ATTN_ROWMAJOR=0 turns it off).
  const bool fused_op = op == Op::kAttnFwd || op == Op::kAttnBwd || op == Op::kAttnFwdIdx ||
                        op == Op::kAttnBwdIdx;
  a.L.rm = false;
  if (fused_op && rowmajor_enabled() && dt == FAST_F32 && H == 2 && dh % 4 != 0 &&
      (H * dh) % 4 == 0 && (H * dh) / 4 <= 64) {
    bool al = true;
    for (int k = 0; k < nrows; ++k)
      if (rows[k] && !aligned(rows[k], 16)) al = false;
    if (al) {
      a.L.rm = true;
      a.L.VE = 4;
      a.L.P = 1;
      a.L.CPH = 0;
      a.L.LPH = 0;
      a.L.G = next_pow2((H * dh) / 4 < 16 ? 16 : (H * dh) / 4);
      a.L.block = wg;
      a.L.SPB = wg / a.L.G;
    }
  }
  // Backward workgroups: ATT_BLOCK_BWD (512) threads for the row-major lanes
  // on large grids, ATT_BLOCK (256) otherwise.  Measured on MI355X: the fp32
  // row-major layer-1 backward of the 1e7-node batch 0.80 ms at 512 against
  // 0.83 at 256; the bf16 head-major one of the large batch 0.92 at 256
  // against 0.93; layer-2 blocks (fewer than 4096 workgroups of 512) 0.079
  // against 0.084 ms at 256, whose last round of workgroups ends sooner.  A
  // segment's lanes and arithmetic do not depend on the workgroup size.
  const bool bwd_op = op == Op::kAttnBwd || op == Op::kAttnBwdIdx;
  if (bwd_op && a.L.block == ATT_BLOCK_BWD && a.L.G <= ATT_BLOCK) {
    const int64_t wgs_large = (g->num_dst + ATT_BLOCK_BWD / a.L.G - 1) / (ATT_BLOCK_BWD / a.L.G);
    if (!(a.L.rm && wgs_large >= 4096)) {
      a.L.block = ATT_BLOCK;
      a.L.SPB = ATT_BLOCK / a.L.G;
    }
  }
  // The fused row-major forward (plain operands) takes 512-thread
  // workgroups on the same large grids: with its per-segment rows streamed,
  // the 1e7-node batch's layer-1 forward 0.383 -> 0.377-0.379 ms.
  if (op == Op::kAttnFwd && a.L.rm && a.L.block == ATT_BLOCK && a.L.G <= ATT_BLOCK) {
    const int64_t wgs_large = (g->num_dst + ATT_BLOCK_BWD / a.L.G - 1) / (ATT_BLOCK_BWD / a.L.G);
    if (wgs_large >= 4096) {
      a.L.block = ATT_BLOCK_BWD;
      a.L.SPB = ATT_BLOCK_BWD / a.L.G;
    }
  }
  // Non-temporal streaming only when every per-edge row starts and ends on a
  // cache line, so no two rows share a line.
  a.L.nt = (size_t(a.L.F) * elem_size(dt)) % CACHE_LINE == 0;
  for (const void* p : {a.K, a.V, static_cast<const void*>(a.dK), static_cast<const void*>(a.dV)})
    if (p && !aligned(p, CACHE_LINE)) a.L.nt = false;
#ifdef FAST_ATTN_FORCE_NT
  a.L.nt = true;   // tuning build: streaming policy whatever the row alignment
#endif
  if (a.L.block > ATT_MAX_BLOCK)
    return fail(FAST_ERR_UNSUPPORTED, "%s: workgroup of %d threads outside the launch bound %d",
                fn, a.L.block, ATT_MAX_BLOCK);
  if (g->num_dst == 0) return ok();
  if (!g->dst_offsets) return fail(FAST_ERR_INVALID_ARG, "%s: dst_offsets is NULL", fn);
  a.N = g->num_dst;
  a.E = g->num_edges;
  a.off = g->dst_offsets;
  const int64_t nb = (a.N + a.L.SPB - 1) / a.L.SPB;
  const dim3 grid{uint32_t(nb)}, block{uint32_t(a.L.block)};
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool fused = op == Op::kAttnFwd || op == Op::kAttnBwd;
  const bool indexed = op == Op::kAttnFwdIdx || op == Op::kAttnBwdIdx;
  const bool done = indexed ? attn_launch_indexed(op, dt, a, grid, block, st)
                    : fused ? attn_launch_fused(op, dt, a, grid, block, st)
                            : attn_launch_unfused(op, dt, a, grid, block, st);
  if (!done)
    return fail(FAST_ERR_UNSUPPORTED, "%s: no kernel for VE=%d P=%d LPH=%d", fn, a.L.VE, a.L.P, a.L.LPH);
  return check_launch(fn);
}

template <typename T, int VE, int P, int LPH, bool NT>
static void launch_fused_nt(Op op, const AttnArgs& a, dim3 grid, dim3 block, hipStream_t st) {
  if (op == Op::kAttnFwd) hipLaunchKernelGGL((k_attn_fwd<T, VE, P, LPH, NT>), grid, block, 0, st, a);
  else hipLaunchKernelGGL((k_attn_bwd<T, VE, P, LPH, NT>), grid, block, 0, st, a);
}

template <typename T, int VE, int P, int LPH>
static void launch_fused(Op op, const AttnArgs& a, dim3 grid, dim3 block, hipStream_t st) {
  if (a.L.nt) launch_fused_nt<T, VE, P, LPH, true>(op, a, grid, block, st);
  else launch_fused_nt<T, VE, P, LPH, false>(op, a, grid, block, st);
}

bool attn_launch_fused(Op op, fast_dtype_t dt, const AttnArgs& a, dim3 grid, dim3 block,
                       hipStream_t st) {
  if (a.L.rm) return attn_launch_rm<false>(op, a, grid, block, st);
  const bool bf = dt == FAST_BF16;
  const int VE = a.L.VE, P = a.L.P, LPH = a.L.LPH;
#define FAST_TRY(T_, VE_, P_, L_)                                                     \
  if (bf == std::is_same<T_, uint16_t>::value && VE == VE_ && P == P_ &&              \
      (L_ == 0 || LPH == L_)) {                                                       \
    launch_fused<T_, VE_, P_, L_>(op, a, grid, block, st);                            \
    return true;                                                                      \
  }
  FAST_ATTN_FAST_SET(FAST_TRY)
  FAST_ATTN_GENERIC_SET(FAST_TRY)
#undef FAST_TRY
  return false;
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
  return attn_run(fn, Op::kAttnFwd, g, H, dh, dtype, a, rows, 4, stream);
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
  return attn_run(fn, Op::kAttnBwd, g, H, dh, dtype, a, rows, 7, stream);
}

// Packed K|V rows: row e of KV holds K_e then V_e (F = H*dh elements each), and
// dKV the gradients in the same layout; the same kernels with a row stride of
// 2F, so that K, V (and dK, dV) move as one stream.
static fast_status_t packed_split(const char* fn, int H, int dh, fast_dtype_t dtype, int64_t* F) {
  if (H < 1 || dh < 1) return fail(FAST_ERR_INVALID_ARG, "%s: H = %d, dh = %d", fn, H, dh);
  if (int64_t(H) * dh > 4096) return fail(FAST_ERR_UNSUPPORTED, "%s: H*dh > 4096", fn);
  if (dtype != FAST_F32 && dtype != FAST_BF16) return fail(FAST_ERR_INVALID_ARG, "%s: bad dtype", fn);
  *F = int64_t(H) * dh;
  return FAST_OK;
}

extern "C" fast_status_t fast_edge_attention_fwd_packed(const fast_tcsr_t* g, int H, int dh,
                                                        fast_dtype_t dtype, const void* Q,
                                                        const void* KV, float scale,
                                                        float neg_slope, void* out, float* lse,
                                                        fast_stream_t stream) {
  const char* fn = "fast_edge_attention_fwd_packed";
  int64_t F = 0;
  fast_status_t s = packed_split(fn, H, dh, dtype, &F);
  if (s != FAST_OK) return s;
  if (has_work(g)) {
    FAST_NEED(Q, fn); FAST_NEED(out, fn);
    if (g->num_edges > 0) FAST_NEED(KV, fn);
  }
  const size_t half = size_t(F) * elem_size(dtype);
  const void* K = KV;
  const void* V = KV ? static_cast<const char*>(KV) + half : nullptr;
  AttnArgs a = {};
  a.scale = scale; a.slope = neg_slope;
  a.Q = Q; a.K = K; a.V = V; a.out = out; a.lse_out = lse;
  a.ldkv = 2 * F;
  const void* rows[] = {Q, K, V, out};
  return attn_run(fn, Op::kAttnFwd, g, H, dh, dtype, a, rows, 4, stream);
}

extern "C" fast_status_t fast_edge_attention_bwd_packed(const fast_tcsr_t* g, int H, int dh,
                                                        fast_dtype_t dtype, const void* Q,
                                                        const void* KV, float scale,
                                                        float neg_slope, const float* lse,
                                                        const void* dout, void* dQ, void* dKV,
                                                        fast_stream_t stream) {
  const char* fn = "fast_edge_attention_bwd_packed";
  int64_t F = 0;
  fast_status_t s = packed_split(fn, H, dh, dtype, &F);
  if (s != FAST_OK) return s;
  if (has_work(g)) {
    FAST_NEED(Q, fn); FAST_NEED(dout, fn); FAST_NEED(dQ, fn);
    if (g->num_edges > 0) { FAST_NEED(KV, fn); FAST_NEED(dKV, fn); }
  }
  const size_t half = size_t(F) * elem_size(dtype);
  const void* K = KV;
  const void* V = KV ? static_cast<const char*>(KV) + half : nullptr;
  void* dK = dKV;
  void* dV = dKV ? static_cast<char*>(dKV) + half : nullptr;
  AttnArgs a = {};
  a.scale = scale; a.slope = neg_slope;
  a.Q = Q; a.K = K; a.V = V; a.dO = dout; a.lse_in = lse; a.dQ = dQ; a.dK = dK; a.dV = dV;
  a.ldkv = 2 * F;
  const void* rows[] = {Q, K, V, dout, dQ, dK, dV};
  return attn_run(fn, Op::kAttnBwd, g, H, dh, dtype, a, rows, 7, stream);
}
