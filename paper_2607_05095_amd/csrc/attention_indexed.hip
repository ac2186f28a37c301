// attention_indexed.hip -- the fused edge softmax + aggregation with indexed
// operands: edge e reads row k_index[e] of K and v_index[e] of V, so K and V
// can stay as the de-duplicated rows of the compressed ids (Sec. 4.2: rows
// are rebuilt through the inverse index; here the operator reads through the
// index instead of a rebuilt per-edge copy).  The backward writes the
// per-edge gradients; the gradient of a shared row is their sum over the
// edges that read it (fast_occurrence_csr + fast_index_add_rows).
#include <type_traits>

#include "attention.h"
#include "attention_rowmajor.h"

namespace fast {

bool attn_launch_indexed(Op op, fast_dtype_t dt, const AttnArgs& a, dim3 grid, dim3 block,
                         hipStream_t st) {
  if (a.L.rm) return attn_launch_rm<true>(op, a, grid, block, st);
  const bool bf = dt == FAST_BF16;
  const int VE = a.L.VE, P = a.L.P, LPH = a.L.LPH;
#define FAST_TRY(T_, VE_, P_, L_)                                                          \
  if (bf == std::is_same<T_, uint16_t>::value && VE == VE_ && P == P_ &&                   \
      (L_ == 0 || LPH == L_)) {                                                            \
    if (op == Op::kAttnFwdIdx) {                                                           \
      if (a.L.nt)                                                                          \
        hipLaunchKernelGGL((k_attn_fwd<T_, VE_, P_, L_, true, true>), grid, block, 0, st, a);  \
      else                                                                                 \
        hipLaunchKernelGGL((k_attn_fwd<T_, VE_, P_, L_, false, true>), grid, block, 0, st, a); \
    } else {                                                                               \
      if (a.L.nt)                                                                          \
        hipLaunchKernelGGL((k_attn_bwd<T_, VE_, P_, L_, true, true>), grid, block, 0, st, a);  \
      else                                                                                 \
        hipLaunchKernelGGL((k_attn_bwd<T_, VE_, P_, L_, false, true>), grid, block, 0, st, a); \
    }                                                                                      \
    return true;                                                                           \
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

static fast_status_t check_rows(const char* fn, const int32_t* idx, int64_t rows) {
  if (idx && rows < 1)
    return fail(FAST_ERR_INVALID_ARG, "%s: an index is given but its operand has %lld rows", fn,
                (long long)rows);
  return FAST_OK;
}

extern "C" fast_status_t fast_edge_attention_fwd_indexed(
    const fast_tcsr_t* g, int H, int dh, fast_dtype_t dtype, const void* Q, const void* K,
    const int32_t* k_index, int64_t k_rows, const void* V, const int32_t* v_index, int64_t v_rows,
    float scale, float neg_slope, void* out, float* lse, fast_stream_t stream) {
  const char* fn = "fast_edge_attention_fwd_indexed";
  if (g && g->num_dst > 0) {
    FAST_NEED(Q, fn); FAST_NEED(out, fn);
    if (g->num_edges > 0) { FAST_NEED(K, fn); FAST_NEED(V, fn); }
  }
  if (check_rows(fn, k_index, k_rows) || check_rows(fn, v_index, v_rows))
    return FAST_ERR_INVALID_ARG;
  AttnArgs a = {};
  a.scale = scale; a.slope = neg_slope;
  a.Q = Q; a.K = K; a.V = V; a.out = out; a.lse_out = lse;
  a.kidx = k_index; a.vidx = v_index; a.k_rows = k_rows; a.v_rows = v_rows;
  const void* rows[] = {Q, K, V, out};
  return attn_run(fn, Op::kAttnFwdIdx, g, H, dh, dtype, a, rows, 4, stream);
}

extern "C" fast_status_t fast_edge_attention_bwd_indexed(
    const fast_tcsr_t* g, int H, int dh, fast_dtype_t dtype, const void* Q, const void* K,
    const int32_t* k_index, int64_t k_rows, const void* V, const int32_t* v_index, int64_t v_rows,
    float scale, float neg_slope, const float* lse, const void* dout, void* dQ, void* dK_edge,
    void* dV_edge, fast_stream_t stream) {
  const char* fn = "fast_edge_attention_bwd_indexed";
  if (g && g->num_dst > 0) {
    FAST_NEED(Q, fn); FAST_NEED(dout, fn); FAST_NEED(dQ, fn);
    if (g->num_edges > 0) {
      FAST_NEED(K, fn); FAST_NEED(V, fn); FAST_NEED(dK_edge, fn); FAST_NEED(dV_edge, fn);
    }
  }
  if (check_rows(fn, k_index, k_rows) || check_rows(fn, v_index, v_rows))
    return FAST_ERR_INVALID_ARG;
  AttnArgs a = {};
  a.scale = scale; a.slope = neg_slope;
  a.Q = Q; a.K = K; a.V = V; a.dO = dout; a.lse_in = lse; a.dQ = dQ; a.dK = dK_edge;
  a.dV = dV_edge;
  a.kidx = k_index; a.vidx = v_index; a.k_rows = k_rows; a.v_rows = v_rows;
  const void* rows[] = {Q, K, V, dout, dQ, dK_edge, dV_edge};
  return attn_run(fn, Op::kAttnBwdIdx, g, H, dh, dtype, a, rows, 7, stream);
}

extern "C" fast_status_t fast_edge_attention_bwd_indexed_coef(
    const fast_tcsr_t* g, int H, int dh, fast_dtype_t dtype, const void* Q, const void* K,
    const int32_t* k_index, int64_t k_rows, const void* V, const int32_t* v_index, int64_t v_rows,
    float scale, float neg_slope, const float* lse, const void* dout, void* dQ, float* g_edge,
    float* alpha_edge, fast_stream_t stream) {
  const char* fn = "fast_edge_attention_bwd_indexed_coef";
  if (g && g->num_dst > 0) {
    FAST_NEED(Q, fn); FAST_NEED(dout, fn); FAST_NEED(dQ, fn);
    if (g->num_edges > 0) {
      FAST_NEED(K, fn); FAST_NEED(V, fn); FAST_NEED(g_edge, fn); FAST_NEED(alpha_edge, fn);
    }
  }
  if ((g_edge && !aligned(g_edge, 4)) || (alpha_edge && !aligned(alpha_edge, 4)))
    return fail(FAST_ERR_UNSUPPORTED, "%s: g_edge/alpha_edge not 4-byte aligned", fn);
  if (check_rows(fn, k_index, k_rows) || check_rows(fn, v_index, v_rows))
    return FAST_ERR_INVALID_ARG;
  AttnArgs a = {};
  a.scale = scale; a.slope = neg_slope;
  a.Q = Q; a.K = K; a.V = V; a.dO = dout; a.lse_in = lse; a.dQ = dQ;
  a.kidx = k_index; a.vidx = v_index; a.k_rows = k_rows; a.v_rows = v_rows;
  a.g_out = g_edge; a.al_out = alpha_edge;
  const void* rows[] = {Q, K, V, dout, dQ};
  return attn_run(fn, Op::kAttnBwdIdx, g, H, dh, dtype, a, rows, 5, stream);
}
