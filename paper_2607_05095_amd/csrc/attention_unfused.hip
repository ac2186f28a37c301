// attention_unfused.hip -- the separate operators: edge softmax forward and
// backward (Sec. 4.3 "Edge Softmax") and attention-weighted aggregation
// forward and backward (Sec. 4.3 "Balanced Aggregate"), with alpha in memory.
#include <type_traits>

#include "attention.h"

namespace fast {

template <typename T, int VE, int P, int LPH>
static void launch_unfused(Op op, const AttnArgs& a, dim3 grid, dim3 block, hipStream_t st) {
  switch (op) {
    case Op::kSoftmaxFwd: hipLaunchKernelGGL((k_softmax_fwd<T, VE, P, LPH>), grid, block, 0, st, a); break;
    case Op::kSoftmaxBwd: hipLaunchKernelGGL((k_softmax_bwd<T, VE, P, LPH>), grid, block, 0, st, a); break;
    case Op::kAggFwd: hipLaunchKernelGGL((k_agg_fwd<T, VE, P, LPH>), grid, block, 0, st, a); break;
    case Op::kAggBwd: hipLaunchKernelGGL((k_agg_bwd<T, VE, P, LPH>), grid, block, 0, st, a); break;
    default: break;
  }
}

bool attn_launch_unfused(Op op, fast_dtype_t dt, const AttnArgs& a, dim3 grid, dim3 block,
                         hipStream_t st) {
  const bool bf = dt == FAST_BF16;
  const int VE = a.L.VE, P = a.L.P, LPH = a.L.LPH;
#define FAST_TRY(T_, VE_, P_, L_)                                                     \
  if (bf == std::is_same<T_, uint16_t>::value && VE == VE_ && P == P_ &&              \
      (L_ == 0 || LPH == L_)) {                                                       \
    launch_unfused<T_, VE_, P_, L_>(op, a, grid, block, st);                          \
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
  return attn_run(fn, Op::kSoftmaxFwd, g, H, dh, dtype, a, rows, 2, stream);
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
  return attn_run(fn, Op::kSoftmaxBwd, g, H, dh, dtype, a, rows, 4, stream);
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
  return attn_run(fn, Op::kAggFwd, g, H, dh, dtype, a, rows, 2, stream);
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
  return attn_run(fn, Op::kAggBwd, g, H, dh, dtype, a, rows, 3, stream);
}
