/*
 * oracle.h -- plain, slow CPU reference of FAST's temporal-subgraph operators.
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists to check the HIP operators;
 * only the test-suite, the smoke check and the CPU-baseline leg of the
 * benchmark load it.  It shares no code, header or constant with the HIP
 * library.  Floating point is accumulated in fp64 (inputs are widened
 * exactly); the time encoding forms its argument in fp32 as stated below.
 *
 * Data model (all arrays row-major, host memory):
 *   sampled CSR temporal subgraph of one layer block (Sec. 4.3, Sec. 5: the
 *   compression engine's `ind_ptr`): off[N+1], edges of destination v are
 *   e in [off[v], off[v+1]); per-edge rows [E,H,dh], per-destination rows
 *   [N,H,dh], per-(edge,head) scalars [E,H], per-(destination,head) [N,H].
 */
#ifndef FAST_ORACLE_H
#define FAST_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* CSR offsets: off[0] = 0, off[v+1] = off[v] + counts[v]. */
void oracle_csr_offsets(const int32_t* counts, int64_t n, int32_t* off);

/* Contract check of a sampled subgraph: violations[5] as documented for
 * fast_check_tcsr (non-monotone offsets; wrong first/last offset; src ids
 * and edge ids outside their bounds; edge times after their destination's
 * time where the offsets are monotone).  NULL arrays count 0. */
void oracle_check_tcsr(const int32_t* off, int64_t N, int64_t E, const int64_t* src_ids,
                       int64_t src_bound, const int64_t* edge_ids, int64_t edge_bound,
                       const float* edge_t, const float* dst_t, int64_t* violations);

/* Within-batch compression (Sec. 4.2, Sec. 5): uni = ascending distinct ids,
 * inv[i] = position of ids[i] in uni.  Returns u = |uni|. */
int64_t oracle_dedup(const int64_t* ids, int64_t n, int64_t* uni, int32_t* inv);

/* Row reconstruction from the compressed ids: slot = slot_map ? slot_map[uni[k]]
 * : uni[k]; a slot in [0, table_rows) copies row_bytes bytes to rows[k], any
 * other slot appends k to miss (ascending).  Returns the number of misses. */
int64_t oracle_gather(const int64_t* uni, int64_t u, const void* table,
                      int64_t table_rows, int64_t row_bytes, const int32_t* slot_map,
                      void* rows, int32_t* miss);

/* Time encoding cos(omega_j * dt + phi_j), dt = t_dst[v] - t_e[e] for e in
 * segment v.  dt and the argument are formed in fp32 (one subtraction, one
 * fused multiply-add); the cosine itself is evaluated in fp64.  te[E*d_t]. */
void oracle_time_encode(const int32_t* off, int64_t N, const float* t_dst,
                        const float* t_e, const float* omega, const float* phi,
                        int d_t, double* te);

/* Occurrence lists (indexed operands, Sec. 4.2): occ_off[num_rows+1] and, for
 * row u, occ[occ_off[u] .. occ_off[u+1]) = the positions p with index[p] == u
 * in ascending order.  Index values outside [0, num_rows) are left out. */
void oracle_occurrence_csr(const int32_t* index, int64_t n, int64_t num_rows, int32_t* occ_off,
                           int32_t* occ);

/* Transposed gather: dst[u, :] = sum over p with index[p] == u of src[p, :]
 * (fp64; rows of D values; 0 for a row no position reads). */
void oracle_index_add_rows(const int32_t* index, int64_t n, int64_t num_rows, int64_t D,
                           const double* src, double* dst);

/* Row gradients from per-edge coefficients: dst[u, h, :] = sum over edges e
 * (segments v by off[N+1], edges in order) with index[e] == u of
 * scal[e, h] * src[v, h, :] (fp64; 0 for a row no edge reads). */
void oracle_index_add_scaled_rows(const int32_t* index, const int32_t* off, int64_t N,
                                  int64_t num_rows, int64_t H, int64_t dh, const double* scal,
                                  const double* src, double* dst);

/* Most-recent-k temporal neighbour sampling (Sec. 6.1) over a T-CSR graph:
 * node v's entries are p in [indptr[v], indptr[v+1]) with neighbour nbr[p],
 * time ts[p] and edge id eid[p], in time order.  For root i (node roots[i],
 * query time root_t[i]) the candidates are the entries with ts < root_t[i];
 * the root's segment holds the last min(k, #candidates) of them in entry
 * order.  Roots outside [0, num_nodes) get empty segments.  Output: off[R+1]
 * and per sampled edge src (neighbour), et (time), ei (edge id); capacity
 * R * k. */
void oracle_sample_recent(const int64_t* indptr, int64_t num_nodes, const int64_t* nbr,
                          const float* ts, const int64_t* eid, const int64_t* roots,
                          const float* root_t, int64_t R, int k, int32_t* off, int64_t* src,
                          float* et, int64_t* ei);

/* SlimCache greedy cache selection (Sec. 4.2, Alg. 1).
 * Counting: for each batch k (ids[batch_off[k]..batch_off[k+1])), every
 * distinct id x in [0, id_bound) of the batch does freq[x] += 1 (freq is
 * accumulated into, not cleared). */
void oracle_access_count(const int64_t* ids, const int64_t* batch_off, int64_t num_batches,
                         int64_t id_bound, int32_t* freq);

/* Selection: node and edge ids ranked by descending frequency (ties by
 * ascending id); while i + j < alpha * (nv + ne), the node head is taken if
 * its count is strictly greater than the edge head's, otherwise the edge
 * head (an exhausted list never wins).  hot_v[0..*n_hot_v) and
 * hot_e[0..*n_hot_e) receive the ids in selection order; capacities nv, ne. */
void oracle_greedy_hot_set(const int32_t* fv, int64_t nv, const int32_t* fe, int64_t ne,
                           double alpha, int64_t* hot_v, int64_t* n_hot_v, int64_t* hot_e,
                           int64_t* n_hot_e);

/* Backward of the time encoding for an upstream gradient dte [E, d_t]:
 *   a = fmaf(omega[j], dt_e, phi[j])  (the forward's fp32 argument)
 *   dphi[j]   = sum_e dte[e,j] * (-sin a)
 *   domega[j] = sum_e dte[e,j] * (-sin a) * dt_e
 * summed in fp64 over every edge of every segment. */
void oracle_time_encode_bwd(const int32_t* off, int64_t N, const float* t_dst,
                            const float* t_e, const float* omega, const float* phi,
                            int d_t, const double* dte, double* domega, double* dphi);

/* Edge softmax forward with per-edge multi-head logits:
 *   pre[e,h]   = scale * <Q[v,h,:], K[e,h,:]>
 *   s[e,h]     = pre > 0 ? pre : slope * pre            (LeakyReLU)
 *   alpha[e,h] = exp(s - m) / Z,  m = max_e s,  Z = sum_e exp(s - m)
 *   lse[v,h]   = m + log Z   (-inf for an empty segment)
 * pre may be NULL. */
void oracle_edge_softmax_fwd(const int32_t* off, int64_t N, int H, int dh,
                             const double* Q, const double* K, double scale,
                             double slope, double* pre, double* alpha, double* lse);

/* Aggregation forward: out[v,h,:] = sum_e alpha[e,h] * V[e,h,:] (0 if empty). */
void oracle_aggregate_fwd(const int32_t* off, int64_t N, int H, int dh,
                          const double* alpha, const double* V, double* out);

/* Aggregation backward for dOut:
 *   dalpha[e,h] = <dOut[v,h,:], V[e,h,:]>,  dV[e,h,:] = alpha[e,h] * dOut[v,h,:] */
void oracle_aggregate_bwd(const int32_t* off, int64_t N, int H, int dh,
                          const double* alpha, const double* V, const double* dout,
                          double* dalpha, double* dV);

/* Edge softmax (and logit) backward:
 *   D[v,h] = sum_e alpha*dalpha,  ds = alpha*(dalpha - D),
 *   g = ds * r * scale with r = 1 if pre > 0 else slope,
 *   dQ[v,h,:] = sum_e g * K[e,h,:],  dK[e,h,:] = g * Q[v,h,:].
 * branch (may be NULL) overrides r per (e,h): 0 = by the sign of pre,
 * 1 = take r = 1, 2 = take r = slope. */
void oracle_edge_softmax_bwd(const int32_t* off, int64_t N, int H, int dh,
                             const double* Q, const double* K, double scale,
                             double slope, const double* alpha, const double* dalpha,
                             const int8_t* branch, double* dQ, double* dK);

#ifdef __cplusplus
}
#endif
#endif
