/*
 * fast.h -- C ABI of the MI355X (gfx950) temporal-subgraph operators of FAST
 * (arXiv 2607.05095): the GPU hot path of one temporal-GNN training step.
 *
 *   fast_csr_offsets          CSR ind_ptr of a sampled block          (Sec. 5)
 *   fast_dedup_gather         uni_ID / inv_Idx + row reconstruction   (Sec. 4.2, Sec. 5)
 *   fast_time_encode          cos(omega * dt + phi) time features     (Sec. 6.1, TGAT)
 *   fast_time_encode_bwd      gradients of omega and phi              (Sec. 6.1)
 *   fast_sample_recent        most-recent-k temporal neighbours       (Sec. 6.1, T-CSR)
 *   fast_access_count         pre-sampling access counts              (Sec. 4.2, Alg. 1)
 *   fast_greedy_hot_set       hot ids under a cache budget + slot map (Sec. 4.2, Alg. 1)
 *   fast_edge_softmax_fwd/bwd per-edge multi-head logits + ESM        (Sec. 4.3)
 *   fast_temporal_aggregate_fwd/bwd  attention-weighted AGG           (Sec. 4.3, Eq. 1)
 *   fast_edge_attention_fwd/bwd      ESM and AGG fused in one kernel  (Sec. 4.3)
 *   fast_edge_attention_fwd/bwd_indexed  the same with K/V read through an
 *                             index into de-duplicated rows           (Sec. 4.2)
 *   fast_occurrence_csr, fast_index_add_rows  the gradient of a shared row
 *                             as the ordered sum over its readers     (Sec. 4.2)
 *   fast_edge_attention_bwd_indexed_coef, fast_index_add_scaled_rows  the
 *                             same from per-edge coefficients         (Sec. 4.2, 4.3)
 *
 * Conventions shared by every entry point
 *   - Memory: every array argument is a DEVICE pointer into HBM owned by the
 *     caller.  The library allocates nothing, frees nothing, never
 *     synchronises the stream and keeps no state other than a thread-local
 *     error message.  Scratch memory, where needed, is a caller-provided
 *     workspace whose size the matching *_workspace() query returns.
 *   - Streams: `stream` is a hipStream_t passed as void* (NULL = the null
 *     stream).  Work is enqueued asynchronously; results are valid once the
 *     stream reaches that point.  Calls on one stream run in order.
 *   - Layout: row-major and contiguous.  Per-edge rows [E,H,dh] follow the
 *     CSR edge order; per-destination rows are [N,H,dh].  Per-(edge,head)
 *     scalars (alpha, dalpha) are fp32 [E,H]; per-(destination,head) lse is
 *     fp32 [N,H].  Row storage is FAST_F32 or FAST_BF16 (bfloat16, stored
 *     as round-to-nearest-even; all arithmetic is fp32).
 *   - Errors: problems the host can see (a NULL required pointer, a negative
 *     size, an unsupported shape or dtype, a misaligned pointer, a workspace
 *     that is too small) return a non-zero status BEFORE anything is
 *     enqueued; a failed launch returns FAST_ERR_HIP.  fast_last_error()
 *     then describes the failure.  No C++ exception crosses this boundary.
 *   - Device-data contract: offsets are non-decreasing with off[0] = 0 and
 *     off[N] = E.  Kernels clamp every offset to [0, E], so a malformed
 *     offsets array gives wrong numbers but never an out-of-bounds access.
 *   - Empty inputs (N = 0, E = 0, n = 0) are valid and write the
 *     documented empty-segment values.
 */
#ifndef FAST_H
#define FAST_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FAST_OK = 0,
  FAST_ERR_INVALID_ARG = 1,  /* NULL required pointer, negative size, bad enum */
  FAST_ERR_UNSUPPORTED = 2,  /* shape/dtype/alignment the library does not handle */
  FAST_ERR_WORKSPACE = 3,    /* ws NULL or ws_bytes smaller than the query */
  FAST_ERR_HIP = 4           /* a HIP launch or runtime call failed */
} fast_status_t;

/* FAST_DTYPE_MAX_ENUM widens the enum's range to every non-negative 32-bit
 * value, so that a C caller's out-of-range value reaches the library as a
 * defined value of the type (and is rejected with FAST_ERR_INVALID_ARG) also
 * in C++, where an enum without it could only hold 0 and 1. */
typedef enum { FAST_F32 = 0, FAST_BF16 = 1, FAST_DTYPE_MAX_ENUM = 0x7fffffff } fast_dtype_t;

typedef void* fast_stream_t; /* hipStream_t */

/* A sampled temporal subgraph of one layer block in CSR-by-destination form
 * (Sec. 4.3: CSR for ESM; Sec. 5: the compression triple's ind_ptr).  Edges
 * of destination v are e in [dst_offsets[v], dst_offsets[v+1]).  All
 * pointers are DEVICE pointers; an operator states which fields it reads and
 * the others may be NULL. */
typedef struct fast_tcsr {
  int64_t num_dst;            /* N >= 0 destination segments                   */
  int64_t num_edges;          /* E >= 0 edges, E < 2^31                        */
  const int32_t* dst_offsets; /* [N+1] int32                                   */
  const int64_t* src_ids;     /* [E] source node id per edge (dedup input)     */
  const float* edge_t;        /* [E] edge timestamps                           */
  const int64_t* edge_ids;    /* [E] edge id per edge (dedup input)            */
  const float* dst_t;         /* [N] destination (query) timestamps            */
} fast_tcsr_t;

/* A temporal graph in T-CSR form (the time-sorted CSR of TGL, on which FAST
 * samples, Sec. 6.1 / Sec. 7): node v's entries are p in
 * [indptr[v], indptr[v+1]), each an event of v with neighbour nbr[p] at
 * time ts[p] and edge id eid[p], in non-decreasing time within each node.
 * All pointers are DEVICE pointers. */
typedef struct fast_temporal_graph {
  int64_t num_nodes;          /* V >= 0                                          */
  int64_t num_entries;        /* M >= 0                                          */
  const int64_t* indptr;      /* [V+1] int64, non-decreasing, indptr[V] = M      */
  const int64_t* nbr;         /* [M] neighbour node id                           */
  const float* ts;            /* [M] event time, sorted within each node         */
  const int64_t* eid;         /* [M] edge (event) id                             */
} fast_temporal_graph_t;

/* Message for the last non-OK status returned on the calling thread ("" if
 * none).  The string stays valid until the next failing call on that thread. */
const char* fast_last_error(void);

/* Library version string, e.g. "fast-mi355x 0.1 gfx950". */
const char* fast_version(void);

/* ------------------------------------------------------------------------
 * CSR offsets (Sec. 5: the compression engine's CSR-style ind_ptr).
 *   offsets[0] = 0, offsets[v+1] = offsets[v] + counts[v]   for v < n
 * counts: [n] int32 >= 0, sum < 2^31.  offsets: [n+1] int32.
 * Workspace: fast_csr_offsets_workspace(n) bytes (never 0).
 * ------------------------------------------------------------------------ */
size_t fast_csr_offsets_workspace(int64_t n);
fast_status_t fast_csr_offsets(const int32_t* counts, int64_t n, int32_t* offsets,
                               void* ws, size_t ws_bytes, fast_stream_t stream);

/* The offsets of several blocks (the layer blocks of one sampled batch, Sec. 5)
 * in one pair of launches: for b < nblocks, offsets[b] receives the offsets of
 * counts[b] ([n[b]]), exactly as fast_csr_offsets would.  counts, n and
 * offsets are HOST arrays of nblocks device pointers / sizes.  Up to 8 blocks
 * of at most 2048 * 2048 counts each share the launches; otherwise the blocks
 * are scanned one after another.  nblocks = 0 does nothing.
 * Workspace: fast_csr_offsets_batched_workspace(nblocks, n) bytes (0 on a
 * negative size or a NULL n). */
size_t fast_csr_offsets_batched_workspace(int nblocks, const int64_t* n);
fast_status_t fast_csr_offsets_batched(int nblocks, const int32_t* const* counts,
                                       const int64_t* n, int32_t* const* offsets, void* ws,
                                       size_t ws_bytes, fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Contract check of a sampled subgraph (the device-data contract above).
 * Counts, into violations[0..5) (device int64, overwritten):
 *   [0] v with off[v+1] < off[v]             (non-monotone offsets)
 *   [1] off[0] != 0 or off[N] != E            (0, 1 or 2)
 *   [2] e with src_ids[e] outside [0, src_bound)    (0 if src_ids is NULL)
 *   [3] e with edge_ids[e] outside [0, edge_bound)  (0 if edge_ids is NULL)
 *   [4] e with edge_t[e] > dst_t[v] for its segment v, i.e. dt < 0, counted
 *       only where the offsets are monotone     (0 if a time array is NULL)
 * Reads every field of g that is not NULL; dst_offsets is required.  Any
 * offsets, even malformed ones, are read in bounds.
 * ------------------------------------------------------------------------ */
fast_status_t fast_check_tcsr(const fast_tcsr_t* g, int64_t src_bound, int64_t edge_bound,
                              int64_t* violations, fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Within-batch de-duplication and row reconstruction (Sec. 4.2 SlimCache
 * compression; Sec. 5 uni_ID / inv_Idx).
 *   uni[0..u)   = the distinct values of ids[0..n), ascending
 *   inv[i]      = the k with uni[k] == ids[i]
 *   *num_unique = u                                  (device int64 scalar)
 *   rows[k]     = table[slot(uni[k])] (D elements, bit-exact copy) where
 *                 slot(x) = slot_map ? slot_map[x] : x
 *   miss[0..m)  = ascending k with slot outside [0, table_rows); rows[k] of a
 *                 missed k is left untouched; *num_miss = m (device int64)
 * ids: [n] int64 in [0, id_bound).  An id outside that range is skipped:
 *   it gets inv = -1 and does not enter uni.
 * table: [table_rows, D] of dtype.  slot_map: NULL or [id_bound] int32.
 *   When rows are requested without a slot_map, id_bound must be <= table_rows.
 * Outputs: uni cap n, inv [n], rows cap n*D (or NULL: dedup only, then
 *   table may be NULL), miss cap n (or NULL; *num_miss is still written
 *   when num_miss != NULL).
 * Limits: n < 2^31, id_bound <= 2^35; a row at most 256 vectors of the
 *   widest access (16, 8, 4 or 2 bytes) that D * element size and the table
 *   and rows pointers' alignment allow -- every D <= 256 qualifies; a wider
 *   row returns FAST_ERR_UNSUPPORTED.
 * Workspace: fast_dedup_gather_workspace(n, id_bound) bytes, 256-byte aligned.
 * ------------------------------------------------------------------------ */
size_t fast_dedup_gather_workspace(int64_t n, int64_t id_bound);
fast_status_t fast_dedup_gather(const int64_t* ids, int64_t n, int64_t id_bound,
                                const void* table, int64_t table_rows, int D,
                                fast_dtype_t dtype, const int32_t* slot_map,
                                int64_t* uni, int32_t* inv, int64_t* num_unique,
                                void* rows, int32_t* miss, int64_t* num_miss,
                                void* ws, size_t ws_bytes, fast_stream_t stream);

/* ------------------------------------------------------------------------
 * fast_dedup_gather without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, results and limits as
 * fast_dedup_gather, minus ws/ws_bytes: its scratch is a fixed array of
 * FAST_NOALLOC_SCRATCH_BYTES in the library's device code, one per GPU, held
 * from the library's first use on that GPU until the process ends.  The call
 * allocates and frees nothing.
 *   - Size limit: problems whose fast_dedup_gather_workspace(n, id_bound)
 *     exceeds FAST_NOALLOC_SCRATCH_BYTES return FAST_ERR_UNSUPPORTED before
 *     anything is enqueued (every dedup of the 1e7-node / 2e8-edge batches
 *     fits: at most 86 MB).
 *   - Device: the stream (NULL = the null stream) must belong to the current
 *     device; the scratch of that device is used (FAST_ERR_INVALID_ARG
 *     otherwise).
 *   - Sharing: every call on one GPU uses the same scratch, which keeps the
 *     last call's contents (each call initialises what it reads).  Calls
 *     that overlap on one GPU -- concurrent streams, or host threads without
 *     ordering between their streams -- race on it and give wrong results;
 *     calls on one stream run in order and are safe.
 * ------------------------------------------------------------------------ */
#define FAST_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
fast_status_t fast_dedup_gather_noalloc(const int64_t* ids, int64_t n, int64_t id_bound,
                                        const void* table, int64_t table_rows, int D,
                                        fast_dtype_t dtype, const int32_t* slot_map,
                                        int64_t* uni, int32_t* inv, int64_t* num_unique,
                                        void* rows, int32_t* miss, int64_t* num_miss,
                                        fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Most-recent-k temporal neighbour sampling (Sec. 6.1: top-k recent
 * sampling, k = 10 in the paper's experiments).  Root i is node roots[i]
 * queried at time root_t[i]; its candidates are the entries of that node
 * with ts < root_t[i] (strictly earlier), and its segment of the sampled
 * block holds the LAST min(k, #candidates) of them in entry order (the most
 * recent, oldest first):
 *   dst_offsets[i+1] - dst_offsets[i] = min(k, #candidates),  dst_offsets[0] = 0
 *   src_ids / edge_t / edge_ids of each sampled edge = nbr / ts / eid
 * A root outside [0, V) gets an empty segment.  The result is the sampled
 * block of one layer in the form fast_tcsr_t describes (with dst_t =
 * root_t); a second hop samples (src_ids, edge_t) of the first.
 * roots [R] int64, root_t [R] fp32: device.  Outputs: dst_offsets [R+1]
 * int32 (its last entry is the number of sampled edges E), src_ids and
 * edge_ids int64, edge_t fp32, capacity R * k each.  Offsets that are out of
 * range are clamped, so a malformed graph never causes an out-of-bounds
 * read; entries that are not time-sorted give unspecified neighbours.
 * Limits: 0 <= k, R < 2^31, R * k < 2^31.
 * Workspace: fast_sample_recent_workspace(R) bytes, 256-byte aligned.
 * ------------------------------------------------------------------------ */
size_t fast_sample_recent_workspace(int64_t num_roots);
fast_status_t fast_sample_recent(const fast_temporal_graph_t* g, const int64_t* roots,
                                 const float* root_t, int64_t num_roots, int k,
                                 int32_t* dst_offsets, int64_t* src_ids, float* edge_t,
                                 int64_t* edge_ids, void* ws, size_t ws_bytes,
                                 fast_stream_t stream);

/* ------------------------------------------------------------------------
 * SlimCache access counting over pre-sampled batches (Sec. 4.2, Alg. 1: the
 * counting loop).  For every batch k, each DISTINCT id x of
 *   ids[batch_offsets[k] .. batch_offsets[k+1])
 * with 0 <= x < id_bound adds 1 to freq[x]; a repeat inside a batch counts
 * once, so freq[x] counts the batches that touch x (the transfers a cached
 * row saves once each batch is compressed).  freq is ACCUMULATED into, so
 * batches may be counted over several calls; the caller zeroes it first.
 * ids: device int64; batch_offsets: HOST int64 [num_batches+1],
 * non-decreasing; freq: device int32 [id_bound].  A few launches per batch.
 * Limits: id_bound < 2^32, num_batches < 2^31 - 1.
 * Workspace: fast_access_count_workspace(id_bound) bytes, 16-byte aligned
 *   (a byte of batch bits per id for up to 32 batches, else a batch stamp
 *   per id; for dense universes, id_bound at most 32 times the mean batch
 *   size, the same space holds up to four byte maps, one per batch).
 * ------------------------------------------------------------------------ */
size_t fast_access_count_workspace(int64_t id_bound);
fast_status_t fast_access_count(const int64_t* ids, const int64_t* batch_offsets,
                                int64_t num_batches, int64_t id_bound, int32_t* freq,
                                void* ws, size_t ws_bytes, fast_stream_t stream);

/* ------------------------------------------------------------------------
 * SlimCache greedy selection of the cached ids (Sec. 4.2, Alg. 1: node and
 * edge ids ranked by descending count, ties by ascending id; the two lists
 * merged under the budget, a node taken only when its count is strictly
 * greater than the edge's, an exhausted list never taken).  The result is
 * the first min(budget, num_nodes + num_edges) ids of the combined order
 * (count descending, edges before nodes at equal count, ascending id).
 *   hot_v[0..*num_hot_v)  selected node ids in ASCENDING id order
 *   slot_v[x]             position of node x in hot_v, or -1 (the cache
 *                         slot map read by fast_dedup_gather); optional
 *   hot_e, num_hot_e, slot_e  the same for edges
 * freq_v [num_nodes], freq_e [num_edges]: device int32 counts (from
 * fast_access_count); counts outside [0, max_freq] are clamped into it, so
 * pass max_freq >= the largest count (the number of batches counted).
 * budget: number of ids to cache (fast_hot_set_budget turns Alg. 1's
 * fraction alpha of all ids into it).
 * hot_v capacity min(budget, num_nodes), hot_e min(budget, num_edges); either
 * hot list and slot map may be NULL.  num_hot_v, num_hot_e: device int64.
 * Limits: num_nodes, num_edges < 2^31; 0 <= max_freq <= 2^24.
 * Workspace: fast_greedy_hot_set_workspace(num_nodes, num_edges, max_freq)
 * bytes, 256-byte aligned.
 * ------------------------------------------------------------------------ */
size_t fast_greedy_hot_set_workspace(int64_t num_nodes, int64_t num_edges, int32_t max_freq);
/* The budget of Alg. 1 (Sec. 4.2): its selection loop runs while
 * i + j < alpha * (num_nodes + num_edges), the product evaluated in fp64, so
 * it takes
 *   *budget = min(num_nodes + num_edges, ceil(fl64(alpha * (num_nodes + num_edges))))
 * ids, and 0 when that product is not positive.  A host computation (no
 * device work, no stream); budget is a HOST pointer.  FAST_ERR_INVALID_ARG
 * for a NULL budget, a NaN alpha, or a count outside [0, 2^52]. */
fast_status_t fast_hot_set_budget(double alpha, int64_t num_nodes, int64_t num_edges,
                                  int64_t* budget);
fast_status_t fast_greedy_hot_set(const int32_t* freq_v, int64_t num_nodes, const int32_t* freq_e,
                                  int64_t num_edges, int32_t max_freq, int64_t budget,
                                  int64_t* hot_v, int64_t* num_hot_v, int32_t* slot_v,
                                  int64_t* hot_e, int64_t* num_hot_e, int32_t* slot_e,
                                  void* ws, size_t ws_bytes, fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Time encoding (Sec. 6.1: TGAT's random Fourier time features).
 *   te[e, j] = cos(fmaf(omega[j], dt_e, phi[j])),  dt_e = dst_t[v] - edge_t[e]
 * for e in segment v.  dt and the argument are fp32 (one subtraction, one
 * fused multiply-add); the cosine of that fp32 argument is accurate to better
 * than 1e-6 absolute (exact Cody-Waite reduction, then the hardware cosine on
 * the reduced angle; library cosf beyond |arg| = 2^16).
 * Reads g->dst_offsets, g->dst_t, g->edge_t.  omega, phi: [d_t] fp32 device.
 * te: [E, d_t] of te_dtype.  d_t >= 1.
 * ------------------------------------------------------------------------ */
fast_status_t fast_time_encode(const fast_tcsr_t* g, const float* omega, const float* phi,
                               int d_t, void* te, fast_dtype_t te_dtype,
                               fast_stream_t stream);

/* The time features of several blocks (the layer blocks of one batch share
 * the encoder's omega and phi, Sec. 6.1) in one launch per 8 blocks: te[b]
 * receives exactly what fast_time_encode(g[b], ...) writes.  g and te are
 * HOST arrays of nblocks pointers; every block is checked as by
 * fast_time_encode before anything is launched for its group of 8, and the
 * widest vector width all te[b] allow is used. */
fast_status_t fast_time_encode_batched(int nblocks, const fast_tcsr_t* const* g,
                                       const float* omega, const float* phi, int d_t,
                                       void* const* te, fast_dtype_t te_dtype,
                                       fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Backward of the time encoding (Sec. 6.1: the encoder's frequencies and
 * phases are trained with the model).  For an upstream gradient dte [E, d_t]:
 *   a_ej      = fmaf(omega[j], dt_e, phi[j])       (the forward's fp32 argument)
 *   domega[j] = sum_e dte[e,j] * (-sin a_ej) * dt_e
 *   dphi[j]   = sum_e dte[e,j] * (-sin a_ej)
 * summed over every edge of the block.  The sine of the fp32 argument, the
 * products and the sums are fp64 (results rounded once to fp32), so a column
 * whose terms nearly cancel keeps its accuracy.  Deterministic: the order of
 * the sums depends only on N and d_t, and repeated calls give bitwise-equal
 * results.  domega, dphi: [d_t] fp32 device, overwritten (zeros when E = 0).
 * Reads g->dst_offsets, g->dst_t, g->edge_t.  dte: [E, d_t] of dte_dtype.
 * Limits: 1 <= d_t, and d_t / v <= 256 for the widest v in {8 (bf16 only),
 * 4, 2, 1} that divides d_t and matches dte's alignment (so d_t <= 256
 * always works, and up to 1024 fp32 / 2048 bf16 when divisible by 4 / 8);
 * otherwise FAST_ERR_UNSUPPORTED.
 * Workspace: fast_time_encode_bwd_workspace(N, d_t) bytes, 8-byte aligned.
 * ------------------------------------------------------------------------ */
size_t fast_time_encode_bwd_workspace(int64_t num_dst, int d_t);
fast_status_t fast_time_encode_bwd(const fast_tcsr_t* g, const float* omega, const float* phi,
                                   int d_t, const void* dte, fast_dtype_t dte_dtype,
                                   float* domega, float* dphi, void* ws, size_t ws_bytes,
                                   fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Edge softmax with per-edge multi-head attention logits (Sec. 4.3 "Edge
 * Softmax": a numerically stable max / sum / divide per destination).
 *   pre[e,h]   = scale * <Q[v,h,:], K[e,h,:]>,  s = pre > 0 ? pre : neg_slope*pre
 *   alpha[e,h] = exp(s - m) / Z,  m = max_{e in v} s,  Z = sum_{e in v} exp(s - m)
 *   lse[v,h]   = m + log Z  (-inf for an empty segment; lse may be NULL)
 * Q: [N,H,dh], K: [E,H,dh] of dtype.  alpha: [E,H] fp32.  Reads g->dst_offsets.
 * Supported: every shape with H <= 64, dh <= 256 and H*dh <= 1024; larger
 * shapes return FAST_ERR_UNSUPPORTED when no lane layout fits.  Row pointers
 * must be aligned to the element size.
 * ------------------------------------------------------------------------ */
fast_status_t fast_edge_softmax_fwd(const fast_tcsr_t* g, int H, int dh, fast_dtype_t dtype,
                                    const void* Q, const void* K, float scale,
                                    float neg_slope, float* alpha, float* lse,
                                    fast_stream_t stream);

/* Backward of fast_edge_softmax_fwd for an upstream gradient dalpha [E,H]:
 *   D[v,h] = sum_e alpha*dalpha,  g = alpha*(dalpha - D) * (pre > 0 ? 1 : neg_slope) * scale
 *   dQ[v,h,:] = sum_e g*K[e,h,:]  (0 for an empty segment),  dK[e,h,:] = g*Q[v,h,:]
 * alpha: the forward's output.  dQ: [N,H,dh], dK: [E,H,dh] of dtype. */
fast_status_t fast_edge_softmax_bwd(const fast_tcsr_t* g, int H, int dh, fast_dtype_t dtype,
                                    const void* Q, const void* K, float scale,
                                    float neg_slope, const float* alpha,
                                    const float* dalpha, void* dQ, void* dK,
                                    fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Attention-weighted temporal aggregation (Sec. 4.3 "Balanced Aggregate";
 * Eq. 1 with AGG = sum of alpha-weighted neighbour messages).
 *   out[v,h,:] = sum_{e in v} alpha[e,h] * V[e,h,:]   (0 for an empty segment)
 * Deterministic: each destination row is reduced by one sub-wavefront, no
 * atomics.  alpha: [E,H] fp32; V: [E,H,dh], out: [N,H,dh] of dtype.
 * ------------------------------------------------------------------------ */
fast_status_t fast_temporal_aggregate_fwd(const fast_tcsr_t* g, int H, int dh,
                                          fast_dtype_t dtype, const float* alpha,
                                          const void* V, void* out, fast_stream_t stream);

/* Backward: dalpha[e,h] = <dout[v,h,:], V[e,h,:]>,  dV[e,h,:] = alpha[e,h]*dout[v,h,:].
 * dalpha: [E,H] fp32; dV: [E,H,dh] of dtype. */
fast_status_t fast_temporal_aggregate_bwd(const fast_tcsr_t* g, int H, int dh,
                                          fast_dtype_t dtype, const float* alpha,
                                          const void* V, const void* dout, float* dalpha,
                                          void* dV, fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Fused edge softmax + aggregation (Sec. 4.3 operators in one pass; alpha is
 * never written to memory).  Equals fast_edge_softmax_fwd followed by
 * fast_temporal_aggregate_fwd: out = AGG(ESM(Q,K), V); lse as in ESM (may be
 * NULL).  Q,out: [N,H,dh]; K,V: [E,H,dh] of dtype.
 * ------------------------------------------------------------------------ */
fast_status_t fast_edge_attention_fwd(const fast_tcsr_t* g, int H, int dh, fast_dtype_t dtype,
                                      const void* Q, const void* K, const void* V,
                                      float scale, float neg_slope, void* out, float* lse,
                                      fast_stream_t stream);

/* Backward of the fused operator for dout [N,H,dh]: equals
 * fast_temporal_aggregate_bwd followed by fast_edge_softmax_bwd, with alpha
 * recomputed from Q and K.  lse: the forward's lse, or NULL to recompute the
 * softmax normaliser.  dQ: [N,H,dh]; dK, dV: [E,H,dh] of dtype. */
fast_status_t fast_edge_attention_bwd(const fast_tcsr_t* g, int H, int dh, fast_dtype_t dtype,
                                      const void* Q, const void* K, const void* V,
                                      float scale, float neg_slope, const float* lse,
                                      const void* dout, void* dQ, void* dK, void* dV,
                                      fast_stream_t stream);

/* ------------------------------------------------------------------------
 * The fused operator on packed K|V rows (Sec. 4.3 operators; the per-edge key
 * and value of Eq. 1 side by side, as a fused K|V projection writes them).
 *   KV: [E, 2, H, dh] of dtype: row e is K[e] (F = H*dh elements) followed by
 *   V[e]; dKV: the same layout for dK and dV.
 * Results equal fast_edge_attention_fwd / _bwd on K = KV[:, 0], V = KV[:, 1]
 * bit for bit (same kernels, rows 2F apart), with the same argument rules and
 * errors; K, V and their gradients then move as one stream each way.
 * ------------------------------------------------------------------------ */
fast_status_t fast_edge_attention_fwd_packed(const fast_tcsr_t* g, int H, int dh,
                                             fast_dtype_t dtype, const void* Q, const void* KV,
                                             float scale, float neg_slope, void* out, float* lse,
                                             fast_stream_t stream);
fast_status_t fast_edge_attention_bwd_packed(const fast_tcsr_t* g, int H, int dh,
                                             fast_dtype_t dtype, const void* Q, const void* KV,
                                             float scale, float neg_slope, const float* lse,
                                             const void* dout, void* dQ, void* dKV,
                                             fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Indexed operands (Sec. 4.2: the compressed batch carries each distinct id
 * once plus an inverse index; here the fused operator reads its K and V rows
 * through such an index instead of from a rebuilt per-edge copy).
 *   edge e reads K[k_index[e]] and V[v_index[e]]   (a NULL index: row e)
 * Otherwise identical to fast_edge_attention_fwd / _bwd.  K: [k_rows, H, dh],
 * V: [v_rows, H, dh] of dtype; k_index, v_index: [E] int32 device; an index
 * value outside [0, rows) reads the nearest valid row.  An index requires
 * rows >= 1.  The backward writes the PER-EDGE gradients dK_edge, dV_edge
 * [E, H, dh] (the gradient of each edge's read); the gradient of a shared
 * row is their sum over the edges that read it: build the occurrence lists
 * of the index with fast_occurrence_csr, then fast_index_add_rows.
 * ------------------------------------------------------------------------ */
fast_status_t fast_edge_attention_fwd_indexed(const fast_tcsr_t* g, int H, int dh,
                                              fast_dtype_t dtype, const void* Q, const void* K,
                                              const int32_t* k_index, int64_t k_rows,
                                              const void* V, const int32_t* v_index,
                                              int64_t v_rows, float scale, float neg_slope,
                                              void* out, float* lse, fast_stream_t stream);
fast_status_t fast_edge_attention_bwd_indexed(const fast_tcsr_t* g, int H, int dh,
                                              fast_dtype_t dtype, const void* Q, const void* K,
                                              const int32_t* k_index, int64_t k_rows,
                                              const void* V, const int32_t* v_index,
                                              int64_t v_rows, float scale, float neg_slope,
                                              const float* lse, const void* dout, void* dQ,
                                              void* dK_edge, void* dV_edge, fast_stream_t stream);

/* Occurrence lists of an index (a stable counting sort by index value):
 *   occ_off[u+1] - occ_off[u] = number of p with index[p] == u,  occ_off[0] = 0
 *   occ[occ_off[u] .. occ_off[u+1]) = those positions p, ascending
 * for u in [0, num_rows).  Positions whose index is outside [0, num_rows) are
 * left out: they fill occ from occ_off[num_rows] on.  index: [n] int32
 * device; occ_off: [num_rows+1] int32; occ: [n] int32.  Bit-exact and
 * deterministic.  Limits: n, num_rows < 2^31 - 1.
 * Workspace: fast_occurrence_csr_workspace(n, num_rows) bytes, 256-byte aligned. */
size_t fast_occurrence_csr_workspace(int64_t n, int64_t num_rows);
fast_status_t fast_occurrence_csr(const int32_t* index, int64_t n, int64_t num_rows,
                                  int32_t* occ_off, int32_t* occ, void* ws, size_t ws_bytes,
                                  fast_stream_t stream);

/* Transposed gather: for every row u in [0, num_rows)
 *   dst[u, :] = sum over j in [occ_off[u], occ_off[u+1]) of src[occ[j], :]
 * in that order, accumulated in fp64 and rounded once to fp32 (0 for a row
 * with no occurrence).  Deterministic: rows with many occurrences are split
 * into fixed pieces whose sums are added in piece order.  src: [n, D] of
 * src_dtype (e.g. the per-edge gradients of the indexed backward); dst:
 * [num_rows, D] fp32, overwritten.  occ_off, occ: from fast_occurrence_csr
 * (values are clamped into range, so malformed lists never read out of
 * bounds).  Limits: n, num_rows < 2^31 - 1, D >= 1.
 * Workspace: fast_index_add_rows_workspace(n, num_rows, D) bytes, 256-byte aligned. */
size_t fast_index_add_rows_workspace(int64_t n, int64_t num_rows, int D);
fast_status_t fast_index_add_rows(const int32_t* occ_off, const int32_t* occ, int64_t n,
                                  int64_t num_rows, int D, fast_dtype_t src_dtype,
                                  const void* src, float* dst, void* ws, size_t ws_bytes,
                                  fast_stream_t stream);

/* ------------------------------------------------------------------------
 * Row gradients of indexed operands in coefficient form.  The backward of
 * edge e of segment v is dK_e[h,:] = g[e,h] * Q[v,h,:] and dV_e[h,:] =
 * alpha[e,h] * dout[v,h,:] (Sec. 4.3: the softmax and aggregation backward,
 * g = alpha (dalpha - D) LReLU'(pre) scale), so a shared row's gradient
 * needs only the two coefficients per edge and head, not the per-edge rows:
 *
 * fast_edge_attention_bwd_indexed_coef: as fast_edge_attention_bwd_indexed
 *   (same arguments and dQ), but writes g_edge [E,H] and alpha_edge [E,H]
 *   (fp32, device) in place of dK_edge and dV_edge.
 *
 * fast_index_add_scaled_rows: for every row u,
 *   dst[u,h,:] = sum over the occurrences e of u (occ_off/occ of the index,
 *                from fast_occurrence_csr) of scal[e,h] * src[v,h,:],
 *   v the segment of edge e in dst_offsets [num_dst+1].  dK rows: scal =
 *   g_edge, src = Q, the occurrence lists of k_index; dV rows: scal =
 *   alpha_edge, src = dout, those of v_index.  Products and sums in fp64,
 *   in occurrence order (long rows cut into pieces as fast_index_add_rows
 *   does), rounded once to fp32; dst [num_rows, H, dh] fp32, overwritten.
 *   src [num_dst, H, dh] of src_dtype, scal [n, H] fp32 (n = edges).
 *   Malformed lists or offsets give wrong sums, never out-of-bounds accesses.
 * Limits: n, num_dst < 2^31, num_rows < 2^31 - 1.
 * Workspace: fast_index_add_scaled_rows_workspace(n, num_rows, H, dh) bytes,
 *   256-byte aligned.
 * ------------------------------------------------------------------------ */
fast_status_t fast_edge_attention_bwd_indexed_coef(
    const fast_tcsr_t* g, int H, int dh, fast_dtype_t dtype, const void* Q, const void* K,
    const int32_t* k_index, int64_t k_rows, const void* V, const int32_t* v_index,
    int64_t v_rows, float scale, float neg_slope, const float* lse, const void* dout, void* dQ,
    float* g_edge, float* alpha_edge, fast_stream_t stream);
size_t fast_index_add_scaled_rows_workspace(int64_t n, int64_t num_rows, int H, int dh);
fast_status_t fast_index_add_scaled_rows(const int32_t* occ_off, const int32_t* occ, int64_t n,
                                         int64_t num_rows, const int32_t* dst_offsets,
                                         int64_t num_dst, int H, int dh,
                                         fast_dtype_t src_dtype, const float* scal,
                                         const void* src, float* dst, void* ws,
                                         size_t ws_bytes, fast_stream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* FAST_H */
