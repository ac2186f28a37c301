/*
 * oracle.c -- plain fp64 CPU reference of FAST's temporal-subgraph operators.
 *
 * TEST INFRASTRUCTURE ONLY (see oracle.h).  Written for a reader checking it
 * against the paper by eye: one loop nest per definition, no blocking, no
 * reordering, no fusion.  Build with -ffp-contract=off so that the only fused
 * multiply-add is the explicit fmaf of the time-encoding argument.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ---- CSR offsets (Sec. 5: CSR-style ind_ptr of the compression triple) ---- */
void oracle_csr_offsets(const int32_t* counts, int64_t n, int32_t* off) {
  off[0] = 0;
  for (int64_t v = 0; v < n; ++v) off[v + 1] = off[v] + counts[v];
}

/* ---- contract check of a sampled subgraph ---- */
void oracle_check_tcsr(const int32_t* off, int64_t N, int64_t E, const int64_t* src_ids,
                       int64_t src_bound, const int64_t* edge_ids, int64_t edge_bound,
                       const float* edge_t, const float* dst_t, int64_t* violations) {
  for (int k = 0; k < 5; ++k) violations[k] = 0;
  for (int64_t v = 0; v < N; ++v)
    if (off[v + 1] < off[v]) violations[0] += 1;
  if (off[0] != 0) violations[1] += 1;
  if (off[N] != E) violations[1] += 1;
  for (int64_t e = 0; e < E; ++e) {
    if (src_ids && (src_ids[e] < 0 || src_ids[e] >= src_bound)) violations[2] += 1;
    if (edge_ids && (edge_ids[e] < 0 || edge_ids[e] >= edge_bound)) violations[3] += 1;
  }
  if (edge_t && dst_t)
    for (int64_t v = 0; v < N; ++v) {
      if (off[v + 1] < off[v]) continue;
      for (int64_t e = off[v]; e < off[v + 1]; ++e)
        if (e >= 0 && e < E && edge_t[e] > dst_t[v]) violations[4] += 1;
    }
}

/* ---- within-batch dedup (Sec. 4.2 compression; Sec. 5 uni_ID / inv_Idx) ---- */
static int cmp_i64(const void* a, const void* b) {
  int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
  return (x > y) - (x < y);
}

int64_t oracle_dedup(const int64_t* ids, int64_t n, int64_t* uni, int32_t* inv) {
  if (n == 0) return 0;
  int64_t* sorted = (int64_t*)malloc((size_t)n * sizeof(int64_t));
  memcpy(sorted, ids, (size_t)n * sizeof(int64_t));
  qsort(sorted, (size_t)n, sizeof(int64_t), cmp_i64);
  int64_t u = 0;
  for (int64_t i = 0; i < n; ++i)
    if (i == 0 || sorted[i] != sorted[i - 1]) uni[u++] = sorted[i];
  free(sorted);
  for (int64_t i = 0; i < n; ++i) {          /* lower_bound of ids[i] in uni */
    int64_t lo = 0, hi = u;
    while (lo < hi) {
      int64_t mid = lo + (hi - lo) / 2;
      if (uni[mid] < ids[i]) lo = mid + 1; else hi = mid;
    }
    inv[i] = (int32_t)lo;
  }
  return u;
}

/* ---- row reconstruction through the cache slot map (Sec. 4.2) ---- */
int64_t oracle_gather(const int64_t* uni, int64_t u, const void* table,
                      int64_t table_rows, int64_t row_bytes, const int32_t* slot_map,
                      void* rows, int32_t* miss) {
  int64_t nmiss = 0;
  for (int64_t k = 0; k < u; ++k) {
    int64_t slot = slot_map ? (int64_t)slot_map[uni[k]] : uni[k];
    if (slot >= 0 && slot < table_rows) {
      if (rows)
        memcpy((char*)rows + k * row_bytes, (const char*)table + slot * row_bytes,
               (size_t)row_bytes);
    } else {
      if (miss) miss[nmiss] = (int32_t)k;
      ++nmiss;
    }
  }
  return nmiss;
}

/* ---- time encoding (Sec. 6.1: TGAT random Fourier time features) ---- */
void oracle_time_encode(const int32_t* off, int64_t N, const float* t_dst,
                        const float* t_e, const float* omega, const float* phi,
                        int d_t, double* te) {
  for (int64_t v = 0; v < N; ++v) {
    for (int64_t e = off[v]; e < off[v + 1]; ++e) {
      float dt = t_dst[v] - t_e[e];
      for (int j = 0; j < d_t; ++j) {
        float arg = fmaf(omega[j], dt, phi[j]);
        te[e * d_t + j] = cos((double)arg);
      }
    }
  }
}

/* ---- indexed operands (Sec. 4.2: rows reconstructed through the inverse
 * index of the compressed ids): occurrence lists and the transposed gather ---- */

/* Occurrence lists of an index: row u lists, in ascending order, every
 * position p with index[p] == u (a stable counting sort by index value).
 * Positions whose index lies outside [0, num_rows) are left out. */
void oracle_occurrence_csr(const int32_t* index, int64_t n, int64_t num_rows, int32_t* occ_off,
                           int32_t* occ) {
  for (int64_t u = 0; u <= num_rows; ++u) occ_off[u] = 0;
  for (int64_t p = 0; p < n; ++p)
    if (index[p] >= 0 && index[p] < num_rows) occ_off[index[p] + 1] += 1;
  for (int64_t u = 0; u < num_rows; ++u) occ_off[u + 1] += occ_off[u];
  int32_t* cursor = (int32_t*)malloc((size_t)(num_rows > 0 ? num_rows : 1) * sizeof(int32_t));
  for (int64_t u = 0; u < num_rows; ++u) cursor[u] = occ_off[u];
  for (int64_t p = 0; p < n; ++p)
    if (index[p] >= 0 && index[p] < num_rows) occ[cursor[index[p]]++] = (int32_t)p;
  free(cursor);
}

/* dst[u] = sum of src[p] over the positions p with index[p] == u (the
 * gradient of a row that several positions read), fp64; 0 if none. */
void oracle_index_add_rows(const int32_t* index, int64_t n, int64_t num_rows, int64_t D,
                           const double* src, double* dst) {
  for (int64_t i = 0; i < num_rows * D; ++i) dst[i] = 0.0;
  for (int64_t p = 0; p < n; ++p) {
    if (index[p] < 0 || index[p] >= num_rows) continue;
    for (int64_t j = 0; j < D; ++j) dst[(int64_t)index[p] * D + j] += src[p * D + j];
  }
}

/* dst[u, h, :] = sum over the edges e with index[e] == u of
 * scal[e, h] * src[v, h, :], v the destination segment of e (off): the
 * gradient of a shared K or V row written as the per-edge coefficient times
 * the row of the segment that edge belongs to (chain rule through the
 * gather; Sec. 4.3 backward), fp64; 0 for a row no edge reads. */
void oracle_index_add_scaled_rows(const int32_t* index, const int32_t* off, int64_t N,
                                  int64_t num_rows, int64_t H, int64_t dh, const double* scal,
                                  const double* src, double* dst) {
  const int64_t D = H * dh;
  for (int64_t i = 0; i < num_rows * D; ++i) dst[i] = 0.0;
  for (int64_t v = 0; v < N; ++v)
    for (int64_t e = off[v]; e < off[v + 1]; ++e) {
      if (index[e] < 0 || index[e] >= num_rows) continue;
      for (int64_t h = 0; h < H; ++h)
        for (int64_t j = 0; j < dh; ++j)
          dst[(int64_t)index[e] * D + h * dh + j] += scal[e * H + h] * src[v * D + h * dh + j];
    }
}

/* ---- most-recent-k temporal neighbour sampling (Sec. 6.1: top-k recent
 * sampling over the T-CSR temporal graph) ---- */
void oracle_sample_recent(const int64_t* indptr, int64_t num_nodes, const int64_t* nbr,
                          const float* ts, const int64_t* eid, const int64_t* roots,
                          const float* root_t, int64_t R, int k, int32_t* off, int64_t* src,
                          float* et, int64_t* ei) {
  int64_t e = 0;
  off[0] = 0;
  for (int64_t i = 0; i < R; ++i) {
    int64_t v = roots[i];
    if (v >= 0 && v < num_nodes) {
      /* candidates: the node's entries strictly earlier than the query time */
      int64_t c = 0;
      for (int64_t p = indptr[v]; p < indptr[v + 1]; ++p)
        if (ts[p] < root_t[i]) c += 1;
      /* keep the last k of them in entry order, i.e. drop the c - k first */
      int64_t skip = c > k ? c - k : 0;
      for (int64_t p = indptr[v]; p < indptr[v + 1]; ++p) {
        if (!(ts[p] < root_t[i])) continue;
        if (skip > 0) {
          skip -= 1;
          continue;
        }
        src[e] = nbr[p];
        et[e] = ts[p];
        ei[e] = eid[p];
        e += 1;
      }
    }
    off[i + 1] = (int32_t)e;
  }
}

/* ---- SlimCache greedy cache selection (Sec. 4.2, Alg. 1) ---- */

/* Counting step: for every batch, each distinct id of the batch adds 1 to its
 * counter, so freq[x] is the number of batches that touch x.  Ids outside
 * [0, id_bound) are ignored. */
void oracle_access_count(const int64_t* ids, const int64_t* batch_off, int64_t num_batches,
                         int64_t id_bound, int32_t* freq) {
  for (int64_t k = 0; k < num_batches; ++k) {
    int64_t n = batch_off[k + 1] - batch_off[k];
    if (n <= 0) continue;
    int64_t* b = (int64_t*)malloc((size_t)n * sizeof(int64_t));
    memcpy(b, ids + batch_off[k], (size_t)n * sizeof(int64_t));
    qsort(b, (size_t)n, sizeof(int64_t), cmp_i64);
    for (int64_t i = 0; i < n; ++i) {
      if (i > 0 && b[i] == b[i - 1]) continue;          /* distinct ids only */
      if (b[i] >= 0 && b[i] < id_bound) freq[b[i]] += 1;
    }
    free(b);
  }
}

typedef struct { int32_t f; int64_t id; } freq_id_t;

/* descending frequency, then ascending id */
static int cmp_freq_desc(const void* a, const void* b) {
  const freq_id_t* x = (const freq_id_t*)a;
  const freq_id_t* y = (const freq_id_t*)b;
  if (x->f != y->f) return x->f > y->f ? -1 : 1;
  return (x->id > y->id) - (x->id < y->id);
}

static freq_id_t* ranked(const int32_t* f, int64_t n) {
  freq_id_t* s = (freq_id_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(freq_id_t));
  for (int64_t i = 0; i < n; ++i) {
    s[i].f = f[i];
    s[i].id = i;
  }
  qsort(s, (size_t)n, sizeof(freq_id_t), cmp_freq_desc);
  return s;
}

/* Selection step: rank node and edge ids by frequency, then take the more
 * frequent head of the two lists while i + j < alpha * (|V| + |E|); a node
 * wins only with a strictly higher count, and an exhausted list never wins.
 * hot_v / hot_e receive the selected ids in selection order. */
void oracle_greedy_hot_set(const int32_t* fv, int64_t nv, const int32_t* fe, int64_t ne,
                           double alpha, int64_t* hot_v, int64_t* n_hot_v, int64_t* hot_e,
                           int64_t* n_hot_e) {
  freq_id_t* sv = ranked(fv, nv);
  freq_id_t* se = ranked(fe, ne);
  int64_t i = 0, j = 0;
  while ((double)(i + j) < alpha * (double)(nv + ne) && i + j < nv + ne) {
    int take_node;
    if (i >= nv) take_node = 0;
    else if (j >= ne) take_node = 1;
    else take_node = sv[i].f > se[j].f;
    if (take_node) {
      hot_v[i] = sv[i].id;
      i += 1;
    } else {
      hot_e[j] = se[j].id;
      j += 1;
    }
  }
  *n_hot_v = i;
  *n_hot_e = j;
  free(sv);
  free(se);
}

/* ---- time-encoding backward (the Sec. 6.1 time features are trainable):
 * the gradient of cos(omega_j * dt + phi_j) taken at the forward's fp32
 * argument, summed over every edge in fp64 ---- */
void oracle_time_encode_bwd(const int32_t* off, int64_t N, const float* t_dst,
                            const float* t_e, const float* omega, const float* phi,
                            int d_t, const double* dte, double* domega, double* dphi) {
  for (int j = 0; j < d_t; ++j) {
    domega[j] = 0.0;
    dphi[j] = 0.0;
  }
  for (int64_t v = 0; v < N; ++v) {
    for (int64_t e = off[v]; e < off[v + 1]; ++e) {
      float dt = t_dst[v] - t_e[e];
      for (int j = 0; j < d_t; ++j) {
        float arg = fmaf(omega[j], dt, phi[j]);
        double dcos = -sin((double)arg);          /* d cos(a) / da */
        dphi[j] += dte[e * d_t + j] * dcos;
        domega[j] += dte[e * d_t + j] * dcos * (double)dt;
      }
    }
  }
}

/* ---- edge softmax forward (Sec. 4.3 "Edge Softmax": max, sum, divide) ---- */
void oracle_edge_softmax_fwd(const int32_t* off, int64_t N, int H, int dh,
                             const double* Q, const double* K, double scale,
                             double slope, double* pre, double* alpha, double* lse) {
  for (int64_t v = 0; v < N; ++v) {
    int64_t e0 = off[v], e1 = off[v + 1];
    for (int h = 0; h < H; ++h) {
      if (e0 == e1) {
        if (lse) lse[v * H + h] = -INFINITY;
        continue;
      }
      /* logits, kept in alpha until normalised */
      for (int64_t e = e0; e < e1; ++e) {
        double dot = 0.0;
        for (int i = 0; i < dh; ++i)
          dot += Q[(v * H + h) * dh + i] * K[(e * H + h) * dh + i];
        double p = scale * dot;
        if (pre) pre[e * H + h] = p;
        alpha[e * H + h] = p > 0.0 ? p : slope * p;
      }
      double m = -INFINITY;
      for (int64_t e = e0; e < e1; ++e)
        if (alpha[e * H + h] > m) m = alpha[e * H + h];
      double Z = 0.0;
      for (int64_t e = e0; e < e1; ++e) Z += exp(alpha[e * H + h] - m);
      for (int64_t e = e0; e < e1; ++e)
        alpha[e * H + h] = exp(alpha[e * H + h] - m) / Z;
      if (lse) lse[v * H + h] = m + log(Z);
    }
  }
}

/* ---- aggregation forward (Sec. 4.3 "Balanced Aggregate"; Eq. 1) ---- */
void oracle_aggregate_fwd(const int32_t* off, int64_t N, int H, int dh,
                          const double* alpha, const double* V, double* out) {
  for (int64_t v = 0; v < N; ++v)
    for (int h = 0; h < H; ++h)
      for (int i = 0; i < dh; ++i) {
        double acc = 0.0;
        for (int64_t e = off[v]; e < off[v + 1]; ++e)
          acc += alpha[e * H + h] * V[(e * H + h) * dh + i];
        out[(v * H + h) * dh + i] = acc;
      }
}

/* ---- aggregation backward ---- */
void oracle_aggregate_bwd(const int32_t* off, int64_t N, int H, int dh,
                          const double* alpha, const double* V, const double* dout,
                          double* dalpha, double* dV) {
  for (int64_t v = 0; v < N; ++v)
    for (int64_t e = off[v]; e < off[v + 1]; ++e)
      for (int h = 0; h < H; ++h) {
        double dot = 0.0;
        for (int i = 0; i < dh; ++i)
          dot += dout[(v * H + h) * dh + i] * V[(e * H + h) * dh + i];
        dalpha[e * H + h] = dot;
        for (int i = 0; i < dh; ++i)
          dV[(e * H + h) * dh + i] = alpha[e * H + h] * dout[(v * H + h) * dh + i];
      }
}

/* ---- edge softmax and logit backward ---- */
void oracle_edge_softmax_bwd(const int32_t* off, int64_t N, int H, int dh,
                             const double* Q, const double* K, double scale,
                             double slope, const double* alpha, const double* dalpha,
                             const int8_t* branch, double* dQ, double* dK) {
  for (int64_t v = 0; v < N; ++v) {
    int64_t e0 = off[v], e1 = off[v + 1];
    for (int h = 0; h < H; ++h) {
      double D = 0.0;
      for (int64_t e = e0; e < e1; ++e) D += alpha[e * H + h] * dalpha[e * H + h];
      for (int i = 0; i < dh; ++i) dQ[(v * H + h) * dh + i] = 0.0;
      for (int64_t e = e0; e < e1; ++e) {
        double dot = 0.0;
        for (int i = 0; i < dh; ++i)
          dot += Q[(v * H + h) * dh + i] * K[(e * H + h) * dh + i];
        double p = scale * dot;
        int b = branch ? branch[e * H + h] : 0;
        double r = (b == 1) ? 1.0 : (b == 2) ? slope : (p > 0.0 ? 1.0 : slope);
        double g = alpha[e * H + h] * (dalpha[e * H + h] - D) * r * scale;
        for (int i = 0; i < dh; ++i) {
          dQ[(v * H + h) * dh + i] += g * K[(e * H + h) * dh + i];
          dK[(e * H + h) * dh + i] = g * Q[(v * H + h) * dh + i];
        }
      }
    }
  }
}
