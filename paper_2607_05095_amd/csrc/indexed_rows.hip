// indexed_rows.hip -- the two reductions that indexed operands need (Sec. 4.2:
// many positions of a batch read one de-duplicated row through the inverse
// index; the gradient of that row is the sum over those positions).
//
// fast_occurrence_csr: for every row, its positions in ascending order -- a
// stable counting sort of the index, done as an LSD radix sort of (key,
// position) pairs over 8-bit digits.  Each pass: per-tile digit histograms,
// one scan of the (digit, tile) counts, and a scatter in which every item
// finds its rank among the tile's items with the same digit from 8 wave
// ballots, in position order -- stable, so after the last pass each row's
// positions are ascending.  Positions whose index is outside the row range
// get the key num_rows and sort behind every valid one.
//
// fast_index_add_rows: dst[u] = sum of src rows over the occurrences of u,
// in occurrence order, accumulated in fp64 and rounded once to fp32.  A row
// with at most IA_PIECE occurrences is summed by one group of lanes; a row
// read by more positions (a hub id of a skewed batch) is summed as a fixed
// three-level tree: pieces of consecutive occurrences, each summed by its own
// group, then (when there are many pieces) groups of consecutive piece sums,
// then the row adds its group (or piece) sums in order -- each level about
// cbrt(count) long, so no group walks a long chain of dependent loads.  The
// tree depends only on the counts, so the result is the same on every run.
#include "scan.h"

namespace fast {

// ------------------------------------------------------------------ radix sort
constexpr int RS_THREADS = 256;
constexpr int RS_WAVES = RS_THREADS / 64;
constexpr int RS_ROUNDS = 8;                        // 64-item rounds per wave
constexpr int RS_TILE = RS_THREADS * RS_ROUNDS;     // 2048 items per tile
constexpr int RS_DIGITS = 256;

inline int64_t rs_tiles(int64_t n) { return (n + RS_TILE - 1) / RS_TILE; }

// Key and value of item i: in the first pass the key comes from the index
// (num_rows for a position outside the row range) and the value is i.
struct RsSrc {
  const int32_t* index;   // first pass
  const int32_t* keys;    // later passes
  const int32_t* vals;
  int32_t num_rows;
  __device__ void get(int64_t i, uint32_t& k, int32_t& v) const {
    if (index) {
      const int32_t x = index[i];
      k = (x >= 0 && x < num_rows) ? uint32_t(x) : uint32_t(num_rows);
      v = int32_t(i);
    } else {
      k = uint32_t(keys[i]);
      v = vals[i];
    }
  }
};

// Items of a tile: wave w takes items [w*512, (w+1)*512) in rounds of 64
// consecutive items, so (wave, round, lane) order is position order.
__device__ __forceinline__ int64_t rs_item(int64_t tile, int w, int r, int lane) {
  return tile * RS_TILE + int64_t(w) * (RS_ROUNDS * 64) + r * 64 + lane;
}

// Lanes of the wave holding the same digit as this lane (inactive lanes excluded).
__device__ __forceinline__ uint64_t digit_match(uint32_t d, bool valid) {
  uint64_t m = __ballot(valid);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const bool bit = (d >> b) & 1u;
    const uint64_t bal = __ballot(bit);
    m &= bit ? bal : ~bal;
  }
  return m;
}

// hist[d * T + tile] = items of the tile whose digit is d.
__global__ void __launch_bounds__(RS_THREADS) k_rs_hist(RsSrc src, int64_t n, int shift,
                                                       uint32_t* hist, int64_t T) {
  __shared__ uint32_t s_h[RS_DIGITS];
  s_h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t tile = blockIdx.x;
#pragma unroll
  for (int k = 0; k < RS_ROUNDS; ++k) {
    const int64_t i = tile * RS_TILE + int64_t(k) * RS_THREADS + threadIdx.x;
    if (i < n) {
      uint32_t key;
      int32_t v;
      src.get(i, key, v);
      atomicAdd(&s_h[(key >> shift) & 255u], 1u);
    }
  }
  __syncthreads();
  hist[int64_t(threadIdx.x) * T + tile] = s_h[threadIdx.x];
}

// base[d * T + tile] (after the scan) = first output slot of the tile's
// items with digit d.  Writes keys (unless NULL) and values.
__global__ void __launch_bounds__(RS_THREADS) k_rs_scatter(RsSrc src, int64_t n, int shift,
                                                          const uint32_t* base, int64_t T,
                                                          int32_t* keys_out, int32_t* vals_out) {
  __shared__ uint32_t s_cnt[RS_WAVES][RS_DIGITS];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t tile = blockIdx.x;
  const uint64_t lt = (uint64_t(1) << lane) - 1;
#pragma unroll
  for (int j = 0; j < RS_WAVES; ++j) s_cnt[j][threadIdx.x] = 0;
  __syncthreads();
  // A: counts per (wave, digit)
  for (int r = 0; r < RS_ROUNDS; ++r) {
    const int64_t i = rs_item(tile, w, r, lane);
    const bool valid = i < n;
    uint32_t key = 0;
    int32_t v = 0;
    if (valid) src.get(i, key, v);
    const uint32_t d = (key >> shift) & 255u;
    const uint64_t m = digit_match(d, valid);
    if (valid && (m & lt) == 0) s_cnt[w][d] += uint32_t(__popcll(m));   // lowest lane of its digit
  }
  __syncthreads();
  // exclusive prefix over the waves, per digit
  {
    uint32_t run = 0;
#pragma unroll
    for (int j = 0; j < RS_WAVES; ++j) {
      const uint32_t c = s_cnt[j][threadIdx.x];
      s_cnt[j][threadIdx.x] = run;
      run += c;
    }
  }
  __syncthreads();
  // B: rank inside the tile and scatter
  for (int r = 0; r < RS_ROUNDS; ++r) {
    const int64_t i = rs_item(tile, w, r, lane);
    const bool valid = i < n;
    uint32_t key = 0;
    int32_t v = 0;
    if (valid) src.get(i, key, v);
    const uint32_t d = (key >> shift) & 255u;
    const uint64_t m = digit_match(d, valid);
    const uint32_t before = s_cnt[w][d];
    if (valid) {
      const int64_t pos = int64_t(base[int64_t(d) * T + tile]) + before + uint32_t(__popcll(m & lt));
      if (keys_out) keys_out[pos] = int32_t(key);
      vals_out[pos] = v;
    }
    if (valid && (m & lt) == 0) s_cnt[w][d] = before + uint32_t(__popcll(m));
  }
}

struct InU32 {
  const uint32_t* p;
  __device__ uint32_t operator()(int64_t i) const { return p[i]; }
};
struct OutU32InPlace {
  uint32_t* p;
  __device__ void operator()(int64_t i, uint32_t prefix, uint32_t) const { p[i] = prefix; }
};

// occ_off[u] = number of sorted keys below u (a lower bound in the sorted
// keys; positions outside the row range carry the key num_rows), u in
// [0, num_rows].  No atomics: a hub row's count costs nothing extra.
__global__ void __launch_bounds__(RS_THREADS) k_occ_offsets(const int32_t* __restrict__ keys,
                                                           int64_t n, int64_t num_rows,
                                                           int32_t* __restrict__ occ_off) {
  const int64_t u = int64_t(blockIdx.x) * RS_THREADS + threadIdx.x;
  if (u > num_rows) return;
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if (int64_t(keys[mid]) < u) lo = mid + 1; else hi = mid;
  }
  occ_off[u] = int32_t(lo);
}


__global__ void __launch_bounds__(RS_THREADS) k_ir_fill(int32_t* p, int64_t n, int32_t v) {
  for (int64_t i = int64_t(blockIdx.x) * RS_THREADS + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * RS_THREADS)
    p[i] = v;
}

struct OccWs {
  int32_t* keys[2];
  int32_t* vals[2];
  uint32_t* hist;
  void* scan_h;
};

static size_t occ_layout(int64_t n, int64_t num_rows, char* base, OccWs* ws) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes, 256);
    return base ? base + o : nullptr;
  };
  const int64_t T = rs_tiles(n);
  char* k0 = take(size_t(n) * 4);
  char* k1 = take(size_t(n) * 4);
  char* v0 = take(size_t(n) * 4);
  char* v1 = take(size_t(n) * 4);
  char* h = take(size_t(T) * RS_DIGITS * 4);
  char* sh = take(scan_workspace(T * RS_DIGITS));
  if (ws) {
    ws->keys[0] = reinterpret_cast<int32_t*>(k0);
    ws->keys[1] = reinterpret_cast<int32_t*>(k1);
    ws->vals[0] = reinterpret_cast<int32_t*>(v0);
    ws->vals[1] = reinterpret_cast<int32_t*>(v1);
    ws->hist = reinterpret_cast<uint32_t*>(h);
    ws->scan_h = sh;
  }
  return off;
}

static uint32_t grid_cap(int64_t n, int64_t per, uint32_t cap = 8192) {
  int64_t g = (n + per - 1) / per;
  if (g < 1) g = 1;
  return uint32_t(g < cap ? g : cap);
}

// ------------------------------------------------------------------ index add
constexpr int IA_THREADS = 256;
constexpr int IA_PIECE = 64;   // occurrences summed by one group
constexpr int IA_UNROLL = 4;   // rows in flight per lane

constexpr int IA_GROUP_MIN = 16;   // fewest pieces per group of the second level

// The smallest power of two p >= lo with p^3 >= c (c < 2^31: p <= 2048).
__device__ __forceinline__ int64_t ia_cbrt_pow2(int64_t c, int64_t lo) {
  int64_t p = lo;
  while (p * p * p < c) p <<= 1;
  return p;
}
// Tree of a row with c > IA_PIECE occurrences: pieces of ia_piece_len(c)
// occurrences and, when there are more than ia_group_len(c) pieces, groups of
// that many consecutive pieces.  For c = 3e5 (a hub of the 1e7-node batch):
// 2344 pieces of 128, 19 groups of 128 pieces.  Functions of c alone.
__device__ __forceinline__ int64_t ia_piece_len(int64_t c) { return ia_cbrt_pow2(c, IA_PIECE); }
__device__ __forceinline__ int64_t ia_group_len(int64_t c) { return ia_cbrt_pow2(c, IA_GROUP_MIN); }

// Pieces of a row (0 for c <= IA_PIECE, which one group sums directly); at
// most 2 c / IA_PIECE.
__device__ __forceinline__ int64_t ia_multi_pieces(int64_t c) {
  if (c <= IA_PIECE) return 0;
  const int64_t p = ia_piece_len(c);
  return (c + p - 1) / p;
}
// Groups of the second level (0 when the row has at most ia_group_len(c)
// pieces); at most 2 pieces / IA_GROUP_MIN.
__device__ __forceinline__ int64_t ia_multi_groups(int64_t c) {
  const int64_t m = ia_multi_pieces(c), g = ia_group_len(c);
  return m > g ? (m + g - 1) / g : 0;
}

// Both counts of row u in one 64-bit item (pieces high, groups low) for one
// scan; item num_rows is 0, so the prefix at num_rows is the pair of totals.
struct InMulti {
  const int32_t* occ_off;
  int64_t n, num_rows;
  __device__ uint64_t operator()(int64_t u) const {
    if (u >= num_rows) return 0u;
    const int64_t c = clamp64(int64_t(occ_off[u + 1]) - occ_off[u], 0, n);
    return (uint64_t(ia_multi_pieces(c)) << 32) | uint64_t(ia_multi_groups(c));
  }
};
struct OutMulti {
  int32_t* multi_off;
  int32_t* group_off;
  __device__ void operator()(int64_t u, uint64_t prefix, uint64_t) const {
    multi_off[u] = int32_t(prefix >> 32);
    group_off[u] = int32_t(prefix & 0xffffffffu);
  }
};

// acc += fp64 rows part[m0 .. m1) (chunk c of VE values, rows of D), in
// order, U rows loaded before they are added.
template <int VE, int U>
__device__ __forceinline__ void ia_sum_partials(const double* __restrict__ part, int64_t m0,
                                                int64_t m1, int D, int c, double (&acc)[VE]) {
  int64_t m = m0;
  for (; m + U <= m1; m += U) {
    double x[U][VE];
#pragma unroll
    for (int r = 0; r < U; ++r)
#pragma unroll
      for (int t = 0; t < VE; ++t) x[r][t] = part[(m + r) * D + c * VE + t];
#pragma unroll
    for (int r = 0; r < U; ++r)
#pragma unroll
      for (int t = 0; t < VE; ++t) acc[t] += x[r][t];
  }
  for (; m < m1; ++m)
#pragma unroll
    for (int t = 0; t < VE; ++t) acc[t] += part[m * D + c * VE + t];
}

// Eight fp32 values of a row sum (the bf16 sources' widest vector).
template <> struct VecIO<float, 8> {
  __device__ static void store(float* p, const float* x) {
    VecIO<float, 4>::store(p, x);
    VecIO<float, 4>::store(p + 4, x + 4);
  }
};

// Row sources of the index-add kernels.  Occurrence j (position p = occ[j])
// contributes, to chunk c (VE values) of its row's sum:
//   PlainRows:  src row p;
//   ScaledRows: coefficient seg_scal[j, head] times src row occ_seg[j] --
//               the coefficient of edge p and the destination segment it
//               belongs to, laid out in occurrence order by k_coef_permute,
//               one head coefficient per element (a chunk spans at most two
//               heads, since VE <= dh).
// Products are formed in fp64 (exact for fp32 factors), sums in fp64.
template <typename T, int VE>
struct PlainRows {
  // rows in flight per lane in the pieces of long rows, whose sums are
  // chains of up to a thousand occurrences: 16 took the hub rows of the
  // 1e7-node batch's layer-1 block (up to 3.1e5 occurrences) from 0.54 to
  // 0.45 ms; the scaled source holds two coefficients more per row and
  // stays at 4 (8 and 16 were slower there)
  static constexpr int PIECE_UNROLL = 16;
  const T* __restrict__ src;
  int D;
  int64_t n;
  struct Item {
    float x[VE];
  };
  __device__ void chunk(int) {}
  __device__ Item fetch(const int32_t* __restrict__ occ, int64_t j, int c) const {
    // each source row is read once per call: streaming (non-temporal)
    // loads, as for the output rows below (1e7-node batch, K / V indices 0.41 /
    // 0.43 -> 0.39 / 0.41 ms; the large batch's V index 1.30 -> 1.21 ms)
    Item it;
    Raw<T, VE> r;
    r.template load<true>(src + clamp64(occ[j], 0, n - 1) * D + c * VE);
    r.unpack(it.x);
    return it;
  }
  __device__ void add(double (&acc)[VE], const Item& it) const {
#pragma unroll
    for (int t = 0; t < VE; ++t) acc[t] += double(it.x[t]);
  }
};

template <typename T, int VE>
struct ScaledRows {
  static constexpr int PIECE_UNROLL = IA_UNROLL;
  const T* __restrict__ src;          // [N, H, dh]
  const float* __restrict__ occ_scal; // [n, H], occurrence order
  const int32_t* __restrict__ occ_seg;// [n], occurrence order
  int D, H, dh;
  int64_t N;
  int h0, h1, split;                  // heads of the chunk; elements t < split use h0
  struct Item {
    float x[VE];
    float s0, s1;
  };
  __device__ void chunk(int c) {
    const int c0 = c * VE;
    h0 = c0 / dh;
    h1 = (c0 + VE - 1) / dh;
    split = (h0 + 1) * dh - c0;
  }
  __device__ Item fetch(const int32_t* __restrict__, int64_t j, int c) const {
    const int64_t v = clamp64(occ_seg[j], 0, N - 1);
    Item it;
    VecIO<T, VE>::load(src + v * D + c * VE, it.x);
    it.s0 = occ_scal[j * H + h0];
    it.s1 = occ_scal[j * H + h1];
    return it;
  }
  __device__ void add(double (&acc)[VE], const Item& it) const {
#pragma unroll
    for (int t = 0; t < VE; ++t) acc[t] = fma(double(t < split ? it.s0 : it.s1), double(it.x[t]), acc[t]);
  }
};

// acc += the contributions of positions occ[j0 .. j1) in order, chunk c;
// IA_UNROLL positions are fetched before they are added (in the same order).
template <int VE, class Src, int U = IA_UNROLL>
__device__ __forceinline__ void ia_sum(const int32_t* __restrict__ occ, int64_t j0, int64_t j1,
                                       int c, const Src& src, double (&acc)[VE]) {
  int64_t j = j0;
  for (; j + U <= j1; j += U) {
    typename Src::Item x[U];
#pragma unroll
    for (int r = 0; r < U; ++r) x[r] = src.fetch(occ, j + r, c);
#pragma unroll
    for (int r = 0; r < U; ++r) src.add(acc, x[r]);
  }
  for (; j < j1; ++j) src.add(acc, src.fetch(occ, j, c));
}

// Pieces of the long rows: one group of `lanes` lanes per piece q in
// [0, multi_off[num_rows]); its sum goes to partial[q].
template <int VE, class Src>
__global__ void __launch_bounds__(IA_THREADS) k_ia_pieces(
    const int32_t* __restrict__ occ_off, const int32_t* __restrict__ occ,
    const int32_t* __restrict__ multi_off, int64_t num_rows, int64_t multi_bound, int64_t n,
    int lanes, int D, Src src, double* __restrict__ partial) {
  const int64_t q = (int64_t(blockIdx.x) * IA_THREADS + threadIdx.x) / lanes;
  const int l = int(threadIdx.x) % lanes;
  if (q >= multi_bound || q >= multi_off[num_rows]) return;
  // the long row u with multi_off[u] <= q < multi_off[u + 1]
  int64_t lo = 0, hi = num_rows - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (multi_off[mid] <= q) lo = mid; else hi = mid - 1;
  }
  const int64_t u = lo, k = q - multi_off[u];
  // offsets and positions are clamped into range, so malformed occurrence
  // lists give wrong sums but never an out-of-bounds access
  const int64_t r0 = clamp64(occ_off[u], 0, n);
  const int64_t r1 = clamp64(occ_off[u + 1], r0, n);
  const int64_t len = ia_piece_len(r1 - r0);
  const int64_t j0 = clamp64(r0 + k * len, r0, r1);
  const int64_t j1 = j0 + len < r1 ? j0 + len : r1;
  const int chunks = D / VE;
  for (int c = l; c < chunks; c += lanes) {
    src.chunk(c);
    double acc[VE];
#pragma unroll
    for (int t = 0; t < VE; ++t) acc[t] = 0.0;
    ia_sum<VE, Src, Src::PIECE_UNROLL>(occ, j0, j1, c, src, acc);
#pragma unroll
    for (int t = 0; t < VE; ++t) partial[q * D + c * VE + t] = acc[t];
  }
}

// Second level of the long rows: one group of `lanes` lanes per group g in
// [0, group_off[num_rows]) of ia_group_len(c) consecutive piece sums, added
// in piece order into partial2[g].
template <int VE>
__global__ void __launch_bounds__(IA_THREADS) k_ia_groups(
    const int32_t* __restrict__ occ_off, const int32_t* __restrict__ multi_off,
    const int32_t* __restrict__ group_off, int64_t num_rows, int64_t multi_bound,
    int64_t group_bound, int64_t n, int lanes, int D, const double* __restrict__ partial,
    double* __restrict__ partial2) {
  const int64_t g = (int64_t(blockIdx.x) * IA_THREADS + threadIdx.x) / lanes;
  const int l = int(threadIdx.x) % lanes;
  if (g >= group_bound || g >= group_off[num_rows]) return;
  // the long row u with group_off[u] <= g < group_off[u + 1]
  int64_t lo = 0, hi = num_rows - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (group_off[mid] <= g) lo = mid; else hi = mid - 1;
  }
  const int64_t u = lo, k = g - group_off[u];
  const int64_t r0 = clamp64(occ_off[u], 0, n);
  const int64_t r1 = clamp64(occ_off[u + 1], r0, n);
  const int64_t len = ia_group_len(r1 - r0);
  const int64_t p0 = clamp64(multi_off[u], 0, multi_bound);
  const int64_t p1 = clamp64(multi_off[u + 1], p0, multi_bound);
  const int64_t m0 = clamp64(p0 + k * len, p0, p1);
  const int64_t m1 = m0 + len < p1 ? m0 + len : p1;
  const int chunks = D / VE;
  for (int c = l; c < chunks; c += lanes) {
    double acc[VE];
#pragma unroll
    for (int t = 0; t < VE; ++t) acc[t] = 0.0;
    ia_sum_partials<VE, 8>(partial, m0, m1, D, c, acc);
#pragma unroll
    for (int t = 0; t < VE; ++t) partial2[g * D + c * VE + t] = acc[t];
  }
}

// One group per row: a short row sums its occurrences directly (zeros for
// none), a long row adds its group sums (or, with few pieces, its piece sums)
// in order.  fp64 sums, rounded once to fp32.
template <int VE, class Src>
__global__ void __launch_bounds__(IA_THREADS) k_ia_rows(
    const int32_t* __restrict__ occ_off, const int32_t* __restrict__ occ,
    const int32_t* __restrict__ multi_off, const int32_t* __restrict__ group_off,
    int64_t num_rows, int64_t multi_bound, int64_t group_bound, int64_t n, int lanes, int D,
    Src src, const double* __restrict__ partial, const double* __restrict__ partial2,
    float* __restrict__ dst) {
  const int64_t u = (int64_t(blockIdx.x) * IA_THREADS + threadIdx.x) / lanes;
  const int l = int(threadIdx.x) % lanes;
  if (u >= num_rows) return;
  const int64_t j0 = clamp64(occ_off[u], 0, n);
  const int64_t j1 = clamp64(occ_off[u + 1], j0, n);
  // piece and group ranges clamped too: the counts of malformed lists may wrap
  const int64_t m0 = clamp64(multi_off[u], 0, multi_bound);
  const int64_t m1 = clamp64(multi_off[u + 1], m0, multi_bound);
  const int64_t g0 = clamp64(group_off[u], 0, group_bound);
  const int64_t g1 = clamp64(group_off[u + 1], g0, group_bound);
  const bool longrow = ia_multi_pieces(j1 - j0) > 0;
  // a long row's sums of the level below: its groups, or its pieces
  const bool grouped = g1 > g0;
  const double* __restrict__ part = grouped ? partial2 : partial;
  const int64_t p0 = grouped ? g0 : m0, p1 = grouped ? g1 : m1;
  const int chunks = D / VE;
  for (int c = l; c < chunks; c += lanes) {
    src.chunk(c);
    double acc[VE];
#pragma unroll
    for (int t = 0; t < VE; ++t) acc[t] = 0.0;
    if (!longrow)
      ia_sum<VE>(occ, j0, j1, c, src, acc);
    else
      ia_sum_partials<VE, IA_UNROLL>(part, p0, p1, D, c, acc);
    float o[VE];
#pragma unroll
    for (int t = 0; t < VE; ++t) o[t] = float(acc[t]);
    // output rows are written once: streamed (scaled sums of the large
    // batch's V index 1.61 -> 1.46 ms with both policies)
    if constexpr (VE == 8) {
      StreamIO<float, 4, true>::store(dst + u * D + c * VE, o);
      StreamIO<float, 4, true>::store(dst + u * D + c * VE + 4, o + 4);
    } else {
      StreamIO<float, VE, true>::store(dst + u * D + c * VE, o);
    }
  }
}

// seg[e] = the segment v with off[v] <= e < off[v + 1]: a binary search in
// the offsets per edge, in edge order (neighbouring threads walk the same
// path); clamped into [0, N) whatever the offsets hold.
__global__ void __launch_bounds__(IA_THREADS) k_edge_seg(const int32_t* __restrict__ off,
                                                        int64_t N, int64_t n,
                                                        int32_t* __restrict__ seg) {
  const int64_t e = int64_t(blockIdx.x) * IA_THREADS + threadIdx.x;
  if (e >= n) return;
  int64_t lo = 0, hi = N - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (int64_t(off[mid]) <= e) lo = mid; else hi = mid - 1;
  }
  seg[e] = int32_t(lo);
}

// Occurrence order for the scaled sums: for every valid occurrence j (below
// occ_off[num_rows]) of edge e = occ[j], occ_seg[j] = seg[e] and
// occ_scal[j, :] = scal[e, :] (positions clamped into range).
__global__ void __launch_bounds__(IA_THREADS) k_coef_permute(
    const int32_t* __restrict__ occ, const int32_t* __restrict__ occ_off, int64_t num_rows,
    int64_t n, const int32_t* __restrict__ seg, const float* __restrict__ scal, int H,
    int32_t* __restrict__ occ_seg, float* __restrict__ occ_scal) {
  const int64_t j = int64_t(blockIdx.x) * IA_THREADS + threadIdx.x;
  if (j >= clamp64(occ_off[num_rows], 0, n)) return;
  const int64_t e = clamp64(occ[j], 0, n - 1);
  occ_seg[j] = seg[e];
  for (int h = 0; h < H; ++h) occ_scal[j * H + h] = scal[e * H + h];
}

struct IaWs {
  int32_t* multi_off;
  int32_t* group_off;
  void* scan;
  double* partial;
  double* partial2;
};

static int64_t ia_multi_bound(int64_t n) { return (2 * n) / IA_PIECE + 1; }
// pieces of rows with groups, over IA_GROUP_MIN / 2
static int64_t ia_group_bound(int64_t n) { return ia_multi_bound(n) * 2 / IA_GROUP_MIN + 1; }

static size_t ia_layout(int64_t n, int64_t num_rows, int D, char* base, IaWs* ws) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes, 256);
    return base ? base + o : nullptr;
  };
  char* mo = take(size_t(num_rows + 1) * 4);
  char* go = take(size_t(num_rows + 1) * 4);
  char* sc = take(scan_workspace<uint64_t>(num_rows + 1));
  char* pa = take(size_t(ia_multi_bound(n)) * size_t(D) * 8);
  char* pb = take(size_t(ia_group_bound(n)) * size_t(D) * 8);
  if (ws) {
    ws->multi_off = reinterpret_cast<int32_t*>(mo);
    ws->group_off = reinterpret_cast<int32_t*>(go);
    ws->scan = sc;
    ws->partial = reinterpret_cast<double*>(pa);
    ws->partial2 = reinterpret_cast<double*>(pb);
  }
  return off;
}

static int pow2_at_least(int x, int cap) {
  int p = 1;
  while (p < x && p < cap) p <<= 1;
  return p;
}

}  // namespace fast

using namespace fast;

extern "C" size_t fast_occurrence_csr_workspace(int64_t n, int64_t num_rows) {
  if (n < 0 || num_rows < 0 || n >= (int64_t(1) << 31) || num_rows >= (int64_t(1) << 31) - 1)
    return 0;
  return occ_layout(n, num_rows, nullptr, nullptr);
}

extern "C" fast_status_t fast_occurrence_csr(const int32_t* index, int64_t n, int64_t num_rows,
                                             int32_t* occ_off, int32_t* occ, void* ws,
                                             size_t ws_bytes, fast_stream_t stream) {
  const char* fn = "fast_occurrence_csr";
  if (n < 0 || num_rows < 0) return fail(FAST_ERR_INVALID_ARG, "%s: negative size", fn);
  if (n >= (int64_t(1) << 31) || num_rows >= (int64_t(1) << 31) - 1)
    return fail(FAST_ERR_UNSUPPORTED, "%s: n or num_rows beyond 2^31", fn);
  if (!occ_off) return fail(FAST_ERR_INVALID_ARG, "%s: occ_off is NULL", fn);
  if (n > 0 && (!index || !occ)) return fail(FAST_ERR_INVALID_ARG, "%s: index/occ is NULL", fn);
  const size_t need = fast_occurrence_csr_workspace(n, num_rows);
  if (!ws || ws_bytes < need)
    return fail(FAST_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu", fn, ws_bytes, need);
  if (!aligned(ws, 256)) return fail(FAST_ERR_UNSUPPORTED, "%s: workspace not 256-byte aligned", fn);
  hipStream_t st = static_cast<hipStream_t>(stream);
  OccWs w;
  occ_layout(n, num_rows, static_cast<char*>(ws), &w);
  if (n == 0) {
    hipLaunchKernelGGL(k_ir_fill, dim3(grid_cap(num_rows + 1, RS_THREADS * 4)), dim3(RS_THREADS), 0,
                       st, occ_off, num_rows + 1, 0);
    return check_launch(fn);
  }
  // positions sorted stably by key, 8 bits per pass (keys <= num_rows)
  int bits = 1;
  while ((int64_t(1) << bits) <= num_rows) ++bits;
  const int passes = (bits + 7) / 8;
  const int64_t T = rs_tiles(n);
  hipError_t e = hipSuccess;
  for (int p = 0; p < passes; ++p) {
    RsSrc src{p == 0 ? index : nullptr, w.keys[(p + 1) & 1], w.vals[(p + 1) & 1], int32_t(num_rows)};
    const bool last = p == passes - 1;
    int32_t* kout = w.keys[p & 1];
    int32_t* vout = last ? occ : w.vals[p & 1];
    hipLaunchKernelGGL(k_rs_hist, dim3(uint32_t(T)), dim3(RS_THREADS), 0, st, src, n, 8 * p, w.hist, T);
    e = scan_launch(InU32{w.hist}, OutU32InPlace{w.hist}, T * RS_DIGITS, w.scan_h, nullptr, nullptr, st);
    if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
    hipLaunchKernelGGL(k_rs_scatter, dim3(uint32_t(T)), dim3(RS_THREADS), 0, st, src, n, 8 * p,
                       w.hist, T, kout, vout);
  }
  // row offsets from the sorted keys
  hipLaunchKernelGGL(k_occ_offsets, dim3(uint32_t((num_rows + RS_THREADS) / RS_THREADS)),
                     dim3(RS_THREADS), 0, st, w.keys[(passes - 1) & 1], n, num_rows, occ_off);
  return check_launch(fn);
}

// Launches the row sums over occurrence lists for a row source: one scan of
// the (piece, group) counts, the long rows' pieces, their groups, then one
// group of lanes per row.
template <int VE, class Src>
static hipError_t ia_launch(const int32_t* occ_off, const int32_t* occ, int64_t n,
                            int64_t num_rows, int D, const Src& src, const IaWs& w, float* dst,
                            hipStream_t st) {
  hipError_t e = scan_launch<InMulti, OutMulti, uint64_t>(
      InMulti{occ_off, n, num_rows}, OutMulti{w.multi_off, w.group_off}, num_rows + 1, w.scan,
      nullptr, nullptr, st);
  if (e != hipSuccess) return e;
  const int lanes = pow2_at_least(D / VE, 64);
  const int64_t groups_per_block = IA_THREADS / lanes;
  const int64_t mb = ia_multi_bound(n), gb = ia_group_bound(n);
  const int64_t np_blocks = (mb + groups_per_block - 1) / groups_per_block;
  const int64_t ng_blocks = (gb + groups_per_block - 1) / groups_per_block;
  const int64_t nr_blocks = (num_rows + groups_per_block - 1) / groups_per_block;
  if (n > 0) {
    hipLaunchKernelGGL((k_ia_pieces<VE, Src>), dim3(uint32_t(np_blocks)), dim3(IA_THREADS), 0, st,
                       occ_off, occ, w.multi_off, num_rows, mb, n, lanes, D, src, w.partial);
    hipLaunchKernelGGL((k_ia_groups<VE>), dim3(uint32_t(ng_blocks)), dim3(IA_THREADS), 0, st,
                       occ_off, w.multi_off, w.group_off, num_rows, mb, gb, n, lanes, D, w.partial,
                       w.partial2);
  }
  hipLaunchKernelGGL((k_ia_rows<VE, Src>), dim3(uint32_t(nr_blocks)), dim3(IA_THREADS), 0, st,
                     occ_off, occ, w.multi_off, w.group_off, num_rows, mb, gb, n, lanes, D, src,
                     w.partial, w.partial2, dst);
  return hipGetLastError();
}

// Widest vector (8 values for bf16 sources, else 4, 2 or 1) that divides D,
// is at most `cap` and fits the alignment of both row pointers.
static int ia_vector(int D, int cap, const void* src, int esz, const float* dst) {
  if (esz == 2 && 8 <= cap && D % 8 == 0 && aligned(src, 16) && aligned(dst, 16)) return 8;
  for (int v : {4, 2})
    if (v <= cap && D % v == 0 && aligned(src, size_t(v) * esz) && aligned(dst, size_t(v) * 4))
      return v;
  return 1;
}

static fast_status_t ia_common_checks(const char* fn, int64_t n, int64_t num_rows, int D,
                                      fast_dtype_t src_dtype) {
  if (n < 0 || num_rows < 0 || D < 1) return fail(FAST_ERR_INVALID_ARG, "%s: bad size", fn);
  if (n >= (int64_t(1) << 31) || num_rows >= (int64_t(1) << 31) - 1)
    return fail(FAST_ERR_UNSUPPORTED, "%s: n or num_rows beyond 2^31", fn);
  if (src_dtype != FAST_F32 && src_dtype != FAST_BF16) return fail(FAST_ERR_INVALID_ARG, "%s: bad dtype", fn);
  return FAST_OK;
}

extern "C" size_t fast_index_add_rows_workspace(int64_t n, int64_t num_rows, int D) {
  if (n < 0 || num_rows < 0 || D < 1 || n >= (int64_t(1) << 31) || num_rows >= (int64_t(1) << 31) - 1)
    return 0;
  return ia_layout(n, num_rows, D, nullptr, nullptr);
}

extern "C" fast_status_t fast_index_add_rows(const int32_t* occ_off, const int32_t* occ,
                                             int64_t n, int64_t num_rows, int D,
                                             fast_dtype_t src_dtype, const void* src, float* dst,
                                             void* ws, size_t ws_bytes, fast_stream_t stream) {
  const char* fn = "fast_index_add_rows";
  if (fast_status_t c = ia_common_checks(fn, n, num_rows, D, src_dtype)) return c;
  if (num_rows == 0) return ok();
  if (!occ_off || !dst) return fail(FAST_ERR_INVALID_ARG, "%s: occ_off/dst is NULL", fn);
  if (n > 0 && (!occ || !src)) return fail(FAST_ERR_INVALID_ARG, "%s: occ/src is NULL", fn);
  const size_t need = fast_index_add_rows_workspace(n, num_rows, D);
  if (!ws || ws_bytes < need)
    return fail(FAST_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu", fn, ws_bytes, need);
  if (!aligned(ws, 256)) return fail(FAST_ERR_UNSUPPORTED, "%s: workspace not 256-byte aligned", fn);
  const int esz = elem_size(src_dtype);
  if (!aligned(src, size_t(esz)) || !aligned(dst, 4))
    return fail(FAST_ERR_UNSUPPORTED, "%s: src/dst misaligned", fn);
  const int VE = ia_vector(D, 8, src, esz, dst);
  hipStream_t st = static_cast<hipStream_t>(stream);
  IaWs w;
  ia_layout(n, num_rows, D, static_cast<char*>(ws), &w);
  hipError_t e = hipSuccess;
#define FAST_IA(T_, VE_) \
  e = ia_launch<VE_>(occ_off, occ, n, num_rows, D, PlainRows<T_, VE_>{static_cast<const T_*>(src), D, n}, w, dst, st)
  if (src_dtype == FAST_F32) {
    if (VE == 4) FAST_IA(float, 4); else if (VE == 2) FAST_IA(float, 2); else FAST_IA(float, 1);
  } else {
    if (VE == 8) FAST_IA(uint16_t, 8); else if (VE == 4) FAST_IA(uint16_t, 4);
    else if (VE == 2) FAST_IA(uint16_t, 2); else FAST_IA(uint16_t, 1);
  }
#undef FAST_IA
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
  return check_launch(fn);
}

static size_t ias_layout(int64_t n, int64_t num_rows, int H, int D, char* base, int32_t** seg,
                         int32_t** occ_seg, float** occ_scal, IaWs* ws) {
  const size_t seg_bytes = align_up(size_t(n) * 4, 256);
  const size_t scal_bytes = align_up(size_t(n) * size_t(H) * 4, 256);
  if (seg) *seg = reinterpret_cast<int32_t*>(base);
  if (occ_seg) *occ_seg = reinterpret_cast<int32_t*>(base + seg_bytes);
  if (occ_scal) *occ_scal = reinterpret_cast<float*>(base + 2 * seg_bytes);
  const size_t head = 2 * seg_bytes + scal_bytes;
  return head + ia_layout(n, num_rows, D, base ? base + head : nullptr, ws);
}

extern "C" size_t fast_index_add_scaled_rows_workspace(int64_t n, int64_t num_rows, int H, int dh) {
  if (H < 1 || dh < 1 || int64_t(H) * dh >= (int64_t(1) << 31)) return 0;
  const int D = H * dh;
  if (n < 0 || num_rows < 0 || n >= (int64_t(1) << 31) || num_rows >= (int64_t(1) << 31) - 1)
    return 0;
  return ias_layout(n, num_rows, H, D, nullptr, nullptr, nullptr, nullptr, nullptr);
}

extern "C" fast_status_t fast_index_add_scaled_rows(
    const int32_t* occ_off, const int32_t* occ, int64_t n, int64_t num_rows,
    const int32_t* dst_offsets, int64_t num_dst, int H, int dh, fast_dtype_t src_dtype,
    const float* scal, const void* src, float* dst, void* ws, size_t ws_bytes,
    fast_stream_t stream) {
  const char* fn = "fast_index_add_scaled_rows";
  if (H < 1 || dh < 1 || int64_t(H) * dh >= (int64_t(1) << 31))
    return fail(FAST_ERR_INVALID_ARG, "%s: bad H = %d or dh = %d", fn, H, dh);
  const int D = H * dh;
  if (fast_status_t c = ia_common_checks(fn, n, num_rows, D, src_dtype)) return c;
  if (num_dst < 0) return fail(FAST_ERR_INVALID_ARG, "%s: negative num_dst", fn);
  if (num_dst >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: num_dst >= 2^31", fn);
  if (n > 0 && num_dst == 0) return fail(FAST_ERR_INVALID_ARG, "%s: edges but no destination", fn);
  if (num_rows == 0) return ok();
  if (!occ_off || !dst) return fail(FAST_ERR_INVALID_ARG, "%s: occ_off/dst is NULL", fn);
  if (n > 0 && (!occ || !src || !scal || !dst_offsets))
    return fail(FAST_ERR_INVALID_ARG, "%s: occ/dst_offsets/scal/src is NULL", fn);
  const size_t need = fast_index_add_scaled_rows_workspace(n, num_rows, H, dh);
  if (!ws || ws_bytes < need)
    return fail(FAST_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu", fn, ws_bytes, need);
  if (!aligned(ws, 256)) return fail(FAST_ERR_UNSUPPORTED, "%s: workspace not 256-byte aligned", fn);
  const int esz = elem_size(src_dtype);
  if (!aligned(src, size_t(esz)) || !aligned(dst, 4) || !aligned(scal, 4))
    return fail(FAST_ERR_UNSUPPORTED, "%s: src/dst/scal misaligned", fn);
  const int VE = ia_vector(D, dh, src, esz, dst);   // a chunk spans at most two heads
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t *seg = nullptr, *occ_seg = nullptr;
  float* occ_scal = nullptr;
  IaWs w;
  ias_layout(n, num_rows, H, D, static_cast<char*>(ws), &seg, &occ_seg, &occ_scal, &w);
  if (n > 0) {
    const dim3 grid{uint32_t((n + IA_THREADS - 1) / IA_THREADS)};
    hipLaunchKernelGGL(k_edge_seg, grid, dim3(IA_THREADS), 0, st, dst_offsets, num_dst, n, seg);
    hipLaunchKernelGGL(k_coef_permute, grid, dim3(IA_THREADS), 0, st, occ, occ_off, num_rows, n, seg,
                       scal, H, occ_seg, occ_scal);
  }
  hipError_t e = hipSuccess;
#define FAST_IAS(T_, VE_)                                                                          \
  e = ia_launch<VE_>(occ_off, occ, n, num_rows, D,                                                 \
                     ScaledRows<T_, VE_>{static_cast<const T_*>(src), occ_scal, occ_seg, D, H, dh, \
                                         num_dst, 0, 0, 0},                                        \
                     w, dst, st)
  if (src_dtype == FAST_F32) {
    if (VE == 4) FAST_IAS(float, 4); else if (VE == 2) FAST_IAS(float, 2); else FAST_IAS(float, 1);
  } else {
    if (VE == 8) FAST_IAS(uint16_t, 8); else if (VE == 4) FAST_IAS(uint16_t, 4);
    else if (VE == 2) FAST_IAS(uint16_t, 2); else FAST_IAS(uint16_t, 1);
  }
#undef FAST_IAS
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
  return check_launch(fn);
}
