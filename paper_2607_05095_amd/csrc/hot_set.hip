// hot_set.hip -- SlimCache's greedy cache selection (Sec. 4.2, Alg. 1) on the
// GPU: access counting over pre-sampled batches, then the choice of the hot
// node and edge ids under a budget of cached rows, and the slot maps that the
// row reconstruction reads.
//
// Counting.  Every batch adds one to the counter of each distinct id it
// touches.  One launch per batch; each id sets its batch's bit in a byte per
// id (atomicOr; up to 32 batches, in groups of 8 with a clear per group) or
// stamps its slot with the batch tag (atomicExch; more batches), and only the
// access that finds the bit clear or replaces an older tag increments the
// counter, so repeats inside a batch count once.  Integer atomics make the
// counts exact whatever the interleaving; an LDS hash per workgroup drops
// most repeats before they reach HBM.
//
// Selection.  Alg. 1 ranks each kind by descending count and merges the two
// lists, a node winning only with a strictly higher count.  The ids it takes
// are therefore the first `budget` ids of one combined order: count
// descending, edges before nodes at equal count, ascending id inside a kind.
// That set is found without a sort: a histogram of the counts gives the
// threshold count T with fewer than `budget` ids above it and enough at or
// above it; all ids above T are taken, and of the ids at exactly T, the
// first R_e edges and R_v nodes in id order.  One scan per kind over a packed
// pair (ids above T, ids at T) then gives every id its position among the
// selected ids (above-T prefix + min(at-T prefix, R)), which is both the slot
// in the id-ordered hot list and the value of the slot map.  When the counts
// are small (fewer than 64 batches counted), the histogram pass also keeps a
// suffix histogram per tile of 4096 ids, so the tile sums of the scan come
// from two of those entries instead of a second read of every count, and it
// stores each id's clamped count as one byte, which the write pass reads in
// place of the four-byte count; node and edge tiles then share each launch.
#include <cmath>
#include <cstdlib>
#include <cstring>

#include "scan.h"

namespace fast {

constexpr int HS_THREADS = 256;
constexpr int HS_LDS_BINS = 4096;  // counts below this are binned in LDS first
constexpr int HS_REG_BINS = 4;     // counts below this are binned in registers

__global__ void __launch_bounds__(HS_THREADS) k_hs_fill_i32(int32_t* p, int64_t n, int32_t v) {
  for (int64_t i = int64_t(blockIdx.x) * HS_THREADS + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * HS_THREADS)
    p[i] = v;
}

static uint32_t grid_for(int64_t n, int64_t per_block_items, uint32_t cap = 16384) {
  int64_t g = (n + per_block_items - 1) / per_block_items;
  if (g < 1) g = 1;
  return uint32_t(g < cap ? g : cap);
}

// ------------------------------------------------------------------ counting
constexpr int HS_CHUNK = 4096;              // ids per workgroup step
constexpr int HS_HASH = 2 * HS_CHUNK;       // LDS hash slots (load <= 1/2)
constexpr int HS_PROBES = 32;
constexpr uint32_t HS_EMPTY = 0xffffffffu;  // never an id: id_bound < 2^32

// Marks id x for batch `tag`; counts it if the batch had not marked it yet.
struct StampCount {
  int32_t tag;
  int32_t* stamp;
  int32_t* freq;
  __device__ void operator()(int64_t x) const {
    // read the stamp in L2 first; a stale read falls through to the exchange,
    // which decides exactly
    if (__hip_atomic_load(&stamp[x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == tag) return;
    if (atomicExch(&stamp[x], tag) != tag) atomicAdd(&freq[x], 1);
  }
};

// The same with one bit per id and batch of a group of up to 8 batches (a
// byte per id, four ids to a 32-bit word): the batch's bit is set by an
// atomic OR, and the access that finds it clear counts the id.  The mask map
// is a quarter of the stamps, so clearing it once per group costs less.
constexpr int AC_GROUP = 8;
struct MaskCount {
  uint32_t bit;        // 1 << (batch index within its group)
  uint32_t* mask32;
  int32_t* freq;
  __device__ void operator()(int64_t x) const {
    uint32_t* w = &mask32[x >> 2];
    const uint32_t b = bit << (8 * (x & 3));
    if (__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & b) return;
    if (!(atomicOr(w, b) & b)) atomicAdd(&freq[x], 1);
  }
};

// A hot id repeats thousands of times in a batch.  Each workgroup takes
// HS_CHUNK ids at a time and drops repeats inside the chunk through an LDS
// hash of 32-bit keys (a plain read first, a compare-and-swap only into an
// empty slot), so only an id's first occurrence in the chunk touches HBM.
// A probe sequence that finds no room also goes to HBM: the stamp there
// decides exactly, the hash is only a filter.
template <typename Act>
__global__ void __launch_bounds__(HS_THREADS) k_access_count(const int64_t* __restrict__ ids,
                                                            int64_t n, int64_t id_bound, Act act) {
  __shared__ uint32_t s_key[HS_HASH];
  for (int64_t c0 = int64_t(blockIdx.x) * HS_CHUNK; c0 < n; c0 += int64_t(gridDim.x) * HS_CHUNK) {
    for (int j = threadIdx.x; j < HS_HASH; j += HS_THREADS) s_key[j] = HS_EMPTY;
    __syncthreads();
    const int m = int(n - c0 < HS_CHUNK ? n - c0 : HS_CHUNK);
    for (int j = threadIdx.x; j < m; j += HS_THREADS) {
      const int64_t x = ids[c0 + j];
      if (x < 0 || x >= id_bound) continue;
      const uint32_t key = uint32_t(x);
      uint32_t h = (key * 0x9E3779B1u) >> 19;          // 13 bits: HS_HASH slots
      bool first = true;
      for (int p = 0; p < HS_PROBES; ++p) {
        const uint32_t k = s_key[h];
        if (k == key) { first = false; break; }
        if (k == HS_EMPTY) {
          const uint32_t old = atomicCAS(&s_key[h], HS_EMPTY, key);
          if (old == HS_EMPTY) break;                   // inserted: first in the chunk
          if (old == key) { first = false; break; }
        }
        h = (h + 1) & (HS_HASH - 1);
      }
      if (first) act(x);
    }
    __syncthreads();
  }
}

// Dense universes (id_bound at most AC_BYTEMAP_RATIO times the mean batch
// size): each batch marks its ids in a byte map with plain stores (repeats
// store the same 1), then a streaming pass adds the maps into freq -- no
// atomics at all.  The workspace (4 bytes per id) holds AC_PLANES such maps:
// a group of up to 4 batches is cleared once, marks one map each, and one
// pass adds all of them (bytes of 0 or 1, so the 32-bit sum of the maps'
// words holds each id's count in its byte).
constexpr int64_t AC_BYTEMAP_RATIO = 32;
constexpr int AC_PLANES = 4;

__global__ void __launch_bounds__(HS_THREADS) k_ac_clear(uint4* p, int64_t n16) {
  for (int64_t i = int64_t(blockIdx.x) * HS_THREADS + threadIdx.x; i < n16;
       i += int64_t(gridDim.x) * HS_THREADS)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

__global__ void __launch_bounds__(HS_THREADS) k_ac_mark(const int64_t* __restrict__ ids, int64_t n,
                                                       int64_t id_bound, uint8_t* map) {
  const int64_t i = int64_t(blockIdx.x) * HS_THREADS + threadIdx.x;
  if (i >= n) return;
  const int64_t x = ids[i];
  if (x >= 0 && x < id_bound) map[x] = 1;
}

// freq[x] += sum over the np maps of map_p[x], four ids per thread (maps
// n4 words apart); bytes past id_bound are never set.
__global__ void __launch_bounds__(HS_THREADS) k_ac_accumulate(const uint32_t* __restrict__ map4,
                                                             int64_t n4, int np, int32_t* freq) {
  for (int64_t t = int64_t(blockIdx.x) * HS_THREADS + threadIdx.x; t < n4;
       t += int64_t(gridDim.x) * HS_THREADS) {
    uint32_t m = 0u;
    for (int p = 0; p < np; ++p) m += map4[int64_t(p) * n4 + t];
    if (m == 0u) continue;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int c = int((m >> (8 * k)) & 0xffu);
      if (c) freq[4 * t + k] += c;
    }
  }
}

static bool use_count_bytemap(int64_t total_ids, int64_t num_batches, int64_t id_bound) {
  static const int mode = [] {
    const char* e = std::getenv("FAST_COUNT_MARK");   // tuning override: bytemap | stamp
    if (!e) return 0;
    return std::strcmp(e, "bytemap") == 0 ? 1 : std::strcmp(e, "stamp") == 0 ? 2 : 0;
  }();
  if (mode) return mode == 1;
  const int64_t mean = num_batches > 0 ? total_ids / num_batches : 0;
  return id_bound <= AC_BYTEMAP_RATIO * (mean > 0 ? mean : 1);
}

// Masks for up to 32 batches (at most four clears of a byte per id, no
// more than the one clear of a 4-byte stamp per id); stamps beyond.
static bool count_masks(int64_t num_batches) {
  static const int mode = [] {
    const char* e = std::getenv("FAST_COUNT_MASKS");   // tuning override: 0 stamps, 1 masks
    return e ? (std::strcmp(e, "0") == 0 ? 0 : 1) : -1;
  }();
  if (mode >= 0) return mode == 1;
  return num_batches <= 4 * AC_GROUP;
}

// ------------------------------------------------------------------ selection
__device__ __forceinline__ int32_t clamp_count(int32_t f, int32_t max_freq) {
  return f < 0 ? 0 : (f > max_freq ? max_freq : f);
}

constexpr int HS_HIST_U = 8;

// hist[c] = number of ids whose clamped count is c, c in [0, max_freq].
// Counts below HS_LDS_BINS go through a per-workgroup LDS histogram (almost
// every id of a large universe has a small count), the rest straight to HBM.
__global__ void __launch_bounds__(HS_THREADS) k_hs_hist(const int32_t* __restrict__ f, int64_t n,
                                                       int32_t max_freq, uint32_t* hist) {
  __shared__ uint32_t s_h[HS_LDS_BINS];
  const int nb = max_freq + 1 < HS_LDS_BINS ? max_freq + 1 : HS_LDS_BINS;
  for (int b = threadIdx.x; b < nb; b += HS_THREADS) s_h[b] = 0;
  __syncthreads();
  // Most ids of a large universe share the few smallest counts: those are
  // counted in registers, so the LDS atomics see only the rare larger ones.
  uint32_t r[HS_REG_BINS] = {};
  auto bin = [&](int32_t raw) {
    const int32_t c = clamp_count(raw, max_freq);
    if (c < HS_REG_BINS) {
#pragma unroll
      for (int b = 0; b < HS_REG_BINS; ++b) r[b] += (c == b);
    } else if (c < nb) {
      atomicAdd(&s_h[c], 1u);
    } else {
      atomicAdd(&hist[c], 1u);
    }
  };
  // four counts per 16-byte load when the array allows it (HS_HIST_U loads
  // in flight per thread before they are binned), then the tail
  const bool vec = (reinterpret_cast<uintptr_t>(f) & 15u) == 0;
  const int64_t n4 = vec ? n / 4 : 0;
  const int4* f4 = reinterpret_cast<const int4*>(f);
  const int64_t stride = int64_t(gridDim.x) * HS_THREADS;
  int64_t i = int64_t(blockIdx.x) * HS_THREADS + threadIdx.x;
  for (; i + (HS_HIST_U - 1) * stride < n4; i += HS_HIST_U * stride) {
    int4 x[HS_HIST_U];
#pragma unroll
    for (int k = 0; k < HS_HIST_U; ++k) x[k] = f4[i + k * stride];
#pragma unroll
    for (int k = 0; k < HS_HIST_U; ++k) {
      bin(x[k].x); bin(x[k].y); bin(x[k].z); bin(x[k].w);
    }
  }
  for (; i < n4; i += stride) {
    const int4 x = f4[i];
    bin(x.x); bin(x.y); bin(x.z); bin(x.w);
  }
  for (int64_t i = 4 * n4 + int64_t(blockIdx.x) * HS_THREADS + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * HS_THREADS)
    bin(f[i]);
#pragma unroll
  for (int b = 0; b < HS_REG_BINS; ++b)
    if (b < nb && r[b]) atomicAdd(&s_h[b], r[b]);
  __syncthreads();
  for (int b = threadIdx.x; b < nb; b += HS_THREADS)
    if (s_h[b]) atomicAdd(&hist[b], s_h[b]);
}

// Threshold of the selection, written by k_hs_threshold.
struct HsParams {
  int32_t T;        // threshold count (max_freq + 1 when nothing is selected)
  int32_t pad;
  int64_t R_v;      // nodes taken among those with count T (lowest ids)
  int64_t R_e;      // edges taken among those with count T (lowest ids)
};

// One workgroup walks the counts from max_freq down, 256 bins at a time, and
// stops at the first count T where the ids at or above it reach the budget.
__global__ void __launch_bounds__(HS_THREADS) k_hs_threshold(
    const uint32_t* __restrict__ hv, const uint32_t* __restrict__ he, int32_t max_freq,
    int64_t budget, int64_t nv, int64_t ne, HsParams* prm, int64_t* num_hot_v,
    int64_t* num_hot_e) {
  __shared__ uint64_t lds4[4];
  __shared__ int64_t s_found[4];   // T, ids above T (both kinds), nodes above T, edges above T
  __shared__ int s_hit;
  const int64_t B = budget < nv + ne ? budget : nv + ne;
  if (threadIdx.x == 0) s_hit = 0;
  __syncthreads();
  uint64_t carry_all = 0, carry_v = 0;
  if (B > 0) {
    for (int64_t top = max_freq; top >= 0; top -= HS_THREADS) {
      const int64_t c = top - int64_t(threadIdx.x);          // descending counts
      const uint64_t w_v = c >= 0 ? hv[c] : 0, w_e = c >= 0 ? he[c] : 0;
      uint64_t tot_all, tot_v;
      const uint64_t ex_all = block_exclusive_scan<uint64_t>(w_v + w_e, lds4, tot_all);
      const uint64_t ex_v = block_exclusive_scan<uint64_t>(w_v, lds4, tot_v);
      const uint64_t above = carry_all + ex_all;   // ids with count > c
      if (c >= 0 && int64_t(above) < B && int64_t(above + w_v + w_e) >= B) {
        s_found[0] = c;
        s_found[1] = int64_t(above);
        s_found[2] = int64_t(carry_v + ex_v);
        s_found[3] = int64_t(above) - int64_t(carry_v + ex_v);
        s_hit = 1;
      }
      __syncthreads();
      if (s_hit) break;
      carry_all += tot_all;
      carry_v += tot_v;
    }
  }
  if (threadIdx.x == 0) {
    HsParams p;
    p.pad = 0;
    if (!s_hit) {                       // empty budget
      p.T = max_freq + 1;
      p.R_v = p.R_e = 0;
      *num_hot_v = 0;
      *num_hot_e = 0;
    } else {
      const int32_t T = int32_t(s_found[0]);
      const int64_t R = B - s_found[1];
      const int64_t at_e = int64_t(he[T]);
      p.T = T;
      p.R_e = R < at_e ? R : at_e;
      p.R_v = R - p.R_e;
      *num_hot_v = s_found[2] + p.R_v;
      *num_hot_e = s_found[3] + p.R_e;
    }
    *prm = p;
  }
}

// Positions of the selected ids, in two passes over the counts with 16-byte
// accesses.  Each id carries a packed pair (high word: its count is above T,
// low word: its count equals T).  Pass A adds the pairs up per tile of
// HS_SEL_TILE ids; the tile sums are scanned (exclusive); pass B recomputes
// the pairs and scans each tile in id order -- four rounds of 1024 ids, four
// consecutive ids per thread -- from the tile's prefix.  An id is selected if
// it is above T, or at T among the first R (of its kind) in id order; its
// position, (ids above T before it) + min(ids at T before it, R), is both its
// slot in the id-ordered hot list and its slot-map value.
constexpr int HS_SEL_ROUNDS = 4;
constexpr int HS_SEL_TILE = HS_THREADS * 4 * HS_SEL_ROUNDS;   // 4096 ids

__device__ __forceinline__ uint64_t sel_pair(int32_t raw, int32_t max_freq, int32_t T) {
  const int32_t c = clamp_count(raw, max_freq);
  return (c > T ? (uint64_t(1) << 32) : 0) | (c == T ? 1u : 0u);
}

// The pairs of ids i0 .. i0+3 (0 for positions at or past n).
__device__ __forceinline__ void sel_pairs4(const int32_t* __restrict__ f, int64_t n, int64_t i0,
                                           bool vec, int32_t max_freq, int32_t T, uint64_t (&p)[4]) {
  if (vec && i0 + 3 < n) {
    const int4 v = *reinterpret_cast<const int4*>(f + i0);
    p[0] = sel_pair(v.x, max_freq, T);
    p[1] = sel_pair(v.y, max_freq, T);
    p[2] = sel_pair(v.z, max_freq, T);
    p[3] = sel_pair(v.w, max_freq, T);
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) p[k] = i0 + k < n ? sel_pair(f[i0 + k], max_freq, T) : 0;
  }
}

__global__ void __launch_bounds__(HS_THREADS) k_sel_tiles(const int32_t* __restrict__ f, int64_t n,
                                                         int32_t max_freq,
                                                         const HsParams* __restrict__ prm,
                                                         uint64_t* __restrict__ tsum) {
  __shared__ uint64_t lds4[4];
  const int32_t T = prm->T;
  const bool vec = (reinterpret_cast<uintptr_t>(f) & 15u) == 0;
  const int64_t base = int64_t(blockIdx.x) * HS_SEL_TILE;
  uint64_t s = 0;
#pragma unroll
  for (int r = 0; r < HS_SEL_ROUNDS; ++r) {
    uint64_t p[4];
    sel_pairs4(f, n, base + (int64_t(r) * HS_THREADS + threadIdx.x) * 4, vec, max_freq, T, p);
    s += p[0] + p[1] + p[2] + p[3];
  }
  uint64_t total;
  block_exclusive_scan<uint64_t>(s, lds4, total);
  if (threadIdx.x == 0) tsum[blockIdx.x] = total;
}

__global__ void __launch_bounds__(HS_THREADS) k_sel_write(
    const int32_t* __restrict__ f, int64_t n, int32_t max_freq, const HsParams* __restrict__ prm,
    bool edges, const uint64_t* __restrict__ tprefix, const uint64_t* __restrict__ tbase,
    int64_t cap, int64_t* __restrict__ hot, int32_t* __restrict__ slot) {
  __shared__ uint64_t lds4[4];
  const int32_t T = prm->T;
  const int64_t R = edges ? prm->R_e : prm->R_v;
  const bool vec = (reinterpret_cast<uintptr_t>(f) & 15u) == 0;
  const bool svec = slot && (reinterpret_cast<uintptr_t>(slot) & 15u) == 0;
  const int64_t base = int64_t(blockIdx.x) * HS_SEL_TILE;
  uint64_t run = tprefix[blockIdx.x] - (tbase ? *tbase : 0u);
  for (int r = 0; r < HS_SEL_ROUNDS; ++r) {     // every thread reaches every block scan
    const int64_t i0 = base + (int64_t(r) * HS_THREADS + threadIdx.x) * 4;
    uint64_t p[4];
    sel_pairs4(f, n, i0, vec, max_freq, T, p);
    uint64_t total;
    uint64_t pre = run + block_exclusive_scan<uint64_t>(p[0] + p[1] + p[2] + p[3], lds4, total);
    int32_t out[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t above = int64_t(pre >> 32), at = int64_t(pre & 0xffffffffu);
      const bool sel = (p[k] >> 32) != 0 || ((p[k] & 1u) != 0 && at < R);
      const int64_t pos = above + (at < R ? at : R);
      out[k] = sel ? int32_t(pos) : -1;
      if (sel && hot && pos < cap) hot[pos] = i0 + k;
      pre += p[k];
    }
    if (slot) {
      if (svec && i0 + 3 < n) {   // streamed, as in the write pass over codes
        __builtin_nontemporal_store(__builtin_bit_cast(u32x4, make_int4(out[0], out[1], out[2], out[3])),
                                    reinterpret_cast<u32x4*>(slot + i0));
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (i0 + k < n) slot[i0 + k] = out[k];
      }
    }
    run += total;
  }
}

// Write pass over one-byte codes: thread t owns the 16 consecutive ids
// base + 16t .. base + 16t + 15 of its tile (one 16-byte load).  Byte-wise
// compares give 16-bit masks of the ids above T and at T, a single 32-bit
// block scan of the packed per-thread counts (above << 16 | at, each at most
// 4096 per tile) places them, the selected ids of a thread are consecutive in
// the hot list, and the tile's slots pass through LDS so that the stores are
// contiguous across lanes.
constexpr int HS_SW_IDS = HS_SEL_TILE / HS_THREADS;   // 16 ids per thread
static_assert(HS_SW_IDS == 16, "one 16-byte load of codes per thread");

// 4-bit mask of the bytes of a whose bit 7 is set (bits 7, 15, 23, 31).
__device__ __forceinline__ uint32_t byte_msb_nibble(uint32_t a) {
  return (((a >> 7) & 0x01010101u) * 0x00204081u) >> 21 & 0xfu;
}

// Masks of the four codes in q (each below 128) above T and equal to T.
__device__ __forceinline__ void code_masks(uint32_t q, int32_t T, uint32_t& gt, uint32_t& eq) {
  const uint32_t hi = q | 0x80808080u;
  const uint32_t g = (hi - uint32_t(T + 1) * 0x01010101u) & 0x80808080u;   // code >= T + 1
  const uint32_t e = (hi - uint32_t(T) * 0x01010101u) & 0x80808080u;       // code >= T
  gt = byte_msb_nibble(g);
  eq = byte_msb_nibble(e & ~g);
}

// Both kinds in one launch, as in the histogram pass; tprefix holds the
// exclusive prefixes over the node tiles and then the edge tiles, so an edge
// tile's prefix is taken relative to tprefix[tiles_v].
struct SelKind {
  const uint8_t* codes;
  int64_t n;
  int64_t cap;
  int64_t* hot;
  int32_t* slot;
};

__global__ void __launch_bounds__(HS_THREADS) k_sel_write_codes(SelKind kv, SelKind ke, int64_t tiles_v,
                                                               const HsParams* __restrict__ prm,
                                                               const uint64_t* __restrict__ tprefix) {
  __shared__ uint32_t lds4[4];
  const bool edges = int64_t(blockIdx.x) >= tiles_v;
  const SelKind& K = edges ? ke : kv;
  if (!K.hot && !K.slot) return;          // uniform over the workgroup
  const uint8_t* __restrict__ codes = K.codes;
  const int64_t n = K.n, cap = K.cap;
  int64_t* __restrict__ hot = K.hot;
  int32_t* __restrict__ slot = K.slot;
  const int64_t tile = edges ? int64_t(blockIdx.x) - tiles_v : int64_t(blockIdx.x);
  // slots of the tile, 16 bytes per entry; entry j sits at j + j / 8 so that
  // both the per-thread writes (4 entries 64 bytes apart) and the striped
  // reads are free of bank conflicts
  __shared__ int4 s_out[HS_SEL_TILE / 4 + HS_SEL_TILE / 32];
  const int32_t T = prm->T;
  const int64_t R = edges ? prm->R_e : prm->R_v;
  const int64_t base = tile * HS_SEL_TILE;
  const int64_t i0 = base + int64_t(threadIdx.x) * HS_SW_IDS;
  const uint4 q = *reinterpret_cast<const uint4*>(codes + i0);   // padded to whole tiles
  uint32_t gt = 0, eq = 0;
  {
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      uint32_t g, e;
      code_masks(w[k], T, g, e);
      gt |= g << (4 * k);
      eq |= e << (4 * k);
    }
  }
  if (i0 + HS_SW_IDS > n) {                 // ids at or past n are never selected
    const int64_t valid = n - i0;
    const uint32_t m = valid <= 0 ? 0u : (1u << valid) - 1u;
    gt &= m;
    eq &= m;
  }
  uint32_t tot;
  const uint32_t ex = block_exclusive_scan<uint32_t>((uint32_t(__popc(gt)) << 16) | uint32_t(__popc(eq)),
                                                     lds4, tot);
  const uint64_t tp = tprefix[blockIdx.x] - (edges ? tprefix[tiles_v] : 0u);   // no borrow: monotone
  const int64_t above = int64_t(tp >> 32) + int64_t(ex >> 16);
  const int64_t at = int64_t(tp & 0xffffffffu) + int64_t(ex & 0xffffu);
  // ids at T are taken while fewer than R of them come before
  uint32_t eqsel = 0;
  if (at + __popc(eq) <= R) {
    eqsel = eq;
  } else if (at < R) {
    uint32_t m = eq;
    for (int64_t left = R - at; left > 0; --left) {
      eqsel |= m & (0u - m);
      m &= m - 1u;
    }
  }
  const uint32_t sel = gt | eqsel;
  const int32_t pos0 = int32_t(above + (at < R ? at : R));
  if (hot) {
    int32_t p = pos0;
    for (uint32_t m = sel; m; m &= m - 1u, ++p)
      if (p < cap) hot[p] = i0 + (__ffs(m) - 1);
  }
  if (!slot) return;
  {
    int32_t p = pos0, o[HS_SW_IDS];
#pragma unroll
    for (int k = 0; k < HS_SW_IDS; ++k) {
      const int32_t b = int32_t((sel >> k) & 1u);
      o[k] = b ? p : -1;
      p += b;
    }
    const int e0 = 4 * threadIdx.x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = e0 + j;
      s_out[e + (e >> 3)] = make_int4(o[4 * j], o[4 * j + 1], o[4 * j + 2], o[4 * j + 3]);
    }
  }
  __syncthreads();
  // The slot map streams out (non-temporal): nothing reads it back in this
  // call, and cached stores left it to be written back by later work
  // (measured on the 1e7-node, 2e8-edge selection: 0.409 -> 0.354 ms; the
  // codes stay cached, the write pass reads them right after they are made).
  const bool svec = (reinterpret_cast<uintptr_t>(slot) & 15u) == 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = j * HS_THREADS + threadIdx.x;
    const int4 v = s_out[e + (e >> 3)];
    const int64_t i = base + 4 * int64_t(e);
    if (svec && i + 3 < n) {
      __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), reinterpret_cast<u32x4*>(slot + i));
    } else {
      if (i < n) slot[i] = v.x;
      if (i + 1 < n) slot[i + 1] = v.y;
      if (i + 2 < n) slot[i + 2] = v.z;
      if (i + 3 < n) slot[i + 3] = v.w;
    }
  }
}

// ------------------------------------------------------------------ tile histograms
// Counts below HS_TH_BINS (max_freq < HS_TH_BINS): one workgroup per tile of
// HS_SEL_TILE ids reads the tile's counts once (16 per thread, all loads
// issued first) and stores the tile's histogram th[tile * nb + c] (nb =
// max_freq + 1, at most 4096 per bin: uint16).  With `codes`, it also stores
// every id's clamped count as one byte, so the selection's write pass reads
// one byte per id instead of four.
constexpr int HS_TH_BINS = 64;

// Bit 7 of each byte of the result is set where that byte of q (a code
// below 128) is nonzero.
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t q) {
  return ((q + 0x7f7f7f7fu) | q) & 0x80808080u;
}

// One launch for both kinds: workgroups [0, tiles_v) take the node tiles,
// the rest the edge tiles; th holds the node rows, then the edge rows.  A
// tile's row is its suffix histogram, th[tile * nb + c] = ids of the tile
// with clamped count >= c, so that the selection reads a tile's (above T,
// at T) pair as two values.  The counts are read once: streaming loads.
__global__ void __launch_bounds__(HS_THREADS) k_hs_tilehist(const int32_t* __restrict__ f_v, int64_t n_v,
                                                           uint8_t* __restrict__ codes_v,
                                                           const int32_t* __restrict__ f_e, int64_t n_e,
                                                           uint8_t* __restrict__ codes_e,
                                                           int64_t tiles_v, int32_t max_freq,
                                                           uint16_t* __restrict__ th) {
  __shared__ uint32_t s_h[HS_TH_BINS];
  const int nb = max_freq + 1;
  const bool edges = int64_t(blockIdx.x) >= tiles_v;
  const int32_t* f = edges ? f_e : f_v;
  const int64_t n = edges ? n_e : n_v;
  uint8_t* codes = edges ? codes_e : codes_v;
  if (threadIdx.x < HS_TH_BINS) s_h[threadIdx.x] = 0u;
  const bool vec = (reinterpret_cast<uintptr_t>(f) & 15u) == 0;
  const int64_t base = (edges ? int64_t(blockIdx.x) - tiles_v : int64_t(blockIdx.x)) * HS_SEL_TILE;
  int32_t c[HS_SEL_ROUNDS][4];
#pragma unroll
  for (int r = 0; r < HS_SEL_ROUNDS; ++r) {
    const int64_t i0 = base + (int64_t(r) * HS_THREADS + threadIdx.x) * 4;
    if (vec && i0 + 3 < n) {
      const int4 v = __builtin_bit_cast(
          int4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(f + i0)));
      c[r][0] = v.x; c[r][1] = v.y; c[r][2] = v.z; c[r][3] = v.w;
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) c[r][k] = i0 + k < n ? f[i0 + k] : 0;
    }
  }
  __syncthreads();
  // Each id's clamped count as one byte; a 4-byte word that runs past n has
  // 0 there, and words wholly past n are not written (the write pass masks
  // every position at or past n).  Almost every id of a large universe has
  // count 0: only the nonzero bytes reach the LDS histogram; bin 0 is implied
  // by the tile's id count.
#pragma unroll
  for (int r = 0; r < HS_SEL_ROUNDS; ++r) {
    const int64_t i0 = base + (int64_t(r) * HS_THREADS + threadIdx.x) * 4;
    if (i0 >= n) continue;
    uint32_t q = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      q |= uint32_t(i0 + k < n ? clamp_count(c[r][k], max_freq) : 0) << (8 * k);
    if (codes) *reinterpret_cast<uint32_t*>(codes + i0) = q;
    for (uint32_t z = nonzero_bytes(q); z; z &= z - 1u)
      atomicAdd(&s_h[(q >> ((__ffs(z) - 1) & ~7)) & 0xffu], 1u);
  }
  __syncthreads();
  if (threadIdx.x < nb) {
    uint32_t v = 0;
    if (threadIdx.x == 0) {
      const int64_t left = n - base;
      v = uint32_t(left < HS_SEL_TILE ? left : HS_SEL_TILE);
    } else {
      for (int b = threadIdx.x; b < nb; ++b) v += s_h[b];
    }
    th[int64_t(blockIdx.x) * nb + threadIdx.x] = uint16_t(v);
  }
}

// hist[c] += sum over tiles of the tile's ids with count c (the difference of
// adjacent entries of its suffix row): the kind's tiles are split among half
// of the grid (the first half takes the nodes, the second the edges), each
// workgroup sums its range in LDS and adds its partial histogram with nb
// global atomics.
__global__ void __launch_bounds__(HS_THREADS) k_hs_tilesum(const uint16_t* __restrict__ th_v,
                                                          int64_t tiles_v,
                                                          const uint16_t* __restrict__ th_e,
                                                          int64_t tiles_e, int nb,
                                                          uint32_t* __restrict__ hv,
                                                          uint32_t* __restrict__ he) {
  __shared__ uint32_t s_h[HS_TH_BINS];
  const int half = gridDim.x / 2;
  const bool edges = int(blockIdx.x) >= half;
  const uint16_t* th = edges ? th_e : th_v;
  const int64_t tiles = edges ? tiles_e : tiles_v;
  const int k = edges ? int(blockIdx.x) - half : int(blockIdx.x);
  if (threadIdx.x < HS_TH_BINS) s_h[threadIdx.x] = 0u;
  __syncthreads();
  // the kind's tiles are split into `half` contiguous ranges; this workgroup
  // reads its range's nb-bin rows as one flat array
  const int64_t t0 = tiles * k / half, t1 = tiles * (k + 1) / half;
  for (int64_t j = t0 * nb + threadIdx.x; j < t1 * nb; j += HS_THREADS) {
    const int c = int(j % nb);
    atomicAdd(&s_h[c], uint32_t(th[j]) - (c + 1 < nb ? uint32_t(th[j + 1]) : 0u));
  }
  __syncthreads();
  if (threadIdx.x < nb && s_h[threadIdx.x]) atomicAdd(&(edges ? he : hv)[threadIdx.x], s_h[threadIdx.x]);
}

// Scan input of the selection from the tiles' suffix rows: tile i's packed
// pair (ids above T, ids at T), over the node tiles and then the edge tiles.
struct InTilePairs {
  const uint16_t* th;
  int nb;
  const HsParams* prm;
  __device__ uint64_t operator()(int64_t i) const {
    const int32_t T = prm->T;
    const uint64_t above = T + 1 < nb ? th[i * nb + T + 1] : 0u;
    const uint64_t at = T < nb ? th[i * nb + T] - above : 0u;
    return (above << 32) | at;
  }
};

struct InU64 {
  const uint64_t* p;
  __device__ uint64_t operator()(int64_t i) const { return p[i]; }
};
struct OutU64InPlace {
  uint64_t* p;
  __device__ void operator()(int64_t i, uint64_t prefix, uint64_t) const { p[i] = prefix; }
};

struct HsWs {
  uint32_t* hv;
  uint32_t* he;
  HsParams* prm;
  uint64_t* tsum_v;   // per-tile pair sums, then their exclusive prefixes
  uint64_t* tsum_e;
  void* scan_v;
  void* scan_e;
  uint16_t* th;       // per-tile suffix rows, node tiles then edge tiles (tiled path only)
  uint64_t* tsum;     // exclusive prefixes over the node tiles then the edge tiles (tiled)
  void* scan;
  uint8_t* codes_v;   // one-byte clamped counts, padded to whole tiles (tiled path only)
  uint8_t* codes_e;
};

static bool use_tile_hist(int32_t max_freq) {
  static const int mode = [] {   // tuning override: FAST_HS_TILE_HIST=0 turns it off
    const char* e = std::getenv("FAST_HS_TILE_HIST");
    return e && e[0] == '0' ? 0 : 1;
  }();
  return mode && max_freq + 1 <= HS_TH_BINS;
}

static bool use_codes(int32_t max_freq) {
  static const int mode = [] {   // tuning override: FAST_HS_CODES=0 turns it off
    const char* e = std::getenv("FAST_HS_CODES");
    return e && e[0] == '0' ? 0 : 1;
  }();
  return mode && use_tile_hist(max_freq);
}

static int64_t sel_tiles(int64_t n) { return (n + HS_SEL_TILE - 1) / HS_SEL_TILE; }

static size_t hs_layout(int64_t nv, int64_t ne, int32_t max_freq, char* base, HsWs* ws) {
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {   // NULL for a region the layout leaves out
    const size_t o = off;
    off += align_up(bytes, 256);
    return base && bytes ? base + o : nullptr;
  };
  char* hv = take(size_t(max_freq + 1) * 4);
  char* he = take(size_t(max_freq + 1) * 4);
  char* pr = take(sizeof(HsParams));
  char* tv = take(size_t(sel_tiles(nv)) * 8);
  char* te = take(size_t(sel_tiles(ne)) * 8);
  char* sv = take(scan_workspace<uint64_t>(sel_tiles(nv)));
  char* se = take(scan_workspace<uint64_t>(sel_tiles(ne)));
  const bool tiled = use_tile_hist(max_freq);
  const int64_t tiles = sel_tiles(nv) + sel_tiles(ne);
  char* th = take(tiled ? size_t(tiles) * size_t(max_freq + 1) * 2 : 0);
  char* ta = take(tiled ? size_t(tiles) * 8 : 0);
  char* sa = take(tiled ? scan_workspace<uint64_t>(tiles) : 0);
  const bool cd = use_codes(max_freq);
  char* cv = take(cd ? size_t(sel_tiles(nv)) * HS_SEL_TILE : 0);
  char* ce = take(cd ? size_t(sel_tiles(ne)) * HS_SEL_TILE : 0);
  if (ws) {
    ws->codes_v = reinterpret_cast<uint8_t*>(cv);
    ws->codes_e = reinterpret_cast<uint8_t*>(ce);
    ws->th = reinterpret_cast<uint16_t*>(th);
    ws->tsum = reinterpret_cast<uint64_t*>(ta);
    ws->scan = sa;
    ws->hv = reinterpret_cast<uint32_t*>(hv);
    ws->he = reinterpret_cast<uint32_t*>(he);
    ws->prm = reinterpret_cast<HsParams*>(pr);
    ws->tsum_v = reinterpret_cast<uint64_t*>(tv);
    ws->tsum_e = reinterpret_cast<uint64_t*>(te);
    ws->scan_v = sv;
    ws->scan_e = se;
  }
  return off;
}

}  // namespace fast

using namespace fast;

static const int32_t HS_MAX_FREQ = (1 << 24);

extern "C" size_t fast_access_count_workspace(int64_t id_bound) {
  if (id_bound < 0 || id_bound >= (int64_t(1) << 32)) return 0;
  return align_up(size_t(id_bound) * 4, 256) + 256;
}

extern "C" fast_status_t fast_access_count(const int64_t* ids, const int64_t* batch_offsets,
                                           int64_t num_batches, int64_t id_bound, int32_t* freq,
                                           void* ws, size_t ws_bytes, fast_stream_t stream) {
  const char* fn = "fast_access_count";
  if (num_batches < 0 || id_bound < 0) return fail(FAST_ERR_INVALID_ARG, "%s: negative size", fn);
  if (num_batches >= (int64_t(1) << 31) - 1)
    return fail(FAST_ERR_UNSUPPORTED, "%s: too many batches", fn);
  if (id_bound >= (int64_t(1) << 32)) return fail(FAST_ERR_UNSUPPORTED, "%s: id_bound >= 2^32", fn);
  if (num_batches == 0 || id_bound == 0) return ok();
  if (!batch_offsets) return fail(FAST_ERR_INVALID_ARG, "%s: batch_offsets is NULL", fn);
  if (batch_offsets[0] < 0) return fail(FAST_ERR_INVALID_ARG, "%s: batch_offsets[0] < 0", fn);
  for (int64_t k = 0; k < num_batches; ++k)
    if (batch_offsets[k + 1] < batch_offsets[k])
      return fail(FAST_ERR_INVALID_ARG, "%s: batch_offsets decrease at %lld", fn, (long long)k);
  if (batch_offsets[num_batches] > batch_offsets[0] && !ids)
    return fail(FAST_ERR_INVALID_ARG, "%s: ids is NULL", fn);
  if (!freq) return fail(FAST_ERR_INVALID_ARG, "%s: freq is NULL", fn);
  const size_t need = fast_access_count_workspace(id_bound);
  if (!ws || ws_bytes < need)
    return fail(FAST_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu", fn, ws_bytes, need);
  if (!aligned(ws, 4) || !aligned(freq, 4))
    return fail(FAST_ERR_UNSUPPORTED, "%s: freq or workspace not 4-byte aligned", fn);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (use_count_bytemap(batch_offsets[num_batches] - batch_offsets[0], num_batches, id_bound)) {
    if (!aligned(ws, 16)) return fail(FAST_ERR_UNSUPPORTED, "%s: workspace not 16-byte aligned", fn);
    uint8_t* map = static_cast<uint8_t*>(ws);
    // AC_PLANES maps of n16 16-byte vectors: within the id_bound * 4 + 256 bytes
    const int64_t n16 = (id_bound + 15) / 16;
    for (int64_t g0 = 0; g0 < num_batches; g0 += AC_PLANES) {
      const int64_t g1 = g0 + AC_PLANES < num_batches ? g0 + AC_PLANES : num_batches;
      if (batch_offsets[g1] == batch_offsets[g0]) continue;
      const int np = int(g1 - g0);
      hipLaunchKernelGGL(k_ac_clear, dim3(grid_for(n16 * np, HS_THREADS * 4)), dim3(HS_THREADS), 0, st,
                         reinterpret_cast<uint4*>(map), n16 * np);
      for (int64_t k = g0; k < g1; ++k) {
        const int64_t n = batch_offsets[k + 1] - batch_offsets[k];
        if (n == 0) continue;
        hipLaunchKernelGGL(k_ac_mark, dim3(uint32_t((n + HS_THREADS - 1) / HS_THREADS)),
                           dim3(HS_THREADS), 0, st, ids + batch_offsets[k], n, id_bound,
                           map + (k - g0) * n16 * 16);
      }
      hipLaunchKernelGGL(k_ac_accumulate, dim3(grid_for(n16 * 4, HS_THREADS * 4)), dim3(HS_THREADS), 0,
                         st, reinterpret_cast<const uint32_t*>(map), n16 * 4, np, freq);
    }
    return check_launch(fn);
  }
  if (count_masks(num_batches)) {
    if (!aligned(ws, 16)) return fail(FAST_ERR_UNSUPPORTED, "%s: workspace not 16-byte aligned", fn);
    uint32_t* mask32 = static_cast<uint32_t*>(ws);
    const int64_t n16 = (id_bound + 15) / 16;          // within the id_bound * 4 + 256 bytes
    for (int64_t g0 = 0; g0 < num_batches; g0 += AC_GROUP) {
      const int64_t g1 = g0 + AC_GROUP < num_batches ? g0 + AC_GROUP : num_batches;
      if (batch_offsets[g1] == batch_offsets[g0]) continue;
      hipLaunchKernelGGL(k_ac_clear, dim3(grid_for(n16, HS_THREADS * 4)), dim3(HS_THREADS), 0, st,
                         reinterpret_cast<uint4*>(mask32), n16);
      for (int64_t k = g0; k < g1; ++k) {
        const int64_t n = batch_offsets[k + 1] - batch_offsets[k];
        if (n == 0) continue;
        hipLaunchKernelGGL((k_access_count<MaskCount>), dim3(grid_for(n, HS_CHUNK)), dim3(HS_THREADS),
                           0, st, ids + batch_offsets[k], n, id_bound,
                           MaskCount{1u << uint32_t(k - g0), mask32, freq});
      }
    }
    return check_launch(fn);
  }
  int32_t* stamp = static_cast<int32_t*>(ws);
  hipLaunchKernelGGL(k_hs_fill_i32, dim3(grid_for(id_bound, HS_THREADS * 8)), dim3(HS_THREADS), 0,
                     st, stamp, id_bound, 0);
  for (int64_t k = 0; k < num_batches; ++k) {
    const int64_t n = batch_offsets[k + 1] - batch_offsets[k];
    if (n == 0) continue;
    hipLaunchKernelGGL((k_access_count<StampCount>), dim3(grid_for(n, HS_CHUNK)), dim3(HS_THREADS), 0,
                       st, ids + batch_offsets[k], n, id_bound, StampCount{int32_t(k + 1), stamp, freq});
  }
  return check_launch(fn);
}

// Alg. 1's loop runs while i + j < alpha * (|V| + |E|), the product taken in
// fp64, and stops when both ranked lists are used up: the number of ids it
// takes is the least integer not below that product, at most |V| + |E|.
extern "C" fast_status_t fast_hot_set_budget(double alpha, int64_t num_nodes, int64_t num_edges,
                                             int64_t* budget) {
  const char* fn = "fast_hot_set_budget";
  if (!budget) return fail(FAST_ERR_INVALID_ARG, "%s: budget is NULL", fn);
  if (num_nodes < 0 || num_edges < 0 || num_nodes > (int64_t(1) << 52) ||
      num_edges > (int64_t(1) << 52))
    return fail(FAST_ERR_INVALID_ARG, "%s: id counts outside [0, 2^52]", fn);
  if (alpha != alpha) return fail(FAST_ERR_INVALID_ARG, "%s: alpha is NaN", fn);
  const int64_t total = num_nodes + num_edges;
  const double x = alpha * double(total);   // exact integer conversion below 2^53
  int64_t b;
  if (!(x > 0.0)) b = 0;
  else if (x >= double(total)) b = total;
  else b = int64_t(std::ceil(x));
  *budget = b;
  return ok();
}

extern "C" size_t fast_greedy_hot_set_workspace(int64_t num_nodes, int64_t num_edges,
                                                int32_t max_freq) {
  if (num_nodes < 0 || num_edges < 0 || max_freq < 0 || max_freq > HS_MAX_FREQ) return 0;
  if (num_nodes >= (int64_t(1) << 32) || num_edges >= (int64_t(1) << 32)) return 0;
  return hs_layout(num_nodes, num_edges, max_freq, nullptr, nullptr);
}

extern "C" fast_status_t fast_greedy_hot_set(const int32_t* freq_v, int64_t num_nodes,
                                             const int32_t* freq_e, int64_t num_edges,
                                             int32_t max_freq, int64_t budget, int64_t* hot_v,
                                             int64_t* num_hot_v, int32_t* slot_v, int64_t* hot_e,
                                             int64_t* num_hot_e, int32_t* slot_e, void* ws,
                                             size_t ws_bytes, fast_stream_t stream) {
  const char* fn = "fast_greedy_hot_set";
  if (num_nodes < 0 || num_edges < 0 || budget < 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: negative size or budget", fn);
  if (max_freq < 0 || max_freq > HS_MAX_FREQ)
    return fail(FAST_ERR_UNSUPPORTED, "%s: max_freq outside [0, 2^24]", fn);
  if (num_nodes >= (int64_t(1) << 31) || num_edges >= (int64_t(1) << 31))
    return fail(FAST_ERR_UNSUPPORTED, "%s: 2^31 or more ids of one kind", fn);
  if (!num_hot_v || !num_hot_e) return fail(FAST_ERR_INVALID_ARG, "%s: NULL num_hot_v/num_hot_e", fn);
  if (num_nodes > 0 && !freq_v) return fail(FAST_ERR_INVALID_ARG, "%s: freq_v is NULL", fn);
  if (num_edges > 0 && !freq_e) return fail(FAST_ERR_INVALID_ARG, "%s: freq_e is NULL", fn);
  const size_t need = fast_greedy_hot_set_workspace(num_nodes, num_edges, max_freq);
  if (!ws || ws_bytes < need)
    return fail(FAST_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu", fn, ws_bytes, need);
  if (!aligned(ws, 256)) return fail(FAST_ERR_UNSUPPORTED, "%s: workspace not 256-byte aligned", fn);
  hipStream_t st = static_cast<hipStream_t>(stream);
  HsWs w;
  hs_layout(num_nodes, num_edges, max_freq, static_cast<char*>(ws), &w);
  const int64_t nbins = int64_t(max_freq) + 1;
  // both count histograms in one fill: he follows hv in the workspace
  const int64_t span = (w.he - w.hv) + nbins;
  hipLaunchKernelGGL(k_hs_fill_i32, dim3(grid_for(span, HS_THREADS)), dim3(HS_THREADS), 0, st,
                     reinterpret_cast<int32_t*>(w.hv), span, 0);
  const bool tiled = use_tile_hist(max_freq);
  const int64_t tv = sel_tiles(num_nodes), te = sel_tiles(num_edges);
  // codes are written only where the layout holds them and a write pass will
  // read them
  const bool cd = use_codes(max_freq);
  uint8_t* cv = cd && (hot_v || slot_v) ? w.codes_v : nullptr;
  uint8_t* ce = cd && (hot_e || slot_e) ? w.codes_e : nullptr;
  if (tiled) {
    if (tv + te > 0)
      hipLaunchKernelGGL(k_hs_tilehist, dim3(uint32_t(tv + te)), dim3(HS_THREADS), 0, st, freq_v,
                         num_nodes, cv, freq_e, num_edges, ce, tv, max_freq, w.th);
    hipLaunchKernelGGL(k_hs_tilesum, dim3(2 * 256), dim3(HS_THREADS), 0, st, w.th, tv,
                       w.th + tv * nbins, te, int(nbins), w.hv, w.he);
  } else {
    if (num_nodes > 0)
      hipLaunchKernelGGL(k_hs_hist, dim3(grid_for(num_nodes, HS_THREADS * 16, 4096)),
                         dim3(HS_THREADS), 0, st, freq_v, num_nodes, max_freq, w.hv);
    if (num_edges > 0)
      hipLaunchKernelGGL(k_hs_hist, dim3(grid_for(num_edges, HS_THREADS * 16, 4096)),
                         dim3(HS_THREADS), 0, st, freq_e, num_edges, max_freq, w.he);
  }
  hipLaunchKernelGGL(k_hs_threshold, dim3(1), dim3(HS_THREADS), 0, st, w.hv, w.he, max_freq,
                     budget, num_nodes, num_edges, w.prm, num_hot_v, num_hot_e);
  const int64_t B = budget < num_nodes + num_edges ? budget : num_nodes + num_edges;
  const bool want_v = num_nodes > 0 && (hot_v || slot_v), want_e = num_edges > 0 && (hot_e || slot_e);
  hipError_t e = hipSuccess;
  if (tiled) {
    // one scan of the tile pairs over the node tiles then the edge tiles
    if (want_v || want_e)
      e = scan_launch<InTilePairs, OutU64InPlace, uint64_t>(InTilePairs{w.th, int(nbins), w.prm},
                                                           OutU64InPlace{w.tsum}, tv + te, w.scan,
                                                           nullptr, nullptr, st);
    if (e == hipSuccess && (want_v || want_e)) {
      if (cd) {
        const SelKind kv{cv, num_nodes, B < num_nodes ? B : num_nodes, want_v ? hot_v : nullptr,
                         want_v ? slot_v : nullptr};
        const SelKind ke{ce, num_edges, B < num_edges ? B : num_edges, want_e ? hot_e : nullptr,
                         want_e ? slot_e : nullptr};
        hipLaunchKernelGGL(k_sel_write_codes, dim3(uint32_t(tv + te)), dim3(HS_THREADS), 0, st, kv,
                           ke, tv, w.prm, w.tsum);
      } else {
        if (want_v)
          hipLaunchKernelGGL(k_sel_write, dim3(uint32_t(tv)), dim3(HS_THREADS), 0, st, freq_v,
                             num_nodes, max_freq, w.prm, false, w.tsum, nullptr,
                             B < num_nodes ? B : num_nodes, hot_v, slot_v);
        if (want_e)
          hipLaunchKernelGGL(k_sel_write, dim3(uint32_t(te)), dim3(HS_THREADS), 0, st, freq_e,
                             num_edges, max_freq, w.prm, true, w.tsum + tv, w.tsum + tv,
                             B < num_edges ? B : num_edges, hot_e, slot_e);
      }
    }
  } else {
    auto select = [&](const int32_t* f, int64_t n, bool edges, uint64_t* tsum, void* scan_ws,
                      int64_t* hot, int32_t* slot) {
      if (n == 0 || (!hot && !slot) || e != hipSuccess) return;
      const int64_t tiles = sel_tiles(n);
      hipLaunchKernelGGL(k_sel_tiles, dim3(uint32_t(tiles)), dim3(HS_THREADS), 0, st, f, n, max_freq,
                         w.prm, tsum);
      e = scan_launch<InU64, OutU64InPlace, uint64_t>(InU64{tsum}, OutU64InPlace{tsum}, tiles,
                                                     scan_ws, nullptr, nullptr, st);
      if (e != hipSuccess) return;
      hipLaunchKernelGGL(k_sel_write, dim3(uint32_t(tiles)), dim3(HS_THREADS), 0, st, f, n, max_freq,
                         w.prm, edges, tsum, nullptr, B < n ? B : n, hot, slot);
    };
    select(freq_v, num_nodes, false, w.tsum_v, w.scan_v, hot_v, slot_v);
    select(freq_e, num_edges, true, w.tsum_e, w.scan_e, hot_e, slot_e);
  }
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
  return check_launch(fn);
}
