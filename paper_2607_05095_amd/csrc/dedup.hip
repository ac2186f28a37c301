// dedup.hip -- within-batch id compression and row reconstruction (Sec. 4.2
// SlimCache: transfer unique ids once plus an inverse index; Sec. 5: the
// uni_ID / inv_Idx triple).
//
// MI355X design: ids live in a bounded universe [0, id_bound), so the sorted
// distinct set is a bitmap over that universe.  Marking is one (checked)
// atomicOr per id; the rank of an id is the exclusive popcount prefix of the
// bitmap words below it plus a popcount inside its word.  This is exact and
// deterministic whatever the id order or thread interleaving, costs
// O(n + id_bound/32) work, and needs no sort.  Rows are then copied with
// 16/8/4-byte vector moves, one thread per vector of a row, from the table
// slot that the optional cache slot map names.
#include "scan.h"

namespace fast {

constexpr int DD_THREADS = 256;

struct DedupWs {
  uint32_t* bitmap;   // [W]
  uint32_t* prefix;   // [W] exclusive popcount prefix per word
  void* scan_w;       // scan workspace over W words
  uint8_t* flags;     // [n] miss flags
  void* scan_n;       // scan workspace over n flags
};

static size_t dedup_layout(int64_t n, int64_t id_bound, char* base, DedupWs* ws) {
  const int64_t W = (id_bound + 31) / 32;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += align_up(bytes, 256);
    return base ? base + o : nullptr;
  };
  char* bm = take(size_t(W) * 4);
  char* pf = take(size_t(W) * 4);
  char* sw = take(scan_workspace(W));
  char* fl = take(size_t(n));
  char* sn = take(scan_workspace(n));
  if (ws) {
    ws->bitmap = reinterpret_cast<uint32_t*>(bm);
    ws->prefix = reinterpret_cast<uint32_t*>(pf);
    ws->scan_w = sw;
    ws->flags = reinterpret_cast<uint8_t*>(fl);
    ws->scan_n = sn;
  }
  return off;
}

__global__ void __launch_bounds__(DD_THREADS) k_fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  for (int64_t i = int64_t(blockIdx.x) * DD_THREADS + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * DD_THREADS)
    p[i] = v;
}

__global__ void __launch_bounds__(DD_THREADS) k_dedup_mark(const int64_t* __restrict__ ids,
                                                           int64_t n, int64_t id_bound,
                                                           uint32_t* bitmap) {
  const int64_t i = int64_t(blockIdx.x) * DD_THREADS + threadIdx.x;
  if (i >= n) return;
  const int64_t id = ids[i];
  if (id < 0 || id >= id_bound) return;
  uint32_t* w = bitmap + (id >> 5);
  const uint32_t bit = 1u << (id & 31);
  // Zipf-hot ids repeat thousands of times: read first so that only the
  // first few occurrences pay for an atomic on the hot word.
  if ((__atomic_load_n(w, __ATOMIC_RELAXED) & bit) == 0) atomicOr(w, bit);
}

struct InPopc {
  const uint32_t* bm;
  __device__ uint32_t operator()(int64_t i) const { return __popc(bm[i]); }
};
struct OutPrefix {
  uint32_t* pf;
  __device__ void operator()(int64_t i, uint32_t prefix, uint32_t) const { pf[i] = prefix; }
};

// uni: every set bit of word w is written at its rank.
__global__ void __launch_bounds__(DD_THREADS) k_dedup_uni(const uint32_t* __restrict__ bitmap,
                                                          const uint32_t* __restrict__ prefix,
                                                          int64_t W, int64_t* __restrict__ uni) {
  const int64_t w = int64_t(blockIdx.x) * DD_THREADS + threadIdx.x;
  if (w >= W) return;
  uint32_t bits = bitmap[w];
  uint32_t r = prefix[w];
  while (bits) {
    const int b = __ffs(bits) - 1;
    uni[r++] = (w << 5) + b;
    bits &= bits - 1;
  }
}

__global__ void __launch_bounds__(DD_THREADS) k_dedup_inv(const int64_t* __restrict__ ids, int64_t n,
                                                          int64_t id_bound,
                                                          const uint32_t* __restrict__ bitmap,
                                                          const uint32_t* __restrict__ prefix,
                                                          int32_t* __restrict__ inv) {
  const int64_t i = int64_t(blockIdx.x) * DD_THREADS + threadIdx.x;
  if (i >= n) return;
  const int64_t id = ids[i];
  if (id < 0 || id >= id_bound) {
    inv[i] = -1;
    return;
  }
  const int64_t w = id >> 5;
  const uint32_t below = bitmap[w] & ((1u << (id & 31)) - 1u);
  inv[i] = int32_t(prefix[w] + __popc(below));
}

// Row copy: thread t of a block moves vector c of row k; a block covers
// `rpb` consecutive rows of `cpr` vectors each.  Rows k >= *num_unique are
// idle.  A slot outside [0, table_rows) flags k as a miss.
template <typename V>
__global__ void __launch_bounds__(DD_THREADS) k_gather_rows(const int64_t* __restrict__ uni,
                                                            const int64_t* __restrict__ num_unique,
                                                            const V* __restrict__ table,
                                                            int64_t table_rows, int cpr, int rpb,
                                                            const int32_t* __restrict__ slot_map,
                                                            V* __restrict__ rows,
                                                            uint8_t* __restrict__ flags) {
  const int64_t u = *num_unique;
  const int r = threadIdx.x / cpr;
  const int c = threadIdx.x - r * cpr;
  if (r >= rpb) return;
  const int64_t k = int64_t(blockIdx.x) * rpb + r;
  if (k >= u) return;
  const int64_t id = uni[k];
  const int64_t slot = slot_map ? int64_t(slot_map[id]) : id;
  const bool hit = slot >= 0 && slot < table_rows;
  if (c == 0 && flags) flags[k] = hit ? 0 : 1;
  if (!hit || !rows) return;
  rows[k * cpr + c] = table[slot * cpr + c];
}

struct InFlags {
  const uint8_t* f;
  const int64_t* num_unique;
  __device__ uint32_t operator()(int64_t i) const { return i < *num_unique ? f[i] : 0u; }
};
struct OutMiss {
  int32_t* miss;
  __device__ void operator()(int64_t i, uint32_t prefix, uint32_t v) const {
    if (v && miss) miss[prefix] = int32_t(i);
  }
};

template <typename V>
static void launch_gather(const int64_t* uni, const int64_t* num_unique, const void* table,
                          int64_t table_rows, int64_t row_bytes, const int32_t* slot_map,
                          void* rows, uint8_t* flags, int64_t cap, hipStream_t st) {
  const int cpr = int(row_bytes / int64_t(sizeof(V)));
  const int rpb = cpr >= DD_THREADS ? 1 : DD_THREADS / cpr;
  const int64_t nb = (cap + rpb - 1) / rpb;
  if (nb == 0) return;
  if (cpr <= DD_THREADS) {
    hipLaunchKernelGGL(k_gather_rows<V>, dim3(uint32_t(nb)), dim3(DD_THREADS), 0, st, uni,
                       num_unique, static_cast<const V*>(table), table_rows, cpr, rpb, slot_map,
                       static_cast<V*>(rows), flags);
  }
}

}  // namespace fast

using namespace fast;

static const int64_t kMaxIdBound = int64_t(1) << 35;

extern "C" size_t fast_dedup_gather_workspace(int64_t n, int64_t id_bound) {
  if (n < 0 || id_bound < 0 || id_bound > kMaxIdBound) return 0;
  return dedup_layout(n, id_bound, nullptr, nullptr);
}

extern "C" fast_status_t fast_dedup_gather(const int64_t* ids, int64_t n, int64_t id_bound,
                                           const void* table, int64_t table_rows, int D,
                                           fast_dtype_t dtype, const int32_t* slot_map,
                                           int64_t* uni, int32_t* inv, int64_t* num_unique,
                                           void* rows, int32_t* miss, int64_t* num_miss,
                                           void* ws, size_t ws_bytes, fast_stream_t stream) {
  const char* fn = "fast_dedup_gather";
  if (n < 0 || id_bound < 0 || table_rows < 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: negative size", fn);
  if (n >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "%s: n >= 2^31", fn);
  if (id_bound > kMaxIdBound) return fail(FAST_ERR_UNSUPPORTED, "%s: id_bound > 2^35", fn);
  if (dtype != FAST_F32 && dtype != FAST_BF16) return fail(FAST_ERR_INVALID_ARG, "%s: bad dtype", fn);
  if (!num_unique) return fail(FAST_ERR_INVALID_ARG, "%s: num_unique is NULL", fn);
  if (n > 0 && (!ids || !uni || !inv)) return fail(FAST_ERR_INVALID_ARG, "%s: NULL ids/uni/inv", fn);
  if (rows && (!table || D <= 0)) return fail(FAST_ERR_INVALID_ARG, "%s: rows requested without a table", fn);
  if (!slot_map && rows && id_bound > table_rows)
    return fail(FAST_ERR_INVALID_ARG, "%s: without a slot map id_bound (%lld) must be <= table_rows (%lld)",
                fn, (long long)id_bound, (long long)table_rows);
  const size_t need = dedup_layout(n, id_bound, nullptr, nullptr);
  if (!ws || ws_bytes < need)
    return fail(FAST_ERR_WORKSPACE, "%s: workspace %zu < %zu bytes", fn, ws_bytes, need);

  hipStream_t st = static_cast<hipStream_t>(stream);
  DedupWs w;
  dedup_layout(n, id_bound, static_cast<char*>(ws), &w);
  const int64_t W = (id_bound + 31) / 32;

  // 1. clear the bitmap, 2. mark ids
  if (W > 0) {
    const int64_t nb = (W + DD_THREADS - 1) / DD_THREADS;
    hipLaunchKernelGGL(k_fill_u32, dim3(uint32_t(nb < 4096 ? nb : 4096)), dim3(DD_THREADS), 0, st,
                       w.bitmap, W, 0u);
  }
  if (n > 0)
    hipLaunchKernelGGL(k_dedup_mark, dim3(uint32_t((n + DD_THREADS - 1) / DD_THREADS)),
                       dim3(DD_THREADS), 0, st, ids, n, id_bound, w.bitmap);
  // 3. word ranks (exclusive popcount prefix) and u
  hipError_t e = scan_launch(InPopc{w.bitmap}, OutPrefix{w.prefix}, W, w.scan_w, num_unique,
                             nullptr, st);
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
  // 4. uni, 5. inv
  if (W > 0)
    hipLaunchKernelGGL(k_dedup_uni, dim3(uint32_t((W + DD_THREADS - 1) / DD_THREADS)),
                       dim3(DD_THREADS), 0, st, w.bitmap, w.prefix, W, uni);
  if (n > 0)
    hipLaunchKernelGGL(k_dedup_inv, dim3(uint32_t((n + DD_THREADS - 1) / DD_THREADS)),
                       dim3(DD_THREADS), 0, st, ids, n, id_bound, w.bitmap, w.prefix, inv);

  // 6. rows through the slot map, miss flags, 7. ordered miss list
  const bool want_miss = miss || num_miss;
  if (rows || want_miss) {
    const int64_t row_bytes = int64_t(D > 0 ? D : 0) * elem_size(dtype);
    uint8_t* flags = want_miss ? w.flags : nullptr;
    if (rows && row_bytes > 0) {
      const bool a16 = row_bytes % 16 == 0 && aligned(table, 16) && aligned(rows, 16);
      const bool a8 = row_bytes % 8 == 0 && aligned(table, 8) && aligned(rows, 8);
      const bool a4 = row_bytes % 4 == 0 && aligned(table, 4) && aligned(rows, 4);
      const int64_t vb = a16 ? 16 : a8 ? 8 : a4 ? 4 : 2;
      if (row_bytes / vb > DD_THREADS)
        return fail(FAST_ERR_UNSUPPORTED, "%s: row of %lld bytes is too wide", fn, (long long)row_bytes);
      if (vb == 16)
        launch_gather<uint4>(uni, num_unique, table, table_rows, row_bytes, slot_map, rows, flags, n, st);
      else if (vb == 8)
        launch_gather<uint2>(uni, num_unique, table, table_rows, row_bytes, slot_map, rows, flags, n, st);
      else if (vb == 4)
        launch_gather<uint32_t>(uni, num_unique, table, table_rows, row_bytes, slot_map, rows, flags, n, st);
      else
        launch_gather<uint16_t>(uni, num_unique, table, table_rows, row_bytes, slot_map, rows, flags, n, st);
    } else {
      // flags only: one 4-byte "row" per id, nothing copied
      launch_gather<uint32_t>(uni, num_unique, nullptr, table_rows, 4, slot_map, nullptr, flags, n, st);
    }
    if (want_miss) {
      e = scan_launch(InFlags{w.flags, num_unique}, OutMiss{miss}, n, w.scan_n, num_miss, nullptr, st);
      if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
    }
  }
  return check_launch(fn);
}
