// dedup.hip -- within-batch id compression and row reconstruction (Sec. 4.2
// SlimCache: transfer unique ids once plus an inverse index; Sec. 5: the
// uni_ID / inv_Idx triple).
//
// MI355X design: ids live in a bounded universe [0, id_bound), so the sorted
// distinct set is a bitmap over that universe; the rank of an id is the
// exclusive popcount prefix of the bitmap words below it plus a popcount
// inside its word.  This is exact and deterministic whatever the id order or
// thread interleaving, and needs no sort.  The bitmap is built one of three
// ways, chosen from (n, id_bound) alone:
//   * byte map (id_bound <= 32 n): every id stores 1 into its own byte with a
//     plain store (racing stores of the same value are benign), then one
//     pass packs 32 bytes into each bitmap word -- O(n + id_bound) bytes,
//     no atomics at all;
//   * buckets (sparse universes): each workgroup merges its 2048 ids per
//     bitmap word in an LDS hash table, counts its merged words per universe
//     bucket (at most 4096 buckets of at most 2^19 ids) and writes them to
//     its own stage region grouped by bucket; one workgroup per bucket then
//     ORs the bucket's runs of every workgroup into an LDS bitmap and writes
//     the bucket's word records, ranked inside the bucket, and a scan over
//     the bucket totals gives each bucket's base rank.  Only LDS atomics;
//     every word record is written once, with no clearing pass;
//   * hashed atomics (universes too large for buckets, or batches with more
//     than 2^24 (bucket, workgroup) counts): the same LDS merge, then one
//     global atomicOr per merged word into a cleared bitmap.
// Rows are then copied with 16/8/4-byte vector moves, one thread per vector
// of a row, from the table slot that the optional cache slot map names (the
// slots are looked up with the unique ids, in the rank pass); rows whose
// vector count does not divide the workgroup are copied in chunks of 16 rows
// whose slots are staged in LDS first.
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "scan.h"

namespace fast {

constexpr int DD_THREADS = 256;

// Byte-map marking when the universe is at most this many times the batch.
constexpr int64_t BYTEMAP_RATIO = 32;

// Bucketed marking: a bucket spans 2^bits ids, bits in [10, 19] chosen so
// that there are about 512 buckets (its bitmap of 32 .. 16384 words fits in
// 64 KB of LDS); at most 4096 buckets, and at most 2^24 (bucket, workgroup)
// counts.
constexpr int BK_MIN_BITS = 10;
constexpr int BK_MAX_BITS = 19;
constexpr int64_t BK_TARGET_BUCKETS = 512;
constexpr int64_t BK_MAX_BUCKETS = 4096;
constexpr int64_t BK_MAX_COUNTS = int64_t(1) << 24;
constexpr int BK_MAX_WORDS = 1 << (BK_MAX_BITS - 5);

// Ids merged per workgroup in the LDS word hash (bucketed and hashed marking).
constexpr int MARK_ITEMS = 8;
constexpr int MARK_IDS = DD_THREADS * MARK_ITEMS;
constexpr int MARK_SLOTS = 2 * MARK_IDS;        // load factor <= 1/2: probing always ends
static_assert(MARK_SLOTS == 4096, "the hash below yields 12 bits");
constexpr uint32_t MARK_EMPTY = 0xffffffffu;     // never a word index (W <= 2^30)

enum MarkPath { MARK_BYTES, MARK_BUCKETS, MARK_HASH };

struct BkPlan {
  int bits = 0;       // 0: no bucketed plan for this universe and batch
  int64_t B = 0;      // buckets
  int64_t nblk = 0;   // merging workgroups (MARK_IDS ids each)
};

static BkPlan bucket_plan(int64_t n, int64_t id_bound) {
  BkPlan p;
  int bits = BK_MIN_BITS;
  while (bits < BK_MAX_BITS && ((id_bound + (int64_t(1) << bits) - 1) >> bits) > BK_TARGET_BUCKETS)
    ++bits;
  const int64_t B = (id_bound + (int64_t(1) << bits) - 1) >> bits;
  const int64_t nblk = (n + MARK_IDS - 1) / MARK_IDS;
  if (B > BK_MAX_BUCKETS || B * nblk > BK_MAX_COUNTS) return p;
  p.bits = bits;
  p.B = B;
  p.nblk = nblk;
  return p;
}

static MarkPath mark_path(int64_t n, int64_t id_bound, BkPlan* plan) {
  static const int mode = [] {
    const char* e = std::getenv("FAST_DEDUP_MARK");   // tuning override: bytemap | bucket | hash
    if (!e) return 0;
    return std::strcmp(e, "bytemap") == 0 ? 1 : std::strcmp(e, "hash") == 0 ? 2
         : std::strcmp(e, "bucket") == 0 ? 3 : 0;
  }();
  const BkPlan p = bucket_plan(n, id_bound);
  if (plan) *plan = p;
  if (mode == 1) return MARK_BYTES;
  if (mode == 2) return MARK_HASH;
  if (mode == 3) return p.bits ? MARK_BUCKETS : MARK_HASH;
  if (id_bound <= BYTEMAP_RATIO * (n > 0 ? n : 1)) return MARK_BYTES;
  return p.bits ? MARK_BUCKETS : MARK_HASH;
}

// Word record w: .x = bits of ids 32w .. 32w+31, .y = number of set bits in
// all words before w (the rank of the word's first id).  Keeping both in one
// 8-byte record makes the inverse lookup of an id a single random load.
struct DedupWs {
  uint8_t* bytemap;   // [32 W] (byte-map marking only)
  uint2* words;       // [W] word records
  void* scan_w;       // scan workspace over W words (byte map, hash)
  uint8_t* flags;     // [n] miss flags
  int32_t* slots;     // [n] table slot of each unique id (with a slot map)
  void* scan_n;       // scan workspace over n flags
  uint16_t* bk_loff;  // [nblk x (B + 1)] start of each bucket's run in workgroup g's stage, then its total
  uint2* bk_stage;    // [nblk x MARK_IDS] each workgroup's (word in bucket, bits), grouped by bucket
  uint32_t* bk_base;  // [B + 1] distinct ids per bucket, then the bucket's base rank (and u)
};

static size_t dedup_layout(int64_t n, int64_t id_bound, char* base, DedupWs* ws) {
  const int64_t W = (id_bound + 31) / 32;
  BkPlan p;
  const MarkPath path = mark_path(n, id_bound, &p);
  const bool bk = path == MARK_BUCKETS;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += align_up(bytes, 256);
    return base ? base + o : nullptr;
  };
  char* by = take(path == MARK_BYTES ? size_t(W) * 32 : 0);
  char* wr = take(size_t(W) * 8);
  char* sw = take(bk ? 0 : scan_workspace(W));
  char* fl = take(size_t(n));
  char* sl = take(size_t(n) * 4);
  char* sn = take(scan_workspace(n));
  char* lo = take(bk ? size_t((p.B + 1) * p.nblk) * 2 : 0);
  char* sg = take(bk ? size_t(p.nblk) * MARK_IDS * 8 : 0);
  char* bb = take(bk ? size_t(p.B + 1) * 4 : 0);
  if (ws) {
    ws->bk_loff = reinterpret_cast<uint16_t*>(lo);
    ws->bk_stage = reinterpret_cast<uint2*>(sg);
    ws->bytemap = reinterpret_cast<uint8_t*>(by);
    ws->words = reinterpret_cast<uint2*>(wr);
    ws->scan_w = sw;
    ws->flags = reinterpret_cast<uint8_t*>(fl);
    ws->slots = reinterpret_cast<int32_t*>(sl);
    ws->scan_n = sn;
    ws->bk_base = reinterpret_cast<uint32_t*>(bb);
  }
  return off;
}

__global__ void __launch_bounds__(64) k_set_i64(int64_t* p, int64_t v) {
  if (threadIdx.x == 0) *p = v;
}

__global__ void __launch_bounds__(DD_THREADS) k_fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  for (int64_t i = int64_t(blockIdx.x) * DD_THREADS + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * DD_THREADS)
    p[i] = v;
}

__global__ void __launch_bounds__(DD_THREADS) k_fill_u128(uint4* p, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * DD_THREADS + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * DD_THREADS)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

__global__ void __launch_bounds__(DD_THREADS) k_dedup_mark_bytes(const int64_t* __restrict__ ids,
                                                                 int64_t n, int64_t id_bound,
                                                                 uint8_t* bytemap) {
  const int64_t i = int64_t(blockIdx.x) * DD_THREADS + threadIdx.x;
  if (i >= n) return;
  const int64_t id = ids[i];
  if (id >= 0 && id < id_bound) bytemap[id] = 1;
}

// bitmap word w <- bytes 32w .. 32w+31 of the byte map (each 0 or 1).  A
// workgroup packs one scan tile of words (SCAN_ITEMS per thread, striped)
// and stores the tile's popcount sum, the reduce step of the rank scan.
__global__ void __launch_bounds__(SCAN_THREADS) k_dedup_pack(const uint4* __restrict__ bytemap,
                                                             int64_t W, uint2* __restrict__ words,
                                                             uint32_t* __restrict__ tsum) {
  __shared__ uint32_t lds4[4];
  const int64_t w0 = int64_t(blockIdx.x) * SCAN_TILE;
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    const int64_t w = w0 + k * SCAN_THREADS + threadIdx.x;
    if (w < W) {
      const uint4 a = bytemap[2 * w], b = bytemap[2 * w + 1];
      const uint32_t q[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
      uint32_t word = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        // bytes b0..b3 in {0,1} at bits 0,8,16,24 -> b0 | b1<<1 | b2<<2 | b3<<3 at bit 24
        const uint32_t nib = ((q[j] & 0x01010101u) * 0x01020408u) >> 24;
        word |= (nib & 0xfu) << (4 * j);
      }
      words[w].x = word;
      c += __popc(word);
    }
  }
  uint32_t total;
  block_exclusive_scan(c, lds4, total);
  if (threadIdx.x == 0) tsum[blockIdx.x] = total;
}

// Marking: each workgroup takes MARK_ITEMS ids per thread and first merges
// them in an LDS hash table keyed by bitmap word (open addressing, LDS
// atomics), so a word receives at most one global atomicOr per workgroup.
// Zipf-hot ids (the hottest is ~12% of a batch) would otherwise serialise
// hundreds of thousands of atomics on one L2 address.
__global__ void __launch_bounds__(DD_THREADS) k_dedup_mark(const int64_t* __restrict__ ids,
                                                           int64_t n, int64_t id_bound,
                                                           uint2* words) {
  __shared__ uint32_t keys[MARK_SLOTS];
  __shared__ uint32_t bits[MARK_SLOTS];
  for (int s = threadIdx.x; s < MARK_SLOTS; s += DD_THREADS) {
    keys[s] = MARK_EMPTY;
    bits[s] = 0u;
  }
  __syncthreads();
  const int64_t base = int64_t(blockIdx.x) * MARK_IDS;
#pragma unroll
  for (int k = 0; k < MARK_ITEMS; ++k) {
    const int64_t i = base + k * DD_THREADS + threadIdx.x;
    if (i >= n) break;
    const int64_t id = ids[i];
    if (id < 0 || id >= id_bound) continue;
    const uint32_t w = uint32_t(id >> 5);
    const uint32_t bit = 1u << (id & 31);
    uint32_t h = (w * 2654435761u) >> (32 - 12);     // Fibonacci hashing into 4096 slots
    for (;;) {
      const uint32_t prev = atomicCAS(&keys[h], MARK_EMPTY, w);
      if (prev == MARK_EMPTY || prev == w) {
        atomicOr(&bits[h], bit);
        break;
      }
      h = (h + 1) & (MARK_SLOTS - 1);
    }
  }
  __syncthreads();
  for (int s = threadIdx.x; s < MARK_SLOTS; s += DD_THREADS) {
    const uint32_t w = keys[s];
    if (w != MARK_EMPTY) atomicOr(&words[w].x, bits[s]);
  }
}

// LDS merge of one workgroup's MARK_IDS ids by bitmap word (the hash table
// of the hashed marking): on return keys[s] holds a word index or
// MARK_EMPTY and bits[s] the OR of that word's bits among the ids.  All ids
// are loaded before the first insertion.
__device__ __forceinline__ void merge_words(const int64_t* __restrict__ ids, int64_t n,
                                            int64_t id_bound, uint32_t* keys, uint32_t* bits) {
  for (int s = threadIdx.x; s < MARK_SLOTS; s += DD_THREADS) {
    keys[s] = MARK_EMPTY;
    bits[s] = 0u;
  }
  const int64_t base = int64_t(blockIdx.x) * MARK_IDS;
  int64_t v[MARK_ITEMS];
#pragma unroll
  for (int k = 0; k < MARK_ITEMS; ++k) {
    const int64_t i = base + k * DD_THREADS + threadIdx.x;
    v[k] = i < n ? ids[i] : int64_t(-1);
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < MARK_ITEMS; ++k) {
    const int64_t id = v[k];
    if (id < 0 || id >= id_bound) continue;
    const uint32_t w = uint32_t(id >> 5);
    const uint32_t bit = 1u << (id & 31);
    uint32_t h = (w * 2654435761u) >> (32 - 12);     // Fibonacci hashing into 4096 slots
    for (;;) {
      const uint32_t prev = atomicCAS(&keys[h], MARK_EMPTY, w);
      if (prev == MARK_EMPTY || prev == w) {
        atomicOr(&bits[h], bit);
        break;
      }
      h = (h + 1) & (MARK_SLOTS - 1);
    }
  }
  __syncthreads();
}

// Bucketed marking, staged form: workgroup g merges its ids by word once,
// counts the merged words per bucket, and writes them to its own stage
// region grouped by bucket, with the start of every bucket's run (and, at
// index B, the total) in its own row loff[g (B + 1) ...] -- one contiguous
// row per workgroup, so the table is written in whole cache lines; a run's
// length is the difference of two neighbouring starts (at most MARK_IDS, so
// 16 bits hold them).  No scan of the counts and no second merge are needed
// before the buckets are marked.
__global__ void __launch_bounds__(DD_THREADS) k_bk_stage(const int64_t* __restrict__ ids, int64_t n,
                                                         int64_t id_bound, int wshift, int B,
                                                         uint16_t* __restrict__ loff,
                                                         uint2* __restrict__ stage) {
  static_assert(MARK_IDS < 65536, "run starts are 16-bit");
  __shared__ uint32_t keys[MARK_SLOTS];
  __shared__ uint32_t bits[MARK_SLOTS];
  __shared__ uint32_t h[BK_MAX_BUCKETS + 1];
  __shared__ uint32_t lds4[4];
  for (int b = threadIdx.x; b < B; b += DD_THREADS) h[b] = 0u;
  merge_words(ids, n, id_bound, keys, bits);
  for (int s = threadIdx.x; s < MARK_SLOTS; s += DD_THREADS) {
    const uint32_t w = keys[s];
    if (w != MARK_EMPTY) atomicAdd(&h[w >> wshift], 1u);
  }
  __syncthreads();
  // exclusive prefix of h over the buckets: thread t owns buckets
  // [t PER, (t + 1) PER); h becomes the run starts, h[B] the total
  constexpr int PER = BK_MAX_BUCKETS / DD_THREADS;
  const int b0 = threadIdx.x * PER;
  uint32_t c[PER], sum = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    c[k] = b0 + k < B ? h[b0 + k] : 0u;
    sum += c[k];
  }
  uint32_t tot;
  uint32_t run = block_exclusive_scan(sum, lds4, tot);
  __syncthreads();                                   // every h read before it is rewritten
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    if (b0 + k < B) h[b0 + k] = run;
    run += c[k];
  }
  if (threadIdx.x == 0) h[B] = tot;
  __syncthreads();
  uint16_t* __restrict__ row = loff + int64_t(blockIdx.x) * (B + 1);
  for (int b = threadIdx.x; b <= B; b += DD_THREADS) row[b] = uint16_t(h[b]);
  __syncthreads();                                   // starts stored before h turns into cursors
  const uint32_t low = (1u << wshift) - 1u;
  uint2* __restrict__ mine = stage + int64_t(blockIdx.x) * MARK_IDS;
  for (int s = threadIdx.x; s < MARK_SLOTS; s += DD_THREADS) {
    const uint32_t w = keys[s];
    if (w != MARK_EMPTY) {
      const uint32_t pos = atomicAdd(&h[w >> wshift], 1u);
      mine[pos] = make_uint2(w & low, bits[s]);
    }
  }
}

// Bucketed marking, one workgroup per bucket of 2^wshift words: OR the
// bucket's run of every workgroup's stage into an LDS bitmap, then write
// every record of the bucket below W with its rank inside the bucket --
// each thread takes 4 consecutive words per block-wide scan (1024 words per
// scan) and stores them as two 16-byte record pairs -- and leave the
// bucket's distinct-id count in total[b].  Buckets are spread over the XCDs
// in contiguous ranges (xcd_tile), so the neighbouring buckets that share
// the cache lines of the run-start rows and of the stage runs read them
// through the same L2.
__global__ void __launch_bounds__(DD_THREADS) k_bk_mark(const uint16_t* __restrict__ loff,
                                                        const uint2* __restrict__ stage, int nblk,
                                                        int B, int wshift, int64_t W,
                                                        uint2* __restrict__ words,
                                                        uint32_t* __restrict__ total) {
  __shared__ uint4 bm4[BK_MAX_WORDS / 4];
  __shared__ uint32_t lds4[4];
  uint32_t* bm = reinterpret_cast<uint32_t*>(bm4);
  const int WB = 1 << wshift;                     // a multiple of 32
  const int b = int(xcd_tile(blockIdx.x, gridDim.x));
  for (int j = threadIdx.x; j < WB; j += DD_THREADS) bm[j] = 0u;
  __syncthreads();
  {
    // thread t ORs the runs of workgroups t, t + 256, ...; the
    // heads of 4 runs are loaded together, then the first 8 entries of all
    // 4 runs, then the ORs (runs hold about 4 entries: n / (nblk B))
    constexpr int G = 4, J = 8;
    for (int g0 = threadIdx.x; g0 < nblk; g0 += G * DD_THREADS) {
      uint32_t cnt[G], at[G];
#pragma unroll
      for (int k = 0; k < G; ++k) {
        const int g = g0 + k * DD_THREADS;
        const uint16_t* r = loff + int64_t(g) * (B + 1) + b;
        at[k] = g < nblk ? r[0] : 0u;
        cnt[k] = g < nblk ? uint32_t(r[1]) - at[k] : 0u;
      }
      uint2 x[G][J];
#pragma unroll
      for (int k = 0; k < G; ++k)
#pragma unroll
        for (int j = 0; j < J; ++j)
          x[k][j] = uint32_t(j) < cnt[k]
                        ? stage[int64_t(g0 + k * DD_THREADS) * MARK_IDS + at[k] + j]
                        : make_uint2(0u, 0u);
#pragma unroll
      for (int k = 0; k < G; ++k)
#pragma unroll
        for (int j = 0; j < J; ++j)
          if (x[k][j].y) atomicOr(&bm[x[k][j].x], x[k][j].y);
#pragma unroll
      for (int k = 0; k < G; ++k)
        for (uint32_t i = J; i < cnt[k]; ++i) {
          const uint2 y = stage[int64_t(g0 + k * DD_THREADS) * MARK_IDS + at[k] + i];
          atomicOr(&bm[y.x], y.y);
        }
    }
  }
  __syncthreads();
  const int64_t w0 = int64_t(b) * WB;
  uint32_t carry = 0;
  for (int j0 = 0; j0 < WB; j0 += 4 * DD_THREADS) {
    const int j = j0 + 4 * threadIdx.x;
    const uint4 x = j < WB ? bm4[j >> 2] : make_uint4(0u, 0u, 0u, 0u);
    const uint32_t p0 = __popc(x.x), p1 = __popc(x.y), p2 = __popc(x.z), p3 = __popc(x.w);
    uint32_t tot;
    const uint32_t r0 = carry + block_exclusive_scan(p0 + p1 + p2 + p3, lds4, tot);
    const uint32_t r1 = r0 + p0, r2 = r1 + p1, r3 = r2 + p2;
    const int64_t w = w0 + j;
    if (j < WB && w + 3 < W) {
      uint4* dst = reinterpret_cast<uint4*>(words + w);   // w is a multiple of 4: 32-byte aligned
      dst[0] = make_uint4(x.x, r0, x.y, r1);
      dst[1] = make_uint4(x.z, r2, x.w, r3);
    } else if (j < WB) {
      if (w < W) words[w] = make_uint2(x.x, r0);
      if (w + 1 < W) words[w + 1] = make_uint2(x.y, r1);
      if (w + 2 < W) words[w + 2] = make_uint2(x.z, r2);
    }
    carry += tot;
  }
  if (threadIdx.x == 0) total[b] = carry;
}

struct InPopc {
  const uint2* wr;
  __device__ uint32_t operator()(int64_t i) const { return __popc(wr[i].x); }
};
struct OutPrefix {   // rewrites the whole record: contiguous 8-byte stores
  uint2* wr;
  __device__ void operator()(int64_t i, uint32_t prefix, uint32_t) const {
    wr[i] = make_uint2(wr[i].x, prefix);
  }
};

// uni: every set bit of word w is written at its rank.  With bucketed
// marking the record holds the rank inside the bucket of 2^wshift words and
// base[] the bucket's base rank; otherwise base is NULL.  With a slot map,
// the unique id's slot is looked up here too (slots[rank]), where the
// lookups of all ids are independent, rather than inside the row copy.
__device__ __forceinline__ void dedup_uni_word(const uint2* __restrict__ words, int64_t w,
                                               const uint32_t* __restrict__ base, int wshift,
                                               int64_t* __restrict__ uni,
                                               const int32_t* __restrict__ slot_map,
                                               int32_t* __restrict__ slots) {
  const uint2 rec = words[w];
  uint32_t bits = rec.x;
  uint32_t r = rec.y + (base ? base[w >> wshift] : 0u);
  while (bits) {
    const int b = __ffs(bits) - 1;
    const int64_t id = (w << 5) + b;
    uni[r] = id;
    if (slots) slots[r] = slot_map[id];
    ++r;
    bits &= bits - 1;
  }
}

// inv: the rank of the id's bit (-1 for an id outside [0, id_bound)).
__device__ __forceinline__ void dedup_inv_id(const int64_t* __restrict__ ids, int64_t i,
                                             int64_t id_bound, const uint2* __restrict__ words,
                                             const uint32_t* __restrict__ base, int wshift,
                                             int32_t* __restrict__ inv) {
  const int64_t id = ids[i];
  if (id < 0 || id >= id_bound) {
    inv[i] = -1;
    return;
  }
  const int64_t w = id >> 5;
  const uint2 rec = words[w];
  const uint32_t below = rec.x & ((1u << (id & 31)) - 1u);
  inv[i] = int32_t(rec.y + (base ? base[w >> wshift] : 0u) + __popc(below));
}

// uni and inv in one launch: workgroups [0, nbw) take 256 words each, the
// rest 256 ids each.  zero_miss, when given, is set to 0 by the first thread
// (a batch that cannot miss), saving a launch of its own.
__global__ void __launch_bounds__(DD_THREADS) k_dedup_uni_inv(const uint2* __restrict__ words,
                                                              int64_t W,
                                                              const uint32_t* __restrict__ base,
                                                              int wshift, int64_t* __restrict__ uni,
                                                              const int64_t* __restrict__ ids,
                                                              int64_t n, int64_t id_bound,
                                                              int32_t* __restrict__ inv,
                                                              const int32_t* __restrict__ slot_map,
                                                              int32_t* __restrict__ slots,
                                                              uint32_t nbw,
                                                              int64_t* __restrict__ zero_miss) {
  if (zero_miss && blockIdx.x == 0 && threadIdx.x == 0) *zero_miss = 0;
  if (blockIdx.x < nbw) {
    const int64_t w = int64_t(blockIdx.x) * DD_THREADS + threadIdx.x;
    if (w < W) dedup_uni_word(words, w, base, wshift, uni, slot_map, slots);
  } else {
    const int64_t i = int64_t(blockIdx.x - nbw) * DD_THREADS + threadIdx.x;
    if (i < n) dedup_inv_id(ids, i, id_bound, words, base, wshift, inv);
  }
}

// Row copy: thread t of a block moves vector c of row k; a block covers
// `rpb` consecutive rows of `cpr` vectors each and strides over row groups,
// so the grid is sized for the machine, not for the worst-case n.  Rows
// k >= *num_unique are idle.  A slot outside [0, table_rows) flags a miss.
// (Several row groups per iteration measured slower than one.)
constexpr int GATHER_U = 1;
#ifndef FAST_GATHER_MAX_WG
#define FAST_GATHER_MAX_WG 8192
#endif

// Row moves with an optional streaming (non-temporal) policy: a gathered row
// is read once and written once per call.  Measured on MI355X, streaming paid
// for 16-byte moves (1e7-node fp32 batch: nodes 0.144 -> 0.125 ms, edges 0.307 -> 0.288
// ms, large nodes 0.171 -> 0.159 ms) and for 8-byte moves (344-byte rows of
// the large batch's edges: the whole call 0.688 -> 0.661 ms with streaming
// loads, step 2.548 -> 2.530 ms).  8-byte moves stream their stores whatever
// NT says: alone the copy runs the same, but it leaves no dirty lines for the
// attention that follows it in the step to write back (large step 2.626 ->
// 2.557 ms, its layer-1 forward 0.486 -> 0.453 ms).
template <typename V, bool NT>
__device__ __forceinline__ V gather_ld(const V* p) {
  if constexpr (NT && sizeof(V) == 16) {
    const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return __builtin_bit_cast(V, x);
  } else if constexpr (NT && sizeof(V) == 8) {
    const u32x2 x = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
    return __builtin_bit_cast(V, x);
  } else {
    return *p;
  }
}
template <typename V, bool NT>
__device__ __forceinline__ void gather_st(V* p, const V& v) {
  if constexpr (NT && sizeof(V) == 16)
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), reinterpret_cast<u32x4*>(p));
  else if constexpr (sizeof(V) == 8)
    __builtin_nontemporal_store(__builtin_bit_cast(u32x2, v), reinterpret_cast<u32x2*>(p));
  else
    *p = v;
}

template <typename V, bool NT>
__global__ void __launch_bounds__(DD_THREADS) k_gather_rows(const int64_t* __restrict__ uni,
                                                            const int64_t* __restrict__ num_unique,
                                                            const V* __restrict__ table,
                                                            int64_t table_rows, int cpr, int rpb,
                                                            const int32_t* __restrict__ slots,
                                                            V* __restrict__ rows,
                                                            uint8_t* __restrict__ flags) {
  const int64_t u = *num_unique;
  const int r = threadIdx.x / cpr;
  const int c = threadIdx.x - r * cpr;
  if (r >= rpb) return;
  const int64_t step = int64_t(gridDim.x) * rpb;
  for (int64_t k0 = int64_t(blockIdx.x) * rpb + r; k0 < u; k0 += step * GATHER_U) {
    int64_t slot[GATHER_U];
#pragma unroll
    for (int j = 0; j < GATHER_U; ++j) {
      const int64_t k = k0 + j * step;
      slot[j] = -1;
      if (k < u) slot[j] = slots ? int64_t(slots[k]) : uni[k];
    }
    V val[GATHER_U];
#pragma unroll
    for (int j = 0; j < GATHER_U; ++j) {
      const bool hit = slot[j] >= 0 && slot[j] < table_rows;
      if (hit && rows) val[j] = gather_ld<V, NT>(table + slot[j] * cpr + c);
    }
#pragma unroll
    for (int j = 0; j < GATHER_U; ++j) {
      const int64_t k = k0 + j * step;
      if (k >= u) break;
      const bool hit = slot[j] >= 0 && slot[j] < table_rows;
      if (c == 0 && flags) flags[k] = hit ? 0 : 1;
      if (hit && rows) gather_st<V, NT>(rows + k * cpr + c, val[j]);
    }
  }
}

// Chunked row copy, for rows whose vector count does not divide the
// workgroup (400-, 344- and 688-byte rows: 25 or 43 vectors, so a row-per-
// lane-group mapping leaves lanes idle and chains slot load -> row load ->
// store for a few rows at a time): a workgroup takes GATHER_CHUNK unique rows
// at a time, stages their slots in LDS with one load per row, then copies the
// chunk's vectors with every thread holding GATHER_UNROLL loads in flight
// before its stores.  Measured on MI355X (whole dedup+gather call): 344-byte
// bf16 rows 0.828 -> 0.721 ms, 688-byte rows through a slot map 0.250 ->
// 0.233 ms, 400-byte rows 0.128 -> 0.126 ms; chunks of 8 / 24 / 32 / 64 rows
// and 8 loads in flight were slower, and 256-byte rows (16 vectors, which
// tile the workgroup exactly) stay faster with the row mapping (0.161 against
// 0.166 ms).
constexpr int GATHER_CHUNK = 16;
constexpr int GATHER_UNROLL = 4;
template <typename V, bool NT, int R>
__global__ void __launch_bounds__(DD_THREADS) k_gather_chunk(const int64_t* __restrict__ uni,
                                                             const int64_t* __restrict__ num_unique,
                                                             const V* __restrict__ table,
                                                             int64_t table_rows, int cpr,
                                                             const int32_t* __restrict__ slots,
                                                             V* __restrict__ rows,
                                                             uint8_t* __restrict__ flags) {
  constexpr int U = GATHER_UNROLL;
  __shared__ int64_t s_slot[R];
  const int64_t u = *num_unique;
  const int nv = R * cpr;
  for (int64_t k0 = int64_t(blockIdx.x) * R; k0 < u; k0 += int64_t(gridDim.x) * R) {
    if (threadIdx.x < R) {
      const int64_t k = k0 + threadIdx.x;
      int64_t sl = -1;
      if (k < u) {
        sl = slots ? int64_t(slots[k]) : uni[k];
        const bool hit = sl >= 0 && sl < table_rows;
        if (flags) flags[k] = hit ? 0 : 1;
        if (!hit) sl = -1;
      }
      s_slot[threadIdx.x] = sl;
    }
    __syncthreads();
    if (rows) {
      for (int v0 = threadIdx.x; v0 < nv; v0 += U * DD_THREADS) {
        V val[U];
        int64_t dst[U];
#pragma unroll
        for (int j = 0; j < U; ++j) {
          const int v = v0 + j * DD_THREADS;
          dst[j] = -1;
          if (v < nv) {
            const int r = v / cpr, c = v - r * cpr;
            const int64_t sl = s_slot[r];
            if (sl >= 0) {
              val[j] = gather_ld<V, NT>(table + sl * cpr + c);
              dst[j] = (k0 + r) * cpr + c;
            }
          }
        }
#pragma unroll
        for (int j = 0; j < U; ++j)
          if (dst[j] >= 0) gather_st<V, NT>(rows + dst[j], val[j]);
      }
    }
    __syncthreads();
  }
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

static bool gather_stream_enabled() {
  static const bool on = [] {
    const char* e = std::getenv("FAST_GATHER_STREAM");   // tuning override: 0 turns it off
    return !(e && std::strcmp(e, "0") == 0);
  }();
  return on;
}

template <typename V>
static void launch_gather(const int64_t* uni, const int64_t* num_unique, const void* table,
                          int64_t table_rows, int64_t row_bytes, const int32_t* slots,
                          void* rows, uint8_t* flags, int64_t cap, hipStream_t st) {
  const int cpr = int(row_bytes / int64_t(sizeof(V)));
  const int rpb = cpr >= DD_THREADS ? 1 : DD_THREADS / cpr;
  int64_t nb = (cap + rpb - 1) / rpb;
  if (nb > FAST_GATHER_MAX_WG) nb = FAST_GATHER_MAX_WG;   // workgroups stride over the rest
  if (nb == 0) return;
  if (DD_THREADS % cpr != 0) {
    int64_t nbc = (cap + GATHER_CHUNK - 1) / GATHER_CHUNK;
    if (nbc > FAST_GATHER_MAX_WG) nbc = FAST_GATHER_MAX_WG;
    if ((sizeof(V) == 16 || sizeof(V) == 8) && gather_stream_enabled())
      hipLaunchKernelGGL((k_gather_chunk<V, true, GATHER_CHUNK>), dim3(uint32_t(nbc)),
                         dim3(DD_THREADS), 0, st, uni, num_unique, static_cast<const V*>(table),
                         table_rows, cpr, slots, static_cast<V*>(rows), flags);
    else
      hipLaunchKernelGGL((k_gather_chunk<V, false, GATHER_CHUNK>), dim3(uint32_t(nbc)),
                         dim3(DD_THREADS), 0, st, uni, num_unique, static_cast<const V*>(table),
                         table_rows, cpr, slots, static_cast<V*>(rows), flags);
    return;
  }
  if (cpr <= DD_THREADS) {
    if (sizeof(V) == 16 && gather_stream_enabled())
      hipLaunchKernelGGL((k_gather_rows<V, true>), dim3(uint32_t(nb)), dim3(DD_THREADS), 0, st, uni,
                         num_unique, static_cast<const V*>(table), table_rows, cpr, rpb, slots,
                         static_cast<V*>(rows), flags);
    else
      hipLaunchKernelGGL((k_gather_rows<V, false>), dim3(uint32_t(nb)), dim3(DD_THREADS), 0, st, uni,
                         num_unique, static_cast<const V*>(table), table_rows, cpr, rpb, slots,
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

// Both entry points: argument checks, then the launches on workspace ws.
static fast_status_t dedup_gather_run(const char* fn, const int64_t* ids, int64_t n,
                                      int64_t id_bound, const void* table, int64_t table_rows,
                                      int D, fast_dtype_t dtype, const int32_t* slot_map,
                                      int64_t* uni, int32_t* inv, int64_t* num_unique, void* rows,
                                      int32_t* miss, int64_t* num_miss, void* ws, size_t ws_bytes,
                                      fast_stream_t stream) {
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
  if (!aligned(ws, 256)) return fail(FAST_ERR_UNSUPPORTED, "%s: workspace not 256-byte aligned", fn);

  hipStream_t st = static_cast<hipStream_t>(stream);
  DedupWs w;
  dedup_layout(n, id_bound, static_cast<char*>(ws), &w);
  const int64_t W = (id_bound + 31) / 32;

  BkPlan p;
  const MarkPath path = mark_path(n, id_bound, &p);
  const uint32_t* base = nullptr;   // bucket base ranks (bucketed marking only)
  const int wshift = path == MARK_BUCKETS ? p.bits - 5 : 0;
  hipError_t e = hipSuccess;
  // 1. mark ids, 2. word ranks (exclusive popcount prefix) and u
  if (path == MARK_BUCKETS) {
    const int B = int(p.B), nblk = int(p.nblk);
    if (nblk > 0) {
      hipLaunchKernelGGL(k_bk_stage, dim3(uint32_t(nblk)), dim3(DD_THREADS), 0, st, ids, n, id_bound,
                         wshift, B, w.bk_loff, w.bk_stage);
    }
    if (B > 0) {
      hipLaunchKernelGGL(k_bk_mark, dim3(uint32_t(B)), dim3(DD_THREADS), 0, st, w.bk_loff,
                         w.bk_stage, nblk, B, wshift, W, w.words, w.bk_base);
    }
    // at most 4096 bucket totals: one workgroup scans them in place
    hipLaunchKernelGGL(k_scan_top<uint32_t>, dim3(1), dim3(SCAN_THREADS), 0, st, w.bk_base, p.B,
                       num_unique, static_cast<int32_t*>(nullptr));
    base = w.bk_base;
  } else {
    if (path == MARK_BYTES) {
      if (W > 0) {
        const int64_t n16 = W * 2;        // 32 W bytes as 16-byte vectors
        const int64_t nb = (n16 + DD_THREADS - 1) / DD_THREADS;
        hipLaunchKernelGGL(k_fill_u128, dim3(uint32_t(nb < 8192 ? nb : 8192)), dim3(DD_THREADS), 0,
                           st, reinterpret_cast<uint4*>(w.bytemap), n16);
      }
      if (n > 0)
        hipLaunchKernelGGL(k_dedup_mark_bytes, dim3(uint32_t((n + DD_THREADS - 1) / DD_THREADS)),
                           dim3(DD_THREADS), 0, st, ids, n, id_bound, w.bytemap);
      if (W > 0)
        hipLaunchKernelGGL(k_dedup_pack, dim3(uint32_t(scan_tiles(W))), dim3(SCAN_THREADS), 0, st,
                           reinterpret_cast<const uint4*>(w.bytemap), W, w.words,
                           static_cast<uint32_t*>(w.scan_w));
      e = scan_finish_launch(InPopc{w.words}, OutPrefix{w.words}, W, w.scan_w, num_unique, nullptr,
                             st);
    } else {
      if (W > 0) {
        const int64_t nb = (2 * W + DD_THREADS - 1) / DD_THREADS;
        hipLaunchKernelGGL(k_fill_u32, dim3(uint32_t(nb < 4096 ? nb : 4096)), dim3(DD_THREADS), 0,
                           st, reinterpret_cast<uint32_t*>(w.words), 2 * W, 0u);
      }
      if (n > 0)
        hipLaunchKernelGGL(k_dedup_mark, dim3(uint32_t((n + MARK_IDS - 1) / MARK_IDS)),
                           dim3(DD_THREADS), 0, st, ids, n, id_bound, w.words);
      e = scan_launch(InPopc{w.words}, OutPrefix{w.words}, W, w.scan_w, num_unique, nullptr, st);
    }
  }
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
  // 3. uni and inv (and the slots of the unique ids, when rows or misses
  // go through a slot map).  Without a slot map and with a row for every id
  // (id_bound <= table_rows) nothing can miss: no flags, no scan, and the
  // miss count is 0.
  const bool all_hit = !slot_map && id_bound <= table_rows;
  const bool want_miss = (miss || num_miss) && !all_hit;
  int32_t* slots = slot_map && (rows || want_miss) ? w.slots : nullptr;
  const int64_t nbw = (W + DD_THREADS - 1) / DD_THREADS, nbi = (n + DD_THREADS - 1) / DD_THREADS;
  int64_t* zero_miss = all_hit ? num_miss : nullptr;
  if (nbw + nbi > 0)
    hipLaunchKernelGGL(k_dedup_uni_inv, dim3(uint32_t(nbw + nbi)), dim3(DD_THREADS), 0, st, w.words, W,
                       base, wshift, uni, ids, n, id_bound, inv, slot_map, slots, uint32_t(nbw),
                       zero_miss);
  else if (zero_miss)
    hipLaunchKernelGGL(k_set_i64, dim3(1), dim3(64), 0, st, zero_miss, int64_t(0));

  // 4. rows from their slots, miss flags, 5. ordered miss list.
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
        launch_gather<uint4>(uni, num_unique, table, table_rows, row_bytes, slots, rows, flags, n, st);
      else if (vb == 8)
        launch_gather<uint2>(uni, num_unique, table, table_rows, row_bytes, slots, rows, flags, n, st);
      else if (vb == 4)
        launch_gather<uint32_t>(uni, num_unique, table, table_rows, row_bytes, slots, rows, flags, n, st);
      else
        launch_gather<uint16_t>(uni, num_unique, table, table_rows, row_bytes, slots, rows, flags, n, st);
    } else {
      // flags only: one 4-byte "row" per id, nothing copied
      launch_gather<uint32_t>(uni, num_unique, nullptr, table_rows, 4, slots, nullptr, flags, n, st);
    }
    if (want_miss) {
      e = scan_launch(InFlags{w.flags, num_unique}, OutMiss{miss}, n, w.scan_n, num_miss, nullptr, st);
      if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
    }
  }
  return check_launch(fn);
}

extern "C" fast_status_t fast_dedup_gather(const int64_t* ids, int64_t n, int64_t id_bound,
                                           const void* table, int64_t table_rows, int D,
                                           fast_dtype_t dtype, const int32_t* slot_map,
                                           int64_t* uni, int32_t* inv, int64_t* num_unique,
                                           void* rows, int32_t* miss, int64_t* num_miss,
                                           void* ws, size_t ws_bytes, fast_stream_t stream) {
  return dedup_gather_run("fast_dedup_gather", ids, n, id_bound, table, table_rows, D, dtype,
                          slot_map, uni, inv, num_unique, rows, miss, num_miss, ws, ws_bytes,
                          stream);
}

// ---------------------------------------------------------------- no allocation
// Scratch of fast_dedup_gather_noalloc: a fixed device array in this code
// object, so the call needs no workspace argument and allocates nothing.
// Every GPU the library runs on holds its own copy until the process ends.
// In host code `scratch` names a host-side stand-in, not device memory: only
// the per-device address from hipGetSymbolAddress is passed to kernels.
static __device__ __align__(256) unsigned char scratch[FAST_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
static fast_status_t scratch_for_current_device(const char* fn, hipStream_t st, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: hipGetDevice: %s", fn, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(FAST_ERR_UNSUPPORTED, "%s: device %d beyond the %d this library tracks", fn, dev,
                kMaxDevices);
  if (st) {   // the kernels run on the stream's device: it must be the current one
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(st, &sdev);
    if (e != hipSuccess)
      return fail(FAST_ERR_HIP, "%s: hipStreamGetDevice: %s", fn, hipGetErrorString(e));
    if (sdev != dev)
      return fail(FAST_ERR_INVALID_ARG, "%s: stream of device %d but device %d is current", fn,
                  int(sdev), dev);
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(FAST_ERR_HIP, "%s: hipGetSymbolAddress(scratch): %s", fn, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FAST_OK;
}

extern "C" fast_status_t fast_dedup_gather_noalloc(const int64_t* ids, int64_t n, int64_t id_bound,
                                                   const void* table, int64_t table_rows, int D,
                                                   fast_dtype_t dtype, const int32_t* slot_map,
                                                   int64_t* uni, int32_t* inv,
                                                   int64_t* num_unique, void* rows, int32_t* miss,
                                                   int64_t* num_miss, fast_stream_t stream) {
  const char* fn = "fast_dedup_gather_noalloc";
  if (n < 0 || id_bound < 0) return fail(FAST_ERR_INVALID_ARG, "%s: negative size", fn);
  if (id_bound > kMaxIdBound) return fail(FAST_ERR_UNSUPPORTED, "%s: id_bound > 2^35", fn);
  const size_t need = dedup_layout(n, id_bound, nullptr, nullptr);
  if (need > size_t(FAST_NOALLOC_SCRATCH_BYTES))
    return fail(FAST_ERR_UNSUPPORTED,
                "%s: n = %lld ids over id_bound = %lld need %zu bytes of scratch, more than the "
                "%zu this variant holds; call fast_dedup_gather with a workspace",
                fn, (long long)n, (long long)id_bound, need, size_t(FAST_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  const fast_status_t s = scratch_for_current_device(fn, static_cast<hipStream_t>(stream), &ws);
  if (s != FAST_OK) return s;
  return dedup_gather_run(fn, ids, n, id_bound, table, table_rows, D, dtype, slot_map, uni, inv,
                          num_unique, rows, miss, num_miss, ws, size_t(FAST_NOALLOC_SCRATCH_BYTES),
                          stream);
}
