// stream_ceiling.hip -- the HBM streaming ceilings of the GPU it runs on,
// for comparison with the operators' achieved bandwidth.  Plain kernels over
// 2 GiB buffers (8x the 256 MB last-level cache): one 16-byte element per
// thread and one element per thread's lifetime (a grid of n / 256
// workgroups), the shape that measured fastest for every pattern on MI355X
// (grid-stride loops with 1k-64k workgroups ran 5-30 % slower).
//   read   : one stream in            write  : one stream out
//   copy   : one in, one out           mix22  : two in, two out (the shape of
//                                               the fused backward's K, V ->
//                                               dK, dV rows)
//   read_nt, write_nt, copy_nt: the first three with streaming
//                               (non-temporal) loads and stores
// Prints one JSON object: bytes moved, median time of `reps` launches, TB/s.
// (The seg10 variants show what the packed forward pays for its output
// rows: its K|V reads alone stream faster than the plain read above.)
//   stream_ceiling [reps] [--variants]
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t err_ = (x);                                                    \
    if (err_ != hipSuccess) {                                                 \
      std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(err_), __LINE__); \
      std::exit(1);                                                           \
    }                                                                         \
  } while (0)

constexpr int THREADS = 256;

__global__ void __launch_bounds__(THREADS) k_read(const u32x4* __restrict__ a, size_t n,
                                                  unsigned* __restrict__ sink) {
  const size_t i = size_t(blockIdx.x) * THREADS + threadIdx.x;
  if (i >= n) return;
  const u32x4 v = a[i];
  if ((v.x ^ v.y ^ v.z ^ v.w) == 0x9e3779b9u) sink[0] = 1u;   // keeps the load
}

__global__ void __launch_bounds__(THREADS) k_write(u32x4* __restrict__ a, size_t n) {
  const size_t i = size_t(blockIdx.x) * THREADS + threadIdx.x;
  if (i >= n) return;
  a[i] = (u32x4){unsigned(i), 1u, 2u, 3u};
}

__global__ void __launch_bounds__(THREADS) k_copy(const u32x4* __restrict__ a,
                                                  u32x4* __restrict__ b, size_t n) {
  const size_t i = size_t(blockIdx.x) * THREADS + threadIdx.x;
  if (i >= n) return;
  b[i] = a[i];
}

// The same three with streaming (non-temporal) loads and stores, the policy
// the library's kernels use for data they touch once.
__global__ void __launch_bounds__(THREADS) k_read_nt(const u32x4* __restrict__ a, size_t n,
                                                     unsigned* __restrict__ sink) {
  const size_t i = size_t(blockIdx.x) * THREADS + threadIdx.x;
  if (i >= n) return;
  const u32x4 v = __builtin_nontemporal_load(a + i);
  if ((v.x ^ v.y ^ v.z ^ v.w) == 0x9e3779b9u) sink[0] = 1u;
}

__global__ void __launch_bounds__(THREADS) k_write_nt(u32x4* __restrict__ a, size_t n) {
  const size_t i = size_t(blockIdx.x) * THREADS + threadIdx.x;
  if (i >= n) return;
  __builtin_nontemporal_store((u32x4){unsigned(i), 1u, 2u, 3u}, a + i);
}

__global__ void __launch_bounds__(THREADS) k_copy_nt(const u32x4* __restrict__ a,
                                                     u32x4* __restrict__ b, size_t n) {
  const size_t i = size_t(blockIdx.x) * THREADS + threadIdx.x;
  if (i >= n) return;
  __builtin_nontemporal_store(__builtin_nontemporal_load(a + i), b + i);
}

__global__ void __launch_bounds__(THREADS) k_mix22(const u32x4* __restrict__ a,
                                                   const u32x4* __restrict__ c,
                                                   u32x4* __restrict__ b, u32x4* __restrict__ d,
                                                   size_t n) {
  const size_t i = size_t(blockIdx.x) * THREADS + threadIdx.x;
  if (i >= n) return;
  u32x4 x = a[i], y = c[i];
  x.x ^= y.y;
  y.x ^= x.w;
  b[i] = x;
  d[i] = y;
}

// Variants of the two-in-two-out traffic (run with --variants): how the two
// streams are laid over a thread's instructions, a wave's lanes, a
// workgroup's waves and the grid's workgroups.  Each moves four 1 GiB streams.
__global__ void __launch_bounds__(THREADS) k_ordered(const u32x4* __restrict__ a,
                                                     const u32x4* __restrict__ c,
                                                     u32x4* __restrict__ b, u32x4* __restrict__ d,
                                                     size_t n) {   // load, store, load, store
  const size_t i = size_t(blockIdx.x) * THREADS + threadIdx.x;
  if (i >= n) return;
  const u32x4 x = a[i];
  b[i] = x;
  d[i] = c[i + (x.x & 0u)];   // the second load's address depends on the first load
}

__global__ void __launch_bounds__(THREADS) k_two_each(const u32x4* __restrict__ a,
                                                      const u32x4* __restrict__ c,
                                                      u32x4* __restrict__ b, u32x4* __restrict__ d,
                                                      size_t n) {   // 4 loads, then 4 stores
  const size_t i = size_t(blockIdx.x) * (2 * THREADS) + threadIdx.x;
  if (i + THREADS >= n + THREADS) return;
  const u32x4 x0 = a[i], y0 = c[i], x1 = a[i + THREADS], y1 = c[i + THREADS];
  b[i] = x0;
  d[i] = y0;
  b[i + THREADS] = x1;
  d[i + THREADS] = y1;
}

__global__ void __launch_bounds__(THREADS) k_by_lanes(const u32x4* __restrict__ a,
                                                      const u32x4* __restrict__ c,
                                                      u32x4* __restrict__ b, u32x4* __restrict__ d,
                                                      size_t n) {   // half a wave per stream pair
  const int lane = threadIdx.x & 63;
  const size_t i = (size_t(blockIdx.x) * THREADS + (threadIdx.x & ~63u)) / 2 + (lane & 31);
  if (i >= n) return;
  if (lane < 32) b[i] = a[i];
  else d[i] = c[i];
}

__global__ void __launch_bounds__(THREADS) k_by_waves(const u32x4* __restrict__ a,
                                                      const u32x4* __restrict__ c,
                                                      u32x4* __restrict__ b, u32x4* __restrict__ d,
                                                      size_t n) {   // alternate waves
  const int w = threadIdx.x >> 6;
  const size_t i = size_t(blockIdx.x) * (THREADS / 2) + (w >> 1) * 64 + (threadIdx.x & 63);
  if (i >= n) return;
  if (w & 1) d[i] = c[i];
  else b[i] = a[i];
}

__global__ void __launch_bounds__(THREADS) k_by_groups(const u32x4* __restrict__ a,
                                                       const u32x4* __restrict__ c,
                                                       u32x4* __restrict__ b, u32x4* __restrict__ d,
                                                       size_t n) {   // alternate workgroups
  const size_t i = size_t(blockIdx.x >> 1) * THREADS + threadIdx.x;
  if (i >= n) return;
  if (blockIdx.x & 1) d[i] = c[i];
  else b[i] = a[i];
}

// Rows of 400 bytes (25 16-byte vectors), one 32-lane group per row and
// lanes 0..24 one vector each: two rows in (K, V), two rows out (dK, dV), the
// access shape of the fused attention backward on fp32 rows of 100.  _sep
// reads and writes four separate arrays; _kv keeps each row's K and V (and
// dK and dV) side by side in one 800-byte row, so that the traffic is one
// stream in and one stream out.
constexpr size_t ROWV = 25;
__global__ void __launch_bounds__(THREADS) k_rows_sep(const u32x4* __restrict__ k,
                                                      const u32x4* __restrict__ v,
                                                      u32x4* __restrict__ dk, u32x4* __restrict__ dv,
                                                      size_t rows) {
  const size_t r = (size_t(blockIdx.x) * THREADS + threadIdx.x) / 32;
  const unsigned l = threadIdx.x & 31u;
  if (r >= rows || l >= ROWV) return;
  const u32x4 x = k[r * ROWV + l], y = v[r * ROWV + l];
  dk[r * ROWV + l] = x;
  dv[r * ROWV + l] = y;
}

__global__ void __launch_bounds__(THREADS) k_rows_kv(const u32x4* __restrict__ kv,
                                                     u32x4* __restrict__ dkv, size_t rows) {
  const size_t r = (size_t(blockIdx.x) * THREADS + threadIdx.x) / 32;
  const unsigned l = threadIdx.x & 31u;
  if (r >= rows || l >= ROWV) return;
  const u32x4 x = kv[r * 2 * ROWV + l], y = kv[r * 2 * ROWV + ROWV + l];
  dkv[r * 2 * ROWV + l] = x;
  dkv[r * 2 * ROWV + ROWV + l] = y;
}

// The forward's shape: the same 800-byte K|V rows read, nothing written per
// row (one 16-byte result per group keeps the loads).
__global__ void __launch_bounds__(THREADS) k_rows_kv_read(const u32x4* __restrict__ kv,
                                                          unsigned* __restrict__ sink, size_t rows) {
  const size_t r = (size_t(blockIdx.x) * THREADS + threadIdx.x) / 32;
  const unsigned l = threadIdx.x & 31u;
  if (r >= rows || l >= ROWV) return;
  const u32x4 x = kv[r * 2 * ROWV + l], y = kv[r * 2 * ROWV + ROWV + l];
  if ((x.x ^ y.y ^ x.z ^ y.w) == 0x9e3779b9u) sink[0] = 1u;
}

// In-place updates: each row (or element) read and written back to the same
// place, as a backward that overwrites K|V with dK|dV would.
__global__ void __launch_bounds__(THREADS) k_rows_kv_inplace(u32x4* __restrict__ kv, size_t rows) {
  const size_t r = (size_t(blockIdx.x) * THREADS + threadIdx.x) / 32;
  const unsigned l = threadIdx.x & 31u;
  if (r >= rows || l >= ROWV) return;
  u32x4 x = kv[r * 2 * ROWV + l], y = kv[r * 2 * ROWV + ROWV + l];
  x.x += 1u;
  y.y += 1u;
  kv[r * 2 * ROWV + l] = x;
  kv[r * 2 * ROWV + ROWV + l] = y;
}

__global__ void __launch_bounds__(THREADS) k_update(u32x4* __restrict__ a, size_t n) {
  const size_t i = size_t(blockIdx.x) * THREADS + threadIdx.x;
  if (i >= n) return;
  u32x4 x = a[i];
  x.x += 1u;
  a[i] = x;
}

// The packed forward's shape: a 32-lane group per 10-row segment reads the
// segment's 800-byte K|V rows in two chunks of 5 (10 loads per lane each)
// and writes one 400-byte row per segment.
constexpr size_t SEG_ROWS = 10, SEG_CH = 5;
__global__ void __launch_bounds__(THREADS) k_seg_kv_fwd(const u32x4* __restrict__ kv,
                                                        u32x4* __restrict__ out, size_t segs) {
  const size_t g = (size_t(blockIdx.x) * THREADS + threadIdx.x) / 32;
  const unsigned l = threadIdx.x & 31u;
  if (g >= segs || l >= ROWV) return;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (size_t c = 0; c < SEG_ROWS; c += SEG_CH) {
    u32x4 x[SEG_CH], y[SEG_CH];
#pragma unroll
    for (size_t i = 0; i < SEG_CH; ++i) {
      const size_t r = g * SEG_ROWS + c + i;
      x[i] = kv[r * 2 * ROWV + l];
      y[i] = kv[r * 2 * ROWV + ROWV + l];
    }
#pragma unroll
    for (size_t i = 0; i < SEG_CH; ++i) acc ^= x[i] + y[i];
  }
  out[g * ROWV + l] = acc;
}

// The same shape with streaming (non-temporal) K|V loads, as the forward
// issues them, and the output row stored normally (OUT = 1), streamed
// (OUT = 2) or not at all (OUT = 0: the loads alone).
template <int OUT>
__global__ void __launch_bounds__(THREADS) k_seg_kv_fwd_nt(const u32x4* __restrict__ kv,
                                                           u32x4* __restrict__ out,
                                                           unsigned* __restrict__ sink, size_t segs) {
  const size_t g = (size_t(blockIdx.x) * THREADS + threadIdx.x) / 32;
  const unsigned l = threadIdx.x & 31u;
  if (g >= segs || l >= ROWV) return;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (size_t c = 0; c < SEG_ROWS; c += SEG_CH) {
    u32x4 x[SEG_CH], y[SEG_CH];
#pragma unroll
    for (size_t i = 0; i < SEG_CH; ++i) {
      const size_t r = g * SEG_ROWS + c + i;
      x[i] = __builtin_nontemporal_load(kv + r * 2 * ROWV + l);
      y[i] = __builtin_nontemporal_load(kv + r * 2 * ROWV + ROWV + l);
    }
#pragma unroll
    for (size_t i = 0; i < SEG_CH; ++i) acc ^= x[i] + y[i];
  }
  if (OUT == 1) out[g * ROWV + l] = acc;
  else if (OUT == 2) __builtin_nontemporal_store(acc, out + g * ROWV + l);
  else if ((acc.x ^ acc.w) == 0x9e3779b9u) sink[0] = 1u;
}

struct Buffers {
  u32x4 *a, *b, *c, *d;
  unsigned* sink;
  size_t n;   // 16-byte elements per buffer
};

template <class Launch>
static float median_ms(Launch launch, int reps) {
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  launch();
  launch();
  CHECK(hipDeviceSynchronize());
  std::vector<float> t;
  for (int r = 0; r < reps; ++r) {
    CHECK(hipEventRecord(e0));
    launch();
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    float ms = 0.f;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    t.push_back(ms);
  }
  CHECK(hipEventDestroy(e0));
  CHECK(hipEventDestroy(e1));
  std::sort(t.begin(), t.end());
  return t[t.size() / 2];
}

int main(int argc, char** argv) {
  const int reps = argc > 1 ? std::atoi(argv[1]) : 15;
  const size_t bytes = size_t(2) << 30;
  Buffers B;
  B.n = bytes / 16;
  CHECK(hipMalloc(&B.a, bytes));
  CHECK(hipMalloc(&B.b, bytes));
  CHECK(hipMalloc(&B.c, bytes));
  CHECK(hipMalloc(&B.d, bytes));
  CHECK(hipMalloc(&B.sink, 64));
  CHECK(hipMemset(B.a, 1, bytes));
  CHECK(hipMemset(B.c, 2, bytes));
  CHECK(hipMemset(B.b, 0, bytes));
  CHECK(hipMemset(B.d, 0, bytes));
  CHECK(hipDeviceSynchronize());
  const size_t half = B.n / 2;
  const dim3 blk(THREADS), g_all(unsigned((B.n + THREADS - 1) / THREADS)),
      g_half(unsigned((half + THREADS - 1) / THREADS));
  struct Row { const char* name; double moved; float ms; };
  std::vector<Row> rows;
  rows.push_back({"read", double(bytes), median_ms([&] {
    hipLaunchKernelGGL(k_read, g_all, blk, 0, 0, B.a, B.n, B.sink); }, reps)});
  rows.push_back({"write", double(bytes), median_ms([&] {
    hipLaunchKernelGGL(k_write, g_all, blk, 0, 0, B.b, B.n); }, reps)});
  rows.push_back({"copy", 2.0 * bytes, median_ms([&] {
    hipLaunchKernelGGL(k_copy, g_all, blk, 0, 0, B.a, B.b, B.n); }, reps)});
  rows.push_back({"read_nt", double(bytes), median_ms([&] {
    hipLaunchKernelGGL(k_read_nt, g_all, blk, 0, 0, B.a, B.n, B.sink); }, reps)});
  rows.push_back({"write_nt", double(bytes), median_ms([&] {
    hipLaunchKernelGGL(k_write_nt, g_all, blk, 0, 0, B.b, B.n); }, reps)});
  rows.push_back({"copy_nt", 2.0 * bytes, median_ms([&] {
    hipLaunchKernelGGL(k_copy_nt, g_all, blk, 0, 0, B.a, B.b, B.n); }, reps)});
  rows.push_back({"mix22", 2.0 * bytes, median_ms([&] {   // four streams of 1 GiB
    hipLaunchKernelGGL(k_mix22, g_half, blk, 0, 0, B.a, B.c, B.b, B.d, half); }, reps)});
  if (argc > 2 && std::strcmp(argv[2], "--variants") == 0) {
    const dim3 g_two(unsigned((half + 2 * THREADS - 1) / (2 * THREADS)));
    const dim3 g_dbl(unsigned(2 * ((half + THREADS - 1) / THREADS)));
    rows.push_back({"mix22_ordered", 2.0 * bytes, median_ms([&] {
      hipLaunchKernelGGL(k_ordered, g_half, blk, 0, 0, B.a, B.c, B.b, B.d, half); }, reps)});
    rows.push_back({"mix22_two_each", 2.0 * bytes, median_ms([&] {
      hipLaunchKernelGGL(k_two_each, g_two, blk, 0, 0, B.a, B.c, B.b, B.d, half); }, reps)});
    rows.push_back({"mix22_by_lanes", 2.0 * bytes, median_ms([&] {
      hipLaunchKernelGGL(k_by_lanes, g_dbl, blk, 0, 0, B.a, B.c, B.b, B.d, half); }, reps)});
    rows.push_back({"mix22_by_waves", 2.0 * bytes, median_ms([&] {
      hipLaunchKernelGGL(k_by_waves, g_dbl, blk, 0, 0, B.a, B.c, B.b, B.d, half); }, reps)});
    rows.push_back({"mix22_by_groups", 2.0 * bytes, median_ms([&] {
      hipLaunchKernelGGL(k_by_groups, g_dbl, blk, 0, 0, B.a, B.c, B.b, B.d, half); }, reps)});
    // 400-byte rows filling 1 GiB per stream (separate) or 2 GiB of 800-byte rows (interleaved)
    const size_t nrow = (bytes / 2) / (16 * ROWV);
    const dim3 g_rows(unsigned((nrow * 32 + THREADS - 1) / THREADS));
    const double moved = 4.0 * double(nrow) * 16 * ROWV;
    rows.push_back({"rows400_sep", moved, median_ms([&] {
      hipLaunchKernelGGL(k_rows_sep, g_rows, blk, 0, 0, B.a, B.c, B.b, B.d, nrow); }, reps)});
    rows.push_back({"rows400_kv", moved, median_ms([&] {
      hipLaunchKernelGGL(k_rows_kv, g_rows, blk, 0, 0, B.a, B.b, nrow); }, reps)});
    rows.push_back({"rows400_kv_inplace", moved, median_ms([&] {
      hipLaunchKernelGGL(k_rows_kv_inplace, g_rows, blk, 0, 0, B.a, nrow); }, reps)});
    rows.push_back({"update_inplace", 2.0 * bytes, median_ms([&] {
      hipLaunchKernelGGL(k_update, g_all, blk, 0, 0, B.a, B.n); }, reps)});
    const size_t nseg = nrow / SEG_ROWS;
    const dim3 g_segs(unsigned((nseg * 32 + THREADS - 1) / THREADS));
    rows.push_back({"seg10_kv_fwd", double(nseg) * (SEG_ROWS * 2 + 1) * 16 * ROWV, median_ms([&] {
      hipLaunchKernelGGL(k_seg_kv_fwd, g_segs, blk, 0, 0, B.a, B.b, nseg); }, reps)});
    rows.push_back({"rows400_kv_read", moved / 2, median_ms([&] {
      hipLaunchKernelGGL(k_rows_kv_read, g_rows, blk, 0, 0, B.a, B.sink, nrow); }, reps)});
    const double seg_in = double(nseg) * SEG_ROWS * 2 * 16 * ROWV, seg_out = double(nseg) * 16 * ROWV;
    rows.push_back({"seg10_kv_fwd_nt", seg_in + seg_out, median_ms([&] {
      hipLaunchKernelGGL(k_seg_kv_fwd_nt<1>, g_segs, blk, 0, 0, B.a, B.b, B.sink, nseg); }, reps)});
    rows.push_back({"seg10_kv_fwd_ntst", seg_in + seg_out, median_ms([&] {
      hipLaunchKernelGGL(k_seg_kv_fwd_nt<2>, g_segs, blk, 0, 0, B.a, B.b, B.sink, nseg); }, reps)});
    rows.push_back({"seg10_kv_read_nt", seg_in, median_ms([&] {
      hipLaunchKernelGGL(k_seg_kv_fwd_nt<0>, g_segs, blk, 0, 0, B.a, B.b, B.sink, nseg); }, reps)});
  }
  CHECK(hipGetLastError());
  std::printf("{");
  for (size_t k = 0; k < rows.size(); ++k)
    std::printf("%s\"%s\": {\"bytes\": %.0f, \"ms\": %.4f, \"TB_per_s\": %.3f}", k ? ", " : "",
                rows[k].name, rows[k].moved, rows[k].ms, rows[k].moved / (rows[k].ms * 1e-3) / 1e12);
  std::printf(", \"reps\": %d, \"buffer_bytes\": %zu}\n", reps, bytes);
  CHECK(hipFree(B.a));
  CHECK(hipFree(B.b));
  CHECK(hipFree(B.c));
  CHECK(hipFree(B.d));
  CHECK(hipFree(B.sink));
  return 0;
}
