// sample.hip -- most-recent-k temporal neighbour sampling (Sec. 6.1: the
// experiments sample the k = 10 most recent neighbours of each root) over a
// T-CSR temporal graph, producing the sampled block in the CSR-by-destination
// form every other operator takes.
//
// A root (node v, query time t) may use only events strictly earlier than t.
// v's entries are in time order, so those events are a prefix of its list;
// a binary search finds its end and the root keeps the last min(k, length)
// entries of it, in entry order.  Three steps: one thread per root searches
// and counts, a scan turns the counts into offsets, and a group of lanes per
// root copies its neighbours, times and edge ids (coalesced: one root's
// entries are contiguous).  The output is a function of the inputs alone.
#include "scan.h"

namespace fast {

constexpr int SR_THREADS = 256;
constexpr int SR_GROUP = 16;   // lanes copying one root's entries

__global__ void __launch_bounds__(SR_THREADS) k_sample_count(
    const int64_t* __restrict__ indptr, int64_t num_nodes, int64_t num_entries,
    const float* __restrict__ ts, const int64_t* __restrict__ roots,
    const float* __restrict__ root_t, int64_t R, int k, int32_t* __restrict__ count,
    int64_t* __restrict__ start) {
  const int64_t i = int64_t(blockIdx.x) * SR_THREADS + threadIdx.x;
  if (i >= R) return;
  const int64_t v = roots[i];
  int32_t c = 0;
  int64_t s = 0;
  if (v >= 0 && v < num_nodes) {
    const int64_t lo = clamp64(indptr[v], 0, num_entries);
    const int64_t hi = clamp64(indptr[v + 1], lo, num_entries);
    const float t = root_t[i];
    int64_t a = lo, b = hi;              // first entry p with !(ts[p] < t)
    while (a < b) {
      const int64_t mid = a + ((b - a) >> 1);
      if (ts[mid] < t) a = mid + 1; else b = mid;
    }
    const int64_t n = a - lo;
    c = int32_t(n < k ? n : k);
    s = a - c;
  }
  count[i] = c;
  start[i] = s;
}

struct InRootCount {
  const int32_t* c;
  __device__ uint32_t operator()(int64_t i) const { return uint32_t(c[i]); }
};
struct OutRootOffset {
  int32_t* off;
  __device__ void operator()(int64_t i, uint32_t prefix, uint32_t) const { off[i] = int32_t(prefix); }
};

// Groups of SR_GROUP lanes, one root each.
__global__ void __launch_bounds__(SR_THREADS) k_sample_fill(
    const int64_t* __restrict__ nbr, const float* __restrict__ ts,
    const int64_t* __restrict__ eid, const int32_t* __restrict__ count,
    const int64_t* __restrict__ start, const int32_t* __restrict__ off, int64_t R,
    int64_t* __restrict__ src_ids, float* __restrict__ edge_t, int64_t* __restrict__ edge_ids) {
  const int64_t i = (int64_t(blockIdx.x) * SR_THREADS + threadIdx.x) / SR_GROUP;
  const int lane = int(threadIdx.x) % SR_GROUP;
  if (i >= R) return;
  const int32_t c = count[i];
  const int64_t s = start[i], o = off[i];
  for (int j = lane; j < c; j += SR_GROUP) {
    src_ids[o + j] = nbr[s + j];
    edge_t[o + j] = ts[s + j];
    edge_ids[o + j] = eid[s + j];
  }
}

struct SrWs {
  int32_t* count;
  int64_t* start;
  void* scan;
};

static size_t sr_layout(int64_t R, char* base, SrWs* ws) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes, 256);
    return base ? base + o : nullptr;
  };
  char* c = take(size_t(R) * 4);
  char* s = take(size_t(R) * 8);
  char* sc = take(scan_workspace(R));
  if (ws) {
    ws->count = reinterpret_cast<int32_t*>(c);
    ws->start = reinterpret_cast<int64_t*>(s);
    ws->scan = sc;
  }
  return off;
}

}  // namespace fast

using namespace fast;

extern "C" size_t fast_sample_recent_workspace(int64_t num_roots) {
  if (num_roots < 0 || num_roots >= (int64_t(1) << 31)) return 0;
  return sr_layout(num_roots, nullptr, nullptr);
}

extern "C" fast_status_t fast_sample_recent(const fast_temporal_graph_t* g, const int64_t* roots,
                                            const float* root_t, int64_t num_roots, int k,
                                            int32_t* dst_offsets, int64_t* src_ids, float* edge_t,
                                            int64_t* edge_ids, void* ws, size_t ws_bytes,
                                            fast_stream_t stream) {
  const char* fn = "fast_sample_recent";
  if (!g) return fail(FAST_ERR_INVALID_ARG, "%s: graph is NULL", fn);
  if (g->num_nodes < 0 || g->num_entries < 0 || num_roots < 0 || k < 0)
    return fail(FAST_ERR_INVALID_ARG, "%s: negative size or k", fn);
  if (num_roots >= (int64_t(1) << 31))   // also with k = 0: the workspace is sized per root
    return fail(FAST_ERR_UNSUPPORTED, "%s: num_roots >= 2^31", fn);
  if (num_roots * int64_t(k) >= (int64_t(1) << 31))
    return fail(FAST_ERR_UNSUPPORTED, "%s: num_roots * k >= 2^31", fn);
  if (!dst_offsets) return fail(FAST_ERR_INVALID_ARG, "%s: dst_offsets is NULL", fn);
  if (num_roots > 0 && (!roots || !root_t))
    return fail(FAST_ERR_INVALID_ARG, "%s: roots/root_t is NULL", fn);
  if (num_roots > 0 && k > 0 && (!src_ids || !edge_t || !edge_ids))
    return fail(FAST_ERR_INVALID_ARG, "%s: NULL src_ids/edge_t/edge_ids", fn);
  if (g->num_nodes > 0 && !g->indptr) return fail(FAST_ERR_INVALID_ARG, "%s: indptr is NULL", fn);
  if (g->num_entries > 0 && (!g->nbr || !g->ts || !g->eid))
    return fail(FAST_ERR_INVALID_ARG, "%s: NULL nbr/ts/eid", fn);
  const size_t need = fast_sample_recent_workspace(num_roots);
  if (!ws || ws_bytes < need)
    return fail(FAST_ERR_WORKSPACE, "%s: workspace of %zu bytes < %zu", fn, ws_bytes, need);
  if (!aligned(ws, 256)) return fail(FAST_ERR_UNSUPPORTED, "%s: workspace not 256-byte aligned", fn);
  hipStream_t st = static_cast<hipStream_t>(stream);
  SrWs w;
  sr_layout(num_roots, static_cast<char*>(ws), &w);
  const int64_t R = num_roots;
  const int kk = (g->num_nodes > 0 && g->num_entries > 0) ? k : 0;   // no entries: all empty
  if (R > 0)
    hipLaunchKernelGGL(k_sample_count, dim3(uint32_t((R + SR_THREADS - 1) / SR_THREADS)),
                       dim3(SR_THREADS), 0, st, g->indptr, g->num_nodes, g->num_entries, g->ts,
                       roots, root_t, R, kk, w.count, w.start);
  hipError_t e = scan_launch(InRootCount{w.count}, OutRootOffset{dst_offsets}, R, w.scan, nullptr,
                             dst_offsets + R, st);
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "%s: %s", fn, hipGetErrorString(e));
  if (R > 0 && kk > 0) {
    const int64_t threads = R * SR_GROUP;
    hipLaunchKernelGGL(k_sample_fill, dim3(uint32_t((threads + SR_THREADS - 1) / SR_THREADS)),
                       dim3(SR_THREADS), 0, st, g->nbr, g->ts, g->eid, w.count, w.start,
                       dst_offsets, R, src_ids, edge_t, edge_ids);
  }
  return check_launch(fn);
}
