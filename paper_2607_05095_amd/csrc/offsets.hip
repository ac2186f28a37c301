// offsets.hip -- CSR offsets of a sampled block (Sec. 5: the compression
// engine's CSR-style ind_ptr): an exclusive scan of per-destination counts.
#include "scan.h"

namespace fast {

struct InCounts {
  const int32_t* c;
  __device__ uint32_t operator()(int64_t i) const { return uint32_t(c[i]); }
};
struct OutOffsets {
  int32_t* off;
  __device__ void operator()(int64_t i, uint32_t prefix, uint32_t) const { off[i] = int32_t(prefix); }
};

}  // namespace fast

using namespace fast;

extern "C" size_t fast_csr_offsets_workspace(int64_t n) {
  return n < 0 ? 0 : scan_workspace(n);
}

extern "C" fast_status_t fast_csr_offsets(const int32_t* counts, int64_t n, int32_t* offsets,
                                          void* ws, size_t ws_bytes, fast_stream_t stream) {
  if (n < 0) return fail(FAST_ERR_INVALID_ARG, "fast_csr_offsets: n = %lld < 0", (long long)n);
  if (n >= (int64_t(1) << 31)) return fail(FAST_ERR_UNSUPPORTED, "fast_csr_offsets: n >= 2^31");
  if (!offsets) return fail(FAST_ERR_INVALID_ARG, "fast_csr_offsets: offsets is NULL");
  if (n > 0 && !counts) return fail(FAST_ERR_INVALID_ARG, "fast_csr_offsets: counts is NULL");
  if (!ws || ws_bytes < scan_workspace(n))
    return fail(FAST_ERR_WORKSPACE, "fast_csr_offsets: workspace %zu < %zu bytes", ws_bytes,
                scan_workspace(n));
  hipError_t e = scan_launch(InCounts{counts}, OutOffsets{offsets}, n, ws, nullptr, offsets + n,
                             static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(FAST_ERR_HIP, "fast_csr_offsets: %s", hipGetErrorString(e));
  return ok();
}
