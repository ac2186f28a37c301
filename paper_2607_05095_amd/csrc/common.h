// common.h -- shared device helpers and host-side status handling of the
// gfx950 operator library.  Wave64 only (CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fast.h"

namespace fast {

// ------------------------------------------------------------------ host side
// Records a formatted message for fast_last_error() and returns `st`.
fast_status_t fail(fast_status_t st, const char* fmt, ...)
    __attribute__((format(printf, 2, 3)));
// FAST_ERR_HIP with the runtime's message if the last launch failed.
fast_status_t check_launch(const char* what);
// Clears the thread's error message (successful call).
fast_status_t ok();

inline bool aligned(const void* p, size_t a) {
  return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0;
}
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int elem_size(fast_dtype_t dt) { return dt == FAST_BF16 ? 2 : 4; }

// Workgroups are dispatched round-robin over the 8 XCDs (block b runs on XCD
// b % 8).  This bijection hands every XCD a contiguous range of logical
// tiles, so neighbouring tiles -- which share the partial cache lines at
// their boundaries -- meet in the same 4 MB L2.
__device__ __forceinline__ uint32_t xcd_tile(uint32_t b, uint32_t nb) {
  const uint32_t q = nb >> 3, r = nb & 7u, x = b & 7u;
  return x * q + (x < r ? x : r) + (b >> 3);
}

// ------------------------------------------------------------------ bf16
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
// fp32 -> bf16 with round-to-nearest-even, two values packed (lo in the low
// half): one v_cvt_pk_bf16_f32 on gfx950.  Its result equals the rounding
// written out -- add 0x7fff plus the lowest kept bit and keep the high half,
// a NaN keeping its sign and payload with the quiet bit set -- for every one
// of the 2^32 fp32 bit patterns (checked exhaustively on MI355X), so the
// instruction replaces a per-element branch on NaN.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16_pack(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}
__device__ __forceinline__ uint32_t bf16_rne(float f) { return bf16_pack(f, 0.f) & 0xffffu; }

// ------------------------------------------------------------------ vectors
// VecIO<T,VE>: VE consecutive elements of storage type T (float, or uint16_t
// holding bf16) moved as one aligned global access and widened to fp32.
template <typename T, int VE> struct VecIO;

template <> struct VecIO<float, 1> {
  __device__ static void load(const float* p, float* x) { x[0] = *p; }
  __device__ static void store(float* p, const float* x) { *p = x[0]; }
};
template <> struct VecIO<float, 2> {
  __device__ static void load(const float* p, float* x) {
    float2 v = *reinterpret_cast<const float2*>(p);
    x[0] = v.x; x[1] = v.y;
  }
  __device__ static void store(float* p, const float* x) {
    *reinterpret_cast<float2*>(p) = make_float2(x[0], x[1]);
  }
};
template <> struct VecIO<float, 4> {
  __device__ static void load(const float* p, float* x) {
    float4 v = *reinterpret_cast<const float4*>(p);
    x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
  }
  __device__ static void store(float* p, const float* x) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  }
};
template <> struct VecIO<uint16_t, 1> {
  __device__ static void load(const uint16_t* p, float* x) { x[0] = __uint_as_float(uint32_t(*p) << 16); }
  __device__ static void store(uint16_t* p, const float* x) { *p = uint16_t(bf16_rne(x[0])); }
};
template <> struct VecIO<uint16_t, 2> {
  __device__ static void load(const uint16_t* p, float* x) {
    uint32_t w = *reinterpret_cast<const uint32_t*>(p);
    x[0] = bf16_lo(w); x[1] = bf16_hi(w);
  }
  __device__ static void store(uint16_t* p, const float* x) {
    *reinterpret_cast<uint32_t*>(p) = bf16_pack(x[0], x[1]);
  }
};
template <> struct VecIO<uint16_t, 4> {
  __device__ static void load(const uint16_t* p, float* x) {
    uint2 w = *reinterpret_cast<const uint2*>(p);
    x[0] = bf16_lo(w.x); x[1] = bf16_hi(w.x); x[2] = bf16_lo(w.y); x[3] = bf16_hi(w.y);
  }
  __device__ static void store(uint16_t* p, const float* x) {
    *reinterpret_cast<uint2*>(p) = make_uint2(bf16_pack(x[0], x[1]), bf16_pack(x[2], x[3]));
  }
};
template <> struct VecIO<uint16_t, 8> {
  __device__ static void load(const uint16_t* p, float* x) {
    uint4 w = *reinterpret_cast<const uint4*>(p);
    x[0] = bf16_lo(w.x); x[1] = bf16_hi(w.x); x[2] = bf16_lo(w.y); x[3] = bf16_hi(w.y);
    x[4] = bf16_lo(w.z); x[5] = bf16_hi(w.z); x[6] = bf16_lo(w.w); x[7] = bf16_hi(w.w);
  }
  __device__ static void store(uint16_t* p, const float* x) {
    *reinterpret_cast<uint4*>(p) = make_uint4(bf16_pack(x[0], x[1]), bf16_pack(x[2], x[3]),
                                              bf16_pack(x[4], x[5]), bf16_pack(x[6], x[7]));
  }
};

// Streaming accesses.  Rows read or written exactly once (K, V, dK, dV,
// time features) may use the non-temporal cache policy (NT = true).  On
// MI355X it raised streaming reads by ~10% when every row covers whole
// 128-byte lines, and lowered them when neighbouring rows share a line (the
// line is evicted before the second row uses it; partial-line streaming
// stores lose write combining).  Callers choose NT from the row alignment.
constexpr int CACHE_LINE = 128;
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename V, bool NT>
__device__ __forceinline__ V ld_stream(const void* p) {
  if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const V*>(p));
  else return *reinterpret_cast<const V*>(p);
}
template <typename V, bool NT>
__device__ __forceinline__ void st_stream(void* p, V v) {
  if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<V*>(p));
  else *reinterpret_cast<V*>(p) = v;
}

// StreamIO<T,VE,NT>: VecIO stores with a selectable cache policy.
template <typename T, int VE, bool NT> struct StreamIO;
template <bool NT> struct StreamIO<float, 1, NT> {
  __device__ static void store(float* p, const float* x) { st_stream<float, NT>(p, x[0]); }
};
template <bool NT> struct StreamIO<float, 2, NT> {
  __device__ static void store(float* p, const float* x) { st_stream<f32x2, NT>(p, f32x2{x[0], x[1]}); }
};
template <bool NT> struct StreamIO<float, 4, NT> {
  __device__ static void store(float* p, const float* x) {
    st_stream<f32x4, NT>(p, f32x4{x[0], x[1], x[2], x[3]});
  }
};
template <bool NT> struct StreamIO<uint16_t, 1, NT> {
  __device__ static void store(uint16_t* p, const float* x) { *p = uint16_t(bf16_rne(x[0])); }
};
template <bool NT> struct StreamIO<uint16_t, 2, NT> {
  __device__ static void store(uint16_t* p, const float* x) {
    st_stream<uint32_t, NT>(p, bf16_pack(x[0], x[1]));
  }
};
template <bool NT> struct StreamIO<uint16_t, 4, NT> {
  __device__ static void store(uint16_t* p, const float* x) {
    st_stream<u32x2, NT>(p, u32x2{bf16_pack(x[0], x[1]), bf16_pack(x[2], x[3])});
  }
};
template <bool NT> struct StreamIO<uint16_t, 8, NT> {
  __device__ static void store(uint16_t* p, const float* x) {
    st_stream<u32x4, NT>(p, u32x4{bf16_pack(x[0], x[1]), bf16_pack(x[2], x[3]),
                                  bf16_pack(x[4], x[5]), bf16_pack(x[6], x[7])});
  }
};

// Raw<T,VE>: the same VE elements kept packed in registers (bf16 pairs in one
// 32-bit register) between the load and their first use, so that a chunk of
// in-flight rows costs VE*sizeof(T)/4 registers per row, not VE.
template <typename T, int VE> struct Raw;
template <int VE> struct Raw<float, VE> {
  float v[VE];
  template <bool NT>
  __device__ void load(const float* p) {
    if constexpr (VE == 1) {
      v[0] = ld_stream<float, NT>(p);
    } else if constexpr (VE == 2) {
      const f32x2 t = ld_stream<f32x2, NT>(p);
      v[0] = t.x; v[1] = t.y;
    } else {
      const f32x4 t = ld_stream<f32x4, NT>(p);
      v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
    }
  }
  __device__ void unpack(float* x) const {
#pragma unroll
    for (int j = 0; j < VE; ++j) x[j] = v[j];
  }
  __device__ void zero() {
#pragma unroll
    for (int j = 0; j < VE; ++j) v[j] = 0.f;
  }
};
template <> struct Raw<uint16_t, 1> {
  uint32_t w;
  template <bool NT>
  __device__ void load(const uint16_t* p) { w = uint32_t(*p) << 16; }
  __device__ void unpack(float* x) const { x[0] = __uint_as_float(w); }
  __device__ void zero() { w = 0u; }
};
template <int VE> struct Raw<uint16_t, VE> {
  static_assert(VE == 2 || VE == 4 || VE == 8, "bf16 vector of 2, 4 or 8");
  uint32_t w[VE / 2];
  template <bool NT>
  __device__ void load(const uint16_t* p) {
    if constexpr (VE == 2) {
      w[0] = ld_stream<uint32_t, NT>(p);
    } else if constexpr (VE == 4) {
      const u32x2 t = ld_stream<u32x2, NT>(p);
      w[0] = t.x; w[1] = t.y;
    } else {
      const u32x4 t = ld_stream<u32x4, NT>(p);
      w[0] = t.x; w[1] = t.y; w[2] = t.z; w[3] = t.w;
    }
  }
  __device__ void unpack(float* x) const {
#pragma unroll
    for (int k = 0; k < VE / 2; ++k) {
      x[2 * k] = bf16_lo(w[k]);
      x[2 * k + 1] = bf16_hi(w[k]);
    }
  }
  __device__ void zero() {
#pragma unroll
    for (int k = 0; k < VE / 2; ++k) w[k] = 0u;
  }
};

// ------------------------------------------------------------------ cross-lane sums
// All-reduce (sum) over aligned groups of `lanes` lanes (a power of two <= 64)
// with DPP row operations and the gfx950 permlane swaps, no LDS traffic.
// Every lane of a group ends with the bitwise-identical sum: each step adds
// a lane's value to its partner's, and x + y == y + x exactly.
__device__ __forceinline__ float dpp_quad_xor1(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, true));
}
__device__ __forceinline__ float dpp_quad_xor2(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, true));
}
__device__ __forceinline__ float dpp_row_half_mirror(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xF, 0xF, true));
}
__device__ __forceinline__ float dpp_row_mirror(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x140, 0xF, 0xF, true));
}
__device__ __forceinline__ float sum_rows16(float x) {  // lanes l and l^16
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_halves32(float x) {  // lanes l and l^32
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float group_sum(float x, int lanes) {
  if (lanes >= 2) x += dpp_quad_xor1(x);
  if (lanes >= 4) x += dpp_quad_xor2(x);
  if (lanes >= 8) x += dpp_row_half_mirror(x);
  if (lanes >= 16) x += dpp_row_mirror(x);
  if (lanes >= 32) x = sum_rows16(x);
  if (lanes >= 64) x = sum_halves32(x);
  return x;
}

__device__ __forceinline__ int64_t clamp64(int64_t x, int64_t lo, int64_t hi) {
  return x < lo ? lo : (x > hi ? hi : x);
}

}  // namespace fast
