// Shared host and device helpers of libfluxmoe (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "fluxmoe.h"

// ------------------------------------------------------------ host side ----

namespace fm {

// Records a message for moe_last_error() and returns `code`.
int fail(int code, const char* fmt, ...);
void clear_error();

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline int esize(int dtype) { return dtype == MOE_F32 ? 4 : dtype == MOE_BF16 ? 2 : 1; }

// Validation helpers: each returns MOE_OK or records and returns an error.
int need(const void* p, const char* name);
int need_aligned(const void* p, const char* name);      // NULL allowed
int need_dtype_float(int dtype, const char* name);

// Checks the launch that was just enqueued.
int check_launch(const char* what);

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
inline int cdiv(long a, long b) { return (int)((a + b - 1) / b); }

}  // namespace fm

#define FM_TRY(expr)            \
  do {                          \
    int rc_ = (expr);           \
    if (rc_ != MOE_OK) return rc_; \
  } while (0)

// ---------------------------------------------------------- device side ----

namespace fm {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

struct bf16 { uint16_t v; };   // storage-only bf16

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// fp32 -> bf16, round to nearest even (inputs are finite).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Two fp32 -> packed bf16 (low half = a), round to nearest even, with the
// gfx950 conversion instruction (same results as f2bf for finite inputs).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pk_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

template <typename T> struct elem;
template <> struct elem<float> {
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ float to_f(float v) { return v; }
  static __device__ __forceinline__ float from_f(float v) { return v; }
};
template <> struct elem<bf16> {
  static __device__ __forceinline__ float to_f(bf16 v) { return bf2f(v.v); }
  static __device__ __forceinline__ bf16 from_f(float v) { return bf16{f2bf(v)}; }
};

__device__ __forceinline__ float to_float(float v) { return v; }
__device__ __forceinline__ float to_float(bf16 v) { return bf2f(v.v); }
template <typename T> __device__ __forceinline__ T from_float(float v);
template <> __device__ __forceinline__ float from_float<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_float<bf16>(float v) { return bf16{f2bf(v)}; }

// 16-byte vector of T: 8 bf16 or 4 fp32.
template <typename T> struct vec16 {
  static constexpr int N = 16 / sizeof(T);
};

// Unpacks a 16-byte chunk into N floats.
__device__ __forceinline__ void unpack16(const u32x4_t& v, float* out, bf16*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(v[i] << 16);
    out[2 * i + 1] = __uint_as_float(v[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void unpack16(const u32x4_t& v, float* out, float*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = __uint_as_float(v[i]);
}
__device__ __forceinline__ u32x4_t pack16(const float* in, bf16*) {
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    v[i] = pk_bf16(in[2 * i], in[2 * i + 1]);
  return v;
}
__device__ __forceinline__ u32x4_t pack16(const float* in, float*) {
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(in[i]);
  return v;
}

// Global-memory accesses through explicit address-space-1 pointers, so that
// the compiler emits global_load/global_store (not flat) even for pointers
// read from device-side tables.
#define FM_GLOBAL __attribute__((address_space(1)))
template <typename T> __device__ __forceinline__ const FM_GLOBAL T* gptr(const T* p) {
  return (const FM_GLOBAL T*)(p);
}
template <typename T> __device__ __forceinline__ FM_GLOBAL T* gptr(T* p) {
  return (FM_GLOBAL T*)(p);
}
// Load of a wave-uniform element of a table that no thread writes while the
// kernel runs, through the scalar cache (constant address space): it neither
// occupies the vector-memory counter nor waits on it.
template <typename T> __device__ __forceinline__ T ld_scalar(const T* p) {
  return *(const __attribute__((address_space(4))) T*)(p);
}
__device__ __forceinline__ u32x4_t ld16(const void* p) {
  return *(const FM_GLOBAL u32x4_t*)(p);
}
__device__ __forceinline__ void st16(void* p, const u32x4_t& v) {
  *(FM_GLOBAL u32x4_t*)(p) = v;
}

// Wave64 helpers.
__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

// (value desc, index asc) order used by every top-k: true if a ranks before b.
__device__ __forceinline__ bool ranks_before(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

}  // namespace fm
