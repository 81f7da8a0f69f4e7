// Device-side helpers shared by the KS kernels: storage-type conversions and
// memory-access wrappers.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace ks {

// Storage types: float (fp32), uint16_t (bfloat16 bit pattern), _Float16 (fp16).
typedef uint16_t bf16_t;

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }
__device__ __forceinline__ float to_f32(_Float16 v) { return (float)v; }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
// fp32 -> bfloat16, round to nearest even; NaNs stay quiet NaNs.
// (Branch-free: both results are formed and one is selected.)
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) {
  const uint32_t u = __float_as_uint(v);
  const uint32_t rne = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  const uint32_t qnan = (u >> 16) | 0x40u;
  return (bf16_t)((u & 0x7fffffffu) > 0x7f800000u ? qnan : rne);
}
// fp32 -> fp16; the conversion instruction rounds to nearest even.
template <> __device__ __forceinline__ _Float16 from_f32<_Float16>(float v) { return (_Float16)v; }

// 16-byte vector type used for global memory traffic.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Streaming (nontemporal) loads: X is read exactly once per launch.
template <typename V>
__device__ __forceinline__ V ld_stream(const V* p) { return __builtin_nontemporal_load(p); }
template <typename V>
__device__ __forceinline__ void st_stream(V* p, V v) { __builtin_nontemporal_store(v, p); }

}  // namespace ks
