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
// fp32 -> bfloat16 and fp16: the conversion instructions (v_cvt_pk_bf16_f32,
// v_cvt_f16_f32) round to nearest even; NaNs stay NaNs.
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) {
  return __builtin_bit_cast(uint16_t, (__bf16)v);
}
template <> __device__ __forceinline__ _Float16 from_f32<_Float16>(float v) { return (_Float16)v; }

// Two fp32 values rounded to the 16-bit storage type T and packed into one
// dword (lo in bits 0..15): one packed conversion for bfloat16.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
template <typename T> __device__ __forceinline__ uint32_t pack2_f32(float lo, float hi);
template <> __device__ __forceinline__ uint32_t pack2_f32<bf16_t>(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
template <> __device__ __forceinline__ uint32_t pack2_f32<_Float16>(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)lo) | ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)hi) << 16);
}

// 16-byte vector type used for global memory traffic.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Wait for the last MFMAs before the epilogue reads their accumulators.
// The compiler's hazard recognizer inserts the wait states it believes an
// MFMA result needs before another instruction reads it, and no more; one
// change that let the packed bf16 conversion read the result of a 16x16x16
// bf16 MFMA at exactly that minimum distance gave wrong first conversions,
// varying from run to run.  This adds 16 wait states (two 8-cycle s_nop)
// between the MFMAs and the epilogue (scheduling barriers keep the code on
// each side), at a cost of 16 cycles per wavefront.
__device__ __forceinline__ void mfma_results_settle() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_nop 7\n\ts_nop 7" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Streaming (nontemporal) loads: X is read exactly once per launch.
template <typename V>
__device__ __forceinline__ V ld_stream(const V* p) { return __builtin_nontemporal_load(p); }
template <typename V>
__device__ __forceinline__ void st_stream(V* p, V v) { __builtin_nontemporal_store(v, p); }

}  // namespace ks
