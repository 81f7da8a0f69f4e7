// Division by a runtime constant as a multiply and a shift, for the index
// decodes of the kernels (host-computed constants; a scalar integer division
// costs tens of instructions on the CU's shared scalar unit).
//
// For d >= 1 take l = ceil(log2 d), m = ceil(2^(31+l) / d) (< 2^32) and
// s = 31 + l; then floor(n / d) = (n * m) >> s for every 0 <= n < 2^31,
// because m*d - 2^(31+l) < d <= 2^l.  The plan verifier compares every decode
// it replays with the plain division.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace ks {

inline void div_magic(uint32_t d, uint32_t* m, int* s) {
  int l = 0;
  while ((1u << l) < d) ++l;
  *s = 31 + l;
  *m = (uint32_t)((((uint64_t)1 << (31 + l)) + d - 1) / d);
}
__host__ __device__ __forceinline__ uint32_t div_fast(uint32_t n, uint32_t m, int s) {
  return (uint32_t)(((uint64_t)n * m) >> s);
}

}  // namespace ks
