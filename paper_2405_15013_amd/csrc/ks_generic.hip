// Generic KS kernel: one thread per output element, any pattern and layout.
//
// Each thread evaluates one entry of Y = X K^T from the packed blocks: for the
// output row m = i*b*d + k*d + j it sums Kv[i*d+j][k][l] * X[., i*c*d + l*d + j]
// over l < c (paper, Section 4.1, row/col index sets of Algorithm 2).  It is the
// fallback for patterns the tiled kernels do not cover (e.g. b or c not a
// multiple of 16 and too large for the VALU kernels); correctness over speed.
#include "ks_epilogue.h"
#include "ks_internal.h"
#include "ks_common.h"

namespace ks {

template <typename T>
__global__ __launch_bounds__(256) void ks_generic_kernel(Problem p) {
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const T* __restrict__ x = static_cast<const T*>(p.x);
  T* __restrict__ y = static_cast<T*>(p.y);
  const int64_t total = (int64_t)p.batch * p.M;
  const int64_t bd = (int64_t)p.b * p.d;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    int64_t beta, m;
    if (p.layout == BSF) { beta = idx / p.M; m = idx - beta * p.M; }
    else { m = idx / p.batch; beta = idx - m * p.batch; }
    const int64_t i = m / bd;
    const int64_t k = (m - i * bd) / p.d;
    const int64_t j = m - i * bd - k * p.d;
    const T* blk = kv + ((i * p.d + j) * p.b + k) * p.c;
    const int64_t n0 = i * p.c * p.d + j;
    float acc = 0.f;
    if (p.layout == BSF) {
      const T* xr = x + beta * p.N + n0;
      for (int l = 0; l < p.c; ++l) acc += to_f32(blk[l]) * to_f32(xr[(int64_t)l * p.d]);
    } else {
      const T* xc = x + n0 * p.batch + beta;
      const int64_t step = (int64_t)p.d * p.batch;
      for (int l = 0; l < p.c; ++l) acc += to_f32(blk[l]) * to_f32(xc[l * step]);
    }
    if (epilogue_on(p)) acc = epilogue_apply<T>(p, acc, (int)m);
    y[idx] = from_f32<T>(acc);
  }
}

hipError_t launch_generic(const Problem& p, const Plan& pl, hipStream_t s) {
  dim3 grid(pl.grid), block(pl.block);
  switch (p.dtype) {
    case F32: hipLaunchKernelGGL(ks_generic_kernel<float>, grid, block, 0, s, p); break;
    case BF16: hipLaunchKernelGGL(ks_generic_kernel<bf16_t>, grid, block, 0, s, p); break;
    case F16: hipLaunchKernelGGL(ks_generic_kernel<_Float16>, grid, block, 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace ks
