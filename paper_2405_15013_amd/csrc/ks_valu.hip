// VALU kernels for KS patterns with small dense blocks (b, c <= 16), e.g. the
// 2 x 2 blocks of butterfly factors (Appendix B.1, Table 5, square dyadic row).
//
// Both follow the output-stationary tiling of Algorithm 2 (Section 4.1): a
// thread owns a set of outputs of one (i, j) block, reads the c inputs they
// depend on once, keeps the b accumulators in registers and writes each output
// once.  With blocks this small the work is a pure stream (2*b*c flops per
// (b + c) elements moved), so the kernels are built for coalesced 16-byte
// nontemporal loads and stores, not for arithmetic.
#include "ks_epilogue.h"
#include "ks_internal.h"
#include "ks_common.h"

namespace ks {

// Vector of VEC storage elements (VEC * sizeof(T) bytes) and its fp32 view.
template <typename T, int VEC> struct Vec;
template <typename T> struct Vec<T, 1> { typedef T type; };
template <> struct Vec<float, 2> { typedef u32x2 type; };
template <> struct Vec<float, 4> { typedef u32x4 type; };
template <> struct Vec<bf16_t, 2> { typedef uint32_t type; };
template <> struct Vec<bf16_t, 4> { typedef u32x2 type; };
template <> struct Vec<bf16_t, 8> { typedef u32x4 type; };
template <> struct Vec<_Float16, 2> { typedef uint32_t type; };
template <> struct Vec<_Float16, 4> { typedef u32x2 type; };
template <> struct Vec<_Float16, 8> { typedef u32x4 type; };

template <typename T, int VEC>
__device__ __forceinline__ void load_vec(const T* p, float (&out)[VEC]) {
  typedef typename Vec<T, VEC>::type V;
  union { V v; T e[VEC]; } u;
  u.v = ld_stream(reinterpret_cast<const V*>(p));
#pragma unroll
  for (int e = 0; e < VEC; ++e) out[e] = to_f32(u.e[e]);
}

template <typename T, int VEC>
__device__ __forceinline__ void store_vec(T* p, const float (&in)[VEC]) {
  typedef typename Vec<T, VEC>::type V;
  union { V v; T e[VEC]; } u;
#pragma unroll
  for (int e = 0; e < VEC; ++e) u.e[e] = from_f32<T>(in[e]);
  st_stream(reinterpret_cast<V*>(p), u.v);
}

// ---------------------------------------------------------------------------
// Batch-size-last.  Block (i, j) reads input rows i*c*d + l*d + j and writes
// output rows i*b*d + k*d + j of the (width, batch) matrices; each row is
// contiguous along the batch, so a thread takes U vectors of VEC consecutive
// batch columns and the whole workgroup shares one (i, j) (blockIdx.y), which
// keeps the block's values in scalar registers.
// ---------------------------------------------------------------------------
template <typename T, int VEC, int BMAX, int CMAX, int U>
__global__ __launch_bounds__(256) void ks_valu_bsl_kernel(Problem p) {
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const T* __restrict__ x = static_cast<const T*>(p.x);
  T* __restrict__ y = static_cast<T*>(p.y);
  const int ij = blockIdx.y;
  const int i = ij / p.d, j = ij - (ij / p.d) * p.d;
  const int b = p.b, c = p.c, d = p.d, batch = p.batch;
  const T* blk = kv + (size_t)ij * b * c;  // workgroup-uniform: read through the scalar cache
  const size_t xrow0 = (size_t)i * c * d + j;  // input row of l = 0
  const size_t yrow0 = (size_t)i * b * d + j;  // output row of k = 0
  const size_t xstep = (size_t)d * batch, ystep = (size_t)d * batch;
  const int nvec = batch / VEC;
  const int v0 = blockIdx.x * (256 * U) + threadIdx.x;
  float xv[U][CMAX][VEC];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int v = v0 + u * 256;
#pragma unroll
    for (int l = 0; l < CMAX; ++l) {
      if (l < c && v < nvec) load_vec<T, VEC>(x + xrow0 * batch + l * xstep + (size_t)v * VEC, xv[u][l]);
    }
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int v = v0 + u * 256;
    if (v >= nvec) continue;
#pragma unroll
    for (int k = 0; k < BMAX; ++k) {
      if (k >= b) continue;
      float acc[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
#pragma unroll
      for (int l = 0; l < CMAX; ++l) {
        if (l < c) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) acc[e] = __builtin_fmaf(to_f32(blk[k * c + l]), xv[u][l][e], acc[e]);
        }
      }
      if (p.bias != nullptr) {
        const float bk = bias_value<T>(p, (int64_t)yrow0 + k * d);
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] += bk;
      }
      if (epilogue_gelu(p)) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] = gelu_f32<T>(acc[e]);
      }
      store_vec<T, VEC>(y + yrow0 * batch + k * ystep + (size_t)v * VEC, acc);
    }
  }
}

// ---------------------------------------------------------------------------
// Batch-size-first.  For a batch row and a given i the inputs of all j form the
// contiguous run [i*c*d, (i+1)*c*d) (l-major, j-minor) and the outputs the run
// [i*b*d, (i+1)*b*d).  A thread owns V consecutive j of one (batch row, i):
// it loads c vectors of V elements at stride d, and writes b such vectors.
// Consecutive lanes take consecutive j-vectors, then the next i, then the next
// batch row, so each wavefront walks memory contiguously.
// ---------------------------------------------------------------------------
template <typename T, int V, int BMAX, int CMAX>
__global__ __launch_bounds__(256) void ks_valu_bsf_kernel(Problem p) {
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const T* __restrict__ x = static_cast<const T*>(p.x);
  T* __restrict__ y = static_cast<T*>(p.y);
  const int b = p.b, c = p.c, d = p.d;
  const int nj = d / V;
  const int per_row = p.a * nj;
  const int64_t total = (int64_t)p.batch * per_row;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int beta = (int)(t / per_row);
  const int r = (int)(t - (int64_t)beta * per_row);
  const int i = r / nj;
  const int j0 = (r - i * nj) * V;
  const T* xs = x + (size_t)beta * p.N + (size_t)i * c * d + j0;
  T* ys = y + (size_t)beta * p.M + (size_t)i * b * d + j0;
  float xv[CMAX][V];
#pragma unroll
  for (int l = 0; l < CMAX; ++l)
    if (l < c) load_vec<T, V>(xs + (size_t)l * d, xv[l]);
  const T* blk = kv + ((size_t)i * d + j0) * b * c;  // block (i, j0); block (i, j0+e) is e*b*c further
#pragma unroll
  for (int k = 0; k < BMAX; ++k) {
    if (k >= b) continue;
    float acc[V];
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] = 0.f;
#pragma unroll
    for (int l = 0; l < CMAX; ++l) {
      if (l < c) {
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] = __builtin_fmaf(to_f32(blk[(size_t)e * b * c + k * c + l]), xv[l][e], acc[e]);
      }
    }
    if (p.bias != nullptr) {
#pragma unroll
      for (int e = 0; e < V; ++e) acc[e] += bias_value<T>(p, (int64_t)(i * b + k) * d + j0 + e);
    }
    if (epilogue_gelu(p)) {
#pragma unroll
      for (int e = 0; e < V; ++e) acc[e] = gelu_f32<T>(acc[e]);
    }
    store_vec<T, V>(ys + (size_t)k * d, acc);
  }
}

namespace {

template <typename T, int VEC>
hipError_t dispatch_valu_bsl(const Problem& p, const Plan& pl, hipStream_t s) {
  dim3 grid(pl.grid, p.a * p.d), block(256);
  const int m = p.b > p.c ? p.b : p.c;
  // The unroll factor must match valu_bsl_unroll(), which sized the grid.
  if (m <= 2) hipLaunchKernelGGL((ks_valu_bsl_kernel<T, VEC, 2, 2, 4>), grid, block, 0, s, p);
  else if (m <= 4) hipLaunchKernelGGL((ks_valu_bsl_kernel<T, VEC, 4, 4, 2>), grid, block, 0, s, p);
  else if (m <= 8) hipLaunchKernelGGL((ks_valu_bsl_kernel<T, VEC, 8, 8, 1>), grid, block, 0, s, p);
  else hipLaunchKernelGGL((ks_valu_bsl_kernel<T, VEC, 16, 16, 1>), grid, block, 0, s, p);
  return hipGetLastError();
}

template <typename T, int V>
hipError_t dispatch_valu_bsf(const Problem& p, const Plan& pl, hipStream_t s) {
  dim3 grid(pl.grid), block(256);
  const int m = p.b > p.c ? p.b : p.c;
  if (m <= 2) hipLaunchKernelGGL((ks_valu_bsf_kernel<T, V, 2, 2>), grid, block, 0, s, p);
  else if (m <= 4) hipLaunchKernelGGL((ks_valu_bsf_kernel<T, V, 4, 4>), grid, block, 0, s, p);
  else if (m <= 8) hipLaunchKernelGGL((ks_valu_bsf_kernel<T, V, 8, 8>), grid, block, 0, s, p);
  else hipLaunchKernelGGL((ks_valu_bsf_kernel<T, V, 16, 16>), grid, block, 0, s, p);
  return hipGetLastError();
}

template <typename T>
hipError_t bsf_by_v(const Problem& p, const Plan& pl, hipStream_t s) {
  switch (pl.vec) {
    case 1: return dispatch_valu_bsf<T, 1>(p, pl, s);
    case 2: return dispatch_valu_bsf<T, 2>(p, pl, s);
    case 4: return dispatch_valu_bsf<T, 4>(p, pl, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_valu_bsl(const Problem& p, const Plan& pl, hipStream_t s) {
  switch (p.dtype) {
    case F32: return pl.vec == 4 ? dispatch_valu_bsl<float, 4>(p, pl, s) : dispatch_valu_bsl<float, 1>(p, pl, s);
    case BF16: return pl.vec == 8 ? dispatch_valu_bsl<bf16_t, 8>(p, pl, s) : dispatch_valu_bsl<bf16_t, 1>(p, pl, s);
    case F16: return pl.vec == 8 ? dispatch_valu_bsl<_Float16, 8>(p, pl, s) : dispatch_valu_bsl<_Float16, 1>(p, pl, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_valu_bsf(const Problem& p, const Plan& pl, hipStream_t s) {
  switch (p.dtype) {
    case F32: return bsf_by_v<float>(p, pl, s);
    case BF16:
      if (pl.vec == 8) return dispatch_valu_bsf<bf16_t, 8>(p, pl, s);
      return bsf_by_v<bf16_t>(p, pl, s);
    case F16:
      if (pl.vec == 8) return dispatch_valu_bsf<_Float16, 8>(p, pl, s);
      return bsf_by_v<_Float16>(p, pl, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ks
