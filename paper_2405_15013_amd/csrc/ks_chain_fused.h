// Fused chain of small-block KS factors (paper Section 1 and Figure 1: a
// product of KS factors such as the butterfly factors of a fast transform;
// Appendix B.1, Table 5), shared by the kernel (ks_chain_fused.hip), the host
// planner (ks_host.cpp) and the host replay (ks_verify.hip).
//
// One workgroup owns a tile of kFusedCols batch columns and keeps the whole
// intermediate vector of each of its columns in LDS, in fp32, for the whole
// chain: X is read from HBM once, every factor is applied LDS -> LDS (the
// output-stationary blocks of Algorithm 2, Section 4.1: a thread reads the c
// inputs of one block (i, j) for its columns and writes its b outputs), and Y
// is written once.  Factors with b == c write in place (the row set of a
// block equals its column set, and blocks are disjoint), otherwise two LDS
// buffers alternate.
//
// LDS layout: row r (an element of the intermediate vector) holds the tile's
// kFusedCols columns at r * kFusedPitch floats (16 columns + 4 pad floats, so
// 16-byte accesses of consecutive rows spread over all banks).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

#include "ks_divide.h"

namespace ks {

constexpr int kFusedMaxFactors = 24;
constexpr int kFusedCols = 16;
constexpr int kFusedPitch = 20;        // floats per LDS row
constexpr int kFusedMaxBC = 8;         // largest b and c of a fused factor
constexpr int kFusedMaxLds = 128 * 1024;
constexpr int kFusedThreads = 1024;                              // threads per workgroup
constexpr int kFusedKPerThread = 4;                              // factor values fetched per thread
constexpr int kFusedKValues = kFusedThreads * kFusedKPerThread;  // largest a*b*c*d of a fused factor (4096)

struct FusedChain {
  int nf;                   // factors, in product order (factor nf-1 is applied first)
  int batch;
  int layout;
  int width_in, width_out;  // a*c*d of factor nf-1, a*b*d of factor 0
  int inplace;              // every factor has b == c: one LDS buffer
  int buf_rows;             // rows of one LDS buffer (the widest vector)
  int a[kFusedMaxFactors], b[kFusedMaxFactors], c[kFusedMaxFactors], d[kFusedMaxFactors];
  uint32_t md[kFusedMaxFactors];  // multiply-shift constants of the division by d
  int sd[kFusedMaxFactors];
  const void* kv[kFusedMaxFactors];
  const void* x;
  void* y;
};

// 16-byte pieces (4 columns each) of one LDS row handled by one work unit of
// a factor with blocks of at most m x m: two for m <= 2, one otherwise (enough
// units for the workgroup's threads, inputs and accumulators within the
// register budget of 1024-thread workgroups).
__host__ __device__ __forceinline__ int fused_pieces(int m) { return m <= 2 ? 2 : 1; }

// Work units of factor f: (block ij, group of pieces), group fastest.
__host__ __device__ __forceinline__ int fused_units(const FusedChain& fc, int f) {
  const int bc = fc.b[f] > fc.c[f] ? fc.b[f] : fc.c[f];
  return fc.a[f] * fc.d[f] * (4 / fused_pieces(bc));
}

// Block (i, j) and piece group g of work unit u of factor f (G = 4 / pieces
// groups per row); the kernel and the host replay share this decode.
__host__ __device__ __forceinline__ void fused_unit(const FusedChain& fc, int f, int G, int u, int* i, int* j,
                                                    int* g) {
  const int ij = u / G;
  *g = u - ij * G;
  *i = (int)div_fast((uint32_t)ij, fc.md[f], fc.sd[f]);
  *j = ij - *i * fc.d[f];
}
// LDS row of input l / output k of block (i, j) of factor f (Section 4.1
// index sets: columns i*c*d + l*d + j, rows i*b*d + k*d + j).
__host__ __device__ __forceinline__ int fused_in_row(const FusedChain& fc, int f, int i, int j, int l) {
  return i * fc.c[f] * fc.d[f] + l * fc.d[f] + j;
}
__host__ __device__ __forceinline__ int fused_out_row(const FusedChain& fc, int f, int i, int j, int k) {
  return i * fc.b[f] * fc.d[f] + k * fc.d[f] + j;
}

// Tile loads and stores, 16-byte form: unit u of a pass over the tile covers
// E = 16 / sizeof(T) consecutive elements.
//  BSL: u -> (row n, column t0 = E * v), global element n*batch + col0 + t0,
//       LDS float n*kFusedPitch + t0 (+1 per element).
//  BSF: u -> (batch row t = u % 16, first element n0 = E * (u / 16)), global
//       element (col0 + t)*width + n0, LDS floats (n0 + e)*kFusedPitch + t.
__host__ __device__ __forceinline__ void fused_vec_unit(int layout, int E, int u, int* row, int* col) {
  if (layout == 1) {  // BSL
    const int pr = kFusedCols / E;
    *row = u / pr;
    *col = (u - *row * pr) * E;
  } else {
    *col = u % kFusedCols;
    *row = (u / kFusedCols) * E;
  }
}

// LDS layout: the vector buffer(s), then two fp32 copies of factor values
// (the factor being applied and the next one).
__host__ __device__ __forceinline__ int fused_kbuf_offset(const FusedChain& fc) {
  return (fc.inplace ? 1 : 2) * fc.buf_rows * kFusedPitch;  // floats
}
__host__ __device__ __forceinline__ int fused_lds_bytes(const FusedChain& fc) {
  return (fused_kbuf_offset(fc) + 2 * kFusedKValues) * 4;
}

}  // namespace ks
