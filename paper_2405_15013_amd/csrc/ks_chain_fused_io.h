// Tile loads and stores of the fused chain kernels (ks_chain_fused.hip and
// ks_chain_mfma.hip): the workgroup's kFusedCols batch columns of X into LDS
// rows as fp32, and LDS rows back into Y in the storage type.
//
// Latency: the tile loads are issued in batches of kFusedLoadBatch 16-byte
// loads per thread before any of them is used (one batch for a 64 KB tile of
// fp32 or a 32 KB tile of 16-bit values).
#pragma once
#include <type_traits>

#include "ks_chain_fused.h"
#include "ks_common.h"
#include "ks_internal.h"

namespace ks {

constexpr int kFusedLoadBatch = 8;

// LDS float index of (row, column) of the tile: rows at kFusedPitch floats.
// The butterfly form passes its own map (16 floats per row, rows swizzled).
struct FusedPitchAddr {
  int pitch = kFusedPitch;
  __device__ __forceinline__ int operator()(int row, int col) const { return row * pitch + col; }
};

// Load the tile's input columns (NC of them) into LDS rows [0, width_in) (fp32).
//  BSL: X is (N, batch); row n of the tile is the run X[n, col0 .. col0+NC).
//  BSF: X is (batch, N); batch row col0+t is the run X[col0+t, 0 .. N).
// VEC: 16-byte accesses (the host checked alignment and that the batch (BSL)
// or N (BSF) is a multiple of the vector).  Columns beyond the batch are
// filled with zeros and never stored.
template <typename T, int LAYOUT, bool VEC, typename A = FusedPitchAddr, int NC = kFusedCols>
__device__ __forceinline__ void fused_load(const FusedChain& fc, float* lds, int col0, A at = A()) {
  const T* __restrict__ x = static_cast<const T*>(fc.x);
  const int N = fc.width_in, B = fc.batch, tid = threadIdx.x;
  constexpr int E = VEC ? 16 / (int)sizeof(T) : 1;  // elements per access
  const int total = N * NC / E;
  for (int base = 0; base < total; base += kFusedThreads * kFusedLoadBatch) {
    typedef typename std::conditional<VEC, u32x4, T>::type W;
    W w[kFusedLoadBatch];
#pragma unroll
    for (int r = 0; r < kFusedLoadBatch; ++r) {
      const int u = base + r * kFusedThreads + tid;
      int row, col;
      if constexpr (VEC) fused_vec_unit(LAYOUT, E, u, &row, &col, NC);
      else if constexpr (LAYOUT == BSL) { row = u / NC; col = u % NC; }
      else { col = u % NC; row = u / NC; }
      const bool ok = u < total && col0 + col < B;
      const int64_t off = LAYOUT == BSL ? (int64_t)row * B + col0 + col : (int64_t)(col0 + col) * N + row;
      if constexpr (VEC) w[r] = ok ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(x + off)) : u32x4{0, 0, 0, 0};
      else w[r] = ok ? x[off] : T(0);
    }
#pragma unroll
    for (int r = 0; r < kFusedLoadBatch; ++r) {
      const int u = base + r * kFusedThreads + tid;
      if (u >= total) break;
      int row, col;
      if constexpr (VEC) fused_vec_unit(LAYOUT, E, u, &row, &col, NC);
      else if constexpr (LAYOUT == BSL) { row = u / NC; col = u % NC; }
      else { col = u % NC; row = u / NC; }
      if constexpr (VEC) {
        const T* e = reinterpret_cast<const T*>(&w[r]);
        if constexpr (LAYOUT == BSL) {
#pragma unroll
          for (int q = 0; q < E; q += 4)
            *reinterpret_cast<f32x4*>(lds + at(row, col + q)) =
                f32x4{to_f32(e[q]), to_f32(e[q + 1]), to_f32(e[q + 2]), to_f32(e[q + 3])};
        } else {
#pragma unroll
          for (int q = 0; q < E; ++q) lds[at(row + q, col)] = to_f32(e[q]);
        }
      } else {
        lds[at(row, col)] = to_f32(w[r]);
      }
    }
  }
}

// Store LDS rows [0, width_out) of the tile's valid columns into Y, rounded to
// the storage type (same layouts and vector rules as fused_load).
template <typename T, int LAYOUT, bool VEC, typename A = FusedPitchAddr, int NC = kFusedCols>
__device__ __forceinline__ void fused_store(const FusedChain& fc, const float* lds, int col0, A at = A()) {
  T* __restrict__ y = static_cast<T*>(fc.y);
  const int M = fc.width_out, B = fc.batch, tid = threadIdx.x;
  constexpr int E = VEC ? 16 / (int)sizeof(T) : 1;
  const int total = M * NC / E;
  for (int u = tid; u < total; u += kFusedThreads) {
    int row, col;
    if constexpr (VEC) fused_vec_unit(LAYOUT, E, u, &row, &col, NC);
    else if constexpr (LAYOUT == BSL) { row = u / NC; col = u % NC; }
    else { col = u % NC; row = u / NC; }
    if (col0 + col >= B) continue;
    const int64_t off = LAYOUT == BSL ? (int64_t)row * B + col0 + col : (int64_t)(col0 + col) * M + row;
    if constexpr (VEC) {
      union { u32x4 w; T e[E]; } o;
#pragma unroll
      for (int q = 0; q < E; ++q)
        o.e[q] = from_f32<T>(LAYOUT == BSL ? lds[at(row, col + q)] : lds[at(row + q, col)]);
      __builtin_nontemporal_store(o.w, reinterpret_cast<u32x4*>(y + off));
    } else {
      y[off] = from_f32<T>(lds[at(row, col)]);
    }
  }
}

}  // namespace ks
