// Masked register-direct MFMA kernel (index arithmetic and decomposition in
// ks_masked_index.h): the MFMA path for patterns whose b or c is not a
// multiple of 16, batch-size-last batches that are not a multiple of the
// 16-byte vector, and buffers that are not 16-byte aligned.
#pragma once
#include "ks_direct.h"
#include "ks_masked_index.h"

namespace ks {
// The problem's and the tile description's fields in scalar registers at
// kernel entry, in one round of kernel-argument loads (as kernarg_fetch of
// Problem in ks_direct.h).
__device__ __forceinline__ void kernarg_fetch(const Problem& p, const MaskedTile& t) {
  asm volatile("" ::KS_PROBLEM_FIELDS(p), "s"(t.mt), "s"(t.kgroups), "s"(t.jgroups), "s"(t.nbt), "s"(t.items),
               "s"(t.nchunks), "s"(t.kvec));
}
}  // namespace ks

namespace ks {

// V consecutive elements of type T (V * sizeof(T) bytes, aligned to that).
template <typename T, int V>
__device__ __forceinline__ void masked_load(const T* p, T (&v)[V]) {
  constexpr int NB = V * (int)sizeof(T);
  if constexpr (NB == 16) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(p);
    __builtin_memcpy(v, &w, 16);
  } else if constexpr (NB == 8) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(p);
    __builtin_memcpy(v, &w, 8);
  } else {
#pragma unroll
    for (int e = 0; e < V; ++e) v[e] = p[e];
  }
}
template <typename T, int V>
__device__ __forceinline__ void masked_store(T* p, const T (&v)[V]) {
  constexpr int NB = V * (int)sizeof(T);
  if constexpr (NB == 16) {
    u32x4 w;
    __builtin_memcpy(&w, v, 16);
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(p));
  } else if constexpr (NB == 8) {
    u32x2 w;
    __builtin_memcpy(&w, v, 8);
    __builtin_nontemporal_store(w, reinterpret_cast<u32x2*>(p));
  } else {
#pragma unroll
    for (int e = 0; e < V; ++e) p[e] = v[e];
  }
}

__device__ __forceinline__ uint32_t masked_bits(float v) { return __float_as_uint(v); }
__device__ __forceinline__ uint32_t masked_bits(bf16_t v) { return v; }
__device__ __forceinline__ uint32_t masked_bits(_Float16 v) { return __builtin_bit_cast(uint16_t, v); }

template <typename T, int LAYOUT, int V, bool EPI>
__global__ __launch_bounds__(256) void ks_masked_kernel(Problem p, MaskedTile t) {
  constexpr int S = sizeof(T);
  constexpr int LP = S == 4 ? 4 : 8;
  constexpr int CH = 4 * LP;
  constexpr int VK = LAYOUT == BSL ? 1 : V;  // K blocks per lane (BSF: one per j of the piece)
  const int lane = threadIdx.x & 63;
  // Spare waves of the last workgroup work on the last item and store
  // nothing: no branch before the loads, one round of kernel-argument loads.
  const int item0 = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool live = item0 < t.items;  // wave-uniform
  const int item = live ? item0 : t.items - 1;
  kernarg_fetch(p, t);
  const int n = lane & 15, g = lane >> 4;
  const MItem it = masked_item(p, t, V, item);
  const T* __restrict__ x = static_cast<const T*>(p.x);
  const T* __restrict__ kv = static_cast<const T*>(p.kv);

  f32x4 acc[1][V];
#pragma unroll
  for (int e = 0; e < V; ++e) acc[0][e] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int ch = 0; ch < t.nchunks; ++ch) {
    const int l0 = ch * CH + LP * g;
    T xs[LP][V];
    T ks[VK][LP];
#pragma unroll
    for (int q = 0; q < LP; ++q) {
      const int64_t off = masked_x_off(p, it, V, l0 + q, n);
      if (off >= 0) {
        masked_load<T, V>(x + off, xs[q]);
      } else {
#pragma unroll
        for (int e = 0; e < V; ++e) xs[q][e] = T(0);
      }
      if (!t.kvec) {
#pragma unroll
        for (int e = 0; e < VK; ++e) {
          const int64_t ko = masked_k_off(p, it, e, n, l0 + q);
          ks[e][q] = ko >= 0 ? kv[ko] : T(0);
        }
      }
    }
    if (t.kvec) {
      // K rows are whole MFMA operands: one LP-element vector per block
      // (LP * sizeof(T) = 16 bytes, aligned), zero in the padding rows.
#pragma unroll
      for (int e = 0; e < VK; ++e) {
        const int64_t ko = masked_k_off(p, it, e, n, l0);
        if (ko >= 0) {
          masked_load<T, LP>(kv + ko, ks[e]);
        } else {
#pragma unroll
          for (int q = 0; q < LP; ++q) ks[e][q] = T(0);
        }
      }
    }
    // MFMA operands in the layout of the register-direct kernels
    uint32_t xw[LP * V * S / 4];
    uint32_t kw[1][VK][LP * S / 4];
    if constexpr (S == 4) {
#pragma unroll
      for (int q = 0; q < LP; ++q) {
#pragma unroll
        for (int e = 0; e < V; ++e) xw[q * V + e] = masked_bits(xs[q][e]);
#pragma unroll
        for (int e = 0; e < VK; ++e) kw[0][e][q] = masked_bits(ks[e][q]);
      }
    } else {
#pragma unroll
      for (int w = 0; w < LP * V / 2; ++w) {
        const int f0 = 2 * w, f1 = 2 * w + 1;  // flat t*V + e
        xw[w] = masked_bits(xs[f0 / V][f0 % V]) | (masked_bits(xs[f1 / V][f1 % V]) << 16);
      }
#pragma unroll
      for (int e = 0; e < VK; ++e)
#pragma unroll
        for (int w = 0; w < LP / 2; ++w)
          kw[0][e][w] = masked_bits(ks[e][2 * w]) | (masked_bits(ks[e][2 * w + 1]) << 16);
    }
    direct_mma<T, LAYOUT, V, 1, LP>(xw, kw, acc);
  }
  if (!live) return;
  // Epilogue (EPI instances only): output feature of (e, r) is row
  // k = k0 + 4g + r of block (i, j0 [+ e in BSF]); padding rows (k >= b) take
  // no bias.
  if constexpr (EPI) {
    constexpr int BV = LAYOUT == BSF ? V : 1;
    const bool has_bias = p.bias != nullptr;
    float bv[4][BV];
    if (has_bias) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int k = it.k0 + 4 * g + r;
#pragma unroll
        for (int e = 0; e < BV; ++e)
          bv[r][e] = k < p.b ? bias_value<T>(p, ((int64_t)it.i * p.b + k) * p.d + it.j0 + e) : 0.0f;
      }
    }
    mfma_results_settle();
    if (has_bias) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int e = 0; e < V; ++e) acc[0][e][r] += bv[r][LAYOUT == BSF ? e : 0];
    }
    if (epilogue_gelu(p)) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int e = 0; e < V; ++e) acc[0][e][r] = gelu_f32<T>(acc[0][e][r]);
    }
  } else {
    mfma_results_settle();
  }
  // outputs k = k0 + 4g + r, columns e of the lane's piece
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t off = masked_y_off(p, it, V, n, g, r);
    if (off < 0) continue;
    T v[V];
#pragma unroll
    for (int e = 0; e < V; ++e) v[e] = from_f32<T>(acc[0][e][r]);
    masked_store<T, V>(static_cast<T*>(p.y) + off, v);
  }
}

// Instances of one storage type: V in {1, 2, 4} (and 8 for 16-bit BSL).
// EPI: the bias / activation epilogue compiled in (calls that need it).
template <typename T>
hipError_t launch_masked_type(const Problem& p, const MaskedTile& t, int V, unsigned grid, hipStream_t s) {
  const dim3 g(grid), b(256);
  const bool epi = has_epilogue(p);
#define KS_MASKED(L, VV)                                                              \
  if (p.layout == L && V == VV) {                                                     \
    if (epi)                                                                          \
      hipLaunchKernelGGL((ks_masked_kernel<T, L, VV, true>), g, b, 0, s, p, t);      \
    else                                                                              \
      hipLaunchKernelGGL((ks_masked_kernel<T, L, VV, false>), g, b, 0, s, p, t);     \
    return hipGetLastError();                                                         \
  }
  KS_MASKED(BSL, 1) KS_MASKED(BSL, 2) KS_MASKED(BSL, 4)
  KS_MASKED(BSF, 1) KS_MASKED(BSF, 2) KS_MASKED(BSF, 4)
  if constexpr (sizeof(T) == 2) {
    KS_MASKED(BSL, 8)
  }
#undef KS_MASKED
  return hipErrorInvalidValue;
}

}  // namespace ks
