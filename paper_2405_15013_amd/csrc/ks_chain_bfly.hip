// Fused dyadic butterfly chain, two register passes (ks_chain_fused.h,
// butterfly form): Y = X (K_1 ... K_L)^T with K_l of pattern
// (2^(l-1), 2, 2, 2^(L-l)), N = 2^L (paper Section 1, Figure 1; Appendix B.1,
// Table 5).
//
// One workgroup of 512 threads owns 16 batch columns, loaded into LDS as
// fp32 (16 floats per row, rows swizzled so that the four units of a
// wavefront hit four bank windows).  Pass A: unit (column n, group g) takes
// the PA = 2^LA rows g*PA .. g*PA + PA-1 of its column into registers and
// applies the factors with d = 1 .. PA/2 there (all their 2 x 2 blocks lie
// inside the group), then writes them back.  Pass B: unit (column n, j)
// takes rows j + PA*r (r < PB) and applies the remaining factors.  Ten
// factors cost two LDS round trips and three barriers.
//
// Factor values: the 16 lanes of a wavefront row work on the 16 columns of
// one unit and need the same blocks, so lane i fetches the unit's i-th block
// of each factor (one 16- or 8-byte load per factor, issued before X) into
// registers and each butterfly takes its block's values from the owning lane
// by DPP row broadcast; the factor values never go through LDS.
#include "ks_chain_fused.h"
#include "ks_chain_fused_io.h"
#include "ks_common.h"
#include "ks_internal.h"

namespace ks {

namespace {

template <typename T> struct BflyRun { typedef u32x4 type; };  // four values
template <> struct BflyRun<bf16_t> { typedef u32x2 type; };
template <> struct BflyRun<_Float16> { typedef u32x2 type; };

// Value of v in lane `src` of this lane's row of 16 (DPP row_newbcast; src
// must fold to a constant).
template <int S>
__device__ __forceinline__ float row_bcast_c(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x150 + S, 0xf, 0xf, true));
}
__device__ __forceinline__ float row_bcast(float v, int src) {
  switch (src) {
    case 0: return row_bcast_c<0>(v);
    case 1: return row_bcast_c<1>(v);
    case 2: return row_bcast_c<2>(v);
    case 3: return row_bcast_c<3>(v);
    case 4: return row_bcast_c<4>(v);
    case 5: return row_bcast_c<5>(v);
    case 6: return row_bcast_c<6>(v);
    case 7: return row_bcast_c<7>(v);
    case 8: return row_bcast_c<8>(v);
    case 9: return row_bcast_c<9>(v);
    case 10: return row_bcast_c<10>(v);
    case 11: return row_bcast_c<11>(v);
    case 12: return row_bcast_c<12>(v);
    case 13: return row_bcast_c<13>(v);
    case 14: return row_bcast_c<14>(v);
    default: return row_bcast_c<15>(v);
  }
}

// One 2 x 2 block applied to (a, b): the block's four values are in lane
// `src` of the row (k, as loaded by that lane).
__device__ __forceinline__ void bfly_apply(const f32x4& k, int src, float& a, float& b) {
  const float k00 = row_bcast(k[0], src), k01 = row_bcast(k[1], src);
  const float k10 = row_bcast(k[2], src), k11 = row_bcast(k[3], src);
  const float a0 = a, b0 = b;
  a = k00 * a0 + k01 * b0;
  b = k10 * a0 + k11 * b0;
}

// LDS map of the butterfly form for the tile load and store.
struct BflyAddr {
  int la;
  __device__ __forceinline__ int operator()(int row, int col) const { return bfly_lds_row(row, la) * 16 + col; }
};

template <typename T, int LAYOUT, bool VEC, int LA, int LB>
__global__ __launch_bounds__(kFusedThreads) void ks_chain_bfly_kernel(FusedChain fc) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  constexpr int PA = 1 << LA, PB = 1 << LB, L = LA + LB;
  static_assert(16 * PA <= kFusedThreads && 16 * PB <= kFusedThreads, "one unit per thread");
  static_assert(PA >= 4 && PB >= 4, "four units per wavefront");
  typedef typename BflyRun<T>::type KW;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col0 = fused_tile((int)blockIdx.x, (int)gridDim.x) * kFusedCols;
  const int n = lane & 15, u = 4 * w + (lane >> 4);  // column, unit

  // Factor blocks, fetched first, straight into registers: at step s of pass
  // A the unit's PA/2 blocks are u*PA/2 + block(r) (PA is a multiple of 2d,
  // and block(r) runs over 0 .. PA/2-1), and lane n of the row holds block
  // u*PA/2 + n; at step s of pass B the block of row j + PA*r is j + block(PA*r)
  // (j < PA <= d leaves the bits above s alone), the butterflies are the r
  // with bit t = s - LA clear, and lane i holds the i-th of them.
  f32x4 ka[LA], kb[LB];
  {
    auto fetch = [&](int q, int blk) {
      const T* kv = static_cast<const T*>(fc.kv[q]) + 4 * blk;
      T e[4];
      if (fc.kvec) {
        const KW w4 = *reinterpret_cast<const KW*>(kv);
        __builtin_memcpy(e, &w4, sizeof(KW));
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) e[t] = kv[t];
      }
      return f32x4{to_f32(e[0]), to_f32(e[1]), to_f32(e[2]), to_f32(e[3])};
    };
    const int ua = 4 * w < PB ? u : 0, ia = n < PA / 2 ? n : 0;
#pragma unroll
    for (int s = 0; s < LA; ++s) ka[s] = fetch(L - 1 - s, ua * (PA / 2) + ia);
    const int jb = 4 * w < PA ? u : 0, ib = n < PB / 2 ? n : 0;
#pragma unroll
    for (int s = LA; s < L; ++s) {
      const int t = s - LA, ri = ((ib >> t) << (t + 1)) | (ib & ((1 << t) - 1));
      kb[s - LA] = fetch(L - 1 - s, jb + bfly_block(PA * ri, s));
    }
  }
  fused_load<T, LAYOUT, VEC>(fc, lds, col0, BflyAddr{LA});
  __syncthreads();

  // Pass A, in place: rows u*PA + r of column n; application steps
  // s = 0 .. LA-1 (factor L-1-s, d = 2^s): block (R >> (s+1), R mod d) mixes
  // rows R and R + d of the group.
  if (4 * w < PB) {
    float x[PA];
#pragma unroll
    for (int r = 0; r < PA; ++r) x[r] = lds[bfly_lds_row(u * PA + r, LA) * 16 + n];
#pragma unroll
    for (int s = 0; s < LA; ++s) {
      const int d = 1 << s;
#pragma unroll
      for (int r = 0; r < PA; ++r)
        if (!(r & d)) bfly_apply(ka[s], bfly_block(r, s), x[r], x[r + d]);
    }
#pragma unroll
    for (int r = 0; r < PA; ++r) lds[bfly_lds_row(u * PA + r, LA) * 16 + n] = x[r];
  }
  __syncthreads();

  // Pass B, in place: rows j + PA*r of column n (j = u); steps s = LA .. L-1
  // (d = 2^s = PA * 2^(s-LA): local partner r + 2^(s-LA)).
  if (4 * w < PA) {
    const int j = u;
    float y[PB];
#pragma unroll
    for (int r = 0; r < PB; ++r) y[r] = lds[bfly_lds_row(j + PA * r, LA) * 16 + n];
#pragma unroll
    for (int s = LA; s < L; ++s) {
      const int t = s - LA, ds = 1 << t;
#pragma unroll
      for (int r = 0; r < PB; ++r)
        if (!(r & ds)) bfly_apply(kb[s - LA], ((r >> (t + 1)) << t) | (r & (ds - 1)), y[r], y[r + ds]);
    }
#pragma unroll
    for (int r = 0; r < PB; ++r) lds[bfly_lds_row(j + PA * r, LA) * 16 + n] = y[r];
  }
  __syncthreads();
  fused_store<T, LAYOUT, VEC>(fc, lds, col0, BflyAddr{LA});
}

template <typename T, int LA, int LB>
hipError_t launch_bfly_l(const FusedChain& fc, bool vec, hipStream_t s) {
  const dim3 grid((fc.batch + kFusedCols - 1) / kFusedCols), block(kFusedThreads);
  const int lds = fused_lds_bytes(fc);
#define KS_BFLY_LAUNCH(L_, V)                                                                                 \
  {                                                                                                          \
    if (lds > 64 * 1024) {                                                                                   \
      static const hipError_t raised = hipFuncSetAttribute(                                                  \
          reinterpret_cast<const void*>(&ks_chain_bfly_kernel<T, L_, V, LA, LB>),                            \
          hipFuncAttributeMaxDynamicSharedMemorySize, kFusedMaxLds);                                         \
      if (raised != hipSuccess) return raised;                                                               \
    }                                                                                                        \
    hipLaunchKernelGGL((ks_chain_bfly_kernel<T, L_, V, LA, LB>), grid, block, lds, s, fc);                   \
    return hipGetLastError();                                                                                \
  }
  if (fc.layout == BSL) {
    if (vec) KS_BFLY_LAUNCH(BSL, true) else KS_BFLY_LAUNCH(BSL, false)
  }
  if (vec) KS_BFLY_LAUNCH(BSF, true) else KS_BFLY_LAUNCH(BSF, false)
#undef KS_BFLY_LAUNCH
}

template <typename T>
hipError_t launch_bfly_t(const FusedChain& fc, bool vec, hipStream_t s) {
  switch (fc.bfly) {
    case 4: return launch_bfly_l<T, 2, 2>(fc, vec, s);
    case 5: return launch_bfly_l<T, 3, 2>(fc, vec, s);
    case 6: return launch_bfly_l<T, 3, 3>(fc, vec, s);
    case 7: return launch_bfly_l<T, 4, 3>(fc, vec, s);
    case 8: return launch_bfly_l<T, 4, 4>(fc, vec, s);
    case 9: return launch_bfly_l<T, 5, 4>(fc, vec, s);
    case 10: return launch_bfly_l<T, 5, 5>(fc, vec, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_chain_bfly(const FusedChain& fc, int dtype, bool vec, hipStream_t s) {
  switch (dtype) {
    case F32: return launch_bfly_t<float>(fc, vec, s);
    case BF16: return launch_bfly_t<bf16_t>(fc, vec, s);
    case F16: return launch_bfly_t<_Float16>(fc, vec, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ks
