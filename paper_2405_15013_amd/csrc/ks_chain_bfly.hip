// Fused dyadic butterfly chain, two register passes (ks_chain_fused.h,
// butterfly form): Y = X (K_1 ... K_L)^T with K_l of pattern
// (2^(l-1), 2, 2, 2^(L-l)), N = 2^L (paper Section 1, Figure 1; Appendix B.1,
// Table 5).
//
// One workgroup of 512 threads owns 16 batch columns, kept in LDS as fp32
// between the passes (16 floats per row, rows swizzled so that the four units
// of a wavefront hit four bank windows).  Pass A: unit (column n, group g)
// takes the PA = 2^LA rows g*PA .. g*PA + PA-1 of its column into registers
// and applies the factors with d = 1 .. PA/2 there (all their 2 x 2 blocks lie
// inside the group).  Pass B: unit (column n, j) takes rows j + PA*r (r < PB)
// and applies the remaining factors.  A wavefront loads the X rows of its own
// pass-A units and, batch-size-last, stores the Y rows of its own pass-B
// units, so the only barrier is the one between the passes (batch-size-first
// a wavefront's output rows are 16-byte runs interleaved with the others' in
// each batch row, and the tile is stored by the shared store after a second
// barrier).
//
// Factor values: the 16 lanes of a wavefront row work on the 16 columns of
// one unit and need the same blocks, so lane i fetches the unit's i-th block
// of each factor (one 16- or 8-byte load per factor: pass A's after the
// wavefront's X loads, pass B's before the barrier) into registers and each
// butterfly takes its block's values from the owning lane by DPP row
// broadcast; the factor values never go through LDS.
#include <type_traits>

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

// LDS map of the butterfly form for the shared tile store.
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

  // Factor blocks go straight into registers: at step s of pass A the unit's
  // PA/2 blocks are u*PA/2 + block(r) (PA is a multiple of 2d, and block(r)
  // runs over 0 .. PA/2-1), and lane n of the row holds block u*PA/2 + n; at
  // step s of pass B the block of row j + PA*r is j + block(PA*r) (j < PA <= d
  // leaves the bits above s alone), the butterflies are the r with bit
  // t = s - LA clear, and lane i holds the i-th of them.  Pass A's blocks are
  // fetched right after the wavefront's X loads, pass B's before the barrier.
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
  // Tile pieces: EP consecutive elements (16 bytes when VEC, else one); in
  // the batch-size-last layout PR pieces make one row of the tile.
  constexpr int EP = VEC ? 16 / (int)sizeof(T) : 1, PR = kFusedCols / EP;
  typedef typename std::conditional<VEC, u32x4, T>::type PW;
  const T* __restrict__ xp = static_cast<const T*>(fc.x);
  T* __restrict__ yp = static_cast<T*>(fc.y);
  const int B = fc.batch;
  auto lds_at = [&](int row, int col) { return lds + bfly_lds_row(row, LA) * 16 + col; };

  // Pass A, rows u*PA + r of column n.  Each wavefront loads exactly the rows
  // of its own four units, as pieces regrouped by column through its own LDS
  // rows, so it starts as soon as its own loads arrive.  Steps s = 0 .. LA-1
  // (factor L-1-s, d = 2^s): block (R >> (s+1), R mod d) mixes rows R and
  // R + d.
  if (4 * w < PB) {
    float x[PA];
    if (LAYOUT == BSL) {
      constexpr int TOT = 4 * PA * PR, NP = (TOT + 63) / 64;  // pieces of the wavefront, per lane
      PW pw[NP];
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        const int p = i * 64 + lane, row = 4 * w * PA + p / PR, col = (p % PR) * EP;
        const bool ok = p < TOT && col0 + col < B;
        const T* src = xp + (int64_t)row * B + col0 + col;
        if constexpr (VEC) pw[i] = ok ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src)) : u32x4{0, 0, 0, 0};
        else pw[i] = ok ? *src : T(0);
      }
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        const int p = i * 64 + lane, row = 4 * w * PA + p / PR, col = (p % PR) * EP;
        if (TOT % 64 && p >= TOT) continue;
        if constexpr (VEC) {
          T e[EP];
          __builtin_memcpy(e, &pw[i], 16);
#pragma unroll
          for (int q = 0; q < EP; q += 4)
            *reinterpret_cast<f32x4*>(lds_at(row, col + q)) = f32x4{to_f32(e[q]), to_f32(e[q + 1]), to_f32(e[q + 2]), to_f32(e[q + 3])};
        } else {
          *lds_at(row, col) = to_f32(pw[i]);
        }
      }
#pragma unroll
      for (int r = 0; r < PA; ++r) x[r] = *lds_at(u * PA + r, n);
    } else {
      // the wavefront's span of vector rows 4w*PA .. +4PA of every batch row
      // t of the tile, as pieces of EP consecutive rows: lane (t, k) takes
      // piece k (16 batch rows x 4 consecutive pieces per load)
      constexpr int KP = 4 * PA / EP, NI = (KP + 3) / 4;
      const int t = lane & 15;
      PW pw[NI];
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int k = 4 * i + (lane >> 4);
        const bool ok = (KP % 4 == 0 || k < KP) && col0 + t < B;
        const T* src = xp + (int64_t)(col0 + t) * (PA * PB) + 4 * w * PA + k * EP;
        if constexpr (VEC) pw[i] = ok ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src)) : u32x4{0, 0, 0, 0};
        else pw[i] = ok ? *src : T(0);
      }
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int k = 4 * i + (lane >> 4);
        if (KP % 4 && k >= KP) continue;
        if constexpr (VEC) {
          T e[EP];
          __builtin_memcpy(e, &pw[i], 16);
#pragma unroll
          for (int q = 0; q < EP; ++q) *lds_at(4 * w * PA + k * EP + q, t) = to_f32(e[q]);
        } else {
          *lds_at(4 * w * PA + k, t) = to_f32(pw[i]);
        }
      }
#pragma unroll
      for (int r = 0; r < PA; ++r) x[r] = *lds_at(u * PA + r, n);
    }
    f32x4 ka[LA];
#pragma unroll
    for (int s = 0; s < LA; ++s) ka[s] = fetch(L - 1 - s, u * (PA / 2) + (n < PA / 2 ? n : 0));
#pragma unroll
    for (int s = 0; s < LA; ++s) {
      const int d = 1 << s;
#pragma unroll
      for (int r = 0; r < PA; ++r)
        if (!(r & d)) bfly_apply(ka[s], bfly_block(r, s), x[r], x[r + d]);
    }
#pragma unroll
    for (int r = 0; r < PA; ++r) *lds_at(u * PA + r, n) = x[r];
  }
  f32x4 kb[LB];
  {
    const int jb = 4 * w < PA ? u : 0, ib = n < PB / 2 ? n : 0;
#pragma unroll
    for (int s = LA; s < L; ++s) {
      const int t = s - LA, ri = ((ib >> t) << (t + 1)) | (ib & ((1 << t) - 1));
      kb[s - LA] = fetch(L - 1 - s, jb + bfly_block(PA * ri, s));
    }
  }
  __syncthreads();

  // Pass B, rows j + PA*r of column n (j = u); steps s = LA .. L-1 (d = 2^s =
  // PA * 2^(s-LA): local partner r + 2^(s-LA)).  The results go back to the
  // wavefront's own rows; batch-size-last it stores them itself as row pieces.
  if (4 * w < PA) {
    const int j = u;
    float y[PB];
#pragma unroll
    for (int r = 0; r < PB; ++r) y[r] = *lds_at(j + PA * r, n);
#pragma unroll
    for (int s = LA; s < L; ++s) {
      const int t = s - LA, ds = 1 << t;
#pragma unroll
      for (int r = 0; r < PB; ++r)
        if (!(r & ds)) bfly_apply(kb[s - LA], ((r >> (t + 1)) << t) | (r & (ds - 1)), y[r], y[r + ds]);
    }
    if constexpr (LAYOUT != BSL) {
#pragma unroll
      for (int r = 0; r < PB; ++r) *lds_at(j + PA * r, n) = y[r];
    } else {
      // pieces of rows 4w + a + PA*r; load i of the lane takes the rows of
      // RPI consecutive r, written just before it
      constexpr int TOT = 4 * PB * PR, NP = (TOT + 63) / 64;
      constexpr int RPI = TOT % 64 ? PB : 16 / PR;
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        if (TOT % 64 == 0 || i == 0) {
#pragma unroll
          for (int r = RPI * i; r < RPI * i + RPI; ++r) *lds_at(j + PA * r, n) = y[r];
        }
        const int p = i * 64 + lane, rho = p / PR, col = (p % PR) * EP;
        const int row = 4 * w + (rho & 3) + PA * (rho >> 2);
        if ((TOT % 64 && p >= TOT) || col0 + col >= B) continue;
        T* dst = yp + (int64_t)row * B + col0 + col;
        if constexpr (VEC) {
          union { u32x4 w4; T e[EP]; } o;
#pragma unroll
          for (int q = 0; q < EP; ++q) o.e[q] = from_f32<T>(*lds_at(row, col + q));
          __builtin_nontemporal_store(o.w4, reinterpret_cast<u32x4*>(dst));
        } else {
          *dst = from_f32<T>(*lds_at(row, col));
        }
      }
    }
  }
  if (LAYOUT == BSF) {
    // a wavefront's output rows interleave with the others' along each batch
    // row: store the whole tile in contiguous runs after a barrier
    __syncthreads();
    fused_store<T, LAYOUT, VEC>(fc, lds, col0, BflyAddr{LA});
  }
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
