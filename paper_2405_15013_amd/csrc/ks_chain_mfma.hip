// Fused chain kernel, MFMA form (ks_chain_fused.h): chains whose factors all
// have square b x b blocks with one b = 16*BT, BT in 1 .. 4 (Monarch-type
// chains; paper Section 1 and Appendix B.1).  The workgroup's tile of 16 or
// 32 batch columns stays in LDS in fp32 for the whole chain; each factor is
// applied in place, one wavefront per block.
//
// Block product: v_mfma_f32_16x16x4_f32 in the register-direct operand
// layout.  Lane (n, g) = (lane % 16, lane / 16) works on column n of the
// tile; for row tile kt, l-chunk ct and t < 4 it supplies A = K[ij][16kt + n]
// [16ct + 4g + t] (element t of one 4-value run of the packed block) and B =
// the tile's value at input row l = 16ct + 4g + t, column n; accumulator r
// of row tile kt is output k = 16kt + 4g + r.  A block's input and output
// rows are the same set (b == c), so the wavefront writes its outputs over
// its inputs once all BT row tiles are accumulated; blocks of one factor use
// disjoint rows, and a barrier separates the factors.
//
// Factor values: each wavefront holds the runs of two blocks in registers
// (ping-pong) and fetches the next block's while it multiplies the current
// one; the last block of a factor fetches the first block of the next factor,
// so its latency overlaps the barrier.
#include <type_traits>

#include "ks_chain_fused.h"
#include "ks_chain_fused_io.h"
#include "ks_common.h"
#include "ks_internal.h"

namespace ks {

namespace {

// A run of four consecutive factor values in the storage type.
template <typename T> struct KRun { typedef u32x4 type; };
template <> struct KRun<bf16_t> { typedef u32x2 type; };
template <> struct KRun<_Float16> { typedef u32x2 type; };

// Element t (0..3) of a run, as fp32.
__device__ __forceinline__ float kelem(const u32x4& w, int t, float) { return __uint_as_float(w[t]); }
__device__ __forceinline__ float kelem(const u32x2& w, int t, bf16_t) {
  return __uint_as_float(((w[t >> 1] >> (16 * (t & 1))) & 0xffffu) << 16);
}
__device__ __forceinline__ float kelem(const u32x2& w, int t, _Float16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)((w[t >> 1] >> (16 * (t & 1))) & 0xffffu));
}

// This lane's runs of one block (kb = the block's packed b x b values):
// kr[kt][ct] = K[16kt + n][16ct + 4g .. 16ct + 4g + 3].  KVEC: one 16- or
// 8-byte load per run (the host checked that the values are aligned to 4
// elements); else element loads.
template <typename T, int BT, bool KVEC>
__device__ __forceinline__ void mfma_kload(typename KRun<T>::type (&kr)[BT][BT], const T* __restrict__ kb, int n,
                                           int g) {
  typedef typename KRun<T>::type KW;
  constexpr int B = 16 * BT;
#pragma unroll
  for (int kt = 0; kt < BT; ++kt)
#pragma unroll
    for (int ct = 0; ct < BT; ++ct) {
      const T* src = kb + (16 * kt + n) * B + 16 * ct + 4 * g;
      if constexpr (KVEC) {
        kr[kt][ct] = *reinterpret_cast<const KW*>(src);
      } else {
        T e[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) e[t] = src[t];
        __builtin_memcpy(&kr[kt][ct], e, sizeof(KW));
      }
    }
}

// One block, in place: addr is this lane's LDS float index of row
// in_row(l = 4g) at column n, step the LDS distance of consecutive l (d rows);
// H column halves of 16 (columns n and 16 + n) share every factor value.
template <typename T, int BT, int H>
__device__ __forceinline__ void mfma_block(const typename KRun<T>::type (&kr)[BT][BT], float* lds, int addr,
                                           int step) {
  f32x4 acc[H][BT];
#pragma unroll
  for (int h = 0; h < H; ++h)
#pragma unroll
    for (int kt = 0; kt < BT; ++kt) acc[h][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float xv[H][BT][4];
#pragma unroll
  for (int h = 0; h < H; ++h)
#pragma unroll
    for (int ct = 0; ct < BT; ++ct)
#pragma unroll
      for (int t = 0; t < 4; ++t) xv[h][ct][t] = lds[addr + 16 * h + (16 * ct + t) * step];
#pragma unroll
  for (int ct = 0; ct < BT; ++ct)
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int kt = 0; kt < BT; ++kt) {
        const float a = kelem(kr[kt][ct], t, T());
#pragma unroll
        for (int h = 0; h < H; ++h)
          acc[h][kt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, xv[h][ct][t], acc[h][kt], 0, 0, 0);
      }
  mfma_results_settle();
#pragma unroll
  for (int h = 0; h < H; ++h)
#pragma unroll
    for (int kt = 0; kt < BT; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) lds[addr + 16 * h + (16 * kt + r) * step] = acc[h][kt][r];
}

// Rows [ij*B, ij*B + B) of the tile for the blocks ij = w, w + W, ... < nb
// of a first factor with d = 1, loaded by wavefront w into LDS (pitch NC + 4)
// as pieces of EP elements (16 bytes when VEC), four blocks' loads in flight
// before any is written.  BSF: a piece is EP consecutive rows of one batch row
// (lanes: 16 batch rows x 4 pieces per load); BSL: EP consecutive columns of
// one row.  Columns beyond the batch are zero.
template <typename T, int LAYOUT, bool VEC, int B, int NC>
__device__ __forceinline__ void wave_load_blocks(const FusedChain& fc, float* lds, int col0, int w, int nb) {
  constexpr int W = kFusedThreads / 64, P = NC + 4, QMAX = 4;
  constexpr int EP = VEC ? 16 / (int)sizeof(T) : 1;
  constexpr int PPB = B * NC / EP;                 // pieces per block
  constexpr int PPL = (PPB + 63) / 64;             // per lane and block
  typedef typename std::conditional<VEC, u32x4, T>::type PW;
  const T* __restrict__ xp = static_cast<const T*>(fc.x);
  const int Bt = fc.batch, N = fc.width_in, lane = threadIdx.x & 63;
  // piece p of a block: (row offset, column) in the tile (fused_block_piece)
  auto piece = [&](int p, int* r, int* c) { fused_block_piece(LAYOUT, B, NC, EP, p, r, c); };
  for (int q0 = w; q0 < nb; q0 += QMAX * W) {
    PW pw[QMAX][PPL];
#pragma unroll
    for (int q = 0; q < QMAX; ++q) {
      const int ij = q0 + q * W;
#pragma unroll
      for (int i = 0; i < PPL; ++i) {
        const int p = i * 64 + lane;
        int r, c;
        piece(p, &r, &c);
        const bool ok = ij < nb && (PPB % 64 == 0 || p < PPB) && col0 + c < Bt;
        const int64_t off = LAYOUT == BSL ? (int64_t)(ij * B + r) * Bt + col0 + c
                                          : (int64_t)(col0 + c) * N + ij * B + r;
        if constexpr (VEC) pw[q][i] = ok ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(xp + off)) : u32x4{0, 0, 0, 0};
        else pw[q][i] = ok ? xp[off] : T(0);
      }
    }
#pragma unroll
    for (int q = 0; q < QMAX; ++q) {
      const int ij = q0 + q * W;
      if (ij >= nb) break;
#pragma unroll
      for (int i = 0; i < PPL; ++i) {
        const int p = i * 64 + lane;
        if (PPB % 64 && p >= PPB) continue;
        int r, c;
        piece(p, &r, &c);
        const int row = ij * B + r;
        if constexpr (VEC) {
          T e[EP];
          __builtin_memcpy(e, &pw[q][i], 16);
          if (LAYOUT == BSL) {
#pragma unroll
            for (int x = 0; x < EP; x += 4)
              *reinterpret_cast<f32x4*>(lds + row * P + c + x) = f32x4{to_f32(e[x]), to_f32(e[x + 1]), to_f32(e[x + 2]), to_f32(e[x + 3])};
          } else {
#pragma unroll
            for (int x = 0; x < EP; ++x) lds[(row + x) * P + c] = to_f32(e[x]);
          }
        } else {
          lds[row * P + c] = to_f32(pw[q][i]);
        }
      }
    }
  }
}

template <typename T, int LAYOUT, bool VEC, int BT, bool KVEC, int NC>
__global__ __launch_bounds__(kFusedThreads) void ks_chain_mfma_kernel(FusedChain fc) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  typedef typename KRun<T>::type KW;
  constexpr int W = kFusedThreads / 64, B = 16 * BT, H = NC / 16, P = NC + 4;
  const int col0 = fused_tile((int)blockIdx.x, (int)gridDim.x) * NC;
  const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, n = lane & 15, g = lane >> 4;
  // Values of block ij of factor f; an index past the factor's last block is
  // clamped to it (fetched, not used).  Every fetch is unconditional, so the
  // count of loads in flight is the same on every path and each wait covers
  // only the block about to be used.
  auto kblock = [&](int f, int ij) {
    const int nb = fused_mfma_blocks(fc, f);
    return static_cast<const T*>(fc.kv[f]) + (int64_t)(ij < nb ? ij : nb - 1) * (B * B);
  };
  // LDS float index of row in_row(4g) of block ij = i*d + j, column n.
  auto lane_addr = [&](int f, int ij) {
    const int d = fc.d[f];
    const int i = (int)div_fast((uint32_t)ij, fc.md[f], fc.sd[f]), j = ij - i * d;
    return (i * B * d + j + 4 * g * d) * P + n;
  };
  KW ka[BT][BT], kb[BT][BT];
  mfma_kload<T, BT, KVEC>(ka, kblock(fc.nf - 1, w), n, g);
  if (fc.d[fc.nf - 1] == 1) {
    // The first factor's blocks are runs of B consecutive rows (d = 1): each
    // wavefront loads exactly the rows of its own blocks (w, w + W, ...) and
    // starts on them without waiting for the others.
    wave_load_blocks<T, LAYOUT, VEC, B, NC>(fc, lds, col0, w, fused_mfma_blocks(fc, fc.nf - 1));
  } else {
    fused_load<T, LAYOUT, VEC, FusedPitchAddr, NC>(fc, lds, col0, FusedPitchAddr{P});
    __syncthreads();
  }
  for (int f = fc.nf - 1; f >= 0; --f) {
    const int nb = fused_mfma_blocks(fc, f), step = fc.d[f] * P;
    for (int ij = w; ij < nb; ij += 2 * W) {
      const int ij1 = ij + W;
      mfma_kload<T, BT, KVEC>(kb, kblock(f, ij1), n, g);
      mfma_block<T, BT, H>(ka, lds, lane_addr(f, ij), step);
      // the wavefront's next block: ij + 2W of this factor, else its first
      // block of the next factor
      const bool here = ij + 2 * W < nb || f == 0;
      mfma_kload<T, BT, KVEC>(ka, here ? kblock(f, ij + 2 * W) : kblock(f - 1, w), n, g);
      if (ij1 < nb) mfma_block<T, BT, H>(kb, lds, lane_addr(f, ij1), step);
    }
    if (w >= nb && f > 0) mfma_kload<T, BT, KVEC>(ka, kblock(f - 1, w), n, g);
    __syncthreads();
  }
  fused_store<T, LAYOUT, VEC, FusedPitchAddr, NC>(fc, lds, col0, FusedPitchAddr{P});
}

template <typename T, int BT, int NC>
hipError_t launch_mfma_nc(const FusedChain& fc, bool vec, hipStream_t s) {
  const dim3 grid((fc.batch + NC - 1) / NC), block(kFusedThreads);
  const int lds = fused_lds_bytes(fc);
#define KS_MFMA_LAUNCH(L, V, KV)                                                                              \
  {                                                                                                          \
    if (lds > 64 * 1024) {                                                                                   \
      static const hipError_t raised = hipFuncSetAttribute(                                                  \
          reinterpret_cast<const void*>(&ks_chain_mfma_kernel<T, L, V, BT, KV, NC>),                         \
          hipFuncAttributeMaxDynamicSharedMemorySize, kFusedMaxLds);                                         \
      if (raised != hipSuccess) return raised;                                                               \
    }                                                                                                        \
    hipLaunchKernelGGL((ks_chain_mfma_kernel<T, L, V, BT, KV, NC>), grid, block, lds, s, fc);                \
    return hipGetLastError();                                                                                \
  }
#define KS_MFMA_LAUNCH_KV(L, V)                                                                               \
  {                                                                                                          \
    if (fc.kvec) KS_MFMA_LAUNCH(L, V, true) else KS_MFMA_LAUNCH(L, V, false)                                 \
  }
  if (fc.layout == BSL) {
    if (vec) KS_MFMA_LAUNCH_KV(BSL, true) else KS_MFMA_LAUNCH_KV(BSL, false)
  }
  if (vec) KS_MFMA_LAUNCH_KV(BSF, true) else KS_MFMA_LAUNCH_KV(BSF, false)
#undef KS_MFMA_LAUNCH_KV
#undef KS_MFMA_LAUNCH
}

// Tiles of 32 columns for blocks of 16 and 32 (ks_host.cpp picks them only there).
template <typename T, int BT>
hipError_t launch_mfma_bt(const FusedChain& fc, bool vec, hipStream_t s) {
  if constexpr (BT <= 2)
    if (fc.cols == 2 * kFusedCols) return launch_mfma_nc<T, BT, 2 * kFusedCols>(fc, vec, s);
  if (fc.cols != kFusedCols) return hipErrorInvalidValue;
  return launch_mfma_nc<T, BT, kFusedCols>(fc, vec, s);
}

template <typename T>
hipError_t launch_mfma_t(const FusedChain& fc, bool vec, hipStream_t s) {
  switch (fused_mfma_bt(fc)) {
    case 1: return launch_mfma_bt<T, 1>(fc, vec, s);
    case 2: return launch_mfma_bt<T, 2>(fc, vec, s);
    case 3: return launch_mfma_bt<T, 3>(fc, vec, s);
    case 4: return launch_mfma_bt<T, 4>(fc, vec, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_chain_mfma(const FusedChain& fc, int dtype, bool vec, hipStream_t s) {
  switch (dtype) {
    case F32: return launch_mfma_t<float>(fc, vec, s);
    case BF16: return launch_mfma_t<bf16_t>(fc, vec, s);
    case F16: return launch_mfma_t<_Float16>(fc, vec, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ks
