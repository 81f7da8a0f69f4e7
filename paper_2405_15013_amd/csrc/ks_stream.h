// Streaming MFMA kernels: the register-direct products (ks_direct.h) with
// every wavefront of one resident round walking an equal share of all batch
// tiles (ks_stream_index.h) as one pipeline of steps (tile, chunk of 16 values
// of l).  The loads of the next PD steps (X from HBM, K from L1/L2) are in
// flight while a step is multiplied, across tile boundaries, so loads, MFMAs
// and stores of different steps overlap inside every wavefront instead of the
// whole chip alternating between load and compute phases.  Outputs of a tile
// are stored when its last chunk is done.
//
// Every storage type takes 16 values of l per chunk (LP = 4 per lane group):
// fp32 with four v_mfma_f32_16x16x4_f32 steps, 16-bit types with one
// v_mfma_f32_16x16x16_{bf16,f16}, so any c that is a multiple of 16 is one
// uniform run of steps.  (The 16-bit path needs a small fraction of the
// 16x16x16 rate to keep up with HBM.)
#pragma once
#include "ks_direct.h"
#include "ks_stream_index.h"

namespace ks {

// VGPRs the steps in flight may take.
constexpr int kStreamRingBudget = 96;

template <typename T, int LAYOUT, int V, bool STRIDED, int MT>
__global__ __launch_bounds__(256) void ks_stream_kernel(Problem p, StreamTile t) {
  constexpr int S = sizeof(T);
  constexpr int LP = 4, CH = 16;
  using Chunk = DChunk<T, LAYOUT, V, STRIDED, MT, LP>;
  constexpr int R = Chunk::NXW + MT * Chunk::VK * Chunk::KW;  // VGPRs of one step
  constexpr int RB0 = kStreamRingBudget / R;
  constexpr int RB = RB0 < 2 ? 2 : (RB0 > 8 ? 8 : RB0);  // ring of steps in flight
  constexpr int PD = RB - 1;                             // steps loaded ahead
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * t.waves + (threadIdx.x >> 6);
  if (w >= t.nwaves) return;  // wave-uniform
  const int n = lane & 15, g = lane >> 4;
  int first, ntiles;
  stream_share(t, w, &first, &ntiles);
  const T* __restrict__ x = static_cast<const T*>(p.x);
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const int c = p.c;
  const int nch = c / CH;
  const int steps = ntiles * nch;
  const int64_t lstride = direct_x_lstride(p);
  const int64_t qstride = direct_x_qstride(p, STRIDED, LP, V, S);
  const int64_t kmstride = (int64_t)16 * c, kestride = (int64_t)p.b * c;
  const bool ntx = t.kgroups == 1;

  auto load_step = [&](Chunk& ch, int s) {
    const int q = s / nch, l0 = (s - q * nch) * CH;
    const DItem it = stream_item(p, t, V, MT, first + q);
    ch.load(x + direct_x_base(p, it, LP, V, n, g), lstride, qstride, kv + direct_k_base(p, it, LP, n, g), kmstride,
            kestride, l0, ntx);
  };

  f32x4 acc[MT][V];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[mt][e] = f32x4{0.f, 0.f, 0.f, 0.f};

  Chunk ring[RB];
#pragma unroll
  for (int u = 0; u < PD; ++u)
    if (u < steps) load_step(ring[u], u);
  // sched_barrier(0): keep the compiler's scheduler from sinking the loads
  // next to their first use.
  __builtin_amdgcn_sched_barrier(0);
  for (int s0 = 0; s0 < steps; s0 += RB) {
#pragma unroll
    for (int u = 0; u < RB; ++u) {
      const int s = s0 + u;
      if (s >= steps) break;
      if (s + PD < steps) load_step(ring[(u + PD) % RB], s + PD);
      __builtin_amdgcn_sched_barrier(0);
      ring[u].mma(acc);
      const int q = s / nch;
      if (s - q * nch == nch - 1) {  // last chunk of tile q
        direct_store<T, LAYOUT, V, STRIDED, MT>(p, stream_item(p, t, V, MT, first + q), n, g, acc);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int e = 0; e < V; ++e) acc[mt][e] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
}

// Wavefronts of one resident round of this instance on the current device:
// compute units x resident workgroups of 256 threads per compute unit x 4
// (queried once per instance and device ordinal).
template <typename T, int LAYOUT, int V, bool STRIDED, int MT>
hipError_t stream_round_waves(int* out) {
  static int cached[16] = {0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const int slot = dev & 15;
  if (cached[slot] == 0) {
    int cus = 0, blocks = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &blocks, reinterpret_cast<const void*>(&ks_stream_kernel<T, LAYOUT, V, STRIDED, MT>), 256, 0);
    if (e != hipSuccess) return e;
    cached[slot] = (cus > 0 ? cus : 1) * (blocks > 0 ? blocks : 1) * 4;
  }
  *out = cached[slot];
  return hipSuccess;
}

template <typename T, int LAYOUT, int V, bool STRIDED, int MT>
hipError_t launch_stream_inst(const Problem& p, const StreamTile& t0, unsigned, hipStream_t s) {
  StreamTile t = t0;
  int round = 0;
  hipError_t e = stream_round_waves<T, LAYOUT, V, STRIDED, MT>(&round);
  if (e != hipSuccess) return e;
  t.waves = 4;
  t.nwaves = t.tiles < round ? t.tiles : round;
  const unsigned grid = (unsigned)((t.nwaves + 3) / 4);
  hipLaunchKernelGGL((ks_stream_kernel<T, LAYOUT, V, STRIDED, MT>), dim3(grid), dim3(256), 0, s, p, t);
  return hipGetLastError();
}

template <typename T, int LAYOUT, int V, bool STRIDED>
hipError_t launch_stream_mt(const Problem& p, const StreamTile& t, int mt, unsigned grid, hipStream_t s) {
  constexpr int MX = direct_mt_max(sizeof(T), LAYOUT, V);
  switch (mt) {
    case 1: return launch_stream_inst<T, LAYOUT, V, STRIDED, 1>(p, t, grid, s);
    case 2: if constexpr (MX >= 2) return launch_stream_inst<T, LAYOUT, V, STRIDED, 2>(p, t, grid, s); break;
    case 3: if constexpr (MX >= 3) return launch_stream_inst<T, LAYOUT, V, STRIDED, 3>(p, t, grid, s); break;
    case 4: if constexpr (MX >= 4) return launch_stream_inst<T, LAYOUT, V, STRIDED, 4>(p, t, grid, s); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

// Instances of one storage type and layout.
template <typename T, int LAYOUT>
hipError_t launch_stream_layout(const Problem& p, const StreamTile& t, int V, bool strided, int mt, unsigned grid,
                                hipStream_t s) {
  if constexpr (LAYOUT == BSL) {
    if (V != kDirectVec || strided) return hipErrorInvalidValue;
    return launch_stream_mt<T, BSL, kDirectVec, false>(p, t, mt, grid, s);
  } else {
    if (strided) {
      if (V != kDirectVec) return hipErrorInvalidValue;
      return launch_stream_mt<T, BSF, kDirectVec, true>(p, t, mt, grid, s);
    }
    switch (V) {
      case 1: return launch_stream_mt<T, BSF, 1, false>(p, t, mt, grid, s);
      case 2: return launch_stream_mt<T, BSF, 2, false>(p, t, mt, grid, s);
      case 4: return launch_stream_mt<T, BSF, 4, false>(p, t, mt, grid, s);
      default: break;
    }
    return hipErrorInvalidValue;
  }
}

}  // namespace ks
