// LDS-DMA MFMA kernel for batch-size-last KS patterns.
//
// The products of the register-direct kernel (paper Section 4.1, Algorithm 2:
// output-stationary work items, the lane operand layout of ks_direct_index.h)
// with X moved HBM -> LDS by the memory unit (global_load_lds_dwordx4) in
// three stage buffers, as in the batch-size-first DMA kernel (ks_dma.h): the
// X bytes of two stages are in flight while a stage is multiplied and they
// occupy no registers, where the register-direct kernel can keep only one
// chunk ahead within its register budget.  In this layout the rows of X are
// contiguous along the batch (Section 4.2's favourable case), so a stage is
// CH whole rows of the tile's batch range: the four wavefronts of a tile
// (RS batch groups x KGW k-groups) load it together, each reads the 16-byte
// units of its own columns as MFMA B operands, and X is read from HBM once
// per tile for all of its k-groups.  K operands are loaded into registers one
// stage ahead; outputs go from the accumulators straight to Y (16-byte rows
// of V batch entries, the register-direct store).
//
// Synchronisation per stage s is that of ks_dma.h: wait until only the DMAs
// of stage s+1 are outstanding, a bare s_barrier, K loads of stage s+1 and
// DMAs of stage s+2 in that pinned order, then LDS operand reads (inline
// ds_read with their own wait) and the MFMAs.
#pragma once
#include "ks_dma.h"

namespace ks {

// K operands of one stage for the batch-size-last layout: one block (i, j),
// MT M-tiles of LP values of l (DmaK with a single j).
template <typename T, int MT, int LP>
using DmaKBsl = DmaK<T, 1, MT, LP>;

// Waves per SIMD the register allocation is fitted to: with the hint the
// accumulators stay in VGPRs (no AGPR copies), which measured 2-5 % faster
// than the default allocation; fp32 with four M-tiles keeps two waves (three
// would spill).
template <typename T, int MT>
constexpr int dma_bsl_waves() {
  return sizeof(T) == 4 ? (MT <= 2 ? 4 : (MT == 3 ? 3 : 2)) : 2;
}

// T: storage type; MT: M-tiles (16 output rows) per wavefront; RS: batch
// groups per tile (KGW = 4 / RS k-groups); EPI: bias / GELU epilogue compiled in.
template <typename T, int MT, int RS, bool EPI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(dma_bsl_waves<T, MT>())))
void ks_dma_bsl_kernel(Problem p, StagedTile t) {
  constexpr int S = sizeof(T);
  constexpr int V = 16 / S;              // batch entries per lane column (one 16-byte unit)
  constexpr int LP = S == 4 ? 4 : 8;     // values of l per lane group (16x16x4 f32, 16x16x32 16-bit)
  constexpr int CH = 4 * LP;             // values of l per stage
  constexpr int W = 4;
  constexpr int UR = 16 * RS;            // 16-byte units per stage row
  constexpr int UD = CH * UR / (64 * W); // DMA instructions per wavefront per stage
  constexpr int STAGE = CH * UR * 16;    // bytes of one stage buffer
  static_assert(UD >= 1 && UD * 64 * W == CH * UR, "a stage is whole DMA instructions per wavefront");
  using Piece = LdsVec<16>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, g = lane >> 4;
  const STile st = dma_bsl_tile(p, t, blockIdx.x);
  const SItem si = dma_bsl_item(t, st, V, MT, w);
  DItem it;
  it.i = st.i;
  it.j0 = si.j0;
  it.k0 = si.k0;
  it.beta0 = si.beta0;
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const int nst = p.c / CH;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;

  // DMA sources: instruction m of this wavefront fills physical units
  // (m*W + w)*64 + lane of the stage buffer.
  const T* __restrict__ xi = static_cast<const T*>(p.x) + (int64_t)st.i * p.c * p.d * p.batch;
  int soff[UD];
#pragma unroll
  for (int m = 0; m < UD; ++m) {
    int r, v;
    dma_bsl_unit_of(t, dma_phys_unit(t, m, w, lane), &r, &v);
    soff[m] = dma_bsl_src(p, t, st, V, r, v);
  }
  const int64_t xstage = (int64_t)CH * p.d * p.batch;  // X elements between the first rows of two stages
  // The DMAs stream X with the nontemporal hint (cache policy bit 1): the
  // tile reads its X once for all its k-groups, and keeping X out of the
  // caches' retention leaves them to K (measured: fp32 batch-size-last 1-3 %
  // faster; the batch-size-first kernel, whose k-group tiles re-read X from
  // L2, got 1-2 % slower with it and keeps the default).
  auto dma = [&](const T* xs, int buf) {
    char* dst = smem + buf * STAGE + w * 1024;
#pragma unroll
    for (int m = 0; m < UD; ++m)
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(xs + soff[m]),
                                       (lds_void_t*)(dst + m * W * 1024), 16, 0, 2);
  };

  // Operand pieces: one 16-byte unit (V batch entries) of stage row LP*g + q.
  uint32_t ooff[LP];
#pragma unroll
  for (int q = 0; q < LP; ++q) ooff[q] = lds0 + dma_bsl_op_byte(t, si, LP, n, g, q);

  const int64_t kmstride = (int64_t)16 * p.c;
  const T* kl = kv + direct_k_base(p, it, LP, n, g);

  f32x4 acc[MT][V];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[mt][e] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One stage (MODE 2: K of stage s+1 and DMA of stage s+2; MODE 1: K of
  // stage s+1 only; MODE 0: nothing), straight-line per mode so that the
  // compiler's waits before the MFMAs see fixed counts.
  int cur = 0;
  const T* xnext = xi + 2 * xstage;
  auto step = [&](auto mode, int s, DmaKBsl<T, MT, LP>& kc, DmaKBsl<T, MT, LP>& kn) {
    constexpr int MODE = decltype(mode)::value;
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (MODE == 0) wait_vmcnt<0>();
    else wait_vmcnt<UD>();
    dma_barrier();
    if constexpr (MODE >= 1) kn.load(kl, kmstride, 0, (s + 1) * CH);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (MODE == 2) {
      dma(xnext, cur == 0 ? 2 : cur - 1);
      xnext += xstage;
    }
    __builtin_amdgcn_sched_barrier(0);
    const uint32_t base = (uint32_t)(cur * STAGE);
    cur = cur == 2 ? 0 : cur + 1;
    typename Piece::type pc[LP];
#pragma unroll
    for (int q = 0; q < LP; ++q) pc[q] = Piece::read(ooff[q] + base);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    uint32_t xw[LP * 4];
#pragma unroll
    for (int q = 0; q < LP; ++q) {
      asm volatile("" : "+v"(pc[q]));  // ordered after the wait above
#pragma unroll
      for (int w2 = 0; w2 < 4; ++w2) xw[q * 4 + w2] = pc[q][w2];
    }
    direct_mma<T, BSL, V, MT, LP>(xw, kc.kw, acc);
  };
  using M0 = std::integral_constant<int, 0>;
  using M1 = std::integral_constant<int, 1>;
  using M2 = std::integral_constant<int, 2>;

  DmaKBsl<T, MT, LP> ka, kb;
  ka.load(kl, kmstride, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
  dma(xi, 0);
  if (nst > 1) dma(xi + xstage, 1);
  __builtin_amdgcn_sched_barrier(0);
  int s = 0;
  for (; s + 3 < nst; s += 2) {
    step(M2(), s, ka, kb);
    step(M2(), s + 1, kb, ka);
  }
  const int left = nst - s;
  if (left == 3) {
    step(M2(), s, ka, kb);
    step(M1(), s + 1, kb, ka);
    step(M0(), s + 2, ka, kb);
  } else if (left == 2) {
    step(M1(), s, ka, kb);
    step(M0(), s + 1, kb, ka);
  } else {
    step(M0(), s, ka, kb);
  }
  // Accumulators -> Y rows (settles the MFMA results, skips columns beyond
  // the batch, applies the epilogue when compiled in).
  direct_store<T, BSL, V, false, MT, EPI>(p, it, n, g, acc);
}

template <typename T, int MT, int RS, bool EPI>
hipError_t launch_dma_bsl_inst(const Problem& p, const StagedTile& t, hipStream_t s) {
  if (t.lds > 64 * 1024) {
    static const hipError_t raised = hipFuncSetAttribute(reinterpret_cast<const void*>(&ks_dma_bsl_kernel<T, MT, RS, EPI>),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, kDmaMaxLds);
    if (raised != hipSuccess) return raised;
  }
  hipLaunchKernelGGL((ks_dma_bsl_kernel<T, MT, RS, EPI>), dim3(t.tiles), dim3(256), t.lds, s, p, t);
  return hipGetLastError();
}

// Instances: MT 1..4 for fp32, 1..2 for 16-bit types (eight accumulator
// chains per M-tile there); RS 1, 2, 4.
template <typename T, bool EPI>
hipError_t launch_dma_bsl_rs(const Problem& p, const StagedTile& t, int mt, hipStream_t s) {
  constexpr int MTMAX = sizeof(T) == 4 ? 4 : 2;
  if (t.W != 4 || mt < 1 || mt > MTMAX) return hipErrorInvalidValue;
#define KS_DMA_BSL_RS(M)                                                   \
  switch (t.RS) {                                                          \
    case 1: return launch_dma_bsl_inst<T, M, 1, EPI>(p, t, s);             \
    case 2: return launch_dma_bsl_inst<T, M, 2, EPI>(p, t, s);             \
    case 4: return launch_dma_bsl_inst<T, M, 4, EPI>(p, t, s);             \
    default: return hipErrorInvalidValue;                                  \
  }
  if (mt == 1) { KS_DMA_BSL_RS(1) }
  if (mt == 2) { KS_DMA_BSL_RS(2) }
  if constexpr (MTMAX == 4) {
    if (mt == 3) { KS_DMA_BSL_RS(3) }
    if (mt == 4) { KS_DMA_BSL_RS(4) }
  }
#undef KS_DMA_BSL_RS
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_dma_bsl_t(const Problem& p, const StagedTile& t, int mt, hipStream_t s) {
  return has_epilogue(p) ? launch_dma_bsl_rs<T, true>(p, t, mt, s) : launch_dma_bsl_rs<T, false>(p, t, mt, s);
}

}  // namespace ks
