// LDS-DMA MFMA kernels for batch-size-first KS patterns.
//
// Same output-stationary tiles and products as the LDS-staged kernels (paper
// Section 4.1, Algorithm 2; tile and item mapping in ks_staged_index.h), with
// the X stages moved from HBM to LDS by the memory unit itself
// (global_load_lds_dwordx4: every lane's 16 bytes land at M0 + 16 * lane), so
// the bytes in flight occupy no registers.  Three stage buffers per
// workgroup: while stage s is multiplied, stages s+1 and s+2 are in flight.
// The paper's weak batch-size-first case (Section 4.2) again becomes
// contiguous row runs: each stage row is X[beta, i*c*d + ls*d .. (ls+LCH)*d).
//
// Synchronisation, per stage s:
//   1. wait until at most UD vector-memory operations are outstanding (the
//      DMAs of stage s+1), so this wavefront's DMAs of stage s and its K loads
//      of stage s have completed;
//   2. s_barrier: every wavefront's DMAs of stage s are in LDS, and every
//      wavefront has finished reading stage s-1, whose buffer is refilled next;
//   3. load K of stage s+1 (registers), then DMA stage s+2;
//   4. read the operands of stage s from LDS and run the MFMAs.
// The vector-memory issue order of step 3 (K loads, then DMAs) is pinned with
// scheduling barriers, which is what makes the count of step 1 exact.  The
// operand reads are issued as inline assembly with their own wait: the
// compiler cannot tell which LDS bytes a DMA writes and would otherwise wait
// for every DMA in flight before using any LDS value.
//
// Outputs leave through the structured epilogue of the staged kernel (LDS
// copy of the output tile, coalesced 16-byte stores; Appendix D.3).
#pragma once
#include <type_traits>

#include "ks_direct.h"
#include "ks_staged_index.h"

namespace ks {

typedef __attribute__((address_space(3))) void lds_void_t;
constexpr int kDmaMaxLds = 128 * 1024;

// vmcnt(N) on gfx9: vmcnt in bits 3:0 and 15:14, expcnt (bits 6:4) and
// lgkmcnt (bits 11:8) left at their maxima (no wait).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// The problem's and the tile description's fields in scalar registers at
// kernel entry, in one statement so that they arrive in one round of
// kernel-argument loads (as kernarg_fetch(Problem) in ks_direct.h).
__device__ __forceinline__ void kernarg_fetch(const Problem& p, const StagedTile& t) {
  asm volatile("" ::KS_PROBLEM_FIELDS(p), "s"(t.tiles), "s"(t.remap), "s"(t.kgt), "s"(t.nbt), "s"(t.mkgt),
               "s"(t.skgt), "s"(t.mnbt), "s"(t.snbt), "s"(t.RS), "s"(t.lRS), "s"(t.JG), "s"(t.lJG), "s"(t.KGW),
               "s"(t.UR), "s"(t.lUR), "s"(t.stage));
}

// Workgroup barrier without a memory fence (a fence would wait for every DMA
// in flight); the empty asm statements keep the compiler from moving memory
// accesses across it, the scheduling barriers keep the scheduler from doing so.
__device__ __forceinline__ void dma_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// One LDS read of NB bytes at LDS byte address addr, outside the compiler's
// tracking (the caller waits with lds_wait before using the value).
template <int NB> struct LdsVec;
template <> struct LdsVec<16> {
  typedef u32x4 type;
  __device__ static __forceinline__ type read(uint32_t addr) {
    type v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
    return v;
  }
};
template <> struct LdsVec<8> {
  typedef u32x2 type;
  __device__ static __forceinline__ type read(uint32_t addr) {
    type v;
    asm volatile("ds_read_b64 %0, %1" : "=v"(v) : "v"(addr));
    return v;
  }
};

// The K operands of one chunk (one stage): MT x V blocks of LP values of l.
template <typename T, int V, int MT, int LP>
struct DmaK {
  static constexpr int KW = LP * (int)sizeof(T) / 4;
  uint32_t kw[MT][V][KW];
  __device__ __forceinline__ void load(const T* __restrict__ kl, int64_t kmstride, int64_t kestride, int l) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int e = 0; e < V; ++e) load_piece<KW * 4, false>(kl + mt * kmstride + e * kestride + l, kw[mt][e]);
  }
};

// V j values per lane (V = min(d, 4)): STRIDED when d > V (pieces of V
// elements at stride d), otherwise the lane's LP x V block is contiguous.
// Register budget per instance: the smallest tiles (MT = NT = 1) are fitted
// to four waves per SIMD (four workgroups per CU), NT = 2 to three, the rest
// to two (the accumulators then live in VGPRs instead of AGPRs).
template <typename T, int V, bool STRIDED, int MT, int LP, int UD, int NT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(MT * NT == 1 ? 4 : ((MT == 1 && NT == 2) ? 3 : 2))))
void ks_dma_kernel(Problem p, StagedTile t) {
  constexpr int S = sizeof(T);
  constexpr int CH = 4 * LP;  // values of l per stage
  constexpr int PE = STRIDED ? V : (LP * V * S < 16 ? LP * V : 16 / S);
  constexpr int NP = LP * V / PE;
  constexpr int PB = PE * S;
  using Piece = LdsVec<PB>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, g = lane >> 4;
  kernarg_fetch(p, t);
  const STile st = dma_tile(t, blockIdx.x);
  const SItem si = dma_item(t, st, V, MT, w);
  DItem it;
  it.i = st.i;
  it.j0 = si.j0;
  it.k0 = si.k0;
  it.beta0 = si.beta0;
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const int nst = p.c / CH;
  const int stage = t.stage;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;

  // DMA sources: instruction m of this wavefront fills physical units
  // (m*W + w)*64 + lane; the lane loads the logical unit stored there (rows
  // beyond the batch read the last row instead).
  const T* __restrict__ xi = static_cast<const T*>(p.x) + (int64_t)st.i * p.c * p.d;
  int soff[UD];
#pragma unroll
  for (int m = 0; m < UD; ++m) {
    int r, v;
    dma_unit_of_fast(t, dma_phys_unit(t, m, w, lane), &r, &v);
    int beta = st.bt * 16 * t.RS * NT + r;
    if (beta >= p.batch) beta = p.batch - 1;
    soff[m] = beta * p.N + v * (16 / S);
  }
  const int xstage = CH * p.d;  // X elements per stage along a row
  // DMA of the stage whose row runs start at xs, into stage buffer buf.
  auto dma = [&](const T* xs, int buf) {
    char* dst = smem + buf * stage + w * 1024;
#pragma unroll
    for (int m = 0; m < UD; ++m)
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(xs + soff[m]),
                                       (lds_void_t*)(dst + m * t.W * 1024), 16, 0, 0);
  };

  // Operand pieces of this lane: LDS byte offsets within a stage buffer (row
  // group 0 of the wavefront; group u is 16*u rows further, and the swizzle
  // depends on the row modulo 16 only).
  uint32_t ooff[NP];
  const uint32_t ugroup = 16 * t.UR * 16;  // bytes of 16 stage rows
  {
    const int r = 16 * NT * si.rs + n;
#pragma unroll
    for (int q = 0; q < NP; ++q)
      ooff[q] = lds0 + dma_lds_byte(t, r, dma_op_byte(p, si, LP, V, STRIDED, PE, S, 0, g, q));
  }

  const int64_t kmstride = (int64_t)16 * p.c, kestride = (int64_t)p.b * p.c;
  const T* kl = kv + direct_k_base(p, it, LP, n, g);

  f32x4 acc[NT][MT][V];
#pragma unroll
  for (int u = 0; u < NT; ++u)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int e = 0; e < V; ++e) acc[u][mt][e] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One stage.  MODE 2: K of stage s+1 and DMA of stage s+2 (steady state);
  // MODE 1: K of stage s+1 only (stage nst-2); MODE 0: nothing (last stage).
  // The modes are separate straight-line code so that the compiler's own
  // wait before the MFMAs sees a fixed number of operations after each K load.
  // Stage s uses buffer cur = s % 3 (kept incrementally), the DMAs of stage
  // s+2 go to buffer (s+2) % 3 from the row runs at xnext.
  int cur = 0;
  const T* xnext = xi + 2 * xstage;
  auto step = [&](auto mode, int s, DmaK<T, V, MT, LP>& kc, DmaK<T, V, MT, LP>& kn) {
    constexpr int MODE = decltype(mode)::value;
    // 1-2: stage s (and its K) complete in every wavefront; stage s-1 read.
    // (The scheduling barrier keeps the wait from being hoisted into the
    // previous stage's MFMAs.)
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (MODE == 0) wait_vmcnt<0>();
    else wait_vmcnt<UD>();
    dma_barrier();
    // 3: K of stage s+1, then the DMAs of stage s+2 (this order is what the
    // count of step 1 relies on).
    if constexpr (MODE >= 1) kn.load(kl, kmstride, kestride, (s + 1) * CH);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (MODE == 2) {
      dma(xnext, cur == 0 ? 2 : cur - 1);
      xnext += xstage;
    }
    __builtin_amdgcn_sched_barrier(0);
    // 4: per row group, operands from LDS, then the MFMAs (the K operands
    // serve all NT groups).
    const uint32_t base = (uint32_t)(cur * stage);
    cur = cur == 2 ? 0 : cur + 1;
#pragma unroll
    for (int u = 0; u < NT; ++u) {
      typename Piece::type pc[NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) pc[q] = Piece::read(ooff[q] + base + u * ugroup);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      uint32_t xw[LP * V * S / 4];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        asm volatile("" : "+v"(pc[q]));  // ordered after the wait above
#pragma unroll
        for (int w2 = 0; w2 < PB / 4; ++w2) xw[q * (PB / 4) + w2] = pc[q][w2];
      }
      direct_mma<T, BSF, V, MT, LP>(xw, kc.kw, acc[u]);
    }
  };
  using M0 = std::integral_constant<int, 0>;
  using M1 = std::integral_constant<int, 1>;
  using M2 = std::integral_constant<int, 2>;

  DmaK<T, V, MT, LP> ka, kb;
  ka.load(kl, kmstride, kestride, 0);
  __builtin_amdgcn_sched_barrier(0);
  dma(xi, 0);
  if (nst > 1) dma(xi + xstage, 1);
  __builtin_amdgcn_sched_barrier(0);
  int s = 0;
  for (; s + 3 < nst; s += 2) {  // both steps are steady-state steps
    step(M2(), s, ka, kb);
    step(M2(), s + 1, kb, ka);
  }
  // The last 1-3 stages (s even, so ka holds K of stage s).
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

  // Structured epilogue: accumulators -> LDS output tile -> contiguous runs.
  // Bias of output feature (mt, e, r4) = row k0 + 16 mt + 4 g + r4 of block
  // (i, j0 + e), shared by the NT row groups; loads issued before the wait
  // for the last MFMA results.
  const bool has_bias = p.bias != nullptr;
  float bv[MT][V][4];
  if (has_bias) {
    const T* bb = static_cast<const T*>(p.bias) + (int64_t)(st.i * p.b + it.k0 + 4 * g) * p.d + it.j0;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
#pragma unroll
        for (int e = 0; e < V; ++e) bv[mt][e][r4] = to_f32(bb[(16 * mt + r4) * p.d + e]);
  }
  mfma_results_settle();
  if (has_bias) {
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int e = 0; e < V; ++e)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) acc[u][mt][e][r4] += bv[mt][e][r4];
  }
  if (epilogue_gelu(p)) {
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int e = 0; e < V; ++e)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) acc[u][mt][e][r4] = gelu_f32<T>(acc[u][mt][e][r4]);
  }
  __syncthreads();  // every wavefront is done with the stage buffers
  char* ycell0 = smem + dma_y_lds_lane(p, t, si, MT, S, n, g);
#pragma unroll
  for (int u = 0; u < NT; ++u)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        // V consecutive j of output row k = k0 + 16*mt + 4*g + r4
        char* cell = ycell0 + u * 16 * t.ypitch + (16 * mt + r4) * p.d * S;
        if constexpr (V == 4) {
          if constexpr (S == 4) {
            *reinterpret_cast<f32x4*>(cell) =
                f32x4{acc[u][mt][0][r4], acc[u][mt][1][r4], acc[u][mt][2][r4], acc[u][mt][3][r4]};
          } else {
            uint32_t wv[2];
#pragma unroll
            for (int e = 0; e < V; e += 2) {
              wv[e / 2] = pack2_f32<T>(acc[u][mt][e][r4], acc[u][mt][e + 1][r4]);
            }
            *reinterpret_cast<u32x2*>(cell) = u32x2{wv[0], wv[1]};
          }
        } else {
#pragma unroll
          for (int e = 0; e < V; ++e) reinterpret_cast<T*>(cell)[e] = from_f32<T>(acc[u][mt][e][r4]);
        }
      }
  __syncthreads();
  // 16-byte units of the output tile (uy = 2^lUY per row): rows beyond the
  // batch are not stored.
  const int nunits = (16 * t.RS * NT) << t.lUY;
  const int rows_valid = p.batch - st.bt * 16 * t.RS * NT;
  T* __restrict__ ytile = static_cast<T*>(p.y) + dma_y_tile_base(p, t, st, MT);
  for (int u = tid; u < nunits; u += 64 * t.W) {
    const int row = u >> t.lUY, v = u & ((1 << t.lUY) - 1);
    if (row >= rows_valid) continue;
    const u32x4 val = *reinterpret_cast<const u32x4*>(smem + row * t.ypitch + v * 16);
    __builtin_nontemporal_store(val, reinterpret_cast<u32x4*>(ytile + dma_y_row(p, row, v, S)));
  }
}

template <typename T, int V, bool STRIDED, int MT, int LP, int UD, int NT>
hipError_t launch_dma_inst(const Problem& p, const StagedTile& t, hipStream_t s) {
  if (t.lds > 64 * 1024) {
    // Opt in to more than 64 KB of dynamic LDS once per instance (a function-
    // local static: initialised exactly once even with concurrent callers).
    static const hipError_t raised = hipFuncSetAttribute(reinterpret_cast<const void*>(&ks_dma_kernel<T, V, STRIDED, MT, LP, UD, NT>),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, kDmaMaxLds);
    if (raised != hipSuccess) return raised;
  }
  hipLaunchKernelGGL((ks_dma_kernel<T, V, STRIDED, MT, LP, UD, NT>), dim3(t.tiles), dim3(256), t.lds, s, p, t);
  return hipGetLastError();
}

// (MT, NT) pairs instantiated: MT * NT <= 4.
template <typename T, int V, bool STRIDED, int LP, int UD>
hipError_t launch_dma_mt(const Problem& p, const StagedTile& t, int mt, hipStream_t s) {
  const int nt = t.NT;
  if (mt == 1 && nt == 1) return launch_dma_inst<T, V, STRIDED, 1, LP, UD, 1>(p, t, s);
  if (mt == 2 && nt == 1) return launch_dma_inst<T, V, STRIDED, 2, LP, UD, 1>(p, t, s);
  if (mt == 1 && nt == 2) return launch_dma_inst<T, V, STRIDED, 1, LP, UD, 2>(p, t, s);
  if (mt == 2 && nt == 2) return launch_dma_inst<T, V, STRIDED, 2, LP, UD, 2>(p, t, s);
  if (mt == 1 && nt == 4) return launch_dma_inst<T, V, STRIDED, 1, LP, UD, 4>(p, t, s);
  return hipErrorInvalidValue;
}

// Instances of one storage type and j-vector mode (V, STRIDED): (MT, NT) with
// MT * NT <= 4, LP (4 for fp32; 8, or 4, for 16-bit types), 2, 4 or 8 DMA
// instructions per wavefront per stage.  One source file per storage type
// and mode, so the instances compile in parallel.
template <typename T, int V, bool STRIDED>
hipError_t launch_dma_mode(const Problem& p, const StagedTile& t, int mt, int lp, hipStream_t s) {
  if (t.W != 4) return hipErrorInvalidValue;
  if constexpr (sizeof(T) == 4) {
    if (lp != 4) return hipErrorInvalidValue;
  }
#define KS_DMA_UD(LPV)                                                              \
  switch (t.UD) {                                                                   \
    case 2: return launch_dma_mt<T, V, STRIDED, LPV, 2>(p, t, mt, s);               \
    case 4: return launch_dma_mt<T, V, STRIDED, LPV, 4>(p, t, mt, s);               \
    case 8: return launch_dma_mt<T, V, STRIDED, LPV, 8>(p, t, mt, s);               \
    default: return hipErrorInvalidValue;                                           \
  }
  if (lp == 4) { KS_DMA_UD(4) }
  if constexpr (sizeof(T) == 2) {
    if (lp == 8) { KS_DMA_UD(8) }
  }
#undef KS_DMA_UD
  return hipErrorInvalidValue;
}

}  // namespace ks
