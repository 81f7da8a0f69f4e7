// Internal interface between the host planner (ks_host.cpp) and the HIP
// kernels.  Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace ks {

enum Layout : int { BSF = 0, BSL = 1 };
enum Dtype : int { F32 = 0, BF16 = 1, F16 = 2, FP8 = 3 };  // FP8: X, K in E4M3, Y in bf16

// Kernel variants (the numbering is the "variant=" field of ks_plan_describe
// and the argument of ks_force_variant).
enum Variant : int {
  V_GENERIC = 0,   // one thread per output element, any pattern
  V_VALU_BSL = 1,  // VALU streaming, batch-size-last, small b and c
  V_VALU_BSF = 2,  // VALU, batch-size-first, small b and c
  V_DIRECT = 3,    // register-direct MFMA, one work item per wavefront, b and c multiples of 16
  V_STAGED = 4,    // LDS-staged MFMA, 4 work items per workgroup share coalesced X stages
  // 5: unused (a persistent streaming variant, measured slower and removed)
  V_DMA = 6,       // LDS-staged MFMA with X moved HBM -> LDS by DMA, three stage buffers (BSF, d >= 4)
  V_MASKED = 7,    // register-direct MFMA with zero-padded tiles and narrow accesses (any b, c, batch, alignment)
  V_FP8 = 8,       // FP8 (E4M3) inputs, bf16 output: the masked decomposition on fp8 MFMAs
  V_COUNT = 9
};

// Problem description shared by all kernels.  Sizes fit in int32 (checked by
// the host: every tensor has < 2^31 elements).
struct Problem {
  int a, b, c, d;
  int batch;
  int N, M;      // a*c*d, a*b*d
  int layout;
  int dtype;
  const void* kv;
  const void* x;
  void* y;
  int align;     // largest power of two (<= 16) dividing the byte addresses of x and y
  const void* bias;  // epilogue (ks_epilogue.h): per-output-feature bias (M values) or null
  int act;           // epilogue activation: 0 none, 1 GELU
};

// Host side: whether the call needs the instances with the epilogue compiled in.
inline bool has_epilogue(const Problem& p) { return p.bias != nullptr || p.act != 0; }

// Launch description produced by the planner.
struct Plan {
  int variant = V_GENERIC;
  // variant-specific tile parameters
  int vec = 1;      // elements per memory vector along the contiguous dimension
  int bt = 0;       // batch rows (BSF) / batch columns (BSL) per work item or tile; stream: tiles per wavefront
  int jg = 1;       // j values per work item (direct) / j-groups per tile (staged)
  int unroll = 1;   // vectors per thread (VALU)
  int waves_m = 1;  // MFMA: 16-row M-tiles per wavefront (MT)
  int waves_n = 1;  // MFMA: k-groups (direct) / k-group tiles (staged)
  int lds_bytes = 0;
  unsigned grid = 1;
  unsigned block = 256;
  int xcd_remap = 0;  // remap blockIdx so neighbouring tiles share an XCD (staged)
  // LDS-staged MFMA
  int rs = 1;       // row (BSF) / column (BSL) groups per tile
  int kgw = 1;      // k-groups per tile
  int lch = 0;      // values of l per stage
  int cps = 1;      // MFMA chunks per stage (LDS-DMA: MFMA lane depth LP)
  int nt = 1;       // LDS-DMA: 16-row groups per wavefront (each K operand serves 16*nt batch rows)
};

// Each launcher enqueues one kernel and returns the hipError_t of the launch.
hipError_t launch_generic(const Problem& p, const Plan& pl, hipStream_t s);
hipError_t launch_valu_bsl(const Problem& p, const Plan& pl, hipStream_t s);
hipError_t launch_valu_bsf(const Problem& p, const Plan& pl, hipStream_t s);
hipError_t launch_direct(const Problem& p, const Plan& pl, hipStream_t s);
hipError_t launch_staged(const Problem& p, const Plan& pl, hipStream_t s);
hipError_t launch_dma(const Problem& p, const Plan& pl, hipStream_t s);
hipError_t launch_masked(const Problem& p, const Plan& pl, hipStream_t s);
hipError_t launch_fp8(const Problem& p, const Plan& pl, hipStream_t s);
struct FusedChain;
hipError_t launch_chain_fused(const FusedChain& fc, int dtype, bool vec, hipStream_t s);

}  // namespace ks

namespace ks {
// Vectors per thread of the batch-size-last VALU kernel for a given block
// shape (shared by the planner, which sizes the grid, and the launcher, which
// picks the kernel instance).
inline int valu_bsl_unroll(int b, int c) {
  const int m = b > c ? b : c;
  return m <= 2 ? 4 : (m <= 4 ? 2 : 1);
}
constexpr int kValuMaxBC = 16;
}  // namespace ks
