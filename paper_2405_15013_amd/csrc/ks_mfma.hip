// MFMA block-GEMM kernel for KS patterns whose blocks are real dense
// contractions (b and c multiples of 16).
//
// Output-stationary tiling (paper, Section 4.1, Algorithm 2; kernel sketch of
// Section 4.2): a workgroup owns the outputs of one i, a group of JG
// consecutive j and a tile of BT batch vectors, i.e. for every j in the group
// the block product
//     Yt[beta][k] = sum_l Xt[beta][l] * Kv[i*d + j][k][l]      (k < b, l < c)
// where Xt[beta][l] = X[beta, i*c*d + l*d + j] and Yt[beta][k] = Y[beta, i*b*d + k*d + j].
// Each element of Y is produced by exactly one workgroup, written once, with no
// atomics and no zero-fill.
//
// Data path per workgroup:
//  1. gather: 16-byte nontemporal loads of the X tile (rows l contiguous along
//     the batch for BSL; runs of j for BSF) into LDS, transposed on the way to
//     Xs[jj][beta][l] with l contiguous, the layout the MFMA operands want;
//  2. block GEMM: MFMA with M = batch, N = k, K = l.  The A operand (X) comes
//     from LDS, the B operand (the packed block, already k-major/l-contiguous in
//     memory) straight from L1/L2.  The accumulation order over l is any fixed
//     permutation that A and B share; fp32 accumulators live in registers.
//  3. epilogue: BSL stores four consecutive batch columns per lane directly
//     into Y's output rows; BSF stages the tile's output segment in LDS and
//     writes it with 16-byte stores (the "structured epilogue" of Appendix D.3).
#include "ks_internal.h"
#include "ks_common.h"
#include "ks_mfma_index.h"

namespace ks {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

// Per-type MFMA step.  A "fragment" is 16 bytes per lane: 4 fp32 values of
// consecutive l for the 16x16x4 fp32 MFMA (one per k-step), or 8 16-bit values
// for the 16x16x32 MFMA.  KC is the number of l consumed per fragment.
template <typename T> struct Mma;
template <> struct Mma<float> {
  static constexpr int KC = 16;
  __device__ static __forceinline__ void step(u32x4 a, u32x4 b, f32x4& acc) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[s]), __uint_as_float(b[s]), acc, 0, 0, 0);
  }
  __device__ static __forceinline__ void tail(u32x2, u32x2, f32x4&) {}
};
template <> struct Mma<bf16_t> {
  static constexpr int KC = 32;
  __device__ static __forceinline__ void step(u32x4 a, u32x4 b, f32x4& acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc,
                                                  0, 0, 0);
  }
  // 16 remaining l (c % 32 == 16): 4 values per lane.
  __device__ static __forceinline__ void tail(u32x2 a, u32x2 b, f32x4& acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, a), __builtin_bit_cast(i16x4, b), acc,
                                                    0, 0, 0);
  }
};
template <> struct Mma<_Float16> {
  static constexpr int KC = 32;
  __device__ static __forceinline__ void step(u32x4 a, u32x4 b, f32x4& acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), acc, 0,
                                                 0, 0);
  }
  __device__ static __forceinline__ void tail(u32x2 a, u32x2 b, f32x4& acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4, a), __builtin_bit_cast(f16x4, b), acc, 0, 0,
                                                0);
  }
};

template <typename T, int LAYOUT, int NT, int MT>
__global__ __launch_bounds__(256) void ks_mfma_kernel(Problem p, MfmaTile t) {
  constexpr int VEC = 16 / (int)sizeof(T);
  constexpr int KC = Mma<T>::KC;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const T* __restrict__ x = static_cast<const T*>(p.x);
  T* __restrict__ y = static_cast<T*>(p.y);
  const int b = p.b, c = p.c, d = p.d, batch = p.batch;
  const int BT = t.bt, JG = t.jg;
  const int P = c + VEC;  // LDS row pitch (elements): 16 bytes of padding
  const TileCoord tc = tile_coord(p, t, blockIdx.x, gridDim.x);
  const int i = tc.i, j0 = tc.j0, beta0 = tc.beta0;

  T* Xs = reinterpret_cast<T*>(smem);  // [JG][BT][P]

  // ---- 1. gather X tile into LDS --------------------------------------------
  {
    const int total = x_chunks(p, t);
    u32x4 buf[kMaxChunks];
#pragma unroll
    for (int u = 0; u < kMaxChunks; ++u) {
      const int q = threadIdx.x + u * 256;
      if (q >= total) break;
      const int64_t src = x_chunk_src(p, t, tc, q);
      buf[u] = src >= 0 ? ld_stream(reinterpret_cast<const u32x4*>(x + src)) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < kMaxChunks; ++u) {
      const int q = threadIdx.x + u * 256;
      if (q >= total) break;
      union { u32x4 v; T e[VEC]; } ch;
      ch.v = buf[u];
#pragma unroll
      for (int e = 0; e < VEC; ++e) Xs[x_chunk_lds(p, t, q, e)] = ch.e[e];
    }
  }
  __syncthreads();

  // ---- 2. block GEMMs --------------------------------------------------------
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, g = lane >> 4;
  const int items = mfma_items(p, t, MT, NT);
  T* Ys = reinterpret_cast<T*>(smem + (size_t)JG * BT * P * sizeof(T));  // BSF: [BT][b*JG + VEC]
  const int PY = b * JG + VEC;
  const int ctail = c % KC;  // 0, or 16 for 16-bit types with c % 32 == 16

  for (int it = wave; it < items; it += 4) {
    const Item itm = mfma_item(p, t, MT, NT, it);
    const int ngi = itm.ngi, mgi = itm.mgi, jj = itm.jj;
    f32x4 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const T* kb = kv + ((size_t)(i * d + j0 + jj) * b + ngi * NT * 16 + n) * c + g * (KC / 4);
    const T* xa = Xs + ((size_t)jj * BT + mgi * MT * 16 + n) * P + g * (KC / 4);
    for (int l0 = 0; l0 + KC <= c; l0 += KC) {
      u32x4 bf[NT], af[MT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) bf[nt] = *reinterpret_cast<const u32x4*>(kb + (size_t)nt * 16 * c + l0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) af[mt] = *reinterpret_cast<const u32x4*>(xa + mt * 16 * P + l0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) Mma<T>::step(af[mt], bf[nt], acc[mt][nt]);
    }
    if (sizeof(T) == 2 && ctail) {
      // last 16 values of l: lanes take 4 each (offset g*4 instead of g*8)
      const int l0 = c - 16;
      const T* kt = kb - g * (KC / 4) + g * 4;
      const T* xt = xa - g * (KC / 4) + g * 4;
      u32x2 bt2[NT], at2[MT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) bt2[nt] = *reinterpret_cast<const u32x2*>(kt + (size_t)nt * 16 * c + l0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) at2[mt] = *reinterpret_cast<const u32x2*>(xt + mt * 16 * P + l0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) Mma<T>::tail(at2[mt], bt2[nt], acc[mt][nt]);
    }

    // ---- 3. epilogue ----------------------------------------------------------
    // acc[mt][nt][r] = Yt[beta = mrow + 4g + r][k = kcol + n]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int bl = (mgi * MT + mt) * 16 + 4 * g;  // tile-local batch index of r = 0
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int k = (ngi * NT + nt) * 16 + n;
        if (LAYOUT == BSL) {
          const int beta = beta0 + bl;
          if (beta < batch) {
            T* dst = y + (size_t)(i * b * d + k * d + j0 + jj) * batch + beta;
            if (sizeof(T) == 4) {
              st_stream(reinterpret_cast<f32x4*>(dst), acc[mt][nt]);
            } else {
              union { u32x2 v; T e[4]; } o;
#pragma unroll
              for (int r = 0; r < 4; ++r) o.e[r] = from_f32<T>(acc[mt][nt][r]);
              st_stream(reinterpret_cast<u32x2*>(dst), o.v);
            }
          }
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) Ys[(bl + r) * PY + k * JG + jj] = from_f32<T>(acc[mt][nt][r]);
        }
      }
    }
  }

  if (LAYOUT == BSF) {
    __syncthreads();
    // Output segment of a batch row: e = k*JG + jj -> column i*b*d + k*d + j0 + jj.
    const int total = y_chunks(p, t);
    for (int q = threadIdx.x; q < total; q += 256) {
      int lds;
      const int64_t dst = y_chunk_dst(p, t, tc, q, &lds);
      if (dst < 0) continue;
      const u32x4 val = *reinterpret_cast<const u32x4*>(Ys + lds);
      st_stream(reinterpret_cast<u32x4*>(y + dst), val);
    }
  }
}

// ---------------------------------------------------------------------------
// Planner.
// ---------------------------------------------------------------------------

namespace {

int nt_for(int ntot) {
  static const int cand[] = {8, 6, 4, 3, 2, 1};
  for (int v : cand)
    if (ntot % v == 0) return v;
  return 1;
}
int mt_for(int nt) { return nt >= 6 ? 1 : (nt >= 3 ? 2 : (nt == 2 ? 4 : 8)); }

// LDS per workgroup: tiles normally stay within 64 KB (two or more workgroups
// per CU); shapes that cannot fit get up to 128 KB of the CU's 160 KB.
constexpr int kLdsBudget = 64 * 1024;
constexpr int kLdsBudgetMax = 128 * 1024;

}  // namespace

namespace {

// Tile shape for a given (NT, MT); false if none fits.
bool plan_mfma_mt(const Problem& p, int NT, int MT, int64_t budget, Plan* pl) {
  const int s = p.dtype == F32 ? 4 : 2;
  const int VEC = 16 / s;
  const int P = p.c + VEC;
  const int ngroups = (p.b / 16) / NT;
  int bt = 16 * MT, jg = 1, mode = LM_BSL;
  int64_t lds = 0;
  if (p.layout == BSL) {
    if (p.batch % VEC) return false;
    // Smallest batch tile giving every wave an item and >= 8 KB of X per tile,
    // then grow while the grid keeps >= 4 workgroups per CU.
    auto items = [&](int t) { return (t / (16 * MT)) * ngroups; };
    auto xbytes = [&](int t) { return (int64_t)t * P * s; };
    if (xbytes(bt) > budget) return false;
    while ((items(bt) < 4 || xbytes(bt) < 8192) && xbytes(bt * 2) <= budget && bt < 512) bt *= 2;
    while (xbytes(bt * 2) <= budget / 2 && bt < 256 &&
           (int64_t)p.a * p.d * ((p.batch + 2 * bt - 1) / (2 * bt)) >= 1024)
      bt *= 2;
    lds = xbytes(bt);
  } else {
    // j-group: all of d when the tile fits, else the largest divisor of d that
    // is a multiple of the vector width.
    auto fits = [&](int j, int t) {
      const int64_t xb = (int64_t)j * t * P * s;
      const int64_t yb = (int64_t)t * (p.b * j + VEC) * s;
      return xb + yb <= budget && (int64_t)p.c * t * j / VEC <= 256 * kMaxChunks;
    };
    jg = 0;
    if (fits(p.d, bt)) jg = p.d;
    if (!jg) {
      for (int j = p.d - 1; j >= VEC; --j)
        if (p.d % j == 0 && j % VEC == 0 && fits(j, bt)) { jg = j; break; }
    }
    if (!jg) return false;
    // Runs of a multiple of the vector width keep the LDS writes conflict-free;
    // otherwise (j-group = all of d) walk the contiguous c*d segment.
    if (jg % VEC == 0) mode = LM_BSF_RUNS;
    else if (jg == p.d && (p.c * p.d) % VEC == 0 && (p.b * p.d) % VEC == 0) mode = LM_BSF_SEG;
    else return false;
    auto items = [&](int t) { return jg * (t / (16 * MT)) * ngroups; };
    while (items(bt) < 4 && fits(jg, bt * 2)) bt *= 2;
    while (fits(jg, bt * 2) && (int64_t)jg * bt * P * s < 16384 &&
           (int64_t)p.a * (p.d / jg) * ((p.batch + 2 * bt - 1) / (2 * bt)) >= 1024)
      bt *= 2;
    lds = (int64_t)jg * bt * P * s + (int64_t)bt * (p.b * jg + VEC) * s;
  }
  const int64_t chunks = (int64_t)p.c * bt * jg / VEC;
  if (chunks > 256 * kMaxChunks || lds > budget) return false;
  const int64_t nbt = (p.batch + bt - 1) / bt;
  const int64_t grid = nbt * p.a * (p.d / jg);
  if (grid > 0x7fffffff) return false;
  pl->variant = V_MFMA;
  pl->vec = VEC;
  pl->bt = bt;
  pl->jg = jg;
  pl->unroll = mode;
  pl->waves_m = MT;
  pl->waves_n = NT;
  pl->lds_bytes = (int)lds;
  pl->grid = (unsigned)grid;
  pl->block = 256;
  pl->xcd_remap = (grid % 8 == 0 && p.layout == BSF && jg < p.d) ? 1 : 0;
  return true;
}

}  // namespace

bool plan_mfma_impl(const Problem& p, bool al16, Plan* pl) {
  if (p.b % 16 || p.c % 16) return false;
  if (!al16) return false;
  const int NT = nt_for(p.b / 16);
  for (int64_t budget : {(int64_t)kLdsBudget, (int64_t)kLdsBudgetMax})
    for (int MT = mt_for(NT); MT >= 1; MT /= 2)
      if (plan_mfma_mt(p, NT, MT, budget, pl)) return true;
  return false;
}

namespace {

template <typename T, int LAYOUT, int NT, int MT>
hipError_t launch_ntmt(const Problem& p, const Plan& pl, const MfmaTile& t, hipStream_t s) {
  if (pl.lds_bytes > 64 * 1024) {
    // Opt in to more than 64 KB of dynamic LDS (once per kernel instance).
    static bool raised = false;
    if (!raised) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&ks_mfma_kernel<T, LAYOUT, NT, MT>),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBudgetMax);
      if (e != hipSuccess) return e;
      raised = true;
    }
  }
  hipLaunchKernelGGL((ks_mfma_kernel<T, LAYOUT, NT, MT>), dim3(pl.grid), dim3(256), pl.lds_bytes, s, p, t);
  return hipGetLastError();
}

// MT ranges over 1 .. mt_for(NT) (powers of two).
template <typename T, int LAYOUT, int NT>
hipError_t launch_nt(const Problem& p, const Plan& pl, const MfmaTile& t, hipStream_t s) {
  constexpr int MTMAX = NT >= 6 ? 1 : (NT >= 3 ? 2 : (NT == 2 ? 4 : 8));
  switch (pl.waves_m) {
    case 1: return launch_ntmt<T, LAYOUT, NT, 1>(p, pl, t, s);
    case 2: if (MTMAX >= 2) return launch_ntmt<T, LAYOUT, NT, (MTMAX >= 2 ? 2 : 1)>(p, pl, t, s); break;
    case 4: if (MTMAX >= 4) return launch_ntmt<T, LAYOUT, NT, (MTMAX >= 4 ? 4 : 1)>(p, pl, t, s); break;
    case 8: if (MTMAX >= 8) return launch_ntmt<T, LAYOUT, NT, (MTMAX >= 8 ? 8 : 1)>(p, pl, t, s); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

template <typename T, int LAYOUT>
hipError_t launch_layout(const Problem& p, const Plan& pl, const MfmaTile& t, hipStream_t s) {
  switch (pl.waves_n) {
    case 8: return launch_nt<T, LAYOUT, 8>(p, pl, t, s);
    case 6: return launch_nt<T, LAYOUT, 6>(p, pl, t, s);
    case 4: return launch_nt<T, LAYOUT, 4>(p, pl, t, s);
    case 3: return launch_nt<T, LAYOUT, 3>(p, pl, t, s);
    case 2: return launch_nt<T, LAYOUT, 2>(p, pl, t, s);
    case 1: return launch_nt<T, LAYOUT, 1>(p, pl, t, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t launch_type(const Problem& p, const Plan& pl, const MfmaTile& t, hipStream_t s) {
  return p.layout == BSL ? launch_layout<T, BSL>(p, pl, t, s) : launch_layout<T, BSF>(p, pl, t, s);
}

}  // namespace

hipError_t launch_mfma(const Problem& p, const Plan& pl, hipStream_t s) {
  MfmaTile t;
  t.bt = pl.bt;
  t.jg = pl.jg;
  t.njg = p.d / pl.jg;
  t.nbt = (p.batch + pl.bt - 1) / pl.bt;
  t.mode = pl.unroll;
  t.remap = pl.xcd_remap;
  t.vec = pl.vec;
  switch (p.dtype) {
    case F32: return launch_type<float>(p, pl, t, s);
    case BF16: return launch_type<bf16_t>(p, pl, t, s);
    case F16: return launch_type<_Float16>(p, pl, t, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ks
