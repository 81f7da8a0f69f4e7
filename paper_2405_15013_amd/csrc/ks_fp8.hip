// FP8 (OCP E4M3) register-direct MFMA kernel: X and K_values hold 8-bit E4M3
// codes, products accumulate in fp32 on v_mfma_f32_16x16x32_fp8_fp8 (8
// values of l per lane and operand), Y is written in bfloat16 (the paper's
// conclusion names low precision as the open limitation of its kernel; its
// half-precision results are in the appendix).
//
// Work decomposition, padding and index arithmetic are the masked kernel's
// (ks_masked_index.h): one wavefront per item, 16 x 16 tiles padded with
// zeros, accesses of V consecutive elements (V bytes of X, 2V bytes of Y).
#include "ks_direct.h"
#include "ks_epilogue.h"
#include "ks_masked_index.h"

namespace ks {

namespace {

// N consecutive bytes (N-byte aligned when N is 2, 4, 8 or 16).
template <int N>
__device__ __forceinline__ void fp8_load(const uint8_t* p, uint8_t (&v)[N]) {
  if constexpr (N == 16) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(p);
    __builtin_memcpy(v, &w, 16);
  } else if constexpr (N == 8) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(p);
    __builtin_memcpy(v, &w, 8);
  } else if constexpr (N == 4) {
    const uint32_t w = *reinterpret_cast<const uint32_t*>(p);
    __builtin_memcpy(v, &w, 4);
  } else if constexpr (N == 2) {
    const uint16_t w = *reinterpret_cast<const uint16_t*>(p);
    __builtin_memcpy(v, &w, 2);
  } else {
    v[0] = p[0];
  }
}

// 4 x 4 transpose of 16-byte pieces across the four 16-lane rows of a
// wavefront: on entry register r of lane row g holds piece M[g][r], on exit
// it holds M[r][g] (for each lane column n).  Two v_permlane16_swap (rows 1
// and 3 of the first operand exchanged with rows 0 and 2 of the second), then
// two v_permlane32_swap (rows 2-3 of the first with rows 0-1 of the second),
// per dword.
__device__ __forceinline__ void fp8_rows_transpose(u32x4 (&m)[4]) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    auto s01 = __builtin_amdgcn_permlane16_swap(m[0][w], m[1][w], false, false);
    auto s23 = __builtin_amdgcn_permlane16_swap(m[2][w], m[3][w], false, false);
    auto s02 = __builtin_amdgcn_permlane32_swap(s01[0], s23[0], false, false);
    auto s13 = __builtin_amdgcn_permlane32_swap(s01[1], s23[1], false, false);
    m[0][w] = s02[0];
    m[1][w] = s13[0];
    m[2][w] = s02[1];
    m[3][w] = s13[1];
  }
}

template <int LAYOUT, int V>
__global__ __launch_bounds__(256) void ks_fp8_kernel(Problem p, MaskedTile t) {
  constexpr int LP = 8;       // values of l per lane and MFMA
  constexpr int CH = 4 * LP;  // values of l per chunk
  constexpr int VK = LAYOUT == BSL ? 1 : V;
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (item >= t.items) return;  // wave-uniform
  const int n = lane & 15, g = lane >> 4;
  const MItem it = masked_item(p, t, V, item);
  // Batch-size-first with V = d, c a multiple of 8 and 16-byte aligned
  // buffers: a lane's X operand (8 values of l x d j) is one run of 8d bytes
  // of its batch row, and (b a multiple of 4) its outputs k0 + 4g .. + 3 one
  // run of 4d bf16.  d = 8: 64-byte runs, four lanes per run
  // (fp8_rows_transpose); d = 1, 2, 4: each lane moves its own run.
  const bool runs = LAYOUT == BSF && V == p.d && p.c % 8 == 0 && p.align >= 16;
  const bool rows8 = runs && V == 8;
  const uint8_t* __restrict__ x = static_cast<const uint8_t*>(p.x);
  const uint8_t* __restrict__ kv = static_cast<const uint8_t*>(p.kv);

  f32x4 acc[V];
#pragma unroll
  for (int e = 0; e < V; ++e) acc[e] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int ch = 0; ch < t.nchunks; ++ch) {
    const int l0 = ch * CH + LP * g;
    uint8_t xs[LP][V];
    uint8_t ks[VK][LP];
    if (rows8) {
      // Rows of d = 8: a lane's operand (8 values of l x 8 j) is the 64-byte
      // run of its batch row from l0*8.  Load x of the wavefront reads, for
      // lane row g, piece g of lane row x's run (four lanes cover one run),
      // then the pieces move to their lanes.
      u32x4 m[4];
      const bool col = masked_col_valid(p, it, V, n);
#pragma unroll
      for (int xr = 0; xr < 4; ++xr) {
        const int lx = ch * CH + LP * xr;
        m[xr] = u32x4{0, 0, 0, 0};
        if (col && lx < p.c)
          m[xr] = *reinterpret_cast<const u32x4*>(x + (int64_t)(it.beta0 + n) * p.N +
                                                  ((int64_t)it.i * p.c + lx) * 8 + 16 * g);
      }
      fp8_rows_transpose(m);
      if constexpr (V == 8) __builtin_memcpy(xs, m, 64);
    } else if (V <= 4 && runs) {
      if constexpr (V <= 4) {
        // the run of values l0 .. l0 + 7 (8V bytes: 8, 16 or two 16-byte loads)
        constexpr int NB = LP * V < 16 ? LP * V : 16;
        const int64_t off = masked_x_off(p, it, V, l0, n);
        if (off >= 0) {
          fp8_load<NB>(x + off, reinterpret_cast<uint8_t(&)[NB]>(xs[0][0]));
          if constexpr (LP * V == 32) fp8_load<16>(x + off + 16, reinterpret_cast<uint8_t(&)[16]>(xs[LP / 2][0]));
        } else {
#pragma unroll
          for (int q = 0; q < LP; ++q)
#pragma unroll
            for (int e = 0; e < V; ++e) xs[q][e] = 0;
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < LP; ++q) {
        const int64_t off = masked_x_off(p, it, V, l0 + q, n);
        if (off >= 0) {
          fp8_load<V>(x + off, xs[q]);
        } else {
#pragma unroll
          for (int e = 0; e < V; ++e) xs[q][e] = 0;
        }
      }
    }
#pragma unroll
    for (int e = 0; e < VK; ++e) {
      if (t.kvec) {  // the lane's 8 values of l are one aligned 8-byte run of row k
        const int64_t ko = masked_k_off(p, it, e, n, l0);
        if (ko >= 0) {
          fp8_load<LP>(kv + ko, ks[e]);
        } else {
#pragma unroll
          for (int q = 0; q < LP; ++q) ks[e][q] = 0;
        }
      } else {
#pragma unroll
        for (int q = 0; q < LP; ++q) {
          const int64_t ko = masked_k_off(p, it, e, n, l0 + q);
          ks[e][q] = ko >= 0 ? kv[ko] : 0;
        }
      }
    }
    // operands: 8 codes per lane, value l0 + q in byte q
    uint64_t kw[VK];
#pragma unroll
    for (int e = 0; e < VK; ++e) {
      uint64_t w = 0;
#pragma unroll
      for (int q = 0; q < LP; ++q) w |= (uint64_t)ks[e][q] << (8 * q);
      kw[e] = w;
    }
#pragma unroll
    for (int e = 0; e < V; ++e) {
      uint64_t xw = 0;
#pragma unroll
      for (int q = 0; q < LP; ++q) xw |= (uint64_t)xs[q][e] << (8 * q);
      acc[e] = __builtin_amdgcn_mfma_f32_16x16x32_fp8_fp8((long)kw[LAYOUT == BSL ? 0 : e], (long)xw, acc[e], 0, 0, 0);
    }
  }
  // Epilogue: output feature of (e, r) is row k = k0 + 4g + r of block
  // (i, j0 [+ e in BSF]); padding rows (k >= b) take no bias.
  constexpr int BV = LAYOUT == BSF ? V : 1;
  const bool has_bias = p.bias != nullptr;
  float bv[4][BV];
  if (has_bias) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int k = it.k0 + 4 * g + r;
#pragma unroll
      for (int e = 0; e < BV; ++e)
        bv[r][e] = k < p.b ? bias_value<bf16_t>(p, ((int64_t)it.i * p.b + k) * p.d + it.j0 + e) : 0.0f;
    }
  }
  mfma_results_settle();
  if (has_bias) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int e = 0; e < V; ++e) acc[e][r] += bv[r][LAYOUT == BSF ? e : 0];
  }
  if (epilogue_gelu(p)) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int e = 0; e < V; ++e) acc[e][r] = gelu_f32(acc[e][r]);
  }
  if (rows8) {
    // Lane row g's outputs k = k0 + 4g + r (r = 0..3, 8 j each) are one
    // 64-byte run of its batch row; after the transpose, store x writes piece
    // g of lane row x's run, so four lanes write 64 contiguous bytes.
    u32x4 m[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      uint16_t v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = from_f32<bf16_t>(acc[e < V ? e : 0][r]);  // V == 8 here
      __builtin_memcpy(&m[r], v, 16);
    }
    fp8_rows_transpose(m);
    if (!masked_col_valid(p, it, V, n)) return;
    bf16_t* yrow = static_cast<bf16_t*>(p.y) + (int64_t)(it.beta0 + n) * p.M + (int64_t)it.i * p.b * 8;
#pragma unroll
    for (int xr = 0; xr < 4; ++xr) {
      const int k = it.k0 + 4 * xr + g;
      if (k < p.b) *reinterpret_cast<u32x4*>(yrow + (int64_t)k * 8) = m[xr];
    }
    return;
  }
  if (V <= 4 && runs && p.b % 4 == 0) {
    // outputs k0 + 4g .. k0 + 4g + 3 (all j): one run of 4V bf16
    const int64_t off = masked_y_off(p, it, V, n, g, 0);
    if (off < 0) return;
    uint16_t v[4 * V];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int e = 0; e < V; ++e) v[r * V + e] = from_f32<bf16_t>(acc[e][r]);
    bf16_t* yo = static_cast<bf16_t*>(p.y) + off;
    if constexpr (V == 1) {
      u32x2 w;
      __builtin_memcpy(&w, v, 8);
      *reinterpret_cast<u32x2*>(yo) = w;
    } else if constexpr (V <= 4) {
#pragma unroll
      for (int h = 0; h < 4 * V / 8; ++h) {
        u32x4 w;
        __builtin_memcpy(&w, v + 8 * h, 16);
        *reinterpret_cast<u32x4*>(yo + 8 * h) = w;
      }
    }
    return;
  }
  // outputs k = k0 + 4g + r in bfloat16
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t off = masked_y_off(p, it, V, n, g, r);
    if (off < 0) continue;
    uint16_t v[V];
#pragma unroll
    for (int e = 0; e < V; ++e) v[e] = from_f32<bf16_t>(acc[e][r]);
    bf16_t* yo = static_cast<bf16_t*>(p.y) + off;
    if constexpr (V == 8) {
      u32x4 w;
      __builtin_memcpy(&w, v, 16);
      if constexpr (LAYOUT == BSL) __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(yo));
      else *reinterpret_cast<u32x4*>(yo) = w;
    } else if constexpr (V == 4) {
      u32x2 w;
      __builtin_memcpy(&w, v, 8);
      if constexpr (LAYOUT == BSL) __builtin_nontemporal_store(w, reinterpret_cast<u32x2*>(yo));
      else *reinterpret_cast<u32x2*>(yo) = w;
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e) yo[e] = v[e];
    }
  }
}

}  // namespace

// Access width V (elements): up to 8 along the batch (BSL) or consecutive j
// (BSF), as the batch / d and the buffers' alignment allow (X pieces of V
// bytes, Y pieces of 2V bytes).  In BSF with V = d = 8 a lane's X operand is
// one contiguous 64-byte run of its batch row (8 values of l x 8 j) and its 4
// output rows one contiguous 64-byte run of Y.
int fp8_vec(const Problem& p) {
  int V = 8;
  for (; V > 1; V /= 2) {
    if (p.layout == BSL && p.batch % V) continue;
    if (p.layout == BSF && p.d % V) continue;
    if (p.align % (2 * V)) continue;
    break;
  }
  return V;
}

bool plan_fp8(const Problem& p, Plan* pl) {
  if (p.dtype != FP8) return false;
  const int V = fp8_vec(p);
  const MaskedTile t = masked_tile(p, V);
  const int64_t items = (int64_t)t.nbt * p.a * t.jgroups * t.kgroups;
  if (items > 0x7fffffff - 3) return false;
  pl->variant = V_FP8;
  pl->vec = V;
  pl->unroll = 0;
  pl->waves_m = 1;
  pl->waves_n = t.kgroups;
  pl->bt = p.layout == BSL ? 16 * V : 16;
  pl->jg = p.layout == BSL ? 1 : V;
  pl->lds_bytes = 0;
  pl->block = 256;
  pl->grid = (unsigned)((items + 3) / 4);
  pl->xcd_remap = 0;
  return true;
}

hipError_t launch_fp8(const Problem& p, const Plan& pl, hipStream_t s) {
  const MaskedTile t = masked_tile(p, pl.vec);
  const dim3 g(pl.grid), b(256);
#define KS_FP8(L, VV)                                                        \
  if (p.layout == L && pl.vec == VV) {                                       \
    hipLaunchKernelGGL((ks_fp8_kernel<L, VV>), g, b, 0, s, p, t);           \
    return hipGetLastError();                                                \
  }
  KS_FP8(BSL, 1) KS_FP8(BSL, 2) KS_FP8(BSL, 4) KS_FP8(BSL, 8)
  KS_FP8(BSF, 1) KS_FP8(BSF, 2) KS_FP8(BSF, 4) KS_FP8(BSF, 8)
#undef KS_FP8
  return hipErrorInvalidValue;
}

}  // namespace ks
