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
#include "ks_masked.h"

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

// One chunk (32 values of l) of a wavefront's operands as loaded, before any
// use of the data, so that the next chunk's loads are in flight while this
// one is multiplied: X as 16 dwords (the lane's 8 values of l x V, or for
// 64-byte row runs the pieces still in their loading lanes), K as MT x VK
// runs of 8 values of l (2 dwords each).
template <int V, int MT, int VK>
struct Fp8Chunk {
  static constexpr int XW = 2 * V;  // dwords of the lane's X operand
  uint32_t xw[XW < 16 ? 16 : XW];
  uint32_t kw[MT][VK][2];
};

template <int LAYOUT, int V, int MT>
__global__ __launch_bounds__(256) void ks_fp8_kernel(Problem p, MaskedTile t) {
  constexpr int LP = 8;       // values of l per lane and MFMA
  constexpr int CH = 4 * LP;  // values of l per chunk
  constexpr int VK = LAYOUT == BSL ? 1 : V;
  using Chunk = Fp8Chunk<V, MT, VK>;
  const int lane = threadIdx.x & 63;
  // Spare waves of the last workgroup work on the last item and store
  // nothing: no branch before the loads, one round of kernel-argument loads.
  const int item0 = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool live = item0 < t.items;  // wave-uniform
  const int item = live ? item0 : t.items - 1;
  kernarg_fetch(p, t);
  const int n = lane & 15, g = lane >> 4;
  const MItem it = masked_item(p, t, V, item);
  // Batch-size-first with V = d, c a multiple of 8 and 16-byte aligned
  // buffers: a lane's X operand (8 values of l x d j) is one run of 8d bytes
  // of its batch row, and (b a multiple of 4) its outputs k0 + 4g .. + 3 of
  // each M-tile one run of 4d bf16.  d = 8: 64-byte runs, four lanes per run
  // (fp8_rows_transpose); d = 1, 2, 4: each lane moves its own run.
  const bool runs = LAYOUT == BSF && V == p.d && p.c % 8 == 0 && p.align >= 16;
  const bool rows8 = runs && V == 8;
  const bool col = masked_col_valid(p, it, V, n);
  const uint8_t* __restrict__ x = static_cast<const uint8_t*>(p.x);
  const uint8_t* __restrict__ kv = static_cast<const uint8_t*>(p.kv);

  // Issue the loads of chunk ch (no use of the loaded data).
  auto load = [&](int ch, Chunk& cb) {
    const int l0 = ch * CH + LP * g;
    if (rows8) {
      // load xr: piece g of lane row xr's 64-byte run (values from ch*CH + 8xr)
#pragma unroll
      for (int xr = 0; xr < 4; ++xr) {
        const int lx = ch * CH + LP * xr;
        u32x4 w = u32x4{0, 0, 0, 0};
        if (col && lx < p.c)
          w = *reinterpret_cast<const u32x4*>(x + (int64_t)(it.beta0 + n) * p.N + ((int64_t)it.i * p.c + lx) * 8 + 16 * g);
#pragma unroll
        for (int w2 = 0; w2 < 4; ++w2) cb.xw[4 * xr + w2] = w[w2];
      }
    } else if (V <= 4 && runs) {
      if constexpr (V <= 4) {
        // the run of values l0 .. l0 + 7 (8V bytes: one or two vectors)
        const int64_t off = masked_x_off(p, it, V, l0, n);
#pragma unroll
        for (int w2 = 0; w2 < 2 * V; ++w2) cb.xw[w2] = 0;
        if (off >= 0) {
          if constexpr (V == 1) {
            const u32x2 w = *reinterpret_cast<const u32x2*>(x + off);
            cb.xw[0] = w[0];
            cb.xw[1] = w[1];
          } else {
#pragma unroll
            for (int h = 0; h < V / 2; ++h) {
              const u32x4 w = *reinterpret_cast<const u32x4*>(x + off + 16 * h);
#pragma unroll
              for (int w2 = 0; w2 < 4; ++w2) cb.xw[4 * h + w2] = w[w2];
            }
          }
        }
      }
    } else {
      uint8_t xs[LP][V];
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
      __builtin_memcpy(cb.xw, xs, LP * V);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int e = 0; e < VK; ++e) {
        // the lane's 8 values of l of K row k0 + 16 mt + n of block (i, j0 + e)
        const int64_t ko = masked_k_off(p, it, e, 16 * mt + n, l0);
        if (t.kvec) {  // one aligned 8-byte run (c a multiple of 8)
          u32x2 w = u32x2{0, 0};
          if (ko >= 0) w = *reinterpret_cast<const u32x2*>(kv + ko);
          cb.kw[mt][e][0] = w[0];
          cb.kw[mt][e][1] = w[1];
        } else {
          uint8_t ks[LP];
#pragma unroll
          for (int q = 0; q < LP; ++q) {
            const int64_t kq = masked_k_off(p, it, e, 16 * mt + n, l0 + q);
            ks[q] = kq >= 0 ? kv[kq] : 0;
          }
          __builtin_memcpy(cb.kw[mt][e], ks, LP);
        }
      }
  };

  // The MFMAs of one chunk: B operand of chain e = the lane's 8 values of l
  // at j (BSF) or batch entry (BSL) e, byte q = value l0 + q.
  f32x4 acc[MT][V];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[mt][e] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](Chunk& cb) {
    uint8_t xs[LP][V];
    if (rows8) {
      if constexpr (V == 8) {
        u32x4 m[4];
#pragma unroll
        for (int xr = 0; xr < 4; ++xr) m[xr] = u32x4{cb.xw[4 * xr], cb.xw[4 * xr + 1], cb.xw[4 * xr + 2], cb.xw[4 * xr + 3]};
        fp8_rows_transpose(m);
        __builtin_memcpy(xs, m, 64);
      }
    } else {
      __builtin_memcpy(xs, cb.xw, LP * V);
    }
#pragma unroll
    for (int e = 0; e < V; ++e) {
      uint64_t xw = 0;
#pragma unroll
      for (int q = 0; q < LP; ++q) xw |= (uint64_t)xs[q][e] << (8 * q);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const uint64_t kw = (uint64_t)cb.kw[mt][LAYOUT == BSL ? 0 : e][0] | ((uint64_t)cb.kw[mt][LAYOUT == BSL ? 0 : e][1] << 32);
        acc[mt][e] = __builtin_amdgcn_mfma_f32_16x16x32_fp8_fp8((long)kw, (long)xw, acc[mt][e], 0, 0, 0);
      }
    }
  };

  for (int ch = 0; ch < t.nchunks; ++ch) {
    Chunk cur;
    load(ch, cur);
    mma(cur);
  }

  if (!live) return;
  // Epilogue: output feature of (mt, e, r) is row k = k0 + 16 mt + 4g + r of
  // block (i, j0 [+ e in BSF]); padding rows (k >= b) take no bias.
  constexpr int BV = LAYOUT == BSF ? V : 1;
  const bool has_bias = p.bias != nullptr;
  float bv[MT][4][BV];
  if (has_bias) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int k = it.k0 + 16 * mt + 4 * g + r;
#pragma unroll
        for (int e = 0; e < BV; ++e)
          bv[mt][r][e] = k < p.b ? bias_value<bf16_t>(p, ((int64_t)it.i * p.b + k) * p.d + it.j0 + e) : 0.0f;
      }
  }
  mfma_results_settle();
  if (has_bias) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int e = 0; e < V; ++e) acc[mt][e][r] += bv[mt][r][LAYOUT == BSF ? e : 0];
  }
  if (epilogue_gelu(p)) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int e = 0; e < V; ++e) acc[mt][e][r] = gelu_f32<bf16_t>(acc[mt][e][r]);
  }

#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    MItem im = it;  // the M-tile's output rows k0 + 16 mt ..
    im.k0 += 16 * mt;
    if (rows8) {
      if constexpr (V == 8) {
        // Lane row g's outputs k = k0 + 4g + r (r = 0..3, 8 j each) are one
        // 64-byte run of its batch row; after the transpose, store xr writes
        // piece g of lane row xr's run, so four lanes write 64 contiguous bytes.
        u32x4 m[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          uint16_t v[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = from_f32<bf16_t>(acc[mt][e][r]);
          __builtin_memcpy(&m[r], v, 16);
        }
        fp8_rows_transpose(m);
        if (col) {
          bf16_t* yrow = static_cast<bf16_t*>(p.y) + (int64_t)(im.beta0 + n) * p.M + (int64_t)im.i * p.b * 8;
#pragma unroll
          for (int xr = 0; xr < 4; ++xr) {
            const int k = im.k0 + 4 * xr + g;
            if (k < p.b) *reinterpret_cast<u32x4*>(yrow + (int64_t)k * 8) = m[xr];
          }
        }
      }
      continue;
    }
    if (V <= 4 && runs && p.b % 4 == 0) {
      if constexpr (V <= 4) {
        // outputs k0 + 4g .. k0 + 4g + 3 (all j): one run of 4V bf16
        const int64_t off = masked_y_off(p, im, V, n, g, 0);
        if (off >= 0) {
          uint16_t v[4 * V];
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int e = 0; e < V; ++e) v[r * V + e] = from_f32<bf16_t>(acc[mt][e][r]);
          bf16_t* yo = static_cast<bf16_t*>(p.y) + off;
          if constexpr (V == 1) {
            u32x2 w;
            __builtin_memcpy(&w, v, 8);
            *reinterpret_cast<u32x2*>(yo) = w;
          } else {
#pragma unroll
            for (int h = 0; h < 4 * V / 8; ++h) {
              u32x4 w;
              __builtin_memcpy(&w, v + 8 * h, 16);
              *reinterpret_cast<u32x4*>(yo + 8 * h) = w;
            }
          }
        }
      }
      continue;
    }
    // outputs k = k0 + 4g + r in bfloat16
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t off = masked_y_off(p, im, V, n, g, r);
      if (off < 0) continue;
      uint16_t v[V];
#pragma unroll
      for (int e = 0; e < V; ++e) v[e] = from_f32<bf16_t>(acc[mt][e][r]);
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

// M-tiles per wavefront: the largest MT in {4, 2, 1} (2 at most for access
// widths of 4 or 8, whose accumulators and operands would otherwise leave one
// wavefront per SIMD) that divides the 16-row tiles of b and leaves at least
// 768 wavefronts; more M-tiles read each X operand once for more output rows.
int fp8_mt(const Problem& p, int V) {
  const int mtmax = V >= 4 ? 2 : 4;
  const int tiles = (p.b + 15) / 16;
  for (int mt = mtmax; mt > 1; mt /= 2) {
    if (tiles % mt) continue;
    const MaskedTile t = masked_tile(p, V, mt);
    if ((int64_t)t.nbt * p.a * t.jgroups * t.kgroups >= 768) return mt;
  }
  return 1;
}

bool plan_fp8(const Problem& p, Plan* pl) {
  if (p.dtype != FP8) return false;
  const int V = fp8_vec(p);
  const int MT = fp8_mt(p, V);
  const MaskedTile t = masked_tile(p, V, MT);
  const int64_t items = (int64_t)t.nbt * p.a * t.jgroups * t.kgroups;
  if (items > 0x7fffffff - 3) return false;
  pl->variant = V_FP8;
  pl->vec = V;
  pl->unroll = 0;
  pl->waves_m = MT;
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
  const MaskedTile t = masked_tile(p, pl.vec, pl.waves_m);
  const dim3 g(pl.grid), b(256);
#define KS_FP8(L, VV, M)                                                     \
  if (p.layout == L && pl.vec == VV && pl.waves_m == M) {                    \
    hipLaunchKernelGGL((ks_fp8_kernel<L, VV, M>), g, b, 0, s, p, t);        \
    return hipGetLastError();                                                \
  }
  KS_FP8(BSL, 1, 1) KS_FP8(BSL, 2, 1) KS_FP8(BSL, 4, 1) KS_FP8(BSL, 8, 1)
  KS_FP8(BSL, 1, 2) KS_FP8(BSL, 2, 2) KS_FP8(BSL, 4, 2) KS_FP8(BSL, 8, 2)
  KS_FP8(BSL, 1, 4) KS_FP8(BSL, 2, 4)
  KS_FP8(BSF, 1, 1) KS_FP8(BSF, 2, 1) KS_FP8(BSF, 4, 1) KS_FP8(BSF, 8, 1)
  KS_FP8(BSF, 1, 2) KS_FP8(BSF, 2, 2) KS_FP8(BSF, 4, 2) KS_FP8(BSF, 8, 2)
  KS_FP8(BSF, 1, 4) KS_FP8(BSF, 2, 4)
#undef KS_FP8
  return hipErrorInvalidValue;
}

}  // namespace ks
