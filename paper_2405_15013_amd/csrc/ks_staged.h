// LDS-staged MFMA kernels for KS patterns whose blocks are dense contractions
// (b and c multiples of 16).
//
// Same output-stationary products as the register-direct kernels (paper
// Section 4.1, Algorithm 2; operand layout in ks_direct.h), but the X values
// of a tile are brought in by the whole workgroup: every stage of LCH values
// of l is read with coalesced 16-byte nontemporal loads into a per-thread
// register stage, written to one of two LDS buffers and read back by the
// wavefronts as MFMA operands (ks_staged_index.h).  This turns the strided
// batch-size-first gathers into contiguous row runs (the paper's weak case,
// Section 4.2), shares one load of X among the k-groups of a tile, and keeps
// one stage of loads in flight per workgroup while the previous one is
// multiplied.  K blocks are read from L1/L2 one stage ahead.  BSL outputs are
// stored straight from the accumulators (ks_direct.h, direct_store); BSF
// outputs go through an LDS copy of the tile and leave as contiguous row runs
// (the "structured epilogue" of Appendix D.3), so no partial cache lines are
// written back.
#pragma once
#include "ks_direct.h"
#include "ks_staged_index.h"

namespace ks {

constexpr int kStagedMaxLds = 128 * 1024;  // LDS per workgroup (of the CU's 160 KB)
constexpr int kStagedUnitsPerThread = 4;  // 16-byte units of a stage per thread (<= 256 per wavefront)

template <int NB>
__device__ __forceinline__ void lds_read_piece(const char* p, uint32_t* w) {
  if constexpr (NB == 16) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(p);
    w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
  } else {
    static_assert(NB == 8, "pieces are 8 or 16 bytes");
    const u32x2 v = *reinterpret_cast<const u32x2*>(p);
    w[0] = v[0]; w[1] = v[1];
  }
}

template <typename T, int LAYOUT, int V, bool STRIDED, int MT, int LP>
struct SChunk {
  static constexpr int S = sizeof(T);
  static constexpr int VK = LAYOUT == BSL ? 1 : V;
  static constexpr int KW = LP * S / 4;
  static constexpr int PE = (LAYOUT == BSL || STRIDED) ? V : (LP * V * S < 16 ? LP * V : 16 / S);
  static constexpr int NP = LP * V / PE;
  static constexpr int PB = PE * S;
  uint32_t kw[MT][VK][KW];

  __device__ __forceinline__ void load_k(const T* __restrict__ kl, int64_t kmstride, int64_t kestride, int l) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int e = 0; e < VK; ++e) load_piece<KW * 4, false>(kl + mt * kmstride + e * kestride + l, kw[mt][e]);
  }
  // X operands from LDS (lane base `ob`, chunk at stage-relative l0) and MFMAs.
  __device__ __forceinline__ void mma(const char* ob, int olstride, int oqstride, int l0, f32x4 (&acc)[MT][V]) const {
    uint32_t xw[LP * V * S / 4];
    const char* o = ob + l0 * olstride;
#pragma unroll
    for (int q = 0; q < NP; ++q) lds_read_piece<PB>(o + q * oqstride, xw + q * (PB / 4));
    direct_mma<T, LAYOUT, V, MT, LP>(xw, kw, acc);
  }
};

template <typename T, int LAYOUT, int V, bool STRIDED, int MT, int CPS>
__global__ __launch_bounds__(512) void ks_staged_kernel(Problem p, StagedTile t) {
  constexpr int S = sizeof(T);
  constexpr int LP = S == 4 ? 4 : 8;
  constexpr int CH = 4 * LP;
  constexpr int UPT = kStagedUnitsPerThread;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int nthr = 64 * t.W;
  const int n = lane & 15, g = lane >> 4;
  const STile st = staged_tile(p, t, blockIdx.x);
  const SItem si = staged_item(p, t, st, V, MT, w);
  DItem it;
  it.i = st.i;
  it.j0 = si.j0;
  it.k0 = si.k0;
  it.beta0 = si.beta0;
  const T* __restrict__ x = static_cast<const T*>(p.x);
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const int c = p.c;
  const int LCH = t.LCH;
  const int nstages = (c + LCH - 1) / LCH;

  // ---- stage loads: units tid + nthr*k of the stage ------------------------
  // X is streamed with nontemporal loads unless other tiles (k-group tiles)
  // read the same stage.
  //
  // Units of a stage: thread tid takes units tid + nthr*k.  A unit's X offset
  // is linear in the stage start (ls * d elements in BSF, ls * d * batch in
  // BSL) and its LDS offset does not depend on the stage, so both are
  // computed once for the full stages and once more for a shorter last stage.
  uint32_t stg[UPT][4];
  const bool ntx = t.kgt == 1;
  const int64_t xls = p.layout == BSL ? (int64_t)p.d * p.batch : p.d;  // X elements per value of l
  int64_t uoff[UPT];
  int ulds[UPT];
  int nunits = 0;
  auto units_for = [&](int nl) {
    const int ur = staged_units_per_row(p, t, V, S, nl);
    nunits = staged_rows(p, t, nl) * ur;
#pragma unroll
    for (int k = 0; k < UPT; ++k) {
      const int u = tid + nthr * k;
      const int r = u / ur, v = u - (u / ur) * ur;
      uoff[k] = u < nunits ? staged_x_unit(p, t, st, V, S, 0, r, v) : 0;
      ulds[k] = staged_lds_unit(t, r, v);
    }
  };
  units_for(c < LCH ? c : LCH);
  auto gload = [&](int ls) {
    if (c - ls < LCH && ls > 0) units_for(c - ls);  // shorter last stage
    const T* xs = x + (int64_t)ls * xls;
#pragma unroll
    for (int k = 0; k < UPT; ++k) {
      if (tid + nthr * k < nunits) {
        if (ntx) load_piece<16, true>(xs + uoff[k], stg[k]);
        else load_piece<16, false>(xs + uoff[k], stg[k]);
      }
    }
  };
  auto lstore = [&](int buf) {
    char* base = smem + buf * t.stage;
#pragma unroll
    for (int k = 0; k < UPT; ++k) {
      if (tid + nthr * k < nunits) {
        const u32x4 v = {stg[k][0], stg[k][1], stg[k][2], stg[k][3]};
        *reinterpret_cast<u32x4*>(base + ulds[k]) = v;
      }
    }
  };

  const int64_t kmstride = (int64_t)16 * c, kestride = (int64_t)p.b * c;
  const T* kl = kv + direct_k_base(p, it, LP, n, g);
  const int ob = staged_op_base(p, t, si, LP, V, S, n, g);
  const int olstride = staged_op_lstride(p, t, S);
  const int oqstride = staged_op_qstride(p, t, STRIDED, SChunk<T, LAYOUT, V, STRIDED, MT, LP>::PE, S);

  f32x4 acc[MT][V];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[mt][e] = f32x4{0.f, 0.f, 0.f, 0.f};

  SChunk<T, LAYOUT, V, STRIDED, MT, LP> kc[CPS], kn[CPS];
  gload(0);
  lstore(0);
  if (nstages > 1) gload(LCH);
#pragma unroll
  for (int q = 0; q < CPS; ++q)
    if ((q + 1) * CH <= c) kc[q].load_k(kl, kmstride, kestride, q * CH);
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();

  for (int s = 0; s < nstages; ++s) {
    const int ls = s * LCH;
    const int nl = c - ls < LCH ? c - ls : LCH;
    const char* buf = smem + (s & 1) * t.stage;
    const bool more = s + 1 < nstages;
    if (more) {
#pragma unroll
      for (int q = 0; q < CPS; ++q)
        if (ls + LCH + (q + 1) * CH <= c) kn[q].load_k(kl, kmstride, kestride, ls + LCH + q * CH);
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the next stage's K loads ahead of this stage's MFMAs
#pragma unroll
    for (int q = 0; q < CPS; ++q)
      if ((q + 1) * CH <= nl) kc[q].mma(buf + ob, olstride, oqstride, q * CH, acc);
    if constexpr (S == 2) {
      if (nl % CH) {  // c % 32 == 16: the last 16 values of l, 16x16x16 steps
        SChunk<T, LAYOUT, V, STRIDED, MT, 4> tc;
        tc.load_k(kv + direct_k_base(p, it, 4, n, g), kmstride, kestride, c - 16);
        const int ob4 = staged_op_base(p, t, si, 4, V, S, n, g);
        const int oq4 = staged_op_qstride(p, t, STRIDED, SChunk<T, LAYOUT, V, STRIDED, MT, 4>::PE, S);
        tc.mma(buf + ob4, olstride, oq4, nl - 16, acc);
      }
    }
    if (more) {
      lstore((s + 1) & 1);
      if (s + 2 < nstages) gload(ls + 2 * LCH);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < CPS; ++q) kc[q] = kn[q];
    }
    __syncthreads();
  }

  if constexpr (LAYOUT == BSL) {
    // Each lane's 4-element runs along the batch already form 256-byte row
    // segments per wavefront store: store straight from the accumulators.
    direct_store<T, LAYOUT, V, STRIDED, MT, true>(p, it, n, g, acc);
  } else {
    // Structured epilogue: accumulators -> LDS output tile -> contiguous runs.
    // (The loop's last barrier guarantees no wavefront still reads X stages.)
    const bool has_bias = p.bias != nullptr;
    float bv[MT][V][4];  // output feature: row k0 + 16 mt + 4 g + r4 of block (i, j0 + e)
    if (has_bias) {
      const T* bb = static_cast<const T*>(p.bias) + (int64_t)(it.i * p.b + it.k0 + 4 * g) * p.d + it.j0;
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
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int e = 0; e < V; ++e)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) acc[mt][e][r4] += bv[mt][e][r4];
    }
    if (epilogue_gelu(p)) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int e = 0; e < V; ++e)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) acc[mt][e][r4] = gelu_f32<T>(acc[mt][e][r4]);
    }
    const int r = 16 * si.rs + n;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        // V consecutive j of output row k: one V*S-byte LDS write
        const int k = it.k0 + 16 * mt + 4 * g + r4;
        char* cell = smem + staged_y_lds(p, t, st, MT, S, r, k, it.j0);
        if constexpr (S == 4) {
          if constexpr (V == 4) {
            *reinterpret_cast<f32x4*>(cell) = f32x4{acc[mt][0][r4], acc[mt][1][r4], acc[mt][2][r4], acc[mt][3][r4]};
          } else if constexpr (V == 2) {
            typedef float f32x2 __attribute__((ext_vector_type(2)));
            *reinterpret_cast<f32x2*>(cell) = f32x2{acc[mt][0][r4], acc[mt][1][r4]};
          } else {
            *reinterpret_cast<float*>(cell) = acc[mt][0][r4];
          }
        } else {
          uint32_t wv[(V + 1) / 2];
#pragma unroll
          for (int e = 0; e < V; e += 2) {
            const uint32_t lo = __builtin_bit_cast(uint16_t, from_f32<T>(acc[mt][e][r4]));
            const uint32_t hi = e + 1 < V ? __builtin_bit_cast(uint16_t, from_f32<T>(acc[mt][e + 1][r4])) : 0u;
            wv[e / 2] = lo | (hi << 16);
          }
          if constexpr (V == 4) {
            *reinterpret_cast<u32x2*>(cell) = u32x2{wv[0], wv[1]};
          } else if constexpr (V == 2) {
            *reinterpret_cast<uint32_t*>(cell) = wv[0];
          } else {
            *reinterpret_cast<uint16_t*>(cell) = (uint16_t)wv[0];
          }
        }
      }
    __syncthreads();
    const int uy = staged_y_units_per_row(p, t, MT, S);
    const int nunits = 16 * t.RS * uy;
    T* __restrict__ y = static_cast<T*>(p.y);
    for (int u = tid; u < nunits; u += nthr) {
      const int row = u / uy, v = u % uy;
      const int64_t off = staged_y_unit(p, t, st, MT, S, row, v);
      if (off < 0) continue;
      const u32x4 val = *reinterpret_cast<const u32x4*>(smem + row * t.ypitch + v * 16);
      __builtin_nontemporal_store(val, reinterpret_cast<u32x4*>(y + off));
    }
  }
}

template <typename T, int LAYOUT, int V, bool STRIDED, int MT, int CPS>
hipError_t launch_staged_inst(const Problem& p, const StagedTile& t, hipStream_t s) {
  if (t.lds > 64 * 1024) {
    // Opt in to more than 64 KB of dynamic LDS (once per instance).
    // Opt in to more than 64 KB of dynamic LDS once per instance (a function-
    // local static: initialised exactly once even with concurrent callers).
    static const hipError_t raised = hipFuncSetAttribute(reinterpret_cast<const void*>(&ks_staged_kernel<T, LAYOUT, V, STRIDED, MT, CPS>),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize, kStagedMaxLds);
    if (raised != hipSuccess) return raised;
  }
  hipLaunchKernelGGL((ks_staged_kernel<T, LAYOUT, V, STRIDED, MT, CPS>), dim3(t.tiles), dim3(64 * t.W), t.lds, s, p,
                     t);
  return hipGetLastError();
}

template <typename T, int LAYOUT, int V, bool STRIDED, int CPS>
hipError_t launch_staged_mt(const Problem& p, const StagedTile& t, int mt, hipStream_t s) {
  constexpr int MX = direct_mt_max(sizeof(T), LAYOUT, V);
  switch (mt) {
    case 1: return launch_staged_inst<T, LAYOUT, V, STRIDED, 1, CPS>(p, t, s);
    case 2: if constexpr (MX >= 2) return launch_staged_inst<T, LAYOUT, V, STRIDED, 2, CPS>(p, t, s); break;
    case 3: if constexpr (MX >= 3) return launch_staged_inst<T, LAYOUT, V, STRIDED, 3, CPS>(p, t, s); break;
    case 4: if constexpr (MX >= 4) return launch_staged_inst<T, LAYOUT, V, STRIDED, 4, CPS>(p, t, s); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

// All instances of one storage type: BSL (V = 4), BSF with d = 1 (two MFMA
// chunks per stage), d = 2 and d = 4 (contiguous), d >= 8 (strided).
template <typename T>
hipError_t launch_staged_type(const Problem& p, const StagedTile& t, int V, bool strided, int mt, int cps,
                              hipStream_t s) {
  if (p.layout == BSL) {
    if (V != kDirectVec || strided || cps != 1) return hipErrorInvalidValue;
    return launch_staged_mt<T, BSL, kDirectVec, false, 1>(p, t, mt, s);
  }
  if (strided) {
    if (V != kDirectVec || cps != 1) return hipErrorInvalidValue;
    return launch_staged_mt<T, BSF, kDirectVec, true, 1>(p, t, mt, s);
  }
  switch (V) {
    case 1:
      if (cps == 2) return launch_staged_mt<T, BSF, 1, false, 2>(p, t, mt, s);
      break;
    case 2:
      if (cps == 1) return launch_staged_mt<T, BSF, 2, false, 1>(p, t, mt, s);
      break;
    case 4:
      if (cps == 1) return launch_staged_mt<T, BSF, 4, false, 1>(p, t, mt, s);
      break;
    default: break;
  }
  return hipErrorInvalidValue;
}

}  // namespace ks
