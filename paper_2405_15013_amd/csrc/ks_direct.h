// Register-direct MFMA kernels for KS patterns whose blocks are dense
// contractions (b and c multiples of 16).
//
// Output-stationary tiling of the paper (Section 4.1, Algorithm 2; kernel
// sketch of Section 4.2), laid out for CDNA4 wavefronts: every wavefront is an
// independent work item (see ks_direct_index.h) that streams the X values of
// its tile from HBM straight into MFMA operand registers with nontemporal
// vector loads of 4 elements (16 bytes fp32, 8 bytes 16-bit; no LDS, no
// barriers), reads the packed b x c block(s) of K from L1/L2 as 16-byte A
// operands, keeps the fp32 accumulators in registers
// over the whole reduction over l, and stores each output once, directly in
// the requested layout (BSL: 4-element runs along the batch; BSF: runs of
// consecutive j, or of consecutive k and j when d <= 4).
//
// The products are Yt^T = Kblock * Xt^T on 16 x 16 MFMA tiles: A = 16 rows k
// of the block, B = the lane's column of X (a batch vector in BSL, a batch row
// in BSF), reduction over l.  The order of l inside a chunk is any fixed
// assignment that A and B share: lane group g holds l = LPL*g .. LPL*g+LPL-1,
// so both operands are contiguous in memory along l (K rows) or get
// assembled from the lane's loaded vectors (X).
//   fp32:    v_mfma_f32_16x16x4_f32, LPL = 4 (one MFMA per l of the lane);
//   16-bit:  v_mfma_f32_16x16x32_{bf16,f16}, LPL = 8, plus one
//            v_mfma_f32_16x16x16 step with LPL = 4 when c % 32 == 16.
// The next chunk of l is loaded while the MFMAs of the current one run.
#pragma once
#include "ks_common.h"
#include "ks_direct_index.h"
#include "ks_epilogue.h"
#include "ks_internal.h"

namespace ks {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));

// Puts the problem's sizes and pointers in scalar registers at kernel entry,
// so that they arrive in the same round of kernel-argument loads as the rest;
// otherwise the compiler fetches them only after the first branches of the
// work-item decode, a second memory round trip before the first load of X.
#define KS_PROBLEM_FIELDS(p)                                                                               \
  "s"(p.a), "s"(p.b), "s"(p.c), "s"(p.d), "s"(p.batch), "s"(p.N), "s"(p.M), "s"(p.layout), "s"(p.align), \
      "s"(p.x), "s"(p.y), "s"(p.kv)
__device__ __forceinline__ void kernarg_fetch(const Problem& p) { asm volatile("" ::KS_PROBLEM_FIELDS(p)); }

// One MFMA step: acc += A * B where each lane supplies LP values of l.
template <typename T, int LP> struct DMma;
template <> struct DMma<float, 4> {
  // four 16x16x4 steps, one per l of the lane (component t of A and of B)
  __device__ static __forceinline__ void run(const uint32_t* a, float bt, int t, f32x4& acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[t]), bt, acc, 0, 0, 0);
  }
};
template <> struct DMma<bf16_t, 8> {
  __device__ static __forceinline__ void run(const uint32_t* a, const uint32_t* b, f32x4& acc) {
    const u32x4 av = {a[0], a[1], a[2], a[3]}, bv = {b[0], b[1], b[2], b[3]};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av), __builtin_bit_cast(bf16x8_t, bv),
                                                  acc, 0, 0, 0);
  }
};
template <> struct DMma<bf16_t, 4> {
  __device__ static __forceinline__ void run(const uint32_t* a, const uint32_t* b, f32x4& acc) {
    const u32x2 av = {a[0], a[1]}, bv = {b[0], b[1]};
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4_t, av), __builtin_bit_cast(i16x4_t, bv),
                                                    acc, 0, 0, 0);
  }
};
template <> struct DMma<_Float16, 8> {
  __device__ static __forceinline__ void run(const uint32_t* a, const uint32_t* b, f32x4& acc) {
    const u32x4 av = {a[0], a[1], a[2], a[3]}, bv = {b[0], b[1], b[2], b[3]};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, av), __builtin_bit_cast(f16x8_t, bv),
                                                 acc, 0, 0, 0);
  }
};
template <> struct DMma<_Float16, 4> {
  __device__ static __forceinline__ void run(const uint32_t* a, const uint32_t* b, f32x4& acc) {
    const u32x2 av = {a[0], a[1]}, bv = {b[0], b[1]};
    acc = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4_t, av), __builtin_bit_cast(f16x4_t, bv),
                                                acc, 0, 0, 0);
  }
};

// Load NB bytes (16 or 8) at p into w[0 .. NB/4).
template <int NB, bool NT>
__device__ __forceinline__ void load_piece(const void* p, uint32_t* w) {
  if constexpr (NB == 16) {
    const u32x4 v = NT ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p))
                       : *reinterpret_cast<const u32x4*>(p);
    w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
  } else {
    static_assert(NB == 8, "pieces are 8 or 16 bytes");
    const u32x2 v = NT ? __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p))
                       : *reinterpret_cast<const u32x2*>(p);
    w[0] = v[0]; w[1] = v[1];
  }
}

template <int NB>
__device__ __forceinline__ void store_piece(void* p, const uint32_t* w) {
  if constexpr (NB == 16) {
    const u32x4 v = {w[0], w[1], w[2], w[3]};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
  } else {
    static_assert(NB == 8, "pieces are 8 or 16 bytes");
    const u32x2 v = {w[0], w[1]};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x2*>(p));
  }
}

// 16-bit element f of a packed dword array.
__device__ __forceinline__ uint32_t half_of(const uint32_t* w, int f) {
  return (f & 1) ? (w[f >> 1] >> 16) : (w[f >> 1] & 0xffffu);
}

// MFMAs of one chunk: xw holds the lane's LP x V block of X (flat t*V + e),
// kw[mt][e] the A operands (LP values of l of K row k0 + 16*mt + m; one block
// in BSL, block j0 + e in BSF).
template <typename T, int LAYOUT, int V, int MT, int LP>
__device__ __forceinline__ void direct_mma(const uint32_t* xw, const uint32_t (&kw)[MT][LAYOUT == BSL ? 1 : V]
                                           [LP * sizeof(T) / 4], f32x4 (&acc)[MT][V]) {
  if constexpr (sizeof(T) == 4) {
#pragma unroll
    for (int t = 0; t < LP; ++t)
#pragma unroll
      for (int e = 0; e < V; ++e) {
        const float bt = __uint_as_float(xw[t * V + e]);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) DMma<T, LP>::run(kw[mt][LAYOUT == BSL ? 0 : e], bt, t, acc[mt][e]);
      }
  } else {
#pragma unroll
    for (int e = 0; e < V; ++e) {
      // B operand of chain e: the lane's LP values of l for column e,
      // flat elements t*V + e, two per dword.
      uint32_t bw[LP / 2];
#pragma unroll
      for (int q = 0; q < LP / 2; ++q) {
        if constexpr (V == 1) {
          bw[q] = xw[q];
        } else {
          bw[q] = half_of(xw, (2 * q) * V + e) | (half_of(xw, (2 * q + 1) * V + e) << 16);
        }
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) DMma<T, LP>::run(kw[mt][LAYOUT == BSL ? 0 : e], bw, acc[mt][e]);
    }
  }
}

// Stores of the lane's outputs: per M-tile 4 x V values, flat r*V + e, as
// pieces of YPE contiguous elements (ks_direct_index.h, direct_y_off).
// EPI instances apply the bias / activation of ks_epilogue.h piece by piece
// between the accumulator copy and the rounding, so that only one piece of
// the tile is live in VGPRs at a time; plain instances (EPI false) carry no
// epilogue code and keep their register budget.
template <typename T, int LAYOUT, int V, bool STRIDED, int MT, bool EPI>
__device__ __forceinline__ void direct_store(const Problem& p, const DItem& it, int n, int g,
                                             const f32x4 (&acc_in)[MT][V]) {
  constexpr int S = sizeof(T);
  constexpr int YPE = (LAYOUT == BSL || STRIDED) ? V : (4 * V * S < 16 ? 4 * V : 16 / S);
  constexpr int YNP = 4 * V / YPE;
  constexpr int YPB = YPE * S;
  // Output feature of accumulator (mt, e, r): row k = k0 + 16 mt + 4 g + r of
  // block (i, j), j = j0 (+ e in BSF).  The bias loads are issued before the
  // wait for the last MFMA results (they depend on the tile only, so every
  // lane's indices are in range).
  constexpr int BV = LAYOUT == BSF ? V : 1;
  bool has_bias = false, gelu = false;
  float bv[MT][BV][4];
  if constexpr (EPI) {
    has_bias = p.bias != nullptr;
    gelu = epilogue_gelu(p);
    if (has_bias) {
      const T* bb = static_cast<const T*>(p.bias) + (int64_t)(it.i * p.b + it.k0 + 4 * g) * p.d + it.j0;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int e = 0; e < BV; ++e) bv[mt][e][r] = to_f32(bb[(16 * mt + r) * p.d + e]);
    }
  }
  mfma_results_settle();
  if (!direct_lane_valid(p, it, V, n)) return;
  f32x4 acc[MT][V];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[mt][e] = acc_in[mt][e];
  T* yl = static_cast<T*>(p.y) + direct_y_base(p, it, V, n, g);
  const int64_t ymstride = direct_y_mstride(p), yqstride = direct_y_qstride(p, STRIDED, V, S);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int q = 0; q < YNP; ++q) {
      float y[YPE];  // flat f = q * YPE + u: accumulator (mt, f % V, f / V)
#pragma unroll
      for (int u = 0; u < YPE; ++u) {
        const int f = q * YPE + u;
        y[u] = acc[mt][f % V][f / V];
      }
      if constexpr (EPI) {
        if (has_bias) {
#pragma unroll
          for (int u = 0; u < YPE; ++u) {
            const int f = q * YPE + u;
            y[u] += bv[mt][LAYOUT == BSF ? f % V : 0][f / V];
          }
        }
        if (gelu) {
#pragma unroll
          for (int u = 0; u < YPE; ++u) y[u] = gelu_f32<T>(y[u]);
        }
      }
      uint32_t w[YPB / 4];
      if constexpr (S == 4) {
#pragma unroll
        for (int u = 0; u < YPE; ++u) w[u] = __float_as_uint(y[u]);
      } else {
#pragma unroll
        for (int u = 0; u < YPE; u += 2) w[u / 2] = pack2_f32<T>(y[u], y[u + 1]);
      }
      store_piece<YPB>(yl + mt * ymstride + q * yqstride, w);
    }
  }
}

// One chunk of the reduction: LP values of l per lane group (4*LP per chunk).
// Pointers passed to load() are the lane's bases (ks_direct_index.h).
template <typename T, int LAYOUT, int V, bool STRIDED, int MT, int LP>
struct DChunk {
  static constexpr int S = sizeof(T);
  static constexpr int VK = LAYOUT == BSL ? 1 : V;  // distinct K blocks per chunk
  static constexpr int NXW = LP * V * S / 4;         // dwords of X per lane
  static constexpr int KW = LP * S / 4;              // dwords of one A operand
  static constexpr int PE = (LAYOUT == BSL || STRIDED) ? V : (LP * V * S < 16 ? LP * V : 16 / S);
  static constexpr int NP = LP * V / PE;             // X pieces
  static constexpr int PB = PE * S;                  // bytes per piece
  uint32_t xw[NXW];
  uint32_t kw[MT][VK][KW];

  // ntx: X is read by this wavefront only (one k-group), so it is streamed
  // with nontemporal loads; otherwise the k-group neighbours re-read it from
  // the caches.
  __device__ __forceinline__ void load(const T* __restrict__ xl, int64_t lstride, int64_t qstride,
                                       const T* __restrict__ kl, int64_t kmstride, int64_t kestride, int l0, bool ntx) {
    const T* xc = xl + (int64_t)l0 * lstride;
    if (ntx) {
#pragma unroll
      for (int q = 0; q < NP; ++q) load_piece<PB, true>(xc + q * qstride, xw + q * (PB / 4));
    } else {
#pragma unroll
      for (int q = 0; q < NP; ++q) load_piece<PB, false>(xc + q * qstride, xw + q * (PB / 4));
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int e = 0; e < VK; ++e) load_piece<KW * 4, false>(kl + mt * kmstride + e * kestride + l0, kw[mt][e]);
  }

  __device__ __forceinline__ void mma(f32x4 (&acc)[MT][V]) const { direct_mma<T, LAYOUT, V, MT, LP>(xw, kw, acc); }
};

template <typename T, int LAYOUT, int V, bool STRIDED, int MT, bool EPI>
__global__ __launch_bounds__(256) void ks_direct_kernel(Problem p, DirectTile t) {
  constexpr int S = sizeof(T);
  constexpr int LP = S == 4 ? 4 : 8;
  constexpr int CH = 4 * LP;  // l values per chunk
  const int lane = threadIdx.x & 63;
  // A wavefront past the last item (spare waves of the last workgroup) works
  // on the last item with in-bounds loads and stores nothing.  No branch
  // precedes the loads, so every kernel argument arrives in one round of
  // scalar loads instead of one round for the item count and another after
  // the exit test.
  const int item0 = blockIdx.x * t.waves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool live = item0 < t.items;  // wave-uniform
  const int item = live ? item0 : t.items - 1;
  kernarg_fetch(p);
  const int n = lane & 15, g = lane >> 4;
  const DItem it = direct_item_fast(p, t, V, MT, item);
  const T* __restrict__ x = static_cast<const T*>(p.x);
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const int c = p.c;
  const int64_t lstride = direct_x_lstride(p);
  const int64_t kmstride = (int64_t)16 * c, kestride = (int64_t)p.b * c;
  const bool ntx = t.kgroups == 1;

  f32x4 acc[MT][V];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[mt][e] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (c >= CH) {
    const T* xl = x + direct_x_base(p, it, LP, V, n, g);
    const T* kl = kv + direct_k_base(p, it, LP, n, g);
    const int64_t qstride = direct_x_qstride(p, STRIDED, LP, V, S);
    DChunk<T, LAYOUT, V, STRIDED, MT, LP> cur, nxt;
    cur.load(xl, lstride, qstride, kl, kmstride, kestride, 0, ntx);
    for (int l0 = 0; l0 + CH <= c; l0 += CH) {
      const bool more = l0 + 2 * CH <= c;
      if (more) nxt.load(xl, lstride, qstride, kl, kmstride, kestride, l0 + CH, ntx);
      __builtin_amdgcn_sched_barrier(0);
      cur.mma(acc);
      if (more) cur = nxt;
    }
    mfma_results_settle();  // before the paths join (the join copies the accumulators)
  }
  if constexpr (S == 2) {
    if (c % CH) {  // c % 32 == 16: last 16 values of l with the 16x16x16 step
      const T* xl = x + direct_x_base(p, it, 4, V, n, g);
      const T* kl = kv + direct_k_base(p, it, 4, n, g);
      const int64_t qstride = direct_x_qstride(p, STRIDED, 4, V, S);
      DChunk<T, LAYOUT, V, STRIDED, MT, 4> tail;
      tail.load(xl, lstride, qstride, kl, kmstride, kestride, c - 16, ntx);
      tail.mma(acc);
      mfma_results_settle();
    }
  }

  if (!live) return;
  direct_store<T, LAYOUT, V, STRIDED, MT, EPI>(p, it, n, g, acc);
}

// The same work item with the reduction length fixed at compile time: NCH
// full chunks (plus the 16-bit tail) are fully unrolled and the loads of up to
// PD chunks ahead are in flight while a chunk is multiplied, PD chosen so the
// chunks in flight take about 32 VGPRs (at least one chunk ahead).  A
// wavefront's time is then about one memory latency plus its MFMAs, instead
// of one latency per chunk; a deeper prefetch (64 VGPRs) measured slower for
// fp32 (fewer resident wavefronts) and the same for 16-bit storage.
template <typename T, int LAYOUT, int V, bool STRIDED, int MT, int NCH, bool TAIL, bool EPI>
__global__ __launch_bounds__(256) void ks_direct_c_kernel(Problem p, DirectTile t) {
  constexpr int S = sizeof(T);
  constexpr int LP = S == 4 ? 4 : 8;
  constexpr int CH = 4 * LP;
  using Chunk = DChunk<T, LAYOUT, V, STRIDED, MT, LP>;
  constexpr int R = Chunk::NXW + MT * Chunk::VK * Chunk::KW;  // VGPRs of one chunk
  constexpr int PD0 = 32 / R;
  constexpr int PD = NCH <= 1 ? 0 : (PD0 < 1 ? 1 : (PD0 > NCH - 1 ? NCH - 1 : PD0));
  const int lane = threadIdx.x & 63;
  // A wavefront past the last item (spare waves of the last workgroup) works
  // on the last item with in-bounds loads and stores nothing.  No branch
  // precedes the loads, so every kernel argument arrives in one round of
  // scalar loads instead of one round for the item count and another after
  // the exit test.
  const int item0 = blockIdx.x * t.waves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool live = item0 < t.items;  // wave-uniform
  const int item = live ? item0 : t.items - 1;
  kernarg_fetch(p);
  const int n = lane & 15, g = lane >> 4;
  const DItem it = direct_item_fast(p, t, V, MT, item);
  const T* __restrict__ x = static_cast<const T*>(p.x);
  const T* __restrict__ kv = static_cast<const T*>(p.kv);
  const int c = p.c;
  const int64_t lstride = direct_x_lstride(p);
  const int64_t kmstride = (int64_t)16 * c, kestride = (int64_t)p.b * c;
  const bool ntx = t.kgroups == 1;

  f32x4 acc[MT][V];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < V; ++e) acc[mt][e] = f32x4{0.f, 0.f, 0.f, 0.f};

  const T* xl = x + direct_x_base(p, it, LP, V, n, g);
  const T* kl = kv + direct_k_base(p, it, LP, n, g);
  const int64_t qstride = direct_x_qstride(p, STRIDED, LP, V, S);
  // sched_barrier(0) keeps the compiler's scheduler from sinking the loads
  // next to their first use, which would serialise one memory latency per
  // chunk.
  Chunk ch[NCH > 0 ? NCH : 1];
#pragma unroll
  for (int q = 0; q <= PD && q < NCH; ++q) ch[q].load(xl, lstride, qstride, kl, kmstride, kestride, q * CH, ntx);
  DChunk<T, LAYOUT, V, STRIDED, MT, 4> tl;
  if constexpr (TAIL) {
    tl.load(x + direct_x_base(p, it, 4, V, n, g), lstride, direct_x_qstride(p, STRIDED, 4, V, S),
            kv + direct_k_base(p, it, 4, n, g), kmstride, kestride, c - 16, ntx);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int q = 0; q < NCH; ++q) {
    if (q + PD + 1 < NCH)
      ch[q + PD + 1].load(xl, lstride, qstride, kl, kmstride, kestride, (q + PD + 1) * CH, ntx);
    __builtin_amdgcn_sched_barrier(0);
    ch[q].mma(acc);
  }
  if constexpr (TAIL) tl.mma(acc);

  if (!live) return;
  direct_store<T, LAYOUT, V, STRIDED, MT, EPI>(p, it, n, g, acc);
}

// Vector width along the batch (BSL) and largest j-run (BSF): 4 elements, i.e.
// 16-byte fp32 or 8-byte 16-bit pieces.
constexpr int kDirectVec = 4;

// Batch entries per lane of the batch-size-last kernels for 16-bit storage:
// 8 (one 16-byte vector per row of X or Y) when the batch is a multiple of 8.
constexpr int kDirectVecBsl16 = 8;

// Largest M-tile count per wave for a (storage type, layout, V) instance set.
constexpr int direct_mt_max(int esize, int layout, int V) {
  return esize == 4 ? ((layout == BSL || V <= 2) ? 4 : 2) : ((layout == BSL || V <= 2) ? 4 : 2);
}

template <typename T, int LAYOUT, int V, bool STRIDED, int MT, bool EPI>
hipError_t launch_direct_inst(const Problem& p, const DirectTile& t, unsigned grid, hipStream_t s) {
  int nch = 0;
  bool tail = false;
  const dim3 g(grid), b(64 * t.waves);
  if (direct_c_specialised(sizeof(T), p.c, &nch, &tail)) {
#define KS_DIRECT_C(N, TL)                                                                          \
  if (nch == N && tail == TL) {                                                                    \
    hipLaunchKernelGGL((ks_direct_c_kernel<T, LAYOUT, V, STRIDED, MT, N, TL, EPI>), g, b, 0, s, p, t); \
    return hipGetLastError();                                                                      \
  }
    if constexpr (sizeof(T) == 4) {
      KS_DIRECT_C(1, false) KS_DIRECT_C(2, false) KS_DIRECT_C(3, false)
      KS_DIRECT_C(4, false) KS_DIRECT_C(6, false) KS_DIRECT_C(8, false)
    } else {
      KS_DIRECT_C(0, true) KS_DIRECT_C(1, false) KS_DIRECT_C(1, true)
      KS_DIRECT_C(2, false) KS_DIRECT_C(3, false) KS_DIRECT_C(4, false)
    }
#undef KS_DIRECT_C
  }
  hipLaunchKernelGGL((ks_direct_kernel<T, LAYOUT, V, STRIDED, MT, EPI>), g, b, 0, s, p, t);
  return hipGetLastError();
}

template <typename T, int LAYOUT, int V, bool STRIDED, bool EPI>
hipError_t launch_direct_mt(const Problem& p, const DirectTile& t, int mt, unsigned grid, hipStream_t s) {
  constexpr int MX = direct_mt_max(sizeof(T), LAYOUT, V);
  switch (mt) {
    case 1: return launch_direct_inst<T, LAYOUT, V, STRIDED, 1, EPI>(p, t, grid, s);
    case 2: if constexpr (MX >= 2) return launch_direct_inst<T, LAYOUT, V, STRIDED, 2, EPI>(p, t, grid, s); break;
    case 3: if constexpr (MX >= 3) return launch_direct_inst<T, LAYOUT, V, STRIDED, 3, EPI>(p, t, grid, s); break;
    case 4: if constexpr (MX >= 4) return launch_direct_inst<T, LAYOUT, V, STRIDED, 4, EPI>(p, t, grid, s); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

// All instances of one storage type, plain (EPI false) or with the epilogue.
template <typename T, bool EPI>
hipError_t launch_direct_type(const Problem& p, const DirectTile& t, int V, bool strided, int mt, unsigned grid,
                              hipStream_t s) {
  if (p.layout == BSL) {
    if (strided) return hipErrorInvalidValue;
    if constexpr (sizeof(T) == 2) {
      if (V == kDirectVecBsl16) return launch_direct_mt<T, BSL, kDirectVecBsl16, false, EPI>(p, t, mt, grid, s);
    }
    if (V != kDirectVec) return hipErrorInvalidValue;
    return launch_direct_mt<T, BSL, kDirectVec, false, EPI>(p, t, mt, grid, s);
  }
  if (strided) {
    if (V != kDirectVec) return hipErrorInvalidValue;
    return launch_direct_mt<T, BSF, kDirectVec, true, EPI>(p, t, mt, grid, s);
  }
  switch (V) {
    case 1: return launch_direct_mt<T, BSF, 1, false, EPI>(p, t, mt, grid, s);
    case 2: return launch_direct_mt<T, BSF, 2, false, EPI>(p, t, mt, grid, s);
    case 4: return launch_direct_mt<T, BSF, 4, false, EPI>(p, t, mt, grid, s);
    default: break;
  }
  return hipErrorInvalidValue;
}

}  // namespace ks
