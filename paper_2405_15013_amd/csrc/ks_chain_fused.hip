// Fused chain kernel (see ks_chain_fused.h for the decomposition).
//
// Latency: a workgroup is the only one on its CU for most chain shapes (one
// tile of 16 columns per CU at batch 4096), so nothing else hides its memory
// latency.  The tile loads are batched (ks_chain_fused_io.h), and each pass's
// values are fetched from global memory into registers one pass ahead and
// parked in the LDS copy after the pass, so the pass loop itself touches only
// LDS.  Chains of square 16 .. 64 blocks run in ks_chain_mfma.hip.
#include <type_traits>

#include "ks_chain_fused.h"
#include "ks_chain_fused_io.h"
#include "ks_common.h"
#include "ks_internal.h"

namespace ks {

namespace {

// Values of pass q (its factors' packed blocks, one after the other): this
// thread's share fetched into registers in the storage type (so that no
// conversion waits for the loads), converted and parked in the LDS copy after
// the pass.  Scalar form: elements tid + kFusedThreads*r.  Vector form
// (fc.kvec): runs of 4 elements 4*(tid + kFusedThreads*r) .. +3, one 16- or
// 8-byte load and one 16-byte LDS write each (no run crosses a factor, whose
// counts are multiples of 4).
template <typename T>
struct FusedK {
  T v[kFusedKPerThread];
  __device__ __forceinline__ void fetch(const FusedChain& fc, int q) {
    // A pass has at most three factors: their value pointers are selected per
    // element (no per-lane indexing into the kernel arguments).
    const int n = fc.pk[q], cnt = fc.pcnt[q], f0 = fc.pf0[q], m = fc.pm[q];
    const T* k0 = static_cast<const T*>(fc.kv[f0]);
    const T* k1 = m > 1 ? static_cast<const T*>(fc.kv[f0 - 1]) : k0;
    const T* k2 = m > 2 ? static_cast<const T*>(fc.kv[f0 - 2]) : k0;
    if (fc.kvec) {
      typedef typename std::conditional<sizeof(T) == 4, u32x4, u32x2>::type W;
#pragma unroll
      for (int r = 0; r < kFusedKPerThread / 4; ++r) {
        const int e = 4 * (r * kFusedThreads + (int)threadIdx.x);
        if (e < n) {
          const int t = e >= 2 * cnt ? 2 : (e >= cnt ? 1 : 0);
          const T* kp = t == 0 ? k0 : (t == 1 ? k1 : k2);
          const W w = *reinterpret_cast<const W*>(kp + (e - t * cnt));
          __builtin_memcpy(&v[4 * r], &w, sizeof(W));
        }
      }
      return;
    }
#pragma unroll
    for (int r = 0; r < kFusedKPerThread; ++r) {
      const int e = r * kFusedThreads + (int)threadIdx.x;
      if (e < n) {
        const int t = e >= 2 * cnt ? 2 : (e >= cnt ? 1 : 0);
        const T* kp = t == 0 ? k0 : (t == 1 ? k1 : k2);
        v[r] = kp[e - t * cnt];
      }
    }
  }
  __device__ __forceinline__ void park(const FusedChain& fc, int q, float* kbuf) const {
    const int n = fc.pk[q];
    if (fc.kvec) {
#pragma unroll
      for (int r = 0; r < kFusedKPerThread / 4; ++r) {
        const int e = 4 * (r * kFusedThreads + (int)threadIdx.x);
        if (e < n)
          *reinterpret_cast<f32x4*>(kbuf + e) =
              f32x4{to_f32(v[4 * r]), to_f32(v[4 * r + 1]), to_f32(v[4 * r + 2]), to_f32(v[4 * r + 3])};
      }
      return;
    }
#pragma unroll
    for (int r = 0; r < kFusedKPerThread; ++r) {
      const int e = r * kFusedThreads + (int)threadIdx.x;
      if (e < n) kbuf[e] = to_f32(v[r]);
    }
  }
};

// Radix pass q (see ks_chain_fused.h): unit (group g, piece) loads the group's
// P rows (4 columns) into registers, applies the pass's factors t = 0 .. M-1
// (p x p blocks, M = log_p P) on register runs, stores the rows in place.
template <int P, int PR>
__device__ __forceinline__ void fused_radix_pass(const FusedChain& fc, int q, float* buf, const float* kbuf) {
  constexpr int M = PR == P ? 1 : (PR * PR == P ? 2 : 3);
  static_assert(M == 1 || M == 2 || (M == 3 && PR * PR * PR == P), "P must be a power of PR");
  const int d0 = fc.d[fc.pf0[q]], cnt = fc.pcnt[q];
  const int units = fused_radix_units(fc, q);
  for (int u = threadIdx.x; u < units; u += kFusedThreads) {
    const int g = u >> 2, piece = u & 3;
    int i, j0;
    fused_radix_group(fc, q, g, &i, &j0);
    float* rows = buf + (i * P * d0 + j0) * kFusedPitch + piece * 4;
    const int rstep = d0 * kFusedPitch;
    f32x4 v[P];
#pragma unroll
    for (int r = 0; r < P; ++r) v[r] = *reinterpret_cast<const f32x4*>(rows + r * rstep);
#pragma unroll
    for (int t = 0; t < M; ++t) {
      const int st = t == 0 ? 1 : (t == 1 ? PR : PR * PR);
      const float* kt = kbuf + t * cnt;
#pragma unroll
      for (int r = 0; r < P; ++r) {
        if ((r / st) % PR != 0) continue;  // digit t of r must be zero
        // the block's PR x PR values: 16-byte LDS reads (blocks start at
        // multiples of PR * PR >= 4 floats of the 16-byte aligned copy)
        const float* kb = kt + fused_radix_block<P, PR>(i, j0, d0, t, r) * (PR * PR);
        float kq[PR * PR];
#pragma unroll
        for (int w = 0; w < PR * PR / 4; ++w) {
          const f32x4 q4 = *reinterpret_cast<const f32x4*>(kb + 4 * w);
          kq[4 * w] = q4[0];
          kq[4 * w + 1] = q4[1];
          kq[4 * w + 2] = q4[2];
          kq[4 * w + 3] = q4[3];
        }
        f32x4 in[PR];
#pragma unroll
        for (int l = 0; l < PR; ++l) in[l] = v[r + l * st];
#pragma unroll
        for (int k = 0; k < PR; ++k) {
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int l = 0; l < PR; ++l) {
            const float kk = kq[k * PR + l];
            acc[0] = __builtin_fmaf(kk, in[l][0], acc[0]);
            acc[1] = __builtin_fmaf(kk, in[l][1], acc[1]);
            acc[2] = __builtin_fmaf(kk, in[l][2], acc[2]);
            acc[3] = __builtin_fmaf(kk, in[l][3], acc[3]);
          }
          v[r + k * st] = acc;
        }
      }
    }
#pragma unroll
    for (int r = 0; r < P; ++r) *reinterpret_cast<f32x4*>(rows + r * rstep) = v[r];
  }
}

// One factor, LDS -> LDS: unit (ij, g) reads the c input rows of block
// (i, j) = (ij / d, ij % d), pieces g*QN .. g*QN+QN-1 (4 columns each), and
// writes the block's b output rows (Section 4.1 index sets:
// inputs i*c*d + l*d + j, outputs i*b*d + k*d + j).  The block's values come
// from the LDS copy kbuf (packed like K_values).  BB x CC is the block shape
// when EXACT, else an upper bound (b, c read at run time).
template <int BB, int CC, int QN, bool EXACT>
__device__ __forceinline__ void fused_factor(const FusedChain& fc, int f, const float* src, float* dst,
                                             const float* kbuf) {
  const int b = EXACT ? BB : fc.b[f], c = EXACT ? CC : fc.c[f], d = fc.d[f];
  constexpr int G = 4 / QN;
  const int units = fc.a[f] * d * G;
  for (int u = threadIdx.x; u < units; u += kFusedThreads) {
    int i, j, g;
    fused_unit(fc, f, G, u, &i, &j, &g);
    const float* blk = kbuf + (i * d + j) * b * c;
    f32x4 xin[CC][QN];
#pragma unroll
    for (int l = 0; l < CC; ++l) {
      if (EXACT || l < c) {
        const float* row = src + fused_in_row(fc, f, i, j, l) * kFusedPitch + g * QN * 4;
#pragma unroll
        for (int q = 0; q < QN; ++q) xin[l][q] = *reinterpret_cast<const f32x4*>(row + 4 * q);
      }
    }
#pragma unroll
    for (int k = 0; k < BB; ++k) {
      if (EXACT || k < b) {
        f32x4 acc[QN];
#pragma unroll
        for (int q = 0; q < QN; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int l = 0; l < CC; ++l) {
          if (EXACT || l < c) {
            const float kk = blk[k * c + l];
#pragma unroll
            for (int q = 0; q < QN; ++q) {
              acc[q][0] = __builtin_fmaf(kk, xin[l][q][0], acc[q][0]);
              acc[q][1] = __builtin_fmaf(kk, xin[l][q][1], acc[q][1]);
              acc[q][2] = __builtin_fmaf(kk, xin[l][q][2], acc[q][2]);
              acc[q][3] = __builtin_fmaf(kk, xin[l][q][3], acc[q][3]);
            }
          }
        }
        float* row = dst + fused_out_row(fc, f, i, j, k) * kFusedPitch + g * QN * 4;
#pragma unroll
        for (int q = 0; q < QN; ++q) *reinterpret_cast<f32x4*>(row + 4 * q) = acc[q];
      }
    }
  }
}

// Factor f with the instance for its block shape (exact 2x2, 4x4, 8x8, else
// bounded by the larger of b and c); fused_pieces() gives the QN the host
// replay assumes.
__device__ __forceinline__ void fused_apply(const FusedChain& fc, int f, const float* src, float* dst,
                                            const float* kbuf) {
  const int b = fc.b[f], c = fc.c[f], m = b > c ? b : c;
  if (b == 2 && c == 2) fused_factor<2, 2, 2, true>(fc, f, src, dst, kbuf);
  else if (b == 4 && c == 4) fused_factor<4, 4, 1, true>(fc, f, src, dst, kbuf);
  else if (b == 8 && c == 8) fused_factor<8, 8, 1, true>(fc, f, src, dst, kbuf);
  else if (m <= 2) fused_factor<2, 2, 2, false>(fc, f, src, dst, kbuf);
  else if (m <= 4) fused_factor<4, 4, 1, false>(fc, f, src, dst, kbuf);
  else fused_factor<8, 8, 1, false>(fc, f, src, dst, kbuf);
}

// Radix pass with its instance (group size P, radix p).
__device__ __forceinline__ void fused_radix_apply(const FusedChain& fc, int q, float* buf, const float* kbuf) {
  const int P = fc.pP[q], p = fc.pp[q];
  if (p == 2) {
    if (P == 8) fused_radix_pass<8, 2>(fc, q, buf, kbuf);
    else if (P == 4) fused_radix_pass<4, 2>(fc, q, buf, kbuf);
    else fused_radix_pass<2, 2>(fc, q, buf, kbuf);
  } else if (p == 4) {
    fused_radix_pass<4, 4>(fc, q, buf, kbuf);
  } else {
    fused_radix_pass<8, 8>(fc, q, buf, kbuf);
  }
}

template <typename T, int LAYOUT, bool VEC>
__global__ __launch_bounds__(kFusedThreads) void ks_chain_fused_kernel(FusedChain fc) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int col0 = fused_tile((int)blockIdx.x, (int)gridDim.x) * kFusedCols;
  // src holds the current vector; single-factor passes with b != c write dst
  float* src = lds;
  float* dst = fc.inplace ? lds : lds + fc.buf_rows * kFusedPitch;
  float* kbuf = lds + fused_kbuf_offset(fc);
  FusedK<T> kr;
  kr.fetch(fc, 0);
  fused_load<T, LAYOUT, VEC>(fc, src, col0);
  kr.park(fc, 0, kbuf);
  __syncthreads();
  for (int q = 0; q < fc.npass; ++q) {
    const bool more = q + 1 < fc.npass;
    if (more) kr.fetch(fc, q + 1);  // in flight during this pass
    if (fused_is_radix(fc, q)) {
      fused_radix_apply(fc, q, src, kbuf);
    } else {
      fused_apply(fc, fc.pf0[q], src, dst, kbuf);
      if (!fc.inplace) {
        float* t = src;
        src = dst;
        dst = t;
      }
    }
    __syncthreads();
    if (more) {
      kr.park(fc, q + 1, kbuf);
      __syncthreads();
    }
  }
  fused_store<T, LAYOUT, VEC>(fc, src, col0);
}

template <typename T>
hipError_t launch_fused_t(const FusedChain& fc, bool vec, hipStream_t s) {
  const dim3 grid((fc.batch + kFusedCols - 1) / kFusedCols), block(kFusedThreads);
  const int lds = fused_lds_bytes(fc);
#define KS_FUSED_LAUNCH(L, V)                                                                                 \
  {                                                                                                          \
    if (lds > 64 * 1024) {                                                                                   \
      static const hipError_t raised = hipFuncSetAttribute(                                                  \
          reinterpret_cast<const void*>(&ks_chain_fused_kernel<T, L, V>),                                    \
          hipFuncAttributeMaxDynamicSharedMemorySize, kFusedMaxLds);                                         \
      if (raised != hipSuccess) return raised;                                                               \
    }                                                                                                        \
    hipLaunchKernelGGL((ks_chain_fused_kernel<T, L, V>), grid, block, lds, s, fc);                           \
    return hipGetLastError();                                                                                \
  }
  if (fc.layout == BSL) {
    if (vec) KS_FUSED_LAUNCH(BSL, true) else KS_FUSED_LAUNCH(BSL, false)
  }
  if (vec) KS_FUSED_LAUNCH(BSF, true) else KS_FUSED_LAUNCH(BSF, false)
#undef KS_FUSED_LAUNCH
}

}  // namespace

hipError_t launch_chain_mfma(const FusedChain& fc, int dtype, bool vec, hipStream_t s);
hipError_t launch_chain_bfly(const FusedChain& fc, int dtype, bool vec, hipStream_t s);

hipError_t launch_chain_fused(const FusedChain& fc, int dtype, bool vec, hipStream_t s) {
  if (fc.mfma) return launch_chain_mfma(fc, dtype, vec, s);
  if (fc.bfly) return launch_chain_bfly(fc, dtype, vec, s);
  switch (dtype) {
    case F32: return launch_fused_t<float>(fc, vec, s);
    case BF16: return launch_fused_t<bf16_t>(fc, vec, s);
    case F16: return launch_fused_t<_Float16>(fc, vec, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ks
