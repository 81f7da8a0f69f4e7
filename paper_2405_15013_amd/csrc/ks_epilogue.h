// Output epilogue shared by every kernel: Y = act(X K^T + bias), for the
// KS layers of a Transformer MLP (paper appendix, ViT-S/16 submodule table:
// "Linear + bias" rows, and the feed-forward block Linear + GELU).  bias holds
// one value per output feature m (the column of Y in BSF, its row in BSL) in
// the storage type; act is KS_ACT_NONE or KS_ACT_GELU (the exact form
// x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2))).  Both are wave-uniform launch
// arguments.  The kernels test them once per tile, not per output: the bias
// of all of a lane's outputs is loaded in one batch, then added, then the
// activation runs over the whole register tile, so a plain ks_matmul pays two
// untaken scalar branches.
#pragma once
#include "ks_common.h"
#include "ks_internal.h"

namespace ks {

constexpr int kActGelu = 1;  // KS_ACT_GELU

__device__ __forceinline__ bool epilogue_on(const Problem& p) { return p.bias != nullptr || p.act != 0; }
__device__ __forceinline__ bool epilogue_gelu(const Problem& p) { return p.act == kActGelu; }

template <typename T>
__device__ __forceinline__ float bias_value(const Problem& p, int64_t m) {
  return to_f32(static_cast<const T*>(p.bias)[m]);
}

// Monomial coefficients of R(u), written by gelu_fit.py (Chebyshev fit of
// degree 9; |R_fit - R| <= 1.3e-7 in log2 units, i.e. a relative error of
// 9e-8 in the normal tail below, for |x| <= 16).
constexpr float kGeluR0 = -1.82569253f;
constexpr float kGeluR1 = 2.88297439f;
constexpr float kGeluR2 = 2.20453787f;
constexpr float kGeluR3 = 0.657676935f;
constexpr float kGeluR4 = -1.50583696f;
constexpr float kGeluR5 = 2.12293911f;
constexpr float kGeluR6 = -78.4830017f;
constexpr float kGeluR7 = 235.065887f;
constexpr float kGeluR8 = -269.774841f;
constexpr float kGeluR9 = 113.810883f;

// Degree 5 (gelu_fit.py, same fit): |R_fit - R| <= 1.2e-5 in log2 units, a
// relative error of 8e-6 in the tail, far below the precision of 16-bit
// outputs (bf16 2^-8, fp16 2^-11); used when the result is stored in 16 bits.
constexpr float kGeluS0 = -1.82723665f;
constexpr float kGeluS1 = 2.93737769f;
constexpr float kGeluS2 = 1.46866286f;
constexpr float kGeluS3 = 5.47383213f;
constexpr float kGeluS4 = -16.3639202f;
constexpr float kGeluS5 = 10.5570784f;

// Exact GELU without branches.  With z = |x| / sqrt 2 and u = 1 / (2 + z),
// the normal tail is Phi(-|x|) = erfc(z) / 2 = u * 2^(-log2(e) x^2 / 2 + R(u))
// where R(u) = log2(exp(z^2) erfc(z) / (2u)) is smooth on (0, 1/2] (fitted
// above).  Since Phi(x) = 1 - Phi(-x), both signs reduce to
// GELU(x) = max(x, 0) - |x| Phi(-|x|).  The tail keeps its relative accuracy
// (no 1 + erf cancellation); x is clamped to [-16, 16] for the tail only,
// where Phi(-16) already underflows, so GELU(+inf) = +inf and GELU(-inf) = -0.
// Cost: 16 VALU operations, one v_rcp_f32 and one v_exp_f32 (12 VALU with
// the degree-5 R for 16-bit outputs, OUT the type the result is stored in).
template <typename OUT = float>
__device__ __forceinline__ float gelu_f32(float x) {
  const float xc = __builtin_amdgcn_fmed3f(x, -16.0f, 16.0f);
  const float ax = __builtin_fabsf(xc);
  const float u = __builtin_amdgcn_rcpf(__builtin_fmaf(ax, 0.70710678118654752f, 2.0f));
  float r;
  if constexpr (sizeof(OUT) == 4) {
    r = kGeluR9;
    r = __builtin_fmaf(r, u, kGeluR8);
    r = __builtin_fmaf(r, u, kGeluR7);
    r = __builtin_fmaf(r, u, kGeluR6);
    r = __builtin_fmaf(r, u, kGeluR5);
    r = __builtin_fmaf(r, u, kGeluR4);
    r = __builtin_fmaf(r, u, kGeluR3);
    r = __builtin_fmaf(r, u, kGeluR2);
    r = __builtin_fmaf(r, u, kGeluR1);
    r = __builtin_fmaf(r, u, kGeluR0);
  } else {
    r = kGeluS5;
    r = __builtin_fmaf(r, u, kGeluS4);
    r = __builtin_fmaf(r, u, kGeluS3);
    r = __builtin_fmaf(r, u, kGeluS2);
    r = __builtin_fmaf(r, u, kGeluS1);
    r = __builtin_fmaf(r, u, kGeluS0);
  }
  // -log2(e)/2 * x^2 + R(u)
  const float t = __builtin_fmaf(xc * -0.72134752044448170f, xc, r);
  const float tail = u * __builtin_amdgcn_exp2f(t);
  return __builtin_fmaf(-ax, tail, __builtin_fmaxf(x, 0.0f));
}

// Single-output form (bias index m), for kernels with one output per thread.
template <typename T>
__device__ __forceinline__ float epilogue_apply(const Problem& p, float v, int64_t m) {
  if (p.bias != nullptr) v += bias_value<T>(p, m);
  if (epilogue_gelu(p)) v = gelu_f32<T>(v);
  return v;
}

}  // namespace ks
