// Output epilogue shared by every kernel: Y = act(X K^T + bias), for the
// KS layers of a Transformer MLP (paper appendix, ViT-S/16 submodule table:
// "Linear + bias" rows, and the feed-forward block Linear + GELU).  bias holds
// one value per output feature m (the column of Y in BSF, its row in BSL) in
// the storage type; act is KS_ACT_NONE or KS_ACT_GELU (the exact form
// x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2))).  Both are wave-uniform launch
// arguments: a plain ks_matmul pays one untaken branch per output.
#pragma once
#include "ks_common.h"
#include "ks_internal.h"

namespace ks {

__device__ __forceinline__ bool epilogue_on(const Problem& p) { return p.bias != nullptr || p.act != 0; }

template <typename T>
__device__ __forceinline__ float epilogue_apply(const Problem& p, float v, int m) {
  if (p.bias != nullptr) v += to_f32(static_cast<const T*>(p.bias)[m]);
  if (p.act == 1) v = 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
  return v;
}

}  // namespace ks
