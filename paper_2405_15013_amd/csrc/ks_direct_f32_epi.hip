// Instances of the register-direct MFMA kernels (ks_direct.h) for float storage
// with the bias / activation epilogue compiled in (ks_matmul_bias_act); a file
// of its own so they compile in parallel with the plain instances.
#include "ks_direct.h"

namespace ks {

hipError_t launch_direct_f32_epi(const Problem& p, const DirectTile& t, int V, bool strided, int mt, unsigned grid,
                                hipStream_t s) {
  return launch_direct_type<float, true>(p, t, V, strided, mt, grid, s);
}

}  // namespace ks
