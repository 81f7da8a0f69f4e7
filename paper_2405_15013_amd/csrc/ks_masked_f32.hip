// Instances of the masked register-direct MFMA kernel (ks_masked.h) for one
// storage type (one file per type so the instances compile in parallel).
#include "ks_masked.h"

namespace ks {

hipError_t launch_masked_f32(const Problem& p, const MaskedTile& t, int V, unsigned grid, hipStream_t s) {
  return launch_masked_type<float>(p, t, V, grid, s);
}

}  // namespace ks
