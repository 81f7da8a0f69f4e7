// Instances of the LDS-staged MFMA kernels (ks_staged.h) for float storage.
// One file per storage type so the instances compile in parallel.
#include "ks_staged.h"

namespace ks {

hipError_t launch_staged_f32(const Problem& p, const StagedTile& t, int V, bool strided, int mt, int cps,
                            hipStream_t s) {
  return launch_staged_type<float>(p, t, V, strided, mt, cps, s);
}

}  // namespace ks
