// Instances of the LDS-staged MFMA kernels (ks_staged.h) for bf16_t storage.
// One file per storage type so the instances compile in parallel.
#include "ks_staged.h"

namespace ks {

hipError_t launch_staged_bf16(const Problem& p, const StagedTile& t, int V, bool strided, int mt, int cps,
                            hipStream_t s) {
  return launch_staged_type<bf16_t>(p, t, V, strided, mt, cps, s);
}

}  // namespace ks
