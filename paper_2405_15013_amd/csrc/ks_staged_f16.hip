// Instances of the LDS-staged MFMA kernels (ks_staged.h) for _Float16 storage.
// One file per storage type so the instances compile in parallel.
#include "ks_staged.h"

namespace ks {

hipError_t launch_staged_f16(const Problem& p, const StagedTile& t, int V, bool strided, int mt, int cps,
                            hipStream_t s) {
  return launch_staged_type<_Float16>(p, t, V, strided, mt, cps, s);
}

}  // namespace ks
