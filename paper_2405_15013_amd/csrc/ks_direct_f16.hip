// Instances of the register-direct MFMA kernels (ks_direct.h) for _Float16 storage.
// One file per storage type so the instances compile in parallel.
#include "ks_direct.h"

namespace ks {

hipError_t launch_direct_f16(const Problem& p, const DirectTile& t, int V, bool strided, int mt, unsigned grid,
                            hipStream_t s) {
  return launch_direct_type<_Float16, false>(p, t, V, strided, mt, grid, s);
}

}  // namespace ks
