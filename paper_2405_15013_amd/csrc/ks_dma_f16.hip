// Instances of the LDS-DMA MFMA kernels (ks_dma.h) for _Float16 storage.
// One file per storage type so the instances compile in parallel.
#include "ks_dma.h"

namespace ks {

hipError_t launch_dma_f16(const Problem& p, const StagedTile& t, bool strided, int mt, int lp, hipStream_t s) {
  return launch_dma_type<_Float16>(p, t, strided, mt, lp, s);
}

}  // namespace ks
