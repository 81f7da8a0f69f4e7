// Instances of the LDS-DMA MFMA kernel (ks_dma.h) for _Float16 storage, d == 1.
#include "ks_dma.h"

namespace ks {

hipError_t launch_dma_f16_v1(const Problem& p, const StagedTile& t, int mt, int lp, hipStream_t s) {
  return launch_dma_mode<_Float16, 1, false>(p, t, mt, lp, s);
}

}  // namespace ks
