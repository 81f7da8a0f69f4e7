// Instances of the batch-size-last LDS-DMA MFMA kernel (ks_dma_bsl.h) for _Float16 storage.
#include "ks_dma_bsl.h"

namespace ks {

hipError_t launch_dma_bsl_f16(const Problem& p, const StagedTile& t, int mt, hipStream_t s) {
  return launch_dma_bsl_t<_Float16>(p, t, mt, s);
}

}  // namespace ks
