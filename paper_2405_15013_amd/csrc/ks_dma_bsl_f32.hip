// Instances of the batch-size-last LDS-DMA MFMA kernel (ks_dma_bsl.h) for float storage.
#include "ks_dma_bsl.h"

namespace ks {

hipError_t launch_dma_bsl_f32(const Problem& p, const StagedTile& t, int mt, hipStream_t s) {
  return launch_dma_bsl_t<float>(p, t, mt, s);
}

}  // namespace ks
