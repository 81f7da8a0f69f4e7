// Instances of the batch-size-last LDS-DMA MFMA kernel (ks_dma_bsl.h) for bf16_t storage.
#include "ks_dma_bsl.h"

namespace ks {

hipError_t launch_dma_bsl_bf16(const Problem& p, const StagedTile& t, int mt, hipStream_t s) {
  return launch_dma_bsl_t<bf16_t>(p, t, mt, s);
}

}  // namespace ks
