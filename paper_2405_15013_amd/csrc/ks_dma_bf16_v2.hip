// Instances of the LDS-DMA MFMA kernel (ks_dma.h) for bf16_t storage, d == 2.
#include "ks_dma.h"

namespace ks {

hipError_t launch_dma_bf16_v2(const Problem& p, const StagedTile& t, int mt, int lp, hipStream_t s) {
  return launch_dma_mode<bf16_t, 2, false>(p, t, mt, lp, s);
}

}  // namespace ks
