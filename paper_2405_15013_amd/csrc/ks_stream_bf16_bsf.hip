// Instances of the streaming MFMA kernels (ks_stream.h) for bf16_t storage,
// BSF layout.  One file per storage type and layout so the instances
// compile in parallel.
#include "ks_stream.h"

namespace ks {

hipError_t launch_stream_bf16_bsf(const Problem& p, const StreamTile& t, int V, bool strided, int mt, unsigned grid,
                                   hipStream_t s) {
  return launch_stream_layout<bf16_t, BSF>(p, t, V, strided, mt, grid, s);
}

}  // namespace ks
