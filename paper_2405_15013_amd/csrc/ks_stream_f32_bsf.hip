// Instances of the streaming MFMA kernels (ks_stream.h) for float storage,
// BSF layout.  One file per storage type and layout so the instances
// compile in parallel.
#include "ks_stream.h"

namespace ks {

hipError_t launch_stream_f32_bsf(const Problem& p, const StreamTile& t, int V, bool strided, int mt, unsigned grid,
                                   hipStream_t s) {
  return launch_stream_layout<float, BSF>(p, t, V, strided, mt, grid, s);
}

}  // namespace ks
