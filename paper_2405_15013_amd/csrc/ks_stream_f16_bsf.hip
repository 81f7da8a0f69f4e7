// Instances of the streaming MFMA kernels (ks_stream.h) for _Float16 storage,
// BSF layout.  One file per storage type and layout so the instances
// compile in parallel.
#include "ks_stream.h"

namespace ks {

hipError_t launch_stream_f16_bsf(const Problem& p, const StreamTile& t, int V, bool strided, int mt, unsigned grid,
                                   hipStream_t s) {
  return launch_stream_layout<_Float16, BSF>(p, t, V, strided, mt, grid, s);
}

}  // namespace ks
