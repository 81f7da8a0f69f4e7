// Work decomposition of the streaming MFMA kernels (ks_stream.h), shared by
// the kernels and by the host-side plan verifier (ks_plan_verify).
//
// The batch tiles of all segments (i, j or j-group, k-group) form one
// flattened sequence, k-group fastest (the k-groups of a tile read the same X
// back to back), then the batch tile (the next tile of a segment reads the
// neighbouring runs of the same rows of X and Y and the same packed K rows),
// then j, then i.  The nwaves wavefronts of a launch (one resident round)
// take equal contiguous shares of it, so they finish together.  Each tile is
// a work item of the register-direct kernels (ks_direct_index.h: 16*V batch
// entries in BSL, 16 batch rows in BSF, 16*MT output rows k), and its outputs
// are written once (paper Section 4.1, Algorithm 2).
#pragma once
#include "ks_direct_index.h"

namespace ks {

struct StreamTile {
  int kgroups;  // b / (16*MT)
  int jgroups;  // BSL: d; BSF: d / V
  int nbt;      // batch tiles
  int tiles;    // kgroups * nbt * jgroups * a
  int nwaves;   // wavefronts of the launch (<= tiles)
  int waves;    // wavefronts per workgroup
};

// Share [first, first + count) of the flattened tiles for wavefront w.
KS_HD void stream_share(const StreamTile& t, int w, int* first, int* count) {
  const int64_t a = (int64_t)w * t.tiles / t.nwaves, b = (int64_t)(w + 1) * t.tiles / t.nwaves;
  *first = (int)a;
  *count = (int)(b - a);
}

// Work item of flattened tile f.
KS_HD DItem stream_item(const Problem& p, const StreamTile& t, int V, int MT, int f) {
  DItem it;
  int rest = f;
  const int kg = rest % t.kgroups;
  rest /= t.kgroups;
  const int bt = rest % t.nbt;
  rest /= t.nbt;
  const int jg = rest % t.jgroups;
  it.i = rest / t.jgroups;
  it.k0 = kg * 16 * MT;
  if (p.layout == BSL) {
    it.j0 = jg;
    it.beta0 = bt * 16 * V;
  } else {
    it.j0 = jg * V;
    it.beta0 = bt * 16;
  }
  return it;
}

}  // namespace ks
