// MFMA block-GEMM kernel (placeholder until the tiled kernel lands).
#include "ks_internal.h"
namespace ks {
bool plan_mfma_impl(const Problem&, bool, Plan*) { return false; }
hipError_t launch_mfma(const Problem&, const Plan&, hipStream_t) { return hipErrorInvalidValue; }
}  // namespace ks
