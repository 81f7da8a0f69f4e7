// ks_chain_noalloc: the chain driver of ks_chain with its intermediates in a
// fixed device array of this library instead of a caller workspace, for
// callers that cannot allocate device memory (code under stream capture,
// serving loops, harnesses that forbid allocation).
//
// The array lives in the library's code object: one copy per GPU, allocated
// by the HIP runtime when the code object is loaded on that GPU and held until
// the process ends.  Host code never uses the array's name as an address (on
// the host it names a stand-in, not device memory): the device address of each
// GPU's copy is looked up once per device with hipGetSymbolAddress, with that
// device current, and kept in a per-device table.
//
// Every call on one GPU uses that GPU's copy, so calls that overlap in time on
// one GPU (several streams or threads at once) race on the intermediates;
// stream-ordered calls do not.  The intermediates are fully overwritten by
// each factor, so nothing needs clearing between calls.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/ks.h"

namespace ks {
ks_status_t chain_impl(const ks_factor_t* factors, int nfactors, const void* X, void* Y, int64_t batch, int layout,
                       int dtype, void* workspace, size_t workspace_bytes, void* stream);
void set_last_hip_error(int e);
}

namespace {

constexpr size_t kScratchBytes = KS_CHAIN_NOALLOC_MAX_WORKSPACE;  // 64 MiB per GPU
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current GPU's copy of the scratch array, looked up on
// the first call on that GPU.
hipError_t scratch_for_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

size_t ks_chain_noalloc_max_workspace(void) { return kScratchBytes; }

ks_status_t ks_chain_noalloc(const ks_factor_t* factors, int nfactors, const void* X, void* Y, int64_t batch,
                             int layout, int dtype, void* stream) {
  // The workspace this chain needs (0 for one factor, or for arguments that
  // ks_chain rejects, which chain_impl then reports) must fit the array.
  const size_t need = ks_chain_workspace_bytes(factors, nfactors, batch, dtype);
  if (need > kScratchBytes) return KS_ERR_SCRATCH_LIMIT;
  void* ws = nullptr;
  if (need > 0 && batch > 0) {
    const hipError_t e = scratch_for_current_device(&ws);
    if (e != hipSuccess) {
      ks::set_last_hip_error((int)e);
      return KS_ERR_HIP;
    }
  }
  return ks::chain_impl(factors, nfactors, X, Y, batch, layout, dtype, ws, ws ? kScratchBytes : 0, stream);
}

}  // extern "C"
