// The entry point that allocates nothing: ckm_round_eval_noalloc runs the
// rounding path of ckm_round_eval_async with its work buffer in a static
// device array instead of a caller buffer. The array lives in this file; so
// does the lookup of its device address, since in host code the array's
// name is only a host-side stand-in for it.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <mutex>

#include "ckm_internal.h"

namespace {

// The work area, one copy per device the library runs on, held until the
// process ends. Every call on a device shares it (see ckm.h).
__device__ __align__(256) unsigned char scratch[CKM_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

namespace ckm {

// Resolves the device address of `scratch` on `device`, which must be the
// current device. Called once per device by graph creation (the library's
// set-up call); later calls only read the kept address.
hipError_t noalloc_setup(int device) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_scratch_ptr[device]) return hipSuccess;
  void* ptr = nullptr;
  const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!ptr) return hipErrorInvalidSymbol;
  g_scratch_ptr[device] = ptr;
  return hipSuccess;
}

void* noalloc_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_mu);
  return g_scratch_ptr[device];
}

}  // namespace ckm

extern "C" ckm_status ckm_round_eval_noalloc(const ckm_graph* g, const double* d_s_frac, int64_t ld, int32_t K,
                                             uint64_t seed, int64_t budget, uint32_t flags, int64_t* d_peak,
                                             int64_t* d_cost, uint8_t* d_feasible, int32_t* d_best_k,
                                             uint64_t* d_best_S, uint64_t* d_best_R, int32_t* d_status,
                                             void* stream) {
  if (!g) return ckm::set_error(CKM_E_INVALID_ARG, "graph is NULL");
  if (K < 1) return ckm::set_error(CKM_E_INVALID_ARG, "K = %d < 1", K);
  if (K > CKM_MAX_CANDIDATES) return ckm::set_error(CKM_E_UNSUPPORTED, "K = %d > %d", K, CKM_MAX_CANDIDATES);
  const ckm::Layout L = ckm::make_layout(g->n, K);
  if (L.total > CKM_NOALLOC_SCRATCH_BYTES)
    return ckm::set_error(CKM_E_UNSUPPORTED, "n = %d, K = %d needs %zu bytes of work area, more than the %zu held",
                          g->n, K, L.total, (size_t)CKM_NOALLOC_SCRATCH_BYTES);
  void* work = ckm::noalloc_scratch(g->device);
  if (!work)
    return ckm::set_error(CKM_E_DEVICE, "no work area resolved for device %d", g->device);
  // The area is passed as an ordinary work buffer of its full size: the row
  // arrays are used when they fit in it, and every stage initializes what it
  // reads, so nothing carried over from an earlier call is read.
  // Every launch goes on the caller's stream (no side stream).
  return ckm::round_eval(g, d_s_frac, ld, K, seed, budget, flags, d_peak, d_cost, d_feasible, d_best_k, d_best_S,
                         d_best_R, d_status, work, CKM_NOALLOC_SCRATCH_BYTES, stream, false);
}
