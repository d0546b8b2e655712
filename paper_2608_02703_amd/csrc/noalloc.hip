// archead_logits_noalloc: archead_logits for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid allocation).  The call's workspace is a fixed
// device array of this library, so the call itself allocates nothing.
//
// The array is a file-scope __device__ object: in host code its name is a
// host-side stand-in, not a device address.  Its device address is taken
// once per device with hipGetSymbolAddress, with that device current, when
// the first handle is created on it (archead_create calls scratch_setup), and
// only that address is passed to kernels.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "archead.h"
#include "internal.h"

namespace {

constexpr int kMaxDevices = 64;

// The static workspace: ARCHEAD_NOALLOC_SCRATCH_BYTES on every device the
// library runs on, held until the process ends.
static __device__ __align__(256) unsigned char scratch[ARCHEAD_NOALLOC_SCRATCH_BYTES];

std::mutex g_mu;
void* g_scratch[kMaxDevices];   // device address of `scratch` per device, or null

}  // namespace

namespace archead {

archead_status scratch_setup(int device) {
  if (device < 0 || device >= kMaxDevices)
    return fail(ARCHEAD_E_UNSUPPORTED, "device index %d out of range", device);
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_scratch[device]) return ARCHEAD_OK;
  void* p = nullptr;
  hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !p)
    return fail(ARCHEAD_E_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
  g_scratch[device] = p;
  return ARCHEAD_OK;
}

}  // namespace archead

using namespace archead;

extern "C" {

archead_status archead_logits_noalloc(const archead_handle* h, const void* x, int64_t M,
                                      int64_t ldx, void* out, archead_dtype out_dtype,
                                      int64_t ldo, void* stream) {
  clear_error();
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "handle is NULL");
  if (M < 0) return fail(ARCHEAD_E_INVALID_ARG, "M = %lld < 0", (long long)M);
  if (M == 0) return ARCHEAD_OK;
  const size_t need = archead_workspace_bytes(h, M, ARCHEAD_OP_LOGITS);
  if (need > size_t(ARCHEAD_NOALLOC_SCRATCH_BYTES))
    return fail(ARCHEAD_E_WORKSPACE,
                "M = %lld needs %zu bytes of workspace; the static workspace holds %zu "
                "(use archead_logits with a caller workspace)",
                (long long)M, need, size_t(ARCHEAD_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    if (h->device >= 0 && h->device < kMaxDevices) ws = g_scratch[h->device];
  }
  if (!ws) return fail(ARCHEAD_E_HIP, "static workspace of device %d is not set up", h->device);
  return archead_logits(h, x, M, ldx, out, out_dtype, ldo, ws,
                        size_t(ARCHEAD_NOALLOC_SCRATCH_BYTES), stream);
}

}  // extern "C"
