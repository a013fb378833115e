// e2ttt_chunk_forward_static (include/e2ttt.h): the forward without
// save_for_backward on a workspace the library owns, for callers that cannot
// allocate device memory.
//
// The workspace is a file-scope device array.  In host code its name stands
// for a host-side shadow, not a device address, so it is never passed to a
// kernel or a copy: the first call on a device (with that device current)
// looks up the device address of that GPU's copy with hipGetSymbolAddress and
// keeps it, and every call uses the kept address.  Every GPU the library runs
// on holds its own copy until the process ends.  The forward writes every
// word of the workspace it reads (scalar kernels, carries, the exchange slots)
// and clears the exchange's sync words with a kernel at the start of each
// call, so a call needs nothing cleared from the previous one.  Calls that
// overlap on one GPU share the array and race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "e2ttt.h"

static __device__ __align__(256) unsigned char scratch[E2TTT_STATIC_WORKSPACE_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of the current GPU's copy of `scratch`, or nullptr.
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}

}  // namespace

extern "C" e2ttt_status e2ttt_chunk_forward_static(const e2ttt_desc* desc, const void* q,
                                                   const void* k, const void* v, const float* eta,
                                                   const float* beta, const float* gamma,
                                                   const float* w_in, const float* m_in, void* out,
                                                   float* w_out, float* m_out, void* stream) {
  if (!desc) return E2TTT_ERR_NULL_ARG;
  const size_t need = e2ttt_workspace_bytes(desc, 0);
  if (need == 0)   // a bad descriptor: the forward reports which check failed
    return e2ttt_chunk_forward(desc, q, k, v, eta, beta, gamma, w_in, m_in, out, w_out, m_out,
                               nullptr, 0, 0, stream);
  if (need > E2TTT_STATIC_WORKSPACE_BYTES) return E2TTT_ERR_WORKSPACE_TOO_SMALL;
  void* ws = scratch_on_current_device();
  if (!ws) return E2TTT_ERR_HIP;
  return e2ttt_chunk_forward(desc, q, k, v, eta, beta, gamma, w_in, m_in, out, w_out, m_out, ws,
                             E2TTT_STATIC_WORKSPACE_BYTES, 0, stream);
}
