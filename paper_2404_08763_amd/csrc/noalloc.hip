// CATS MLP forward for callers that cannot allocate device memory (code
// under graph capture, tight serving loops, harnesses that forbid
// hipMalloc): the same kernels as cats_mlp_forward, with the workspace taken
// from a fixed device array that the library holds on every GPU it runs on.
//
// The array lives in this translation unit.  Its name is a host-side
// stand-in in host code, so its device address is looked up once per device
// (with that device current) and only that address is ever handed to a
// kernel.
#include <hip/hip_runtime.h>

#include <mutex>

#include "cats.h"

namespace cats {
// records the message returned by cats_last_error() and returns st
cats_status report_error(cats_status st, const char* msg);
}  // namespace cats

namespace {

__device__ __align__(256) unsigned char scratch[CATS_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

struct ScratchTable {
  std::mutex mu;
  void* ptr[kMaxDevices] = {};
};

ScratchTable& table() {
  static ScratchTable* t = new ScratchTable();  // lives until process exit
  return *t;
}

}  // namespace

extern "C" cats_status cats_mlp_forward_noalloc(const cats_layer* layer, const float* x, int32_t B, float t,
                                                const float* residual, float* y, const cats_forward_aux* aux,
                                                void* stream) {
  if (!layer) return cats::report_error(CATS_ERR_NULL, "layer is NULL");
  // the size rule of the allocating entry point; a call that needs more
  // than the fixed array is rejected before any device work
  const size_t need = cats_workspace_bytes(layer->d, layer->m, B, 0);
  if (need == 0) return cats_mlp_forward(layer, x, B, t, residual, y, aux, nullptr, 0, stream);  // its shape error
  if (need > CATS_NOALLOC_SCRATCH_BYTES)
    return cats::report_error(CATS_ERR_WORKSPACE,
                              "this block and batch need more scratch memory than the fixed "
                              "CATS_NOALLOC_SCRATCH_BYTES array; use cats_mlp_forward with a workspace");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return cats::report_error(CATS_ERR_HIP, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return cats::report_error(CATS_ERR_RANGE, "device ordinal out of range");
  void* p = nullptr;
  {
    ScratchTable& T = table();
    std::lock_guard<std::mutex> lk(T.mu);
    if (!T.ptr[dev]) {
      // this device's copy of the array (set-up on the first call on the
      // device, which is current)
      void* q = nullptr;
      e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return cats::report_error(CATS_ERR_HIP, hipGetErrorString(e));
      if (!q) return cats::report_error(CATS_ERR_HIP, "no device address for the scratch array");
      T.ptr[dev] = q;
    }
    p = T.ptr[dev];
  }
  return cats_mlp_forward(layer, x, B, t, residual, y, aux, p, CATS_NOALLOC_SCRATCH_BYTES, stream);
}
