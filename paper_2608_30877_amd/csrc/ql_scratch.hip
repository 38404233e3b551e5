// Allocation-free variant of the stack entry point, for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid hipMalloc).  The stack's workspace lives in a
// file-scope device array of fixed size instead of a caller buffer.
//
// Each GPU the library runs on holds its own copy of `scratch` (allocated
// with the code object, kept until the process ends).  In host code the
// array's name is only a host-side stand-in, so its device address is
// looked up once per device with hipGetSymbolAddress, with that device
// current, and only that address is ever handed to kernels.
//
// Every call on one GPU shares that GPU's array and leaves its contents
// behind.  No part of it needs to start at zero: everything a call reads for
// its real rows is written earlier in the same call (padding rows of a tile
// may read stale values, which never reach a stored row).  Calls that
// overlap on one GPU -- on different streams, or from different host
// threads -- race on the array.
#include <mutex>

#include "../../include/qlinear.h"
#include "ql_internal.h"

static constexpr size_t kScratchBytes = (size_t)128 << 20;   // 128 MiB per device

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;

std::once_flag g_once[kMaxDevices];
void* g_addr[kMaxDevices];
hipError_t g_err[kMaxDevices];

// device address of `scratch` on the current device
int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return QL_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return QL_ERR_UNSUPPORTED;
  std::call_once(g_once[dev], [dev]() {
    void* p = nullptr;
    g_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_addr[dev] = g_err[dev] == hipSuccess ? p : nullptr;
  });
  if (g_err[dev] != hipSuccess || !g_addr[dev]) return QL_ERR_HIP;
  *out = g_addr[dev];
  return QL_OK;
}

}  // namespace

extern "C" {

size_t qlayer_stack_scratch_capacity(void) { return kScratchBytes; }

int qlayer_stack_forward_noalloc(const ql_layer* layers, int32_t n_layers, float* h, int64_t M,
                                 int64_t d, int64_t d_ff, int32_t group, float eps,
                                 ql_stream_t stream) {
  const size_t need = qlayer_stack_workspace_bytes(M, d, d_ff, group);
  if (need == 0) return group != 128 ? QL_ERR_UNSUPPORTED : QL_ERR_ARG;  // invalid shape
  if (need > kScratchBytes) return QL_ERR_SCRATCH;
  void* ws = nullptr;
  const int rc = scratch_address(&ws);
  if (rc) return rc;
  return qlayer_stack_forward(layers, n_layers, h, M, d, d_ff, group, eps, ws, kScratchBytes,
                              stream);
}

}  // extern "C"
