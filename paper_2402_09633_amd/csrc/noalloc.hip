// Scratch memory of the no-allocation entry point (gnn_infer_noalloc).
//
// Callers that may not allocate device memory (code under stream capture,
// tight serving loops) run the inference in one fixed array of this file
// instead of the handle's workspace cache.  The array is a file-scope device
// variable: each GPU that loads this file's code object holds its own copy
// until the process ends, at its own address.  Its address is looked up once
// per device with hipGetSymbolAddress (the array's name in host code is not a
// device address) and kept here; the kernels receive that address as their
// workspace argument, exactly as they receive a cached workspace.
//
// Every call on one device shares the array and finds the previous call's
// contents in it.  The inference path never reads workspace memory it has
// not written in the same call (its counters and flags are cleared by fill
// kernels), so stale contents do no harm; calls that overlap on one device
// race on the array.
#include <mutex>
#include <string>

#include "../../include/gnn.h"
#include "gnn_internal.h"

namespace gnn {
namespace {

// 512 MiB: events up to about 50k hits and 330k edges at H = 128 in fp32
// (workspace 378 MB; 255 MB in bf16).  The host side keeps a shadow of
// every device variable at full size (address space only, never touched),
// which is one reason to keep the array modest.
constexpr size_t kScratchBytes = size_t(512) << 20;
static_assert(kScratchBytes == GNN_NOALLOC_SCRATCH_BYTES, "header and array disagree");

__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_ptr[kMaxDevices] = {};

}  // namespace

int noalloc_scratch(int device, void **ptr, size_t *bytes) {
  if (device < 0 || device >= kMaxDevices)
    return set_error(GNN_E_UNSUPPORTED, "device ordinal beyond the scratch table");
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[device]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      const std::string why = e != hipSuccess ? hipGetErrorString(e) : "NULL address";
      return set_error(GNN_E_HIP,
                       ("hipGetSymbolAddress of the scratch array failed: " + why).c_str());
    }
    g_ptr[device] = p;
  }
  *ptr = g_ptr[device];
  *bytes = kScratchBytes;
  return GNN_OK;
}

}  // namespace gnn
