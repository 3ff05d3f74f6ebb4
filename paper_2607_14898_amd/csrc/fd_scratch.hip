// Fixed per-device workspace of fd_decode_chunk_noalloc.
//
// The decode's activation buffers (residual streams, GEMM operands, the MLP
// hidden, per-call RoPE tables) normally live in the workspace each cache
// allocates at creation. For callers that cannot allocate, the same buffers
// can come from this file-scope device array instead. Each GPU that loads it
// holds its own copy for the life of the process; in host code `scratch` is
// only a stand-in for the symbol, so its device address is looked up once per
// device (with that device current) and kept.
#include "fd_kernels.h"

#include <mutex>

namespace fd {
namespace {

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

}  // namespace

hipError_t noalloc_scratch(int device, void** ptr) {
  *ptr = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[device]) {
    int prev = 0;
    hipError_t e = hipGetDevice(&prev);
    if (e != hipSuccess) return e;
    if (prev != device && (e = hipSetDevice(device)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (prev != device) (void)hipSetDevice(prev);
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_addr[device] = p;
  }
  *ptr = g_addr[device];
  return hipSuccess;
}

}  // namespace fd
