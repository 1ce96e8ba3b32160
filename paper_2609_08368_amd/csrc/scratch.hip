// Device memory of the allocation-free decode entry point (rl_attn_decode_noalloc):
// one statically sized array per device, in the library's code object, so a
// call that may not allocate (stream capture, serving loops, harnesses that
// forbid hipMalloc) still has room for its plan and split partials.
//
// The array's name is only meaningful in device code. Host code asks the
// runtime for its device address once per device (scratch_address) and passes
// that pointer to the kernels, to hipMemsetAsync and to copies; every GPU
// holds its own copy at its own address. The array keeps whatever the last call
// wrote: the planner rewrites every field it reads, and the error word in the
// first 256 bytes starts at zero (static storage, and cleared again when the
// address is first taken outside stream capture) and is cleared by
// rl_attn_check_device_errors after it is read. Calls that overlap on one
// device share the array and race.
#include <map>
#include <mutex>

#include "kernels.hpp"

static __device__ __align__(256) char scratch[rl::kScratchBytes];

namespace rl {

namespace {

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_ptrs;   // device -> address of its copy of the array

}  // namespace

hipError_t scratch_address(hipStream_t stream, void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_ptrs.find(dev);
  if (it == g_scratch_ptrs.end()) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // the current device's copy
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    // the error word starts at zero; a memset is not recorded into a graph
    // being captured (there the static zero initialisation stands)
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    e = hipStreamIsCapturing(stream, &cs);
    if (e != hipSuccess) return e;
    if (cs == hipStreamCaptureStatusNone) {
      e = hipMemsetAsync(p, 0, kScratchErrBytes, stream);
      if (e != hipSuccess) return e;
    }
    it = g_scratch_ptrs.emplace(dev, p).first;
  }
  *ptr = it->second;
  return hipSuccess;
}

bool scratch_address_if_set_up(void** ptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_ptrs.find(dev);
  if (it == g_scratch_ptrs.end()) return false;
  *ptr = it->second;
  return true;
}

}  // namespace rl
