// Allocation-free variant of tm_orthogonalize (bf16, batched).
//
// The cached-workspace entry points grow a per-(device, stream) workspace with
// hipMalloc.  Callers that cannot allocate (code under HIP graph capture, tight
// serving loops, harnesses that forbid allocation) call
// tm_orthogonalize_noalloc instead: its workspace is the file-scope device
// array `scratch` below, TM_NOALLOC_SCRATCH_BYTES per GPU, which the loader
// places in device memory with the code object and which each GPU keeps until
// the process ends.
//
// In host code the name `scratch` is a host-side stand-in, not a device
// address.  The device address is resolved once per device, with that device
// current, by hipGetSymbolAddress on the entry point's first call there, and
// only that address is handed to the kernels.
//
// Every call on one GPU shares that GPU's array and leaves its contents
// behind.  Nothing in it has to start at zero: the first phase of every call
// writes the zero-padded copy of its input, and every later buffer (Gram,
// polynomial, scale vector, partial sums) is written in full before it is
// read.  Calls that overlap in time on one GPU (different streams, or other
// threads) race on the array.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>

#include "tm_internal.h"
#include "turbomuon.h"

namespace tmk {
tm_status check_batched_bf16(void* X, int64_t m, int64_t n, int64_t batch, int iters,
                             const float* coeffs, int precond);
tm_status run_batched_bf16_in(void* X, int64_t m, int64_t n, int64_t batch, int iters,
                              const float* coeffs, int precond, void* stream, char* ws,
                              uint64_t ws_bytes);
tm_status fail_with(tm_status s, const char* msg);
}  // namespace tmk

static __device__ __align__(256) char scratch[TM_NOALLOC_SCRATCH_BYTES];

namespace {

std::mutex g_scratch_mu;
std::map<int, char*> g_scratch_ptr;   // device -> device address of its `scratch`

// Device address of the current device's `scratch` (resolved on first use).
tm_status scratch_of_current_device(char** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return tmk::fail_with(TM_ERR_HIP, "hipGetDevice failed");
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it == g_scratch_ptr.end()) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return tmk::fail_with(TM_ERR_HIP, "hipGetSymbolAddress of the static scratch failed");
    }
    it = g_scratch_ptr.emplace(dev, static_cast<char*>(p)).first;
  }
  *out = it->second;
  return TM_OK;
}

}  // namespace

extern "C" tm_status tm_orthogonalize_noalloc(void* X, int64_t m, int64_t n, int64_t batch,
                                              int iters, const float* coeffs, int precond,
                                              void* stream) {
  tm_status s = tmk::check_batched_bf16(X, m, n, batch, iters, coeffs, precond);
  if (s != TM_OK || batch == 0) return s;
  char* ws = nullptr;
  s = scratch_of_current_device(&ws);
  if (s != TM_OK) return s;
  return tmk::run_batched_bf16_in(X, m, n, batch, iters, coeffs, precond, stream, ws,
                                  uint64_t(TM_NOALLOC_SCRATCH_BYTES));
}
