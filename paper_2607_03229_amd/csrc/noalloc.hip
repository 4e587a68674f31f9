// Placeholder-index check that allocates nothing: its per-row hit counters live in a
// file-scope device array instead of a caller-provided buffer, for callers that cannot
// allocate device memory (code under stream capture, serving loops, harnesses that forbid
// allocation).  It shares the kernels of mpipe_merge_check_indices.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/mpipe.h"
#include "internal.h"

namespace mpipe {
mpipe_status set_error(mpipe_status s, const std::string& m);
}

namespace {

constexpr int64_t kMaxRows = MPIPE_CHECK_NOALLOC_MAX_ROWS;
constexpr int kMaxDevices = 64;

// One int32 hit counter per row of the LLM input buffer.  Every GPU the library runs on
// holds its own copy until the process ends.  In host code `scratch` names a host-side
// stand-in, never the device memory: the device address comes from hipGetSymbolAddress.
static __device__ __align__(256) int32_t scratch[kMaxRows];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};   // device address of `scratch` on each device, once looked up

// The device address of `scratch` on the current device, looked up on the first call
// made on that device (with it current) and kept.
mpipe_status scratch_ptr(int32_t** out) {
  int dev = 0;
  hipError_t r = hipGetDevice(&dev);
  if (r != hipSuccess)
    return mpipe::set_error(MPIPE_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(r));
  if (dev < 0 || dev >= kMaxDevices)
    return mpipe::set_error(MPIPE_ERR_UNSUPPORTED, "device index beyond the supported 64");
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (r != hipSuccess || !p)
      return mpipe::set_error(MPIPE_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") +
                                                 hipGetErrorString(r));
    g_ptr[dev] = p;
  }
  *out = static_cast<int32_t*>(g_ptr[dev]);
  return MPIPE_OK;
}

}  // namespace

extern "C" mpipe_status mpipe_merge_check_indices_noalloc(const int64_t* idx, int64_t n_merged,
                                                          int64_t n_rows, int32_t* status,
                                                          void* stream) {
  if (n_merged < 0 || n_rows < 0) return mpipe::set_error(MPIPE_ERR_INVALID_ARG, "negative size");
  if (n_rows > kMaxRows)
    return mpipe::set_error(MPIPE_ERR_WORKSPACE,
                            "n_rows " + std::to_string(n_rows) + " exceeds the " +
                                std::to_string(kMaxRows) + " rows of the built-in scratch");
  if (!status || (n_merged > 0 && !idx))
    return mpipe::set_error(MPIPE_ERR_INVALID_ARG, "null device buffer");
  int32_t* marks = nullptr;
  const mpipe_status st = scratch_ptr(&marks);
  if (st != MPIPE_OK) return st;
  // the counters of rows [0, n_rows) are cleared by a fill kernel before they are marked
  const hipError_t r =
      mpipe::check_indices(idx, n_merged, n_rows, marks, status, reinterpret_cast<hipStream_t>(stream));
  if (r != hipSuccess)
    return mpipe::set_error(MPIPE_ERR_HIP, std::string("check_indices: ") + hipGetErrorString(r));
  return MPIPE_OK;
}
