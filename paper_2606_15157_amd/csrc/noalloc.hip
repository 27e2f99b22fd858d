// rkv_prefill_evict_noalloc: the prefill eviction pass for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).
// Its workspace is `scratch`, a file-scope device array of kScratchBytes that every GPU the
// library runs on holds until the process ends; everything else is rkv_prefill_evict.
//
// The array's name is a host-side stand-in in host code: its device address on the current GPU
// comes from hipGetSymbolAddress, taken once per device on the first call there and kept per
// device (each GPU holds its own copy at its own address).  Only that address is handed to
// kernels.  Every call on one GPU shares the array, which keeps the last call's contents: the
// pass itself re-initialises what must start cleared (status word, row-sum marks, repair
// flags) at the start of every call, and calls that overlap on one GPU (other streams,
// threads) race on it.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "rkv_internal.h"

namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;   // 64 MiB: a 32-layer 8K route of one sequence
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

}  // namespace

extern "C" int rkv_prefill_evict_noalloc(const rkv_plan* plan, const rkv_shape* shape, const rkv_prefill_io* io,
                                         uint32_t* status_out, void* stream) {
  size_t need = 0;
  int st = rkv_prefill_workspace_size(plan, shape, &need);
  if (st) return st;
  if (need > kScratchBytes)
    return rkv::fail(RKV_ERR_WORKSPACE, "the call needs a " + std::to_string(need) +
                                            "-byte workspace, above the no-allocation scratch of " +
                                            std::to_string(kScratchBytes) + " bytes; use rkv_prefill_evict");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return rkv::fail(RKV_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return rkv::fail(RKV_ERR_UNSUPPORTED, "device index above 63");
  void* ptr = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[dev]) {
      e = hipGetSymbolAddress(&g_scratch[dev], HIP_SYMBOL(scratch));
      if (e != hipSuccess) {
        g_scratch[dev] = nullptr;
        return rkv::fail(RKV_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
      }
    }
    ptr = g_scratch[dev];
  }
  st = rkv_prefill_evict(plan, shape, io, ptr, kScratchBytes, stream);
  if (st || !status_out) return st;
  // the status word (first word of the workspace) into the caller's buffer, by a copy kernel
  rkv::CopyLaunch C;
  C.n_tasks = 1;
  C.task[0] = {ptr, status_out, (int64_t)sizeof(uint32_t)};
  int err = rkv::launch_copies(C, stream);
  if (err) return rkv::fail(RKV_ERR_HIP, std::string("kernel launch failed: ") + hipGetErrorString((hipError_t)err));
  return RKV_OK;
}
