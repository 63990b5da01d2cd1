// The traced decode for callers that cannot allocate device memory: the
// log-sum-exp partials of the decoding trace live in a library-owned static
// device array instead of a caller-provided scratch buffer.
//
// Each GPU holds its own copy of the array (PD_TRACE_STATIC_BYTES) for the
// life of the process.  Host code never passes the array's name to a kernel
// (in host code it is only a stand-in for the symbol): the device address is
// taken once per device with hipGetSymbolAddress, with that device current,
// and kept in g_addr.  Calls on one GPU share its array, so calls that
// overlap in time on one GPU race.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "kernels.h"
#include "../../include/pdec.h"

namespace {

constexpr size_t kScratchBytes = PD_TRACE_STATIC_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (nullptr on failure, with
// the error recorded).
void* scratch_address(int32_t* status) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *status = pdec::fail_with(PD_E_DEVICE, (std::string("hipGetDevice: ") + hipGetErrorString(e)).c_str());
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
      *status = pdec::fail_with(PD_E_DEVICE, (std::string("hipGetSymbolAddress: ") + hipGetErrorString(e)).c_str());
      return nullptr;
    }
    g_addr[dev] = p;
  }
  return g_addr[dev];
}

}  // namespace

extern "C" pd_status pd_decode_traced_static(pd_ctx* ctx, int32_t mode, int32_t block, int32_t horizon,
                                             int32_t max_iters, const int32_t* tgt_m, int32_t* out_ids,
                                             int32_t out_ld, int32_t* out_len, int32_t* out_k, int32_t* out_flags,
                                             void* dev_records, int64_t capacity, void* stream) {
  int32_t st = PD_OK;
  void* p = scratch_address(&st);
  if (p == nullptr) return st;
  return pdec::decode_traced_on(ctx, mode, block, horizon, max_iters, tgt_m, out_ids, out_ld, out_len, out_k,
                                out_flags, dev_records, capacity, p, kScratchBytes,
                                "the static trace scratch (PD_TRACE_STATIC_BYTES per GPU)", stream);
}
